"""Pins for the oracle's LC1 readout input over the packed buffer (CPU only).

App. E.3: DINOv2's LC1 readout joins the normalised CLS token with the mean of
the normalised surviving visual tokens.  The oracle applies LayerNorm (biased
variance, eps inside the root, affine) to each packed row and averages the
non-CLS rows of each sequence.  Pinned against torch's layer_norm and mean in
fp64, invariances of LayerNorm (row shift; permuting the visual rows),
constant rows (LayerNorm gives beta) and the one-visual-token and CLS-only
cases.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W


def torch_reference(x64, cu, gamma, beta, eps):
    out = []
    g, b = torch.from_numpy(gamma.astype(np.float64)), torch.from_numpy(beta.astype(np.float64))
    for i in range(len(cu) - 1):
        y = torch.nn.functional.layer_norm(torch.from_numpy(x64[cu[i]:cu[i + 1]]), (x64.shape[1],), g, b, eps)
        out.append(torch.cat([y[0], y[1:].mean(dim=0)]).numpy())
    return np.stack(out)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_matches_torch_layer_norm_and_mean(dtype):
    rng = np.random.default_rng(1)
    lens = np.array([2, 5, 197, 64, 3, 120])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    C = 96
    x = (rng.standard_normal((int(cu[-1]), C)) * 3 + rng.standard_normal(C)).astype(np.float32)
    xs = W.f32_to_bf16_bits(x) if dtype == "bf16" else x
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = rng.standard_normal(C).astype(np.float32)
    got = oracle.lc1_readout(xs, cu, gamma, beta, 1e-6, dtype)
    want = torch_reference(oracle.widen(xs, dtype).astype(np.float64), cu, gamma, beta, 1e-6)
    assert np.allclose(got, want, rtol=0, atol=1e-12)


def test_row_shift_and_visual_permutation_invariance():
    rng = np.random.default_rng(2)
    lens = np.array([10, 40])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    C = 64
    x = (np.round(rng.standard_normal((50, C)) * 256) / 256).astype(np.float32)  # shifts below stay exact
    gamma, beta = np.ones(C, np.float32), np.zeros(C, np.float32)
    base = oracle.lc1_readout(x, cu, gamma, beta, 1e-6, "f32")
    shifted = x + rng.integers(-4, 5, (50, 1)).astype(np.float32)     # exact shifts in fp32
    assert np.allclose(oracle.lc1_readout(shifted, cu, gamma, beta, 1e-6, "f32"), base, rtol=0, atol=1e-9)
    perm = x.copy()
    perm[11:50] = x[11:50][rng.permutation(39)]
    assert np.allclose(oracle.lc1_readout(perm, cu, gamma, beta, 1e-6, "f32"), base, rtol=0, atol=1e-12)
    # with unit gamma and zero beta every normalised row has mean 0 and variance var / (var + eps)
    y_cls = base[:, :C]
    assert np.allclose(y_cls.mean(axis=1), 0, atol=1e-12)
    var = x[cu[:-1]].astype(np.float64).var(axis=1)
    assert np.allclose((y_cls ** 2).mean(axis=1), var / (var + 1e-6), rtol=1e-12)


def test_constant_rows_give_beta_and_single_token_cases():
    C = 32
    rng = np.random.default_rng(3)
    beta = rng.standard_normal(C).astype(np.float32)
    gamma = rng.standard_normal(C).astype(np.float32)
    x = np.repeat(rng.standard_normal((4, 1)).astype(np.float32), C, axis=1)
    cu = np.array([0, 2, 3, 4], np.int32)                            # 1 visual, 0 visual, 0 visual
    got = oracle.lc1_readout(x, cu, gamma, beta, 1e-6, "f32")
    assert np.allclose(got[0, :C], beta, atol=1e-12) and np.allclose(got[0, C:], beta, atol=1e-12)
    assert np.all(np.isnan(got[1, C:])) and np.allclose(got[1, :C], beta, atol=1e-12)
    x2 = rng.standard_normal((2, C)).astype(np.float32)
    one = oracle.lc1_readout(x2, np.array([0, 2], np.int32), gamma, beta, 1e-6, "f32")
    cls_of_second = oracle.lc1_readout(x2[1:], np.array([0, 1], np.int32), gamma, beta, 1e-6, "f32")
    assert np.allclose(one[0, C:], cls_of_second[0, :C], rtol=0, atol=0)   # mean of one row is that row
