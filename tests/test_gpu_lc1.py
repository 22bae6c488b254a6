"""GPU parity for dora_lc1_readout against the fp64 oracle.

The kernel computes in fp32; each image's outputs must lie within a bound
derived from its arithmetic (`fp32_bound`): row sums of at most 32 values
per lane plus a 6-level butterfly (38 roundings per element), the centred
second moment likewise, the reciprocal square root and the affine step (a
few roundings each), and the mean over the rows (at most n/8 sequential
adds per wave, 8 across waves, one scale).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import to_dev

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def fp32_bound(x64, cu, gamma, beta, eps):
    tol = []
    for b in range(len(cu) - 1):
        r = x64[cu[b]:cu[b + 1]]
        mu = r.mean(axis=1, keepdims=True)
        rstd = 1.0 / np.sqrt(((r - mu) ** 2).mean(axis=1, keepdims=True) + eps)
        a = np.abs((r - mu) * rstd * gamma)
        y = np.abs(a) + np.abs(beta)
        n = r.shape[0]
        tol.append(U * (100 * a.max() + 40 * np.abs(r).max() * rstd.max() * np.abs(gamma).max()
                        + (n / 8 + 14) * y.max()))
    return np.array(tol)


def compare(dora, x, cu, gamma, beta, dtype, eps=1e-6):
    out, st = dora.dora_lc1_readout(to_dev(x), to_dev(cu), to_dev(gamma), to_dev(beta), eps)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    got = out.cpu().numpy().astype(np.float64)
    want = oracle.lc1_readout(x, cu, gamma, beta, eps, dtype)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    tol = fp32_bound(oracle.widen(x, dtype), cu, gamma.astype(np.float64), beta.astype(np.float64), eps)
    err = np.where(nan, 0.0, np.abs(got - want))
    assert np.all(err <= tol[:, None]), (err.max(), tol.min())
    return err.max()


# Row shapes: 768/384/1024/2048 bf16 and 192/1024 f32 fill their lane groups
# exactly; 64, 8, 200, 520 and 1000 bf16 and 100 f32 leave some lanes' last
# piece past the row's end (16-, 32- and 64-lane groups, 1 to 3 pieces a lane).
@pytest.mark.parametrize("C,dtype", [(768, "bf16"), (1024, "bf16"), (384, "bf16"), (192, "f32"), (64, "bf16"),
                                     (2048, "bf16"), (1024, "f32"), (8, "bf16"), (200, "bf16"), (520, "bf16"),
                                     (1000, "bf16"), (100, "f32")])
def test_ragged_sequences(gpu, C, dtype):
    rng = np.random.default_rng(C)
    lens = np.array([1, 2, 3, 8, 9, 16, 17, 31, 197, 257, 1000])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    x = (rng.standard_normal((int(cu[-1]), C)) * rng.uniform(0.5, 2, C) + rng.standard_normal(C)).astype(np.float32)
    xs = W.f32_to_bf16_bits(x) if dtype == "bf16" else x
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = (0.1 * rng.standard_normal(C)).astype(np.float32)
    err = compare(gpu, xs, cu, gamma, beta, dtype)
    print(f"[lc1] C={C} {dtype} max err {err:.2e}", flush=True)


@pytest.mark.parametrize("name", ["dinov2_b14_bf16", "deit_b_bf16"])
def test_workload_full_size(gpu, name):
    w = W.WORKLOADS[name]
    keep = W.generate(w, parts=("keep",))[0].keep
    x, gamma, beta = W.readout_rows(w, keep)
    cu = np.concatenate([[0], np.cumsum(keep)]).astype(np.int32)
    err = compare(gpu, x, cu, gamma, beta, w.dtype)
    print(f"[lc1] {name} max err {err:.2e}", flush=True)


def test_invalid_sequences_set_status(gpu):
    rng = np.random.default_rng(3)
    C = 64
    x = rng.standard_normal((20, C)).astype(np.float32)
    g, b = np.ones(C, np.float32), np.zeros(C, np.float32)
    for cu in ([0, 5, 5, 20], [0, 5, 21, 20], [1, 5, 10, 20]):
        out, st = gpu.dora_lc1_readout(to_dev(x), to_dev(np.array(cu, np.int32)), to_dev(g), to_dev(b))
        torch.cuda.synchronize()
        o = out.cpu().numpy()
        assert int(st.item()) & gpu.DORA_DEV_CU_SEQLENS, cu
        bad = [i for i in range(3) if not (cu[i] >= 0 and cu[i + 1] > cu[i] and cu[i + 1] <= 20 and (i or cu[0] == 0))]
        assert np.all(np.isnan(o[bad])), cu


def run_lc1(dora, x, cu, gamma, beta, eps=1e-6, **kw):
    out, st = dora.dora_lc1_readout(to_dev(x), to_dev(cu), to_dev(gamma), to_dev(beta), eps, **kw)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    return out.cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("lens,C,dtype", [
    ([1, 2, 600], 768, "bf16"),                    # only CLS; 2 rows over 3 parts (one empty); a long row
    ([577] * 4 + [70] * 4, 768, "bf16"),           # skewed, few images: 5 parts per image
    ([300, 1, 299, 5, 1000, 64], 192, "f32"),
    ([129] * 16, 1024, "bf16"),
])
def test_split_and_single_workgroup_paths(gpu, lens, C, dtype):
    """With a workspace a sequence's rows are split over several workgroups
    and a second kernel adds their sums in part order; without one, one
    workgroup per sequence.  Both meet the fp32 bound against the oracle, the
    split result repeats bit for bit on a reused workspace, and a fresh
    workspace gives the same bits."""
    rng = np.random.default_rng(sum(lens) + C)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    x = (rng.standard_normal((int(cu[-1]), C)) * rng.uniform(0.5, 2, C) + rng.standard_normal(C)).astype(np.float32)
    xs = W.f32_to_bf16_bits(x) if dtype == "bf16" else x
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = (0.1 * rng.standard_normal(C)).astype(np.float32)
    want = oracle.lc1_readout(xs, cu, gamma, beta, 1e-6, dtype)
    tol = fp32_bound(oracle.widen(xs, dtype), cu, gamma.astype(np.float64), beta.astype(np.float64), 1e-6)
    ws = gpu.new_lc1_workspace(len(lens), C)
    outs = [run_lc1(gpu, xs, cu, gamma, beta, workspace=ws) for _ in range(3)]
    outs.append(run_lc1(gpu, xs, cu, gamma, beta))
    single = run_lc1(gpu, xs, cu, gamma, beta, single=True)
    nan = np.isnan(want)
    for got in outs + [single]:
        assert np.array_equal(np.isnan(got), nan)
        err = np.where(nan, 0.0, np.abs(got - want))
        assert np.all(err <= tol[:, None]), (err.max(), tol.min())
    for got in outs[1:]:
        assert np.array_equal(got, outs[0], equal_nan=True)
    print(f"[lc1] split lens={lens[:4]}... C={C} {dtype} ok", flush=True)


def test_vit_b384_skewed_batch(gpu):
    """64 images of 577 tokens, half keeping 90-100 % and half 8-15 %."""
    w = W.WORKLOADS["vit_b384_skew_bf16"]
    keep = W.generate(w, parts=("keep",))[0].keep
    x, gamma, beta = W.readout_rows(w, keep)
    cu = np.concatenate([[0], np.cumsum(keep)]).astype(np.int32)
    err = compare(gpu, x, cu, gamma, beta, w.dtype)
    print(f"[lc1] vit_b384_skew_bf16 max err {err:.2e}", flush=True)


def test_invalid_sequence_on_the_split_path(gpu):
    """An empty sequence among long ones, with a workspace (so the rows are
    split over several workgroups): its row is NaN with DORA_DEV_CU_SEQLENS,
    and the valid sequences still meet the bound against the oracle."""
    rng = np.random.default_rng(4)
    C = 256
    cu = np.array([0, 300, 300, 900], np.int32)                            # sequence 1 is empty
    x = W.f32_to_bf16_bits(rng.standard_normal((900, C)).astype(np.float32))
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = (0.1 * rng.standard_normal(C)).astype(np.float32)
    assert 900 // (64 * 3) >= 2                                            # the host picks a split > 1
    out, st = gpu.dora_lc1_readout(to_dev(x), to_dev(cu), to_dev(gamma), to_dev(beta), 1e-6,
                                   workspace=gpu.new_lc1_workspace(3, C))
    torch.cuda.synchronize()
    assert int(st.item()) & gpu.DORA_DEV_CU_SEQLENS
    o = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isnan(o[1]))
    for b in (0, 2):
        seg = np.array([0, cu[b + 1] - cu[b]], np.int32)
        xb = x[cu[b]:cu[b + 1]]
        want = oracle.lc1_readout(xb, seg, gamma, beta, 1e-6, "bf16")[0]
        tol = fp32_bound(oracle.widen(xb, "bf16"), seg, gamma.astype(np.float64), beta.astype(np.float64), 1e-6)
        assert np.all(np.abs(o[b] - want) <= tol[0]), b


@pytest.mark.parametrize("with_ws", [False, True])
def test_many_short_sequences(gpu, with_ws):
    """3000 sequences of 1 to 40 rows (more images than workgroups fit at
    once), with and without a workspace."""
    rng = np.random.default_rng(3000 + with_ws)
    C = 768
    lens = rng.integers(1, 41, 3000)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    x = W.f32_to_bf16_bits((rng.standard_normal((int(cu[-1]), C)) + rng.standard_normal(C)).astype(np.float32))
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = (0.1 * rng.standard_normal(C)).astype(np.float32)
    want = oracle.lc1_readout(x, cu, gamma, beta, 1e-6, "bf16")
    tol = fp32_bound(oracle.widen(x, "bf16"), cu, gamma.astype(np.float64), beta.astype(np.float64), 1e-6)
    kw = {"workspace": gpu.new_lc1_workspace(len(lens), C)} if with_ws else {}
    got = run_lc1(gpu, x, cu, gamma, beta, **kw)
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    err = np.where(nan, 0.0, np.abs(got - want))
    assert np.all(err <= tol[:, None]), (err.max(), tol.min())


def test_constant_rows_without_eps(gpu):
    """eps = 0: a constant row has zero variance, so its normalised values are
    0/0 = NaN, in the kernel (0 times the reciprocal square root of 0) as in
    the oracle; a sequence without such a row stays finite."""
    rng = np.random.default_rng(5)
    C = 256
    x = rng.standard_normal((12, C)).astype(np.float32)
    x[0] = 3.0   # CLS of sequence 0 constant
    x[6] = -1.5  # a visual row of sequence 1 constant
    cu = np.array([0, 4, 9, 12], np.int32)
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = (0.1 * rng.standard_normal(C)).astype(np.float32)
    want = oracle.lc1_readout(x, cu, gamma, beta, 0.0, "f32")
    got = run_lc1(gpu, x, cu, gamma, beta, eps=0.0)
    assert np.all(np.isnan(want[0, :C])) and np.all(np.isnan(want[1, C:])) and np.all(np.isfinite(want[2]))
    assert np.array_equal(np.isnan(got), np.isnan(want))
    ok = ~np.isnan(want)
    assert np.max(np.abs(got[ok] - want[ok])) < 1e-4
