"""Seeded random configurations against the oracle: shapes, dtypes, dense and
packed layouts and keep counts drawn at random (valid inputs only), beyond
the hand-picked cases of the other GPU tests."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import assert_attn_close, cu_of, to_dev, to_host_bits, widen

pytestmark = pytest.mark.gpu


def random_select_case(seed):
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.integers(1, 300))
    N = int(rng.choice([1, 2, 7, 64, 65, 197, 300, 577, 1024, 2048]))
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    C = int(rng.choice([8, 16, 24, 64, 384, 768, 1024])) if dtype == "bf16" else int(rng.choice([4, 8, 12, 192, 768]))
    packed = rng.random() < 0.5
    if packed:
        n = rng.integers(1, N + 1, B)
        cu_in = cu_of(n)
        total = int(cu_in[-1])
        scores = rng.standard_normal(total).astype(np.float32)
        tokens = W._normal(rng, (total, C), dtype)
    else:
        n = np.full(B, N)
        cu_in = None
        scores = rng.standard_normal((B, N)).astype(np.float32)
        tokens = W._normal(rng, (B, N, C), dtype)
    if rng.random() < 0.3:
        scores = np.round(scores).astype(np.float32)          # many ties
    keep = np.array([rng.integers(1, m + 1) for m in n], np.int32)
    return scores, keep, tokens, cu_in, N


@pytest.mark.parametrize("seed", range(24))
def test_random_select_pack(gpu, seed):
    scores, keep, tokens, cu_in, N = random_select_case(seed)
    print(f"[random] select seed {seed}: B={len(keep)} N={N} C={tokens.shape[-1]} {tokens.dtype} "
          f"packed={cu_in is not None}", flush=True)
    want = oracle.select_pack(scores, keep, tokens, cu_in=cu_in, N=N)
    assert want[3] == 0
    idx, cu, packed, st = gpu.dora_select_pack(to_dev(scores), to_dev(keep), to_dev(tokens),
                                               cu_in=None if cu_in is None else to_dev(cu_in), N=N,
                                               cap_rows=int(keep.sum()))
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert np.array_equal(cu.cpu().numpy(), want[1]) and np.array_equal(idx.cpu().numpy(), want[0])
    assert np.array_equal(to_host_bits(packed), want[2])


@pytest.mark.parametrize("seed", range(16))
def test_random_attention(gpu, seed):
    rng = np.random.default_rng(2000 + seed)
    B = int(rng.integers(1, 40))
    lens = rng.integers(1, int(rng.choice([16, 64, 200, 600])) + 1, B)
    H = int(rng.integers(1, 17))
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    q, k, v = W.random_qkv(rng, lens, H, dtype)
    cu = cu_of(lens)
    print(f"[random] attention seed {seed}: B={B} max len={lens.max()} H={H} {dtype}", flush=True)
    tq, tk, tv, tcu = to_dev(q), to_dev(k), to_dev(v), to_dev(cu)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = gpu.dora_varlen_attn(tq, tk, tv, tcu, int(lens.max()), dev_status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert_attn_close(widen(out), oracle.varlen_attn(q, k, v, cu, dtype), dtype, f"seed {seed}")


@pytest.mark.parametrize("seed", range(6))
def test_random_residual(gpu, seed):
    scores, keep, tokens, cu_in, N = random_select_case(100 + seed)
    rng = np.random.default_rng(3000 + seed)
    dtype = "bf16" if tokens.dtype == np.uint16 else "f32"
    addend = W._normal(rng, tokens.shape, dtype)
    want = oracle.select_pack_residual(scores, keep, tokens, addend, dtype, cu_in=cu_in, N=N)
    assert want[3] == 0
    idx, cu, packed, st = gpu.dora_select_pack_residual(
        to_dev(scores), to_dev(keep), to_dev(tokens), to_dev(addend),
        cu_in=None if cu_in is None else to_dev(cu_in), N=N, cap_rows=int(keep.sum()))
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert np.array_equal(idx.cpu().numpy(), want[0]) and np.array_equal(to_host_bits(packed), want[2])


@pytest.mark.parametrize("seed", range(6))
def test_random_pl_sample(gpu, seed):
    import test_gpu_pl as pl
    rng = np.random.default_rng(4000 + seed)
    B = int(rng.integers(1, 200))
    N = int(rng.choice([2, 5, 64, 197, 577, 1500]))
    packed = rng.random() < 0.5
    n = rng.integers(1, N + 1, B) if packed else np.full(B, N)
    cu = cu_of(n) if packed else None
    shape = (int(n.sum()),) if packed else (B, N)
    s = (rng.standard_normal(shape) * rng.uniform(0.1, 4)).astype(np.float32)
    g = rng.gumbel(size=shape).astype(np.float32)
    k = np.array([rng.integers(0, m) for m in n], np.int32)
    print(f"[random] pl seed {seed}: B={B} N={N} packed={packed}", flush=True)
    pl.check(gpu, s, g, k, cu=cu, N=N if packed else None)


@pytest.mark.parametrize("seed", range(12))
def test_random_lc1(gpu, seed):
    """Row widths that fill their lane groups and widths that leave a padded
    last piece, with and without a workspace (the split path)."""
    import test_gpu_lc1 as lc
    rng = np.random.default_rng(5000 + seed)
    dtype = "bf16" if rng.random() < 0.7 else "f32"
    C = int(rng.choice([8, 64, 200, 384, 520, 768, 1000, 1024])) if dtype == "bf16" \
        else int(rng.choice([4, 100, 192, 516, 768]))
    lens = rng.integers(1, int(rng.choice([8, 200, 1500])) + 1, int(rng.integers(1, 64)))
    cu = cu_of(lens)
    x = (rng.standard_normal((int(cu[-1]), C)) * rng.uniform(0.2, 3, C) + rng.standard_normal(C)).astype(np.float32)
    xs = W.f32_to_bf16_bits(x) if dtype == "bf16" else x
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = (0.1 * rng.standard_normal(C)).astype(np.float32)
    split = rng.random() < 0.5
    print(f"[random] lc1 seed {seed}: B={len(lens)} C={C} {dtype} workspace={split}", flush=True)
    if not split:
        lc.compare(gpu, xs, cu, gamma, beta, dtype)
        return
    want = oracle.lc1_readout(xs, cu, gamma, beta, 1e-6, dtype)
    tol = lc.fp32_bound(oracle.widen(xs, dtype), cu, gamma.astype(np.float64), beta.astype(np.float64), 1e-6)
    got = lc.run_lc1(gpu, xs, cu, gamma, beta, workspace=gpu.new_lc1_workspace(len(lens), C))
    nan = np.isnan(want)
    assert np.array_equal(np.isnan(got), nan)
    err = np.where(nan, 0.0, np.abs(got - want))
    assert np.all(err <= tol[:, None]), (err.max(), tol.min())
