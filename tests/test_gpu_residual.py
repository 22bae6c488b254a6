"""GPU parity for dora_select_pack_residual: bit-exact against the oracle.

Deletion after the attention residual (Sec. 3.1, Eq. (1)): the packed rows
are the kept rows of h + a, each element the exact sum rounded once to the
storage type.  Indices, boundaries and every bit of the packed rows must
match the oracle (NaN outputs, from inf + -inf, only in position).  Full-size
workloads are compared element by element in the launch configuration the
benchmark times.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import to_dev, to_host_bits

pytestmark = pytest.mark.gpu


def dtype_of(x):
    return "bf16" if x.dtype == np.uint16 else "f32"


def run_gpu(dora, scores, keep, h, a, cu_in=None, N=None, cap=None, guard=0):
    B = len(keep)
    th, ta = to_dev(h), to_dev(a)
    C = h.shape[-1]
    total = int(np.sum(keep)) if cap is None else cap
    idx = torch.full((total + guard,), -7, dtype=torch.int32, device="cuda")
    cu = torch.full((B + 1,), -7, dtype=torch.int32, device="cuda")
    packed = torch.zeros((total + guard, C), dtype=th.dtype, device="cuda")
    word = packed.view(torch.int16 if th.dtype == torch.bfloat16 else torch.int32)
    if guard:
        word[total:].fill_(0x2B2B)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    dora.dora_select_pack_residual(to_dev(scores), to_dev(keep.astype(np.int32)), th, ta,
                                   cu_in=None if cu_in is None else to_dev(cu_in), N=N, idx_out=idx,
                                   cu_out=cu, packed_out=packed, cap_rows=total, dev_status=st)
    torch.cuda.synchronize()
    canary = True
    if guard:
        canary = bool(torch.all(word[total:] == 0x2B2B).item()) and bool(torch.all(idx[total:] == -7).item())
    return (idx[:total].cpu().numpy(), cu.cpu().numpy(), to_host_bits(packed[:total]), int(st.item()), canary)


def same_bits(got, want):
    """Bitwise equality, except that a NaN only has to be a NaN."""
    if got.dtype == np.uint16:
        gn = ((got & 0x7F80) == 0x7F80) & ((got & 0x7F) != 0)
        wn = ((want & 0x7F80) == 0x7F80) & ((want & 0x7F) != 0)
        gv, wv = got, want
    else:
        gn, wn = np.isnan(got), np.isnan(want)
        gv, wv = got.view(np.uint32), want.view(np.uint32)
    return np.array_equal(gn, wn) and np.array_equal(gv[~gn], wv[~wn])


def check_round(dora, scores, keep, h, a, cu_in=None, N=None):
    idx_o, cu_o, packed_o, st_o = oracle.select_pack_residual(scores, keep, h, a, dtype_of(h), cu_in=cu_in, N=N)
    assert st_o == 0
    idx_g, cu_g, packed_g, st_g, _ = run_gpu(dora, scores, keep, h, a, cu_in=cu_in, N=N)
    assert st_g == 0
    assert np.array_equal(cu_g, cu_o)
    assert np.array_equal(idx_g, idx_o)
    assert same_bits(packed_g, packed_o)
    return idx_o, cu_o, packed_o


@pytest.mark.parametrize("name", ["deit_tiny_fp32", "deit_s_bf16", "deit_b_bf16", "vit_b384_skew_bf16"])
def test_workload_full_size(gpu, name):
    w = W.WORKLOADS[name]
    r = W.generate(w, parts=("keep", "scores", "tokens", "attn_out"))[0]
    print(f"[residual] {name} B={w.B} N={w.N} C={w.C} sum_keep={r.total_keep}", flush=True)
    check_round(gpu, r.scores, r.keep, r.tokens, r.attn_out)


def test_cascade_rounds_on_packed_input(gpu):
    """Each round adds its attention output to the previous round's packed rows."""
    w = W.WORKLOADS["vit_l_cascade_bf16"]
    rounds = W.generate(w, parts=("keep", "scores", "tokens", "attn_out"))
    h, cu_in, N = rounds[0].tokens, None, w.N
    for i, r in enumerate(rounds):
        print(f"[residual] cascade round {i} sum_keep={r.total_keep}", flush=True)
        _, cu, packed = check_round(gpu, r.scores, r.keep, h, r.attn_out, cu_in=cu_in, N=N)
        h, cu_in, N = packed, cu, int(r.keep.max())


def wide_bits(rng, shape, dtype):
    """Finite values over the whole exponent range (subnormals, zeros, both signs)."""
    n = int(np.prod(shape))
    if dtype == "bf16":
        e = rng.integers(0, 255, n, dtype=np.uint16)
        return ((rng.integers(0, 2, n, dtype=np.uint16) << 15) | (e << 7)
                | rng.integers(0, 128, n, dtype=np.uint16)).reshape(shape)
    e = rng.integers(0, 255, n, dtype=np.uint32)
    return ((rng.integers(0, 2, n, dtype=np.uint32) << 31) | (e << 23)
            | rng.integers(0, 1 << 23, n, dtype=np.uint32)).view(np.float32).reshape(shape)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_rounding_edges(gpu, dtype):
    """Wide exponents, exact cancellations, ties to even, subnormal sums and
    overflow to infinity, in one ragged batch."""
    rng = np.random.default_rng(11 if dtype == "bf16" else 12)
    B, n, C = 7, 61, 40 if dtype == "bf16" else 20
    h = wide_bits(rng, (B, n, C), dtype)
    a = wide_bits(rng, (B, n, C), dtype)
    # Addends near h's own magnitude (carries, cancellations, ties) for half of the images.
    if dtype == "bf16":
        a[:3] = (h[:3] & 0xFF80) | rng.integers(0, 128, h[:3].shape, dtype=np.uint16)
        a[3, :, :] = h[3] ^ 0x8000                                   # exact cancellation
        a[4, :, :8] = 0x7F7F                                         # the largest finite value
        h[4, :, :8] = rng.choice(np.array([0x7F7F, 0x7B00, 0x7F00, 0x3F80], np.uint16), (n, 8))
        h[5], a[5] = h[5] & 0x807F, a[5] & 0x807F                    # subnormal + subnormal
    else:
        with np.errstate(over="ignore"):
            a[:3] = -h[:3] * np.float32(1 + 2 ** -20)
        a[3] = -h[3]
        a[4, :, :4] = np.float32(3.4028235e38)
        h[4, :, :4] = rng.choice(np.array([3.4028235e38, 1e38, 2e38, 1.0], np.float32), (n, 4))
        h[5] = (h[5].view(np.uint32) & 0x807FFFFF).view(np.float32)
        a[5] = (a[5].view(np.uint32) & 0x807FFFFF).view(np.float32)
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = np.array([n, 1, 30, n, n, 17, 45], np.int32)
    check_round(gpu, scores, keep, h, a)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_negative_zero_addend_equals_select_pack(gpu, dtype):
    rng = np.random.default_rng(13)
    B, n, C = 11, 197, 64
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = rng.integers(1, n + 1, B).astype(np.int32)
    h = wide_bits(rng, (B, n, C), dtype)
    mz = np.full_like(h, 0x8000) if dtype == "bf16" else np.full_like(h, -0.0)
    i1, c1, p1, s1, _ = run_gpu(gpu, scores, keep, h, mz)
    th = to_dev(h)
    i0, c0, p0, s0 = gpu.dora_select_pack(to_dev(scores), to_dev(keep), th)
    torch.cuda.synchronize()
    assert s1 == int(s0.item()) == 0
    tot = int(keep.sum())
    assert np.array_equal(i1, i0[:tot].cpu().numpy()) and np.array_equal(c1, c0.cpu().numpy())
    assert np.array_equal(p1.view(np.uint8), to_host_bits(p0[:tot]).view(np.uint8))


@pytest.mark.parametrize("n", [1, 2, 64, 65, 577, 2048])
@pytest.mark.parametrize("C,dtype", [(8, "bf16"), (4, "f32"), (1024, "bf16")])
def test_sizes_and_row_widths(gpu, n, C, dtype):
    rng = np.random.default_rng(n * 7 + C)
    B = 5
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = rng.integers(1, n + 1, B).astype(np.int32)
    keep[0], keep[-1] = 1, n
    h, a = (W._normal(rng, (B, n, C), dtype) for _ in range(2))
    print(f"[residual] n={n} C={C} {dtype}", flush=True)
    check_round(gpu, scores, keep, h, a)


def test_dense_and_packed_input_agree(gpu):
    rng = np.random.default_rng(14)
    B, n, C = 6, 197, 96
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = rng.integers(1, n + 1, B).astype(np.int32)
    h, a = (W._normal(rng, (B, n, C), "bf16") for _ in range(2))
    dense = run_gpu(gpu, scores, keep, h, a)
    cu_in = (np.arange(B + 1) * n).astype(np.int32)
    packed = run_gpu(gpu, scores.reshape(-1), keep, h.reshape(-1, C), a.reshape(-1, C), cu_in=cu_in, N=n)
    for x, y in zip(dense[:4], packed[:4]):
        assert np.array_equal(np.asarray(x), np.asarray(y))


def test_capacity_overflow_never_writes_past_cap(gpu):
    rng = np.random.default_rng(15)
    B, n, C = 8, 100, 16
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = np.full(B, 90, np.int32)
    h, a = (W._normal(rng, (B, n, C), "bf16") for _ in range(2))
    idx, cu, packed, st, canary = run_gpu(gpu, scores, keep, h, a, cap=500, guard=64)
    assert st & gpu.DORA_DEV_CAPACITY and canary
    idx_o, _, packed_o, _ = oracle.select_pack_residual(scores, keep, h, a, "bf16")
    assert np.array_equal(idx, idx_o[:500]) and np.array_equal(packed, packed_o[:500])


def test_keep_out_of_range_sets_status(gpu):
    rng = np.random.default_rng(16)
    B, n, C = 6, 40, 4
    scores = rng.standard_normal((B, n)).astype(np.float32)
    h, a = (W._normal(rng, (B, n, C), "f32") for _ in range(2))
    for bad in (0, n + 1):
        keep = np.full(B, 10, np.int32)
        keep[3] = bad
        *_, st, canary = run_gpu(gpu, scores, keep, h, a, cap=B * n, guard=8)
        assert st & gpu.DORA_DEV_KEEP_RANGE and canary
