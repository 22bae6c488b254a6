"""GPU parity for dora_select_pack: bit-exact against the oracle.

Indices, sequence boundaries and packed rows must match the oracle exactly
(integer / byte work).  Covers every workload shape at full size (the launch
configuration the benchmark times), cascaded rounds on packed input,
adversarial score patterns, size edges and the device error word.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import to_dev, to_host_bits

pytestmark = pytest.mark.gpu


def run_gpu(dora, scores, keep, tokens, cu_in=None, N=None, cap=None, guard=0):
    """Call the library; returns host copies (idx, cu, packed bits, status, canary ok)."""
    B = len(keep)
    ts, tk = to_dev(scores), to_dev(keep.astype(np.int32))
    tt = to_dev(tokens)
    C = tokens.shape[-1]
    total = int(np.sum(keep)) if cap is None else cap
    idx = torch.full((total + guard,), -7, dtype=torch.int32, device="cuda")
    cu = torch.full((B + 1,), -7, dtype=torch.int32, device="cuda")
    packed = torch.zeros((total + guard, C), dtype=tt.dtype, device="cuda")
    if guard:
        packed[total:].view(torch.int16 if tt.dtype == torch.bfloat16 else torch.int32).fill_(0x2B2B)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    dora.dora_select_pack(ts, tk, tt, cu_in=None if cu_in is None else to_dev(cu_in), N=N,
                          idx_out=idx, cu_out=cu, packed_out=packed, cap_rows=total, dev_status=st)
    torch.cuda.synchronize()
    canary = True
    if guard:
        tail = to_host_bits(packed[total:])
        canary = bool(np.all(tail.view(np.uint16 if tail.dtype == np.uint16 else np.int32) == 0x2B2B)) and \
            bool(torch.all(idx[total:] == -7).item())
    return (idx[:total].cpu().numpy(), cu.cpu().numpy(), to_host_bits(packed[:total]),
            int(st.item()), canary)


def check_round(dora, scores, keep, tokens, cu_in=None, N=None):
    idx_o, cu_o, packed_o, st_o = oracle.select_pack(scores, keep, tokens, cu_in=cu_in, N=N)
    assert st_o == 0
    idx_g, cu_g, packed_g, st_g, _ = run_gpu(dora, scores, keep, tokens, cu_in=cu_in, N=N)
    assert st_g == 0
    assert np.array_equal(cu_g, cu_o)
    assert np.array_equal(idx_g, idx_o)
    assert np.array_equal(packed_g, packed_o)
    return idx_g, cu_g, packed_g


@pytest.mark.parametrize("name", ["deit_tiny_fp32", "deit_s_bf16", "deit_b_bf16", "vit_b384_skew_bf16"])
def test_workload_full_size(gpu, name):
    w = W.WORKLOADS[name]
    r = W.generate(w, parts=("keep", "scores", "tokens"))[0]
    print(f"[select_pack] {name} B={w.B} N={w.N} C={w.C} sum_keep={r.total_keep}", flush=True)
    check_round(gpu, r.scores, r.keep, r.tokens)


def test_cascade_three_rounds_on_packed_input(gpu):
    w = W.WORKLOADS["vit_l_cascade_bf16"]
    rounds = W.generate(w, parts=("keep", "scores", "tokens"))
    tokens, cu_in, N = rounds[0].tokens, None, w.N
    for i, r in enumerate(rounds):
        print(f"[select_pack] cascade round {i} sum_keep={r.total_keep}", flush=True)
        idx, cu, packed = check_round(gpu, r.scores, r.keep, tokens, cu_in=cu_in, N=N)
        tokens, cu_in, N = packed, cu, int(r.keep.max())


def adversarial_scores(rng, B, n):
    pats = []
    pats.append(np.full(n, 0.5, np.float32))                               # all ties
    pats.append(np.where(rng.random(n) < 0.5, -0.0, 0.0).astype(np.float32))  # signed zeros
    a = rng.choice(np.array([np.nan, np.inf, -np.inf, 1.0, -1.0, 0.0], np.float32), n)
    pats.append(a)                                                          # specials
    pats.append(np.full(n, np.nan, np.float32))                            # all NaN
    pats.append(np.linspace(3, -3, n).astype(np.float32))                  # decreasing
    pats.append(np.linspace(-3, 3, n).astype(np.float32))                  # increasing
    x = rng.integers(-3, 3, n).astype(np.float32)                          # few distinct values
    pats.append(x)
    d = np.frombuffer(rng.integers(0, 2 ** 32, n, dtype=np.uint32).tobytes(), np.float32).copy()
    pats.append(d)                                                          # random bit patterns
    e = (1.0 + np.arange(n) * 2 ** -23).astype(np.float32)                 # adjacent floats
    pats.append(rng.permutation(e))
    out = np.stack([pats[i % len(pats)] for i in range(B)])
    return out


@pytest.mark.parametrize("n", [1, 2, 63, 64, 65, 128, 197, 300, 577, 1024, 1500, 2048])
def test_adversarial_patterns_all_sizes(gpu, n):
    rng = np.random.default_rng(n)
    B = 27
    scores = adversarial_scores(rng, B, n)
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    keep[0], keep[1 % B] = 1, n                                             # extremes
    tokens = rng.integers(0, 2 ** 16, size=(B, n, 8)).astype(np.uint16)     # 16-byte bf16 rows
    print(f"[select_pack] adversarial n={n}", flush=True)
    check_round(gpu, scores, keep, tokens)


@pytest.mark.parametrize("C,dtype", [(4, np.float32), (8, np.uint16), (2048, np.float32), (24, np.uint16)])
def test_row_widths(gpu, C, dtype):
    rng = np.random.default_rng(C)
    B, n = 9, 197
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    if dtype == np.float32:
        tokens = rng.standard_normal((B, n, C)).astype(np.float32)
    else:
        tokens = rng.integers(0, 2 ** 16, size=(B, n, C)).astype(np.uint16)
    check_round(gpu, scores, keep, tokens)


@pytest.mark.parametrize("C,dtype", [(262144, np.float32), (524288, np.uint16)])
def test_widest_rows(gpu, C, dtype):
    """Rows of 1 MB, the widest the library takes (4096 16-byte pieces per
    thread block step): a short batch, bit-exact."""
    rng = np.random.default_rng(C + 1)
    B, n = 3, 5
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = np.array([5, 1, 3], np.int32)
    if dtype == np.float32:
        tokens = rng.standard_normal((B, n, C)).astype(np.float32)
    else:
        tokens = rng.integers(0, 2 ** 16, size=(B, n, C)).astype(np.uint16)
    check_round(gpu, scores, keep, tokens)


def test_many_images(gpu):
    rng = np.random.default_rng(77)
    B, n = 3000, 50
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    tokens = rng.integers(0, 2 ** 16, size=(B, n, 8)).astype(np.uint16)
    check_round(gpu, scores, keep, tokens)


def test_deterministic(gpu):
    w = W.WORKLOADS["deit_s_bf16"]
    r = W.generate(w, parts=("keep", "scores", "tokens"))[0]
    a = run_gpu(gpu, r.scores, r.keep, r.tokens)
    b = run_gpu(gpu, r.scores, r.keep, r.tokens)
    for x, y in zip(a[:3], b[:3]):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("n", [40, 577])  # one-wave and four-wave selection
def test_keep_out_of_range_sets_status(gpu, n):
    rng = np.random.default_rng(3)
    B = 6
    scores = rng.standard_normal((B, n)).astype(np.float32)
    tokens = rng.standard_normal((B, n, 4)).astype(np.float32)
    for bad in (0, n + 1, -5):
        keep = np.full(B, 10, np.int32)
        keep[3] = bad
        *_, st, canary = run_gpu(gpu, scores, keep, tokens, cap=B * n, guard=8)
        assert st & gpu.DORA_DEV_KEEP_RANGE and canary


@pytest.mark.parametrize("n,kb,cap", [(100, 90, 500), (600, 540, 3000)])  # one-wave and four-wave selection
def test_capacity_overflow_never_writes_past_cap(gpu, n, kb, cap):
    rng = np.random.default_rng(4)
    B = 8
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = np.full(B, kb, np.int32)
    tokens = rng.integers(0, 2 ** 16, size=(B, n, 16)).astype(np.uint16)
    idx, cu, packed, st, canary = run_gpu(gpu, scores, keep, tokens, cap=cap, guard=64)
    assert st & gpu.DORA_DEV_CAPACITY
    assert canary
    idx_o, cu_o, packed_o, _ = oracle.select_pack(scores, keep, tokens)
    assert np.array_equal(idx, idx_o[:cap]) and np.array_equal(packed, packed_o[:cap])


def test_invalid_cu_in_sets_status(gpu):
    rng = np.random.default_rng(5)
    lens = np.array([5, 9, 3])
    cu_in = np.array([0, 5, 14, 17], np.int32)
    scores = rng.standard_normal(17).astype(np.float32)
    tokens = rng.standard_normal((17, 4)).astype(np.float32)
    keep = np.array([2, 2, 2], np.int32)
    for bad in ([0, 5, 4, 17], [1, 5, 14, 17], [0, 5, 14, 18], [0, 5, 5, 17]):
        *_, st, canary = run_gpu(gpu, scores, keep, tokens, cu_in=np.array(bad, np.int32), N=12,
                                 cap=6, guard=4)
        assert st & gpu.DORA_DEV_CU_IN, bad
        assert canary
    *_, st, _ = run_gpu(gpu, scores, keep, tokens, cu_in=cu_in, N=9)
    assert st == 0
    *_, st, _ = run_gpu(gpu, scores, keep, tokens, cu_in=cu_in, N=8, cap=6)   # segment longer than N
    assert st & gpu.DORA_DEV_CU_IN


@pytest.mark.parametrize("n", [257, 300, 577])
def test_digit_prefix_ties_every_keep_count(gpu, n):
    """Rows over 256 tokens select one 8-bit digit of the key at a time.
    Scores whose bit patterns share every prefix of 1, 2 and 3 bytes with
    many others (4 choices per byte, so about n / 4 keys per bucket at each
    pass, and many exact ties), one image for every keep count 1..n."""
    rng = np.random.default_rng(700 + n)
    byte_vals = np.array([0x3F, 0x40, 0xBF, 0xC0], np.uint32)                # both signs, around 1.0 and 2.0
    low_vals = np.array([0x00, 0x01, 0x80, 0xFF], np.uint32)
    bits = (byte_vals[rng.integers(0, 4, n)] << 24) | (low_vals[rng.integers(0, 4, n)] << 16) \
        | (low_vals[rng.integers(0, 4, n)] << 8) | low_vals[rng.integers(0, 4, n)]
    row = bits.astype(np.uint32).view(np.float32)
    scores = np.tile(row, (n, 1))
    keep = np.arange(1, n + 1, dtype=np.int32)
    tokens = rng.integers(0, 2 ** 16, size=(n, n, 8)).astype(np.uint16)
    print(f"[select_pack] digit prefix ties n={n}", flush=True)
    check_round(gpu, scores, keep, tokens)


@pytest.mark.parametrize("B", [2049, 8192, 65536])
def test_large_batch_block_scan(gpu, B):
    """Past 2048 images one workgroup scans the keep counts into cu_seqlens
    before the gather (Sec. 3.5 "Inference": the packed buffer's
    boundaries); the results stay bit-exact."""
    rng = np.random.default_rng(B)
    n = 197
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    tokens = rng.integers(0, 2 ** 16, size=(B, n, 8)).astype(np.uint16)
    print(f"[select_pack] large batch B={B} sum_keep={int(keep.sum())}", flush=True)
    check_round(gpu, scores, keep, tokens)


def test_large_batch_packed_input_rounds(gpu):
    """Two chained rounds on packed input with 8192 images."""
    rng = np.random.default_rng(8193)
    B, n = 8192, 100
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    tokens = rng.integers(0, 2 ** 16, size=(B, n, 8)).astype(np.uint16)
    idx, cu, packed = check_round(gpu, scores, keep, tokens)
    keep2 = np.maximum(1, (keep * rng.uniform(0.3, 1.0, B)).astype(np.int32))
    scores2 = rng.standard_normal(int(keep.sum())).astype(np.float32)
    check_round(gpu, scores2, keep2, packed, cu_in=cu, N=n)


def test_large_batch_errors_write_nothing_past_cap(gpu):
    """The scanned path keeps the error contract: a bad keep count sets its
    bit, and nothing lands past the capacity."""
    rng = np.random.default_rng(4097)
    B, n = 4096, 40
    scores = rng.standard_normal((B, n)).astype(np.float32)
    tokens = rng.integers(0, 2 ** 16, size=(B, n, 8)).astype(np.uint16)
    keep = np.full(B, 10, np.int32)
    keep[3000] = 0
    *_, st, canary = run_gpu(gpu, scores, keep, tokens, cap=B * 10, guard=8)
    assert st & gpu.DORA_DEV_KEEP_RANGE and canary
    keep = np.full(B, 30, np.int32)
    idx, cu, packed, st, canary = run_gpu(gpu, scores, keep, tokens, cap=1000, guard=16)
    assert st & gpu.DORA_DEV_CAPACITY and canary
    idx_o, cu_o, packed_o, _ = oracle.select_pack(scores, keep, tokens)
    assert np.array_equal(idx, idx_o[:1000]) and np.array_equal(packed, packed_o[:1000])
    assert np.array_equal(cu, cu_o)
