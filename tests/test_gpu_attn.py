"""GPU parity for dora_varlen_attn against the fp64 oracle.

bf16 inputs: max |err| <= 2e-2 and mean |err| <= 2e-3; fp32 inputs:
max |err| <= 1e-5.  Every case compares every output element with the
oracle, the full-size workloads included (in the launch configuration the
benchmark times).
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import assert_attn_close, cu_of, to_dev, to_host_bits, widen

pytestmark = pytest.mark.gpu


def gpu_attn(dora, q, k, v, cu, max_seqlen=None, scale=0.0, out_fill=None):
    tq, tk, tv = to_dev(q), to_dev(k), to_dev(v)
    tcu = to_dev(np.asarray(cu, np.int32))
    lens = np.diff(cu)
    ms = int(max(1, lens.max())) if max_seqlen is None else max_seqlen
    out = torch.empty_like(tq)
    if out_fill is not None:
        out.view(torch.int16 if out.dtype == torch.bfloat16 else torch.int32).fill_(out_fill)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    dora.dora_varlen_attn(tq, tk, tv, tcu, ms, out=out, softmax_scale=scale, dev_status=st)
    torch.cuda.synchronize()
    return out, int(st.item())


def full_compare(dora, q, k, v, cu, dtype, scale=None, what=""):
    out, st = gpu_attn(dora, q, k, v, cu, scale=0.0 if scale is None else scale)
    assert st == 0
    want = oracle.varlen_attn(q, k, v, cu, dtype, scale=scale)
    return assert_attn_close(widen(out), want, dtype, what)


def qkv(rng, lens, H, dtype, scale_in=1.0):
    tot = int(np.sum(lens))
    arr = [(rng.standard_normal((tot, H, 64)) * scale_in).astype(np.float32) for _ in range(3)]
    return [W.f32_to_bf16_bits(a) if dtype == "bf16" else a for a in arr]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ragged_tile_edges(gpu, dtype):
    lens = np.array([1, 2, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 191, 255, 256, 257, 300])
    rng = np.random.default_rng(31)
    q, k, v = qkv(rng, lens, 3, dtype)
    print(f"[attn] ragged edges {dtype}", flush=True)
    full_compare(gpu, q, k, v, cu_of(lens), dtype, what="ragged")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_query_chunk_and_stage_edges(gpu, dtype):
    """Lengths around the 192-query chunks and the 256-key stages, several
    chunks and stages in one sequence, and heads that wrap a DMA round."""
    lens = np.array([191, 192, 193, 255, 256, 257, 383, 384, 385, 511, 512, 513, 575, 576, 577, 768, 769])
    rng = np.random.default_rng(41)
    q, k, v = qkv(rng, lens, 5, dtype)
    print(f"[attn] chunk/stage edges {dtype}", flush=True)
    full_compare(gpu, q, k, v, cu_of(lens), dtype, what="chunk edges")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_empty_sequences(gpu, dtype):
    lens = np.array([0, 5, 0, 0, 130, 0, 1, 0])
    rng = np.random.default_rng(32)
    q, k, v = qkv(rng, lens, 2, dtype)
    full_compare(gpu, q, k, v, cu_of(lens), dtype, what="empty")


def test_deit_tiny_fp32_workload(gpu):
    w = W.WORKLOADS["deit_tiny_fp32"]
    r = W.generate(w, parts=("keep", "qkv"))[0]
    mx, _ = full_compare(gpu, r.q, r.k, r.v, cu_of(r.keep), "f32", what=w.name)
    print(f"[attn] {w.name} max err {mx:.2e}", flush=True)


def test_deit_s_bf16_workload(gpu):
    w = W.WORKLOADS["deit_s_bf16"]
    r = W.generate(w, parts=("keep", "qkv"))[0]
    mx, mean = full_compare(gpu, r.q, r.k, r.v, cu_of(r.keep), "bf16", what=w.name)
    print(f"[attn] {w.name} max err {mx:.2e} mean {mean:.2e}", flush=True)


def test_deit_b_bf16_full_size(gpu):
    """The headline batch (B = 256, H = 12), every output element."""
    w = W.WORKLOADS["deit_b_bf16"]
    r = W.generate(w, parts=("keep", "qkv"))[0]
    mx, mean = full_compare(gpu, r.q, r.k, r.v, cu_of(r.keep), "bf16", what=w.name)
    print(f"[attn] {w.name} max err {mx:.2e} mean {mean:.2e}", flush=True)


def test_vit_b384_skew_full_size(gpu):
    """The skewed ViT-B/384 batch (sequences of 46-577 tokens), every element."""
    w = W.WORKLOADS["vit_b384_skew_bf16"]
    r = W.generate(w, parts=("keep", "qkv"))[0]
    mx, mean = full_compare(gpu, r.q, r.k, r.v, cu_of(r.keep), "bf16", what=w.name)
    print(f"[attn] {w.name} max err {mx:.2e} mean {mean:.2e}", flush=True)


def test_vit_l_cascade_rounds_full_size(gpu):
    """Each of the three ViT-L rounds (H = 16), every element."""
    w = W.WORKLOADS["vit_l_cascade_bf16"]
    for i, r in enumerate(W.generate(w, parts=("keep", "qkv"))):
        mx, mean = full_compare(gpu, r.q, r.k, r.v, cu_of(r.keep), "bf16", what=f"{w.name} round {i}")
        print(f"[attn] {w.name} round {i} max err {mx:.2e} mean {mean:.2e}", flush=True)


def test_long_sequence_and_many_heads(gpu):
    rng = np.random.default_rng(33)
    lens = np.array([2048])
    q, k, v = qkv(rng, lens, 1, "bf16")
    full_compare(gpu, q, k, v, cu_of(lens), "bf16", what="len 2048")
    lens = np.array([77, 200, 5])
    q, k, v = qkv(rng, lens, 16, "bf16")
    full_compare(gpu, q, k, v, cu_of(lens), "bf16", what="H=16")
    lens = np.array([40, 3, 193])  # 256 heads (the most a plan item can name), one sequence of two chunks
    q, k, v = qkv(rng, lens, 256, "bf16")
    full_compare(gpu, q, k, v, cu_of(lens), "bf16", what="H=256")
    lens = np.array([1])
    q, k, v = qkv(rng, lens, 1, "f32")
    full_compare(gpu, q, k, v, cu_of(lens), "f32", what="H=1, one token")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_large_logits_online_rescale(gpu, dtype):
    # Logits with std ~ 8 force many running-max updates across key blocks.
    lens = np.array([300, 129, 64])
    rng = np.random.default_rng(34)
    q, k, v = qkv(rng, lens, 2, dtype, scale_in=1.0)
    qs = (W.bf16_bits_to_f32(q) if dtype == "bf16" else q) * 8.0
    q = W.f32_to_bf16_bits(qs) if dtype == "bf16" else qs.astype(np.float32)
    full_compare(gpu, q, k, v, cu_of(lens), dtype, what="large logits")


def test_custom_scale(gpu):
    lens = np.array([50, 70])
    rng = np.random.default_rng(35)
    q, k, v = qkv(rng, lens, 2, "f32")
    full_compare(gpu, q, k, v, cu_of(lens), "f32", scale=0.3, what="scale 0.3")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_single_token_returns_v_exactly(gpu, dtype):
    lens = np.ones(37, dtype=np.int64)
    rng = np.random.default_rng(36)
    q, k, v = qkv(rng, lens, 4, dtype)
    out, st = gpu_attn(gpu, q, k, v, cu_of(lens))
    assert st == 0 and np.array_equal(to_host_bits(out), v)


def test_segment_permutation_is_bit_exact(gpu):
    lens = np.array([3, 197, 1, 140, 66, 128])
    rng = np.random.default_rng(37)
    q, k, v = qkv(rng, lens, 3, "bf16")
    cu = cu_of(lens)
    base, _ = gpu_attn(gpu, q, k, v, cu)
    base = to_host_bits(base)
    perm = np.array([4, 1, 5, 0, 3, 2])
    cat = lambda a: np.concatenate([a[cu[b]:cu[b + 1]] for b in perm])
    out, st = gpu_attn(gpu, cat(q), cat(k), cat(v), cu_of(lens[perm]))
    assert st == 0 and np.array_equal(to_host_bits(out), cat(base))


def test_plan_reuse_and_determinism(gpu):
    lens = np.array([197, 64, 65, 1, 130])
    rng = np.random.default_rng(38)
    q, k, v = (to_dev(a) for a in qkv(rng, lens, 3, "bf16"))
    cu = to_dev(cu_of(lens))
    ws = gpu.new_workspace(len(lens), 3, 197)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    gpu.dora_varlen_attn_plan(cu, 3, 197, int(lens.sum()), ws, st)
    outs = [gpu.dora_varlen_attn_execute(q, k, v, cu, 197, ws, dev_status=st) for _ in range(4)]
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    first = to_host_bits(outs[0])
    for o in outs[1:]:
        assert np.array_equal(to_host_bits(o), first)


def test_plan_mismatch_sets_status(gpu):
    lens = np.array([10, 20])
    rng = np.random.default_rng(39)
    q, k, v = (to_dev(a) for a in qkv(rng, lens, 2, "bf16"))
    cu = to_dev(cu_of(lens))
    ws = gpu.new_workspace(2, 2, 64)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    gpu.dora_varlen_attn_plan(cu, 2, 64, 30, ws, st)
    out = torch.zeros_like(q)
    gpu.dora_varlen_attn_execute(q, k, v, cu, 32, ws, out=out, dev_status=st)   # different max_seqlen
    torch.cuda.synchronize()
    assert int(st.item()) & gpu.DORA_DEV_PLAN
    assert torch.all(out.view(torch.int16) == 0)


def test_invalid_offsets_set_status(gpu):
    rng = np.random.default_rng(40)
    q, k, v = qkv(rng, [30], 2, "bf16")
    for bad in ([0, 10, 5, 30], [2, 10, 20, 30], [0, 10, 20, 31], [0, 10, 20, 30]):
        cu = np.array(bad, np.int32)
        ms = 9 if bad == [0, 10, 20, 30] else 30                    # last case: lengths above max_seqlen
        out, st = gpu_attn(gpu, q, k, v, cu, max_seqlen=ms, out_fill=0x1234)
        assert st & gpu.DORA_DEV_CU_SEQLENS, bad
        assert np.all(to_host_bits(out) == 0x1234), bad


def test_maximum_sequence_length(gpu):
    """One sequence of DORA_MAX_SEQLEN tokens (86 query chunks, 64 key
    stages), every output row against the oracle."""
    n = gpu.DORA_MAX_SEQLEN
    rng = np.random.default_rng(42)
    q, k, v = qkv(rng, [n], 1, "bf16")
    cu = cu_of([n])
    out, st = gpu_attn(gpu, q, k, v, cu)
    assert st == 0
    want = oracle.varlen_attn_rows(q, k, v, cu, np.arange(n), "bf16")
    mx, mean = assert_attn_close(widen(out), want, "bf16", "len 16384")
    print(f"[attn] len {n} max err {mx:.2e} mean {mean:.2e}", flush=True)


def test_maximum_sequence_length_f32(gpu):
    """The fp32 kernel on one sequence of DORA_MAX_SEQLEN tokens (256 key
    blocks per 64-query part), every output row against the oracle at 1e-5."""
    n = gpu.DORA_MAX_SEQLEN
    rng = np.random.default_rng(44)
    q, k, v = qkv(rng, [n], 1, "f32")
    cu = cu_of([n])
    out, st = gpu_attn(gpu, q, k, v, cu)
    assert st == 0
    want = oracle.varlen_attn_rows(q, k, v, cu, np.arange(n), "f32")
    mx, mean = assert_attn_close(widen(out), want, "f32", "len 16384 f32")
    print(f"[attn] f32 len {n} max err {mx:.2e} mean {mean:.2e}", flush=True)


def test_maximum_sequence_count(gpu):
    """8192 short sequences (the most one plan orders), lengths 1..4, H = 2."""
    rng = np.random.default_rng(43)
    lens = rng.integers(1, 5, 8192)
    q, k, v = qkv(rng, lens, 2, "bf16")
    full_compare(gpu, q, k, v, cu_of(lens), "bf16", what="8192 sequences")
