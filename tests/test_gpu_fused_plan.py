"""GPU checks of dora_select_pack_plan (select/pack with the attention plan
built in the same launch).

The select/pack results must equal the oracle's bit for bit, as for
dora_select_pack; the plan must be the item list the documented queue order
gives (longer sequences first, then lower image index; heads, then query
chunks), and attention executed on it must equal, bit for bit, attention
executed on a plan that dora_varlen_attn_plan made from the same boundaries
(every item is computed on its own, so the queue order cannot change a
result).  Error cases check the device status word and that an empty plan
writes nothing.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import assert_attn_close, to_dev, to_host_bits, widen

pytestmark = pytest.mark.gpu

Q_TILE = 192       # queries per item, as the library's workspace layout defines
HDR_BYTES = 2048   # plan header: sizes, a row of zeros, eight queue counters
ITEMS_OFF = HDR_BYTES
QUEUE_INTS = [64 + 32 * q for q in range(8)]   # one counter per 128-byte line
EXIT_INT = 64 + 32 * 8                          # the exit counter, on the line after them


SUB_QUEUES = 8      # item i is served by sub-queue i % 8


def n_chunks(k):
    return (int(k) + Q_TILE - 1) // Q_TILE


def item_slot(base, groups, ch, gi, c):
    """Slot of chunk c of group gi in a class of `groups` (sequence, head)
    groups of ch chunks starting at `base`: full blocks of 8 groups put a
    group's chunks 8 slots apart (one sub-queue, consecutive tickets), the
    groups past the last full block follow chunk after chunk."""
    full = groups // SUB_QUEUES * SUB_QUEUES
    if gi < full:
        return base + ch * (gi // SUB_QUEUES) * SUB_QUEUES + c * SUB_QUEUES + gi % SUB_QUEUES
    return base + ch * full + (gi - full) * ch + c


def expected_items(keep, H, max_seqlen):
    """Plan items in slot order as int2 pairs (first row, len << 17 | h << 9 | chunk):
    sequences in queue order (longer first, then lower index), grouped in
    classes of equal chunk count, each (sequence, head) group's chunks placed
    by item_slot."""
    keep = np.asarray(keep, np.int64)
    cu = np.concatenate([[0], np.cumsum(keep)])
    order = sorted(range(len(keep)), key=lambda b: (-keep[b], b))
    total = H * sum(n_chunks(k) for k in keep)
    out = np.full((total, 2), -1, np.int64)
    base = 0
    for ch in sorted({n_chunks(k) for k in keep}, reverse=True):
        members = [b for b in order if n_chunks(keep[b]) == ch]
        groups = len(members) * H
        for rank, b in enumerate(members):
            k = int(keep[b])
            for h in range(H):
                for c in range(ch):
                    out[item_slot(base, groups, ch, rank * H + h, c)] = (int(cu[b]), (k << 17) | (h << 9) | c)
        base += groups * ch
    assert np.all(out >= 0)
    return out


def assert_groups_share_a_subqueue(items):
    """Every (sequence, head) group's chunks sit in one sub-queue at
    consecutive tickets (slots 8 apart), except at most 7 groups per class
    past its last full block of 8, whose chunks are adjacent."""
    slots = {}
    for i, (row, y) in enumerate(items.tolist()):
        slots.setdefault((row, (y >> 9) & 0xFF), []).append((y & 0x1FF, i))
    tail = {}
    for (row, h), v in slots.items():
        idx = [i for _, i in sorted(v)]
        if len(idx) == 1:
            continue
        steps = set(np.diff(idx).tolist())
        assert steps in ({SUB_QUEUES}, {1}), (row, h, idx)
        if steps == {1}:
            tail[len(idx)] = tail.get(len(idx), 0) + 1
    assert all(n < SUB_QUEUES for n in tail.values()), tail


def read_plan(ws):
    hdr = ws[:HDR_BYTES].view(torch.int32).cpu().numpy()
    n = int(hdr[2])
    items = ws[ITEMS_OFF:ITEMS_OFF + 8 * n].view(torch.int32).cpu().numpy().astype(np.int64).reshape(-1, 2)
    return hdr, n, items


def fused(dora, r, H, max_seqlen, total, cu_in=None, N=None, ws=None, packed_fill=None):
    B = len(r.keep)
    ts = to_dev(np.ascontiguousarray(r.scores))
    tt = to_dev(r.tokens)
    cap = max(int(np.sum(np.maximum(r.keep, 0))), 1)
    ws = dora.new_workspace(B, H, max_seqlen) if ws is None else ws
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx, cu, packed, _ = dora.dora_select_pack_plan(
        ts, to_dev(r.keep.astype(np.int32)), tt, H, max_seqlen, total, ws,
        cu_in=None if cu_in is None else to_dev(cu_in), N=N, cap_rows=cap, dev_status=st)
    torch.cuda.synchronize()
    return idx, cu, packed, ws, int(st.item())


@pytest.mark.parametrize("name", ["deit_b_bf16", "vit_b384_skew_bf16", "deit_tiny_fp32"])
def test_fused_plan_matches_oracle_and_separate_plan(gpu, name):
    w = W.WORKLOADS[name]
    r = W.generate(w, parts=("keep", "scores", "tokens", "qkv"))[0]
    total = r.total_keep
    print(f"[fused] {name} B={w.B} H={w.H} sum_keep={total}", flush=True)
    idx, cu, packed, ws, st = fused(gpu, r, w.H, w.N, total)
    assert st == 0
    idx_o, cu_o, packed_o, st_o = oracle.select_pack(r.scores, r.keep, r.tokens)
    assert st_o == 0
    assert np.array_equal(cu.cpu().numpy(), cu_o)
    assert np.array_equal(idx[:total].cpu().numpy(), idx_o)
    assert np.array_equal(to_host_bits(packed[:total]), packed_o)

    hdr, n, items = read_plan(ws)
    assert np.array_equal(items, expected_items(r.keep, w.H, w.N))
    assert_groups_share_a_subqueue(items)

    q, k, v = (to_dev(a) for a in (r.q, r.k, r.v))
    st_t = torch.zeros(1, dtype=torch.int32, device="cuda")
    out_fused = gpu.dora_varlen_attn_execute(q, k, v, cu, w.N, ws, dev_status=st_t)
    ws2 = gpu.new_workspace(w.B, w.H, w.N)
    gpu.dora_varlen_attn_plan(cu, w.H, w.N, total, ws2, st_t)
    out_sep = gpu.dora_varlen_attn_execute(q, k, v, cu, w.N, ws2, dev_status=st_t)
    torch.cuda.synchronize()
    assert int(st_t.item()) == 0
    assert np.array_equal(to_host_bits(out_fused), to_host_bits(out_sep))
    # the plan kernel's plan: the same items, the same class and sub-queue placement
    _, n2, items2 = read_plan(ws2)
    assert n2 == n and sorted(map(tuple, items2.tolist())) == sorted(map(tuple, items.tolist()))
    assert np.all(np.diff([n_chunks(k) for k in (items2[:, 1] >> 17)]) <= 0)
    assert_groups_share_a_subqueue(items2)
    # and against the oracle, every element
    want = oracle.varlen_attn(r.q, r.k, r.v, cu_o, w.dtype)
    assert_attn_close(widen(out_fused), want, w.dtype, name)


def test_fused_plan_on_cascade_round(gpu):
    """Packed input (a later pruning round): cu_in from the previous round."""
    w = W.WORKLOADS["vit_l_cascade_bf16"]
    rounds = W.generate(w, batch=48, parts=("keep", "scores", "tokens"))
    r0, r1 = rounds[0], rounds[1]
    _, cu0, packed0, _, st = fused(gpu, r0, w.H, w.N, r0.total_keep)
    assert st == 0
    r1.tokens = to_host_bits(packed0[:r0.total_keep])
    cu_in = cu0.cpu().numpy()
    idx, cu, packed, ws, st = fused(gpu, r1, w.H, w.N, r1.total_keep, cu_in=cu_in, N=w.N)
    assert st == 0
    idx_o, cu_o, packed_o, st_o = oracle.select_pack(r1.scores, r1.keep, r1.tokens, cu_in=cu_in, N=w.N)
    assert st_o == 0
    assert np.array_equal(cu.cpu().numpy(), cu_o)
    assert np.array_equal(idx[:r1.total_keep].cpu().numpy(), idx_o)
    assert np.array_equal(to_host_bits(packed[:r1.total_keep]), packed_o)
    _, n, items = read_plan(ws)
    assert np.array_equal(items, expected_items(r1.keep, w.H, w.N))


def test_fused_plan_replaces_a_stale_plan(gpu):
    """A second fused call on the same workspace fully replaces the first plan."""
    w = W.WORKLOADS["deit_s_bf16"]
    rs = [W.generate(w, seed=s, batch=16, parts=("keep", "scores", "tokens"))[0] for s in (11, 12)]
    ws = gpu.new_workspace(16, w.H, w.N)
    for r in rs:
        _, _, _, ws, st = fused(gpu, r, w.H, w.N, r.total_keep, ws=ws)
        assert st == 0
        hdr, n, items = read_plan(ws)
        assert n == len(expected_items(r.keep, w.H, w.N))
        assert np.array_equal(items, expected_items(r.keep, w.H, w.N))
        assert int(hdr[EXIT_INT]) == 0 and all(int(hdr[i]) == 0 for i in QUEUE_INTS)   # counters reset
        assert np.all(hdr[32:64] == 0)                         # the row of zeros


@pytest.mark.parametrize("case", ["keep_above_max_seqlen", "keep_zero", "sum_above_total"])
def test_fused_plan_errors_leave_an_empty_plan(gpu, case):
    w = W.WORKLOADS["deit_s_bf16"]
    r = W.generate(w, seed=3, batch=8, parts=("keep", "scores", "tokens", "qkv"))[0]
    max_seqlen, total = w.N, r.total_keep
    want_bits = gpu.DORA_DEV_CU_SEQLENS
    if case == "keep_above_max_seqlen":
        max_seqlen = int(r.keep.max()) - 1
    elif case == "keep_zero":
        r.keep = r.keep.copy()
        r.keep[5] = 0
        want_bits |= gpu.DORA_DEV_KEEP_RANGE
    else:
        total = r.total_keep - 1
    print(f"[fused] error case {case}", flush=True)
    _, cu, _, ws, st = fused(gpu, r, w.H, max_seqlen, total)
    assert st & want_bits == want_bits
    hdr, n, _ = read_plan(ws)
    assert n == 0
    rows = max(total, 1)
    q = to_dev(np.zeros((rows, w.H, 64), np.uint16))
    out = torch.full_like(q, 0).view(torch.int16).fill_(0x1234).view(torch.bfloat16)
    st_t = torch.zeros(1, dtype=torch.int32, device="cuda")
    gpu.dora_varlen_attn_execute(q, q, q, cu, max_seqlen, ws, out=out, dev_status=st_t)
    torch.cuda.synchronize()
    assert int(st_t.item()) == 0
    assert np.all(to_host_bits(out) == 0x1234)


def test_fused_plan_large_batch(gpu):
    """8192 images: the keep counts are scanned first and the plan kernel
    builds the plan from cu_seqlens.  Select/pack stays bit-exact; the plan
    holds exactly the documented items, longer sequences first (equal
    lengths in any order); attention on it equals attention on a separately
    made plan bit for bit, and the oracle on every element."""
    rng = np.random.default_rng(8192)
    B, N, H = 8192, 64, 2

    class R:
        pass
    r = R()
    r.keep = rng.integers(1, N + 1, size=B).astype(np.int32)
    r.scores = rng.standard_normal((B, N)).astype(np.float32)
    r.tokens = rng.integers(0, 2 ** 16, size=(B, N, 8)).astype(np.uint16)
    total = int(r.keep.sum())
    idx, cu, packed, ws, st = fused(gpu, r, H, N, total)
    assert st == 0
    idx_o, cu_o, packed_o, st_o = oracle.select_pack(r.scores, r.keep, r.tokens)
    assert st_o == 0
    assert np.array_equal(cu.cpu().numpy(), cu_o)
    assert np.array_equal(idx[:total].cpu().numpy(), idx_o)
    assert np.array_equal(to_host_bits(packed[:total]), packed_o)
    hdr, n, items = read_plan(ws)
    want = expected_items(r.keep, H, N)
    assert n == len(want)
    chunks = [n_chunks(k) for k in (items[:, 1] >> 17)]
    assert np.all(np.diff(chunks) <= 0)                       # classes of equal chunk count, longest first
    assert sorted(map(tuple, items.tolist())) == sorted(map(tuple, want.tolist()))
    assert_groups_share_a_subqueue(items)
    q, k, v = W.random_qkv(rng, r.keep, H, "bf16")
    tq, tk, tv = to_dev(q), to_dev(k), to_dev(v)
    st_t = torch.zeros(1, dtype=torch.int32, device="cuda")
    out_fused = gpu.dora_varlen_attn_execute(tq, tk, tv, cu, N, ws, dev_status=st_t)
    ws2 = gpu.new_workspace(B, H, N)
    gpu.dora_varlen_attn_plan(cu, H, N, total, ws2, st_t)
    out_sep = gpu.dora_varlen_attn_execute(tq, tk, tv, cu, N, ws2, dev_status=st_t)
    torch.cuda.synchronize()
    assert int(st_t.item()) == 0
    assert np.array_equal(to_host_bits(out_fused), to_host_bits(out_sep))
    assert_attn_close(widen(out_fused), oracle.varlen_attn(q, k, v, cu_o, "bf16"), "bf16", "8192 images")


@pytest.mark.parametrize("case", ["keep_zero", "keep_above_max_seqlen"])
def test_fused_plan_large_batch_errors(gpu, case):
    """The same error contract past 2048 images: an empty plan and the bits."""
    rng = np.random.default_rng(4099)
    B, N, H = 4096, 40, 2

    class R:
        pass
    r = R()
    r.keep = np.full(B, 10, np.int32)
    r.scores = rng.standard_normal((B, N)).astype(np.float32)
    r.tokens = rng.integers(0, 2 ** 16, size=(B, N, 8)).astype(np.uint16)
    max_seqlen, want_bits = N, gpu.DORA_DEV_CU_SEQLENS
    if case == "keep_zero":
        r.keep[2222] = 0
        want_bits |= gpu.DORA_DEV_KEEP_RANGE
    else:
        max_seqlen = 9
    _, _, _, ws, st = fused(gpu, r, H, max_seqlen, int(r.keep.sum()))
    assert st & want_bits == want_bits
    _, n, _ = read_plan(ws)
    assert n == 0
