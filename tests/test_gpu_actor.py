"""GPU parity for the deterministic actor decode (dora_actor_gate,
dora_actor_decode): bit-exact against the oracle.

Gate decisions, the gate-on numbering and list, keep counts and negated
scores are integer / bit work, compared exactly.  Covers batch sizes around
the gate kernel's 1024-image chunks, ties, NaN and infinite logits and
probabilities, packed input with short and invalid segments, too few logit
rows, M = 126 (DINOv2-B/14's grid), and the whole chain gate -> decode ->
select/pack -> attention on the device with no host synchronisation.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import assert_attn_close, to_dev, to_host_bits, widen

pytestmark = pytest.mark.gpu


def special_probs(rng, B):
    p = rng.random(B).astype(np.float32)
    pick = rng.random(B)
    p[pick < 0.05] = 0.5
    p[(pick >= 0.05) & (pick < 0.08)] = np.nextafter(np.float32(0.5), np.float32(0))
    p[(pick >= 0.08) & (pick < 0.10)] = np.nan
    return p


def tricky_logits(rng, rows, M):
    x = rng.choice(np.array([-1.0, 0.0, 0.5, 2.0], np.float32), (rows, M))
    x[::3] = rng.standard_normal((len(x[::3]), M)).astype(np.float32)
    sp = rng.random((rows, M))
    x[sp < 0.01] = np.nan
    x[(sp > 0.5) & (sp < 0.51)] = np.inf
    x[(sp > 0.6) & (sp < 0.61)] = -np.inf
    return x


def run_gate(dora, p, M, N, cu=None):
    on_rank, on_list, n_on, st = dora.dora_actor_gate(to_dev(p), M, N, cu_in=None if cu is None else to_dev(cu))
    torch.cuda.synchronize()
    return on_rank.cpu().numpy(), on_list.cpu().numpy(), int(n_on.item()), int(st.item())


@pytest.mark.parametrize("B", [1, 7, 256, 1023, 1024, 1025, 5000])
def test_gate_and_decode_dense(gpu, B):
    rng = np.random.default_rng(B)
    N, M = 197, 96
    p = special_probs(rng, B)
    print(f"[actor] dense B={B}", flush=True)
    r_g, l_g, n_g, st = run_gate(gpu, p, M, N)
    r_o, l_o, n_o = oracle.actor_gate(p, np.full(B, N, np.int32), M)
    assert st == 0 and n_g == n_o
    assert np.array_equal(r_g, r_o) and np.array_equal(l_g, l_o)
    logits = tricky_logits(rng, max(n_o, 1), M)
    removal = rng.standard_normal((B, N)).astype(np.float32)
    removal.flat[rng.integers(0, B * N, 50)] = np.nan
    keep, ks, st = gpu.dora_actor_decode(to_dev(logits), to_dev(r_g), N, removal_scores=to_dev(removal))
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert np.array_equal(keep.cpu().numpy(), oracle.actor_budget(logits, np.full(B, N, np.int32), r_o))
    assert np.array_equal(ks.cpu().numpy().view(np.uint32), oracle.negate(removal).view(np.uint32))


def test_packed_segments_short_and_invalid(gpu):
    rng = np.random.default_rng(21)
    B, N, M = 700, 197, 96
    n = rng.integers(1, N + 1, B).astype(np.int32)
    n[:40] = np.arange(1, 41)                                      # every short count, gate never legal below 6
    cu = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    p = special_probs(rng, B)
    r_g, l_g, n_g, st = run_gate(gpu, p, M, N, cu)
    r_o, l_o, n_o = oracle.actor_gate(p, n, M)
    assert st == 0 and n_g == n_o and np.array_equal(r_g, r_o) and np.array_equal(l_g, l_o)
    logits = tricky_logits(rng, n_o + 5, M)
    removal = rng.standard_normal(int(cu[-1]) + 3).astype(np.float32)  # a few rows past the last segment
    keep, ks, st = gpu.dora_actor_decode(to_dev(logits), to_dev(r_g), N, removal_scores=to_dev(removal),
                                         cu_in=to_dev(cu))
    torch.cuda.synchronize()
    assert int(st.item()) == 0
    assert np.array_equal(keep.cpu().numpy(), oracle.actor_budget(logits, n, r_o))
    assert np.array_equal(ks.cpu().numpy().view(np.uint32), oracle.negate(removal).view(np.uint32))
    # invalid segments: gate closed, keep 0, DORA_DEV_CU_IN from both kernels
    bad = cu.copy()
    bad[5] = bad[4]                                                # empty segment 4
    bad[9] = bad[8] + N + 1                                        # segment 8 longer than N
    r_b, _, _, st = run_gate(gpu, np.ones(B, np.float32), M, N, bad)
    assert st & gpu.DORA_DEV_CU_IN and r_b[4] == -1 and r_b[8] == -1
    keep, _, st = gpu.dora_actor_decode(to_dev(logits), to_dev(r_g), N, cu_in=to_dev(bad))
    torch.cuda.synchronize()
    k = keep.cpu().numpy()
    assert int(st.item()) & gpu.DORA_DEV_CU_IN and k[4] == 0 and k[8] == 0


def test_missing_logit_rows_leave_images_unpruned(gpu):
    rng = np.random.default_rng(22)
    B, N, M = 64, 197, 96
    p = np.ones(B, np.float32)
    r_g, _, n_g, _ = run_gate(gpu, p, M, N)
    assert n_g == B
    logits = rng.standard_normal((40, M)).astype(np.float32)     # rows for the first 40 gate-on images only
    keep, _, st = gpu.dora_actor_decode(to_dev(logits), to_dev(r_g), N)
    torch.cuda.synchronize()
    assert int(st.item()) & gpu.DORA_DEV_ACTOR
    k = keep.cpu().numpy()
    want = oracle.actor_budget(np.concatenate([logits, np.zeros((B - 40, M), np.float32)]), np.full(B, N, np.int32),
                               r_g)
    assert np.array_equal(k[:40], want[:40]) and np.all(k[40:] == N)


def test_dinov2_grid_and_in_place_negation(gpu):
    rng = np.random.default_rng(23)
    B, N, M = 300, 257, 126
    p = special_probs(rng, B)
    r_g, _, n_g, _ = run_gate(gpu, p, M, N)
    logits = tricky_logits(rng, max(n_g, 1), M)
    removal = rng.standard_normal((B, N)).astype(np.float32)
    t = to_dev(removal)
    keep, ks, st = gpu.dora_actor_decode(to_dev(logits), to_dev(r_g), N, removal_scores=t, scores_out=t)
    torch.cuda.synchronize()
    assert int(st.item()) == 0 and ks.data_ptr() == t.data_ptr()
    r_o, _, _ = oracle.actor_gate(p, np.full(B, N, np.int32), M)
    assert np.array_equal(keep.cpu().numpy(), oracle.actor_budget(logits, np.full(B, N, np.int32), r_o))
    assert np.array_equal(t.cpu().numpy().view(np.uint32), oracle.negate(removal).view(np.uint32))


def test_chain_on_device_matches_the_oracle_chain(gpu):
    """gate -> decode -> select/pack + plan -> attention with no host sync in
    between, against the oracle's chain, on the DeiT-B workload shape."""
    w = W.WORKLOADS["deit_b_bf16"]
    M = W.budget_outputs(w)
    p, logits, removal = W.actor_outputs(w)
    r = W.generate(w, parts=("keep", "tokens"))[0]
    # oracle chain
    n = np.full(w.B, w.N, np.int32)
    r_o, _, n_o = oracle.actor_gate(p, n, M)
    keep_o = oracle.actor_budget(logits[:max(n_o, 1)], n, r_o)
    ks_o = oracle.negate(removal)
    idx_o, cu_o, packed_o, st_o = oracle.select_pack(ks_o, keep_o, r.tokens)
    assert st_o == 0
    tot = int(keep_o.sum())
    rng = np.random.default_rng(24)
    q, k, v = W.random_qkv(rng, np.diff(cu_o), w.H, "bf16")
    # device chain: the only host reads come after the last launch
    on_rank, on_list, n_on, st = gpu.dora_actor_gate(to_dev(p), M, w.N)
    keep, ks, _ = gpu.dora_actor_decode(to_dev(logits), on_rank, w.N, removal_scores=to_dev(removal),
                                        dev_status=st)
    cap = w.B * w.N
    ws = gpu.new_workspace(w.B, w.H, w.N)
    tq, tk, tv = to_dev(q), to_dev(k), to_dev(v)
    idx, cu, packed, _ = gpu.dora_select_pack_plan(ks, keep, to_dev(r.tokens), w.H, w.N, tot, ws, cap_rows=cap,
                                                   dev_status=st)
    out = gpu.dora_varlen_attn_execute(tq, tk, tv, cu, w.N, ws, dev_status=st)
    torch.cuda.synchronize()
    assert int(st.item()) == 0 and int(n_on.item()) == n_o
    assert np.array_equal(keep.cpu().numpy(), keep_o) and np.array_equal(cu.cpu().numpy(), cu_o)
    assert np.array_equal(idx[:tot].cpu().numpy(), idx_o)
    assert np.array_equal(to_host_bits(packed[:tot]), packed_o)
    got = widen(out)
    want = oracle.varlen_attn(q, k, v, cu_o, "bf16")
    assert_attn_close(got, want, "bf16", "chain")
    print(f"[actor] chain: {n_o} of {w.B} gates open, sum keep {tot}", flush=True)
