"""Pins for the oracle's decode of the deterministic actor (CPU only).

At deployment the gate opens when its probability is at least 0.5 and some
budget is legal, the budget is the legal one with the largest logit, and the
selector removes the k highest-scoring visual tokens (Sec. 3.2 "Sampling and
deployment"; App. A.3).  The grid is {2, 4, ..., N0 - 4} with M = (N0 - 4)/2
outputs and the legal budgets leave at least four visual tokens (App. A.2,
Eq. (legal budgets), Table 3).  Each check gets the expected answer another
way: the paper's table, the set definitions enumerated in Python, torch's
argmax over masked logits, NumPy's compaction and negation.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def legal_set(n_tok, M):
    """B_l from the definitions: the grid {2, ..., 2M} cut at N_l - 4, N_l = n_tok - 1."""
    grid = set(range(2, 2 * M + 1, 2))
    return {k for k in grid if k <= (n_tok - 1) - 4}


@pytest.mark.parametrize("bb", json.load(open(os.path.join(GOLDEN, "actor_budget_grids.json")))["backbones"],
                         ids=lambda b: b["name"])
def test_table3_budget_grids(bb):
    """An unpruned image (N_l = N0) reaches exactly the printed grid B_0."""
    N0, M = bb["N0"], bb["M"]
    assert M == (N0 - 4) // 2
    n_tok = np.full(M, N0 + 1, np.int32)                  # one image per budget output, CLS included
    on_rank, _, n_on = oracle.actor_gate(np.ones(M, np.float32), n_tok, M)
    assert n_on == M
    keep = oracle.actor_budget(np.eye(M, dtype=np.float32), n_tok, on_rank)   # image m: logit 1 at output m
    budgets = n_tok - keep
    assert list(budgets) == list(range(bb["B0_first"], bb["B0_last"] + 1, 2))


@pytest.mark.parametrize("M", [96, 126, 3])
def test_gate_and_reachable_budgets_match_the_set_definitions(M):
    """For every token count, the gate opens iff B_l is non-empty, and the
    budgets a one-hot logit can select are exactly B_l."""
    for n in range(1, 2 * M + 12):
        on_rank, _, n_on = oracle.actor_gate(np.ones(1, np.float32), np.array([n], np.int32), M)
        legal = legal_set(n, M)
        assert (n_on == 1) == bool(legal), n
        if not legal:
            continue
        keep = oracle.actor_budget(np.eye(M, dtype=np.float32), np.full(M, n, np.int32), np.arange(M, dtype=np.int32))
        assert set((n - keep).tolist()) == legal, n
        assert np.all(keep - 1 >= 4)                      # at least four visual tokens survive


def test_budget_is_torch_argmax_over_masked_logits():
    rng = np.random.default_rng(1)
    B, M = 4000, 96
    n_tok = rng.integers(1, 198, B).astype(np.int32)
    n_tok[:50] = 197
    logits = rng.choice(np.array([-1.0, 0.0, 0.5, 2.0], np.float32), (B, M))      # many ties
    logits[::7] = rng.standard_normal((len(logits[::7]), M)).astype(np.float32)
    sp = rng.random((B, M))
    logits[sp < 0.01] = np.nan
    logits[(sp > 0.5) & (sp < 0.51)] = np.inf
    logits[(sp > 0.6) & (sp < 0.61)] = -np.inf
    logits[3] = -np.inf
    on_rank, _, _ = oracle.actor_gate(np.ones(B, np.float32), n_tok, M)
    keep = oracle.actor_budget(logits, n_tok, on_rank)
    t = torch.from_numpy(logits[np.maximum(on_rank, 0)])            # image b's row is on_rank[b]
    legal = torch.arange(M)[None, :] < torch.from_numpy(np.array([len(legal_set(n, M)) for n in n_tok]))[:, None]
    m = torch.argmax(t.masked_fill(~legal, -np.inf), dim=1).numpy()
    on = on_rank >= 0
    assert np.array_equal(keep[on], (n_tok - 2 * (m + 1))[on])
    assert np.array_equal(keep[~on], n_tok[~on])


def test_gate_threshold_and_special_probabilities():
    p = np.array([0.5, np.nextafter(np.float32(0.5), np.float32(0)), np.nan, np.inf, -np.inf, 1.0, 0.0],
                 np.float32)
    on_rank, on_list, n_on = oracle.actor_gate(p, np.full(len(p), 197, np.int32), 96)
    assert list(on_rank) == [0, -1, -1, 1, -1, 2, -1]
    assert list(on_list) == [0, 3, 5, -1, -1, -1, -1] and n_on == 3


def test_compaction_is_numpy_flatnonzero():
    rng = np.random.default_rng(2)
    B = 5000
    p = rng.random(B).astype(np.float32)
    n_tok = rng.integers(1, 30, B).astype(np.int32)
    on_rank, on_list, n_on = oracle.actor_gate(p, n_tok, 96)
    on = (p >= 0.5) & np.array([bool(legal_set(n, 96)) for n in n_tok])
    want = np.flatnonzero(on)
    assert n_on == len(want)
    assert np.array_equal(on_list[:n_on], want) and np.all(on_list[n_on:] == -1)
    assert np.array_equal(on_rank[on], np.arange(n_on)) and np.all(on_rank[~on] == -1)


def test_negate_is_numpy_negative_bitwise():
    rng = np.random.default_rng(3)
    s = rng.integers(0, 2 ** 32, 100000, dtype=np.uint32).view(np.float32)   # every class of value
    got = oracle.negate(s)
    assert np.array_equal(got.view(np.uint32), np.negative(s).view(np.uint32))


def test_decode_then_select_removes_the_highest_removal_scores():
    """End to end on the oracle: after the decode, select/pack removes exactly
    the k highest removal scores of each gate-on image (lowest position kept
    on ties, since -s ties where s ties) and nothing of a gate-off image."""
    rng = np.random.default_rng(4)
    B, N, M = 40, 197, 96
    p = rng.random(B).astype(np.float32)
    n_tok = np.full(B, N, np.int32)
    on_rank, _, n_on = oracle.actor_gate(p, n_tok, M)
    logits = rng.standard_normal((B, M)).astype(np.float32)
    keep = oracle.actor_budget(logits, n_tok, on_rank)
    s = rng.standard_normal((B, N)).astype(np.float32)
    idx, cu, _, st = oracle.select_pack(oracle.negate(s), keep, np.zeros((B, N, 4), np.float32))
    assert st == 0
    for b in range(B):
        kept = set(idx[cu[b]:cu[b + 1]].tolist())
        removed = set(range(N)) - kept
        k = N - keep[b]
        assert 0 in kept and len(removed) == k
        if on_rank[b] < 0:
            assert k == 0
        else:
            order = sorted(range(1, N), key=lambda j: (-s[b, j], -j))
            assert removed == set(order[:k])
