"""Pins for the oracle's Plackett-Luce deletion by Gumbel-top-k (CPU only).

Training draws exactly k distinct tokens without replacement from a
Plackett-Luce distribution over the selector's scores and keeps the drawing
order for the ordered log-probability of App. A.3, Eq. (app-actor-pl).  The
oracle draws by perturbing the scores with Gumbel noise and taking the k
largest keys in decreasing order.  The checks below fix it from outside:
probabilities of all orders summing to one (brute force), k = 1 reducing to
torch's log_softmax, uniform scores giving (n-k)!/n!, NumPy's lexsort for the
order, select/pack deleting the same set, and sampled frequencies matching
the log-probabilities.
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle


def all_orders_mass(s, k):
    n = s.shape[0]
    orders = list(itertools.permutations(range(1, n), k))
    order = np.array([o for o in orders for _ in [0]], np.int32).reshape(-1)
    cu = (np.arange(len(orders) + 1) * k).astype(np.int32)
    lp, st = oracle.pl_logprob(np.tile(s, (len(orders), 1)), order, cu)
    assert st == 0
    return np.exp(lp).sum()


@pytest.mark.parametrize("n", [2, 4, 6])
def test_probabilities_of_all_orders_sum_to_one(n):
    rng = np.random.default_rng(n)
    s = (rng.standard_normal(n) * 2).astype(np.float32)
    for k in range(0, n):
        assert abs(all_orders_mass(s, k) - 1.0) < 1e-12, k


def test_one_draw_is_log_softmax():
    rng = np.random.default_rng(1)
    B, n = 50, 30
    s = (rng.standard_normal((B, n)) * 3).astype(np.float32)
    order = rng.integers(1, n, B).astype(np.int32)
    lp, st = oracle.pl_logprob(s, order, np.arange(B + 1, dtype=np.int32))
    want = torch.log_softmax(torch.from_numpy(s[:, 1:].astype(np.float64)), dim=1).numpy()
    assert st == 0 and np.allclose(lp, want[np.arange(B), order - 1], rtol=0, atol=1e-12)


def test_uniform_scores_give_falling_factorial():
    n = 197
    for k in (0, 1, 2, 50, 192, 196):
        order = np.arange(1, k + 1, dtype=np.int32)[::-1].copy()
        lp, _ = oracle.pl_logprob(np.full((1, n), 0.7, np.float32), order, np.array([0, k], np.int32))
        want = -sum(math.log(n - 1 - t) for t in range(k))
        assert abs(lp[0] - want) < 1e-9 * max(1.0, abs(want)), k


def test_order_is_lexsort_of_keys():
    rng = np.random.default_rng(2)
    B, n = 300, 64
    s = rng.standard_normal((B, n)).astype(np.float32)
    g = rng.gumbel(size=(B, n)).astype(np.float32)
    s[:20] = np.round(s[:20])                                   # ties in the keys
    g[:20] = 0.0
    k = rng.integers(0, n, B).astype(np.int32)
    order, cu, lp, st = oracle.pl_sample(s, g, k)
    assert st == 0 and np.array_equal(cu[1:], np.cumsum(k))
    key = s + g                                                  # float32 sum, as the oracle forms it
    pos = np.arange(1, n)
    for b in range(B):
        want = pos[np.lexsort((-pos, -key[b, 1:]))][:k[b]]     # larger key first, then higher position
        assert np.array_equal(order[cu[b]:cu[b + 1]], want), b


def test_drawn_set_is_what_select_pack_deletes():
    """Same total order: select/pack with keep-scores -(s + g) and keep = n - k
    keeps exactly the positions the sample did not draw, NaN and ties included."""
    rng = np.random.default_rng(3)
    B, n = 400, 40
    s = rng.choice(np.array([-1.0, 0.0, 0.0, 1.0, 2.5], np.float32), (B, n))
    g = rng.choice(np.array([0.0, 0.5, -0.0], np.float32), (B, n))
    s[::9, 3] = np.nan
    k = rng.integers(0, n, B).astype(np.int32)
    order, cu, _, st = oracle.pl_sample(s, g, k)
    idx, cuk, _, st2 = oracle.select_pack(-(s + g), n - k, np.zeros((B, n, 4), np.float32))
    assert st == st2 == 0
    for b in range(B):
        kept = set(idx[cuk[b]:cuk[b + 1]].tolist())
        assert kept.isdisjoint(order[cu[b]:cu[b + 1]].tolist())
        assert len(kept) + k[b] == n


def test_sampled_orders_follow_their_probabilities():
    """Gumbel-top-k is a Plackett-Luce sampler: the frequency of each full
    order of 3 draws out of 4 visual tokens matches exp(log-probability)."""
    n, k, B = 5, 3, 200000
    s = np.array([0.0, 1.0, -0.5, 0.3, 2.0], np.float32)
    rng = np.random.default_rng(4)
    g = rng.gumbel(size=(B, n)).astype(np.float32)
    order, cu, lp, st = oracle.pl_sample(np.tile(s, (B, 1)), g, np.full(B, k, np.int32))
    assert st == 0
    drawn = order.reshape(B, k)
    orders = list(itertools.permutations(range(1, n), k))
    want_lp, _ = oracle.pl_logprob(np.tile(s, (len(orders), 1)), np.array(orders, np.int32).reshape(-1),
                                   (np.arange(len(orders) + 1) * k).astype(np.int32))
    for o, wl in zip(orders, want_lp):
        cnt = int(np.sum(np.all(drawn == np.array(o), axis=1)))
        p = math.exp(wl)
        assert abs(cnt - B * p) < 5 * math.sqrt(B * p * (1 - p)) + 1, (o, cnt, B * p)
    # each sample's own log-probability is that of its order
    first = {tuple(r): lp[i] for i, r in enumerate(drawn[:2000])}
    for o, wl in zip(orders, want_lp):
        if o in first:
            assert abs(first[o] - wl) < 1e-12
