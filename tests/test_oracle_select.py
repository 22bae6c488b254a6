"""Pins for the oracle's selection, boundaries and packing (CPU only).

The paper fixes: CLS always kept, the keep-1 highest-scoring visual tokens
kept (Sec. 3.2 "Sampling and deployment"; App. A.3), survivor order preserved
(Sec. 3.1, Eq. (1)), images packed with explicit boundaries (Sec. 3.5).
Ties, NaN and signed zero follow the stated readings (lower position wins,
NaN lowest, -0 == +0).  Each check below computes the expected answer some
other way than the oracle's sort.
"""
import itertools
import json
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def brute_keep_masks(scores: np.ndarray, keep: np.ndarray) -> np.ndarray:
    """Counting definition: visual position j survives iff fewer than keep-1
    visual positions are strictly preferred to it.  i is preferred to j when
    i is a number and j is NaN, or both numbers and s_i > s_j, or they are
    equal (or both NaN) and i < j.  Returns bool [B, n]; CLS column True."""
    B, n = scores.shape
    s = scores[:, 1:].astype(np.float64)
    isn = np.isnan(s)
    val = np.where(isn, 0.0, s)
    pos = np.arange(1, n)
    a_num, b_num = ~isn[:, :, None], ~isn[:, None, :]
    a_val, b_val = val[:, :, None], val[:, None, :]
    earlier = (pos[:, None] < pos[None, :])[None]
    same = (a_num & b_num & (a_val == b_val)) | (~a_num & ~b_num)
    pref = (a_num & ~b_num) | (a_num & b_num & (a_val > b_val)) | (same & earlier)
    beaten_by = pref.sum(axis=1)                       # [B, n-1] for each j
    out = np.zeros((B, n), dtype=bool)
    out[:, 0] = True
    out[:, 1:] = beaten_by < (keep[:, None] - 1)
    return out


def masks_from_idx(idx, cu, B, n):
    m = np.zeros((B, n), dtype=bool)
    for b in range(B):
        m[b, idx[cu[b]:cu[b + 1]]] = True
    return m


def run(scores, keep, C=2, dtype=np.float32, seed=0):
    B, n = scores.shape
    tokens = np.random.default_rng(seed).standard_normal((B, n, C)).astype(dtype)
    idx, cu, packed, st = oracle.select_pack(scores, keep, tokens)
    assert st == 0
    return idx, cu, packed, tokens


VALUES = [-np.inf, -1.0, -0.0, 0.0, 1.0, np.inf, np.nan]


def test_exhaustive_tiny_against_counting_definition():
    # n = 6: CLS + 5 visual tokens, each from 7 special values, every keep count.
    pats = np.array(list(itertools.product(VALUES, repeat=5)), dtype=np.float32)
    P = pats.shape[0]
    n = 6
    scores = np.concatenate([np.full((P, 1), 3.0, np.float32), pats], axis=1)
    scores = np.repeat(scores, n, axis=0)
    keep = np.tile(np.arange(1, n + 1, dtype=np.int32), P)
    idx, cu, packed, tokens = run(scores, keep)
    got = masks_from_idx(idx, cu, scores.shape[0], n)
    want = brute_keep_masks(scores, keep)
    assert np.array_equal(got, want)


def test_exhaustive_heavy_ties_n8():
    rng = np.random.default_rng(11)
    n = 8
    B = 4000
    scores = rng.choice(np.array([-2.0, -0.0, 0.0, 0.5, np.nan], np.float32), size=(B, n))
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    idx, cu, _, _ = run(scores, keep)
    assert np.array_equal(masks_from_idx(idx, cu, B, n), brute_keep_masks(scores, keep))


def test_matches_numpy_stable_argsort_without_nan():
    rng = np.random.default_rng(5)
    B, n = 64, 197
    scores = rng.standard_normal((B, n)).astype(np.float32)
    scores[:, 50:60] = 0.25                            # a block of exact ties
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    idx, cu, _, _ = run(scores, keep)
    for b in range(B):
        order = np.argsort(-scores[b, 1:], kind="stable") + 1
        want = np.sort(np.concatenate([[0], order[: keep[b] - 1]]))
        assert np.array_equal(idx[cu[b]:cu[b + 1]], want)


def test_invariants_random():
    rng = np.random.default_rng(7)
    B, n = 128, 197
    scores = rng.standard_normal((B, n)).astype(np.float32)
    scores[rng.random((B, n)) < 0.05] = np.nan
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    idx, cu, _, _ = run(scores, keep)
    for b in range(B):
        seg = idx[cu[b]:cu[b + 1]]
        assert len(seg) == keep[b] and seg[0] == 0
        assert np.all(np.diff(seg) > 0) and seg[-1] < n
        kept = set(seg.tolist()) - {0}
        dropped = set(range(1, n)) - kept
        for i in kept:
            for j in dropped:
                si, sj = scores[b, i], scores[b, j]
                ok = (not np.isnan(si) and np.isnan(sj)) or (si > sj) or \
                     ((si == sj or (np.isnan(si) and np.isnan(sj))) and i < j)
                assert ok, (b, i, j, si, sj)


def test_special_cases():
    rng = np.random.default_rng(3)
    n = 33
    s = rng.standard_normal((1, n)).astype(np.float32)
    idx, _, _, _ = run(s, np.array([n], np.int32))
    assert np.array_equal(idx, np.arange(n))                       # keep all -> identity
    idx, _, _, _ = run(s, np.array([1], np.int32))
    assert np.array_equal(idx, [0])                                # keep one -> CLS
    const = np.full((1, n), 0.7, np.float32)
    idx, _, _, _ = run(const, np.array([10], np.int32))
    assert np.array_equal(idx, np.arange(10))                      # all equal -> prefix
    dec = np.linspace(5, -5, n).astype(np.float32)[None]
    idx, _, _, _ = run(dec, np.array([7], np.int32))
    assert np.array_equal(idx, np.arange(7))                       # falling -> prefix
    inc = np.linspace(-5, 5, n).astype(np.float32)[None]
    idx, _, _, _ = run(inc, np.array([7], np.int32))
    assert np.array_equal(idx, np.concatenate([[0], np.arange(n - 6, n)]))   # rising -> tail


def test_cls_score_is_ignored():
    rng = np.random.default_rng(4)
    s = rng.standard_normal((2, 20)).astype(np.float32)
    s[0, 0], s[1, 0] = -np.inf, np.inf
    s[1, 1:] = s[0, 1:]
    idx, cu, _, _ = run(s, np.array([5, 5], np.int32))
    assert np.array_equal(idx[0:5], idx[5:10])


def test_golden_hand_cases():
    cases = json.load(open(os.path.join(GOLDEN, "select_hand.json")))["cases"]
    for c in cases:
        s = np.array([[float(x) for x in c["scores"]]], np.float32)
        idx, cu, _, _ = run(s, np.array([c["keep"]], np.int32))
        assert idx.tolist() == c["expected"], c["why"]


def test_boundaries_and_pack_closed_form():
    rng = np.random.default_rng(9)
    B, n, C = 17, 41, 24
    scores = rng.standard_normal((B, n)).astype(np.float32)
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    tokens = rng.integers(0, 2 ** 16, size=(B, n, C)).astype(np.uint16)
    idx, cu, packed, st = oracle.select_pack(scores, keep, tokens)
    assert st == 0
    assert cu[0] == 0 and np.array_equal(cu[1:], np.cumsum(keep))
    for b in range(B):
        for r in range(keep[b]):
            assert np.array_equal(packed[cu[b] + r], tokens[b, idx[cu[b] + r]])


def test_packed_input_equals_dense_input():
    """A cascaded round on packed input equals the same selection on dense rows."""
    rng = np.random.default_rng(12)
    B, C = 9, 8
    lens = rng.integers(1, 30, size=B).astype(np.int32)
    cu_in = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    scores = rng.standard_normal(int(cu_in[-1])).astype(np.float32)
    tokens = rng.standard_normal((int(cu_in[-1]), C)).astype(np.float32)
    keep = np.array([rng.integers(1, l + 1) for l in lens], np.int32)
    idx, cu, packed, st = oracle.select_pack(scores, keep, tokens, cu_in=cu_in)
    assert st == 0
    for b in range(B):
        s = scores[cu_in[b]:cu_in[b + 1]][None]
        t = tokens[cu_in[b]:cu_in[b + 1]][None]
        i1, c1, p1, st1 = oracle.select_pack(s, keep[b:b + 1], t)
        assert st1 == 0
        assert np.array_equal(idx[cu[b]:cu[b + 1]], i1)
        assert np.array_equal(packed[cu[b]:cu[b + 1]], p1)


def test_error_codes():
    s = np.zeros((2, 5), np.float32)
    t = np.zeros((2, 5, 2), np.float32)
    assert oracle.select_pack(s, np.array([0, 3], np.int32), t)[3] == oracle.BAD_KEEP
    assert oracle.select_pack(s, np.array([6, 3], np.int32), t)[3] == oracle.BAD_KEEP
    bad_cu = np.array([0, 7, 5], np.int32)
    st = oracle.select_pack(np.zeros(7, np.float32), np.array([1, 1], np.int32),
                            np.zeros((7, 2), np.float32), cu_in=bad_cu, N=7)[3]
    assert st & oracle.BAD_SEGMENTS
