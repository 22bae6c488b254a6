"""The seeded generators produce the stated shapes and distributions."""
import numpy as np

import workloads as W


def test_reproducible_and_shapes():
    w = W.WORKLOADS["deit_s_bf16"]
    a, b = W.generate(w)[0], W.generate(w)[0]
    assert np.array_equal(a.keep, b.keep) and np.array_equal(a.q, b.q)
    assert a.scores.shape == (64, 197) and a.scores.dtype == np.float32
    assert a.tokens.shape == (64, 197, 384) and a.tokens.dtype == np.uint16
    assert a.q.shape == (a.total_keep, 6, 64)
    assert np.all((a.keep >= np.rint(0.4 * 197)) & (a.keep <= 197))


def test_keep_rules_small_batches():
    t = W.generate(W.WORKLOADS["deit_tiny_fp32"])[0]
    assert t.q.dtype == np.float32 and np.all((t.keep >= 20) & (t.keep <= 197))
    wb = W.WORKLOADS["deit_b_bf16"]
    keep = W._draw_keep(W.Workload(wb.name, wb.seed, 20000, wb.N, wb.H, wb.dtype, wb.keep_rule),
                        np.random.default_rng(0), np.full(20000, 197))
    r = keep / 197.0
    assert r.min() >= 0.3 - 1e-9 and r.max() <= 1.0
    assert abs(r.mean() - 0.70) < 0.01             # 0.3 + 0.7 * E[Beta(4,3)] = 0.7
    s = W.generate(W.WORKLOADS["vit_b384_skew_bf16"])[0]
    hi, lo = s.keep[s.keep > 300], s.keep[s.keep <= 300]
    assert len(hi) == 32 and len(lo) == 32
    assert hi.min() >= np.rint(0.9 * 577) and lo.max() <= np.rint(0.15 * 577) and lo.min() >= np.rint(0.08 * 577)


def test_cascade_rounds_chain_lengths():
    rounds = W.generate(W.WORKLOADS["vit_l_cascade_bf16"], batch=16)
    assert len(rounds) == 3
    assert rounds[0].tokens is not None and rounds[1].tokens is None
    for prev, cur in zip(rounds, rounds[1:]):
        assert np.array_equal(cur.n_in, prev.keep)
        assert cur.scores.shape == (int(prev.keep.sum()),)
        assert np.all(cur.keep <= cur.n_in) and np.all(cur.keep >= 1)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.5, 3.0e38, np.inf], np.float32)
    got = W.bf16_bits_to_f32(W.f32_to_bf16_bits(x))
    assert got[0] == 1.0                            # tie -> even
    assert got[1] == 1.0 + 2 ** -6                  # tie -> even (upwards)
    assert got[2] == -1.5 and np.isinf(got[4])
