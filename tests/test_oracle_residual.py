"""Pins for the oracle's deletion after the attention residual (CPU only).

Sec. 3.1, Eq. (1): the attention residual H + Attention(LayerNorm(H)) is
formed over all tokens and the deleted rows are removed from that sum before
the MLP.  The oracle forms each element as the exact sum of the two stored
values rounded once, to nearest with ties to even, into the storage format.
The checks below get the expected bits some other way: torch's and NumPy's
own conversions and additions, hand-worked ties, overflow and subnormal
cases, and the -0 addend, which must reduce to plain ``select_pack``.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as W


def bf16_bits_of(x):
    """torch's fp32 -> bf16 conversion (round to nearest even), as uint16."""
    return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16).view(torch.int16) \
        .numpy().view(np.uint16)


def wide_f32(rng, n):
    """fp32 values over the whole exponent range, subnormals and zeros included."""
    mant = rng.integers(0, 1 << 23, n, dtype=np.uint32)
    expo = rng.integers(0, 255, n, dtype=np.uint32)              # 255 (inf/NaN) excluded
    sign = rng.integers(0, 2, n, dtype=np.uint32) << 31
    return (sign | (expo << 23) | mant).view(np.float32)


def test_rounding_matches_torch_bf16_conversion():
    rng = np.random.default_rng(1)
    x = np.concatenate([wide_f32(rng, 400000), rng.standard_normal(100000).astype(np.float32)])
    assert np.array_equal(oracle.round_to_format(x.astype(np.float64), "bf16"), bf16_bits_of(x))


def test_rounding_matches_torch_on_exact_ties():
    # fp32 values whose low 16 bits are exactly 0x8000 sit halfway between two
    # bf16 values; the even neighbour must win, in the normal and subnormal range.
    rng = np.random.default_rng(2)
    hi = rng.integers(0, 0x7F7F, 50000, dtype=np.uint32)
    x = ((hi << 16) | 0x8000).view(np.float32)
    got = oracle.round_to_format(x.astype(np.float64), "bf16")
    assert np.array_equal(got, bf16_bits_of(x))
    assert np.array_equal(got & 1, np.zeros_like(got))          # even significand


def test_rounding_matches_numpy_fp32_cast():
    rng = np.random.default_rng(3)
    # fp64 values over the fp32 range and below it (to exercise the subnormal
    # quantum) and with random low bits (so most are not representable).
    x = np.ldexp(rng.uniform(1.0, 2.0, 300000), rng.integers(-160, 128, 300000)) * rng.choice([-1.0, 1.0], 300000)
    with np.errstate(over="ignore"):
        want = x.astype(np.float32)
    assert np.array_equal(oracle.round_to_format(x, "f32").view(np.uint32), want.view(np.uint32))


def test_hand_worked_roundings():
    """Closed-form cases, worked by hand from the bf16 format (8 significand
    bits, exponents -126..127, subnormal quantum 2^-133)."""
    ulp1 = 2.0 ** -7                                              # bf16 spacing in [1, 2)
    cases = [
        (1.0 + ulp1 / 2, 1.0),                                    # tie, 1.0 has the even significand
        (1.0 + 3 * ulp1 / 2, 1.0 + 2 * ulp1),                     # tie, rounds up to the even one
        (1.0 + ulp1 / 2 + 2.0 ** -30, 1.0 + ulp1),                # just past the tie
        (-(1.0 + ulp1 / 2), -1.0),                                # ties are symmetric in sign
        (2.0 ** -133 * 1.5, 2.0 ** -132),                         # subnormal tie -> even multiple (2)
        (2.0 ** -133 * 2.5, 2.0 ** -132),                         # subnormal tie -> even multiple (2)
        (2.0 ** -134, 0.0),                                       # half the smallest subnormal: tie to 0
        (2.0 ** -134 * 1.01, 2.0 ** -133),
        ((2 - 2.0 ** -7) * 2.0 ** 127, (2 - 2.0 ** -7) * 2.0 ** 127),  # largest finite bf16
        ((2 - 2.0 ** -8) * 2.0 ** 127, np.inf),                   # tie above it: odd max rounds up to inf
        ((2 - 2.0 ** -8) * 2.0 ** 127 - 2.0 ** 100, (2 - 2.0 ** -7) * 2.0 ** 127),
        (-0.0, -0.0),
    ]
    x = np.array([c[0] for c in cases])
    want = np.array([c[1] for c in cases], dtype=np.float32)
    got = oracle.round_to_format(x, "bf16")
    want_bits = (want.view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(got, want_bits), [(c, hex(g)) for c, g in zip(cases, got)]


def test_bf16_residual_matches_torch_bf16_add():
    """torch's CPU bf16 addition adds in fp32 and rounds once to bf16; with 24
    >= 2*8+2 significand bits that double rounding is innocuous, so it is the
    correctly rounded sum too."""
    rng = np.random.default_rng(4)
    n = 300000
    h = bf16_bits_of(wide_f32(rng, n))
    a = bf16_bits_of(np.concatenate([wide_f32(rng, n // 2), rng.standard_normal(n - n // 2).astype(np.float32)]))
    a[:1000] = h[:1000] ^ 0x8000                                  # exact cancellation -> +0
    th = torch.from_numpy(h.view(np.int16)).view(torch.bfloat16)
    ta = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    want = (th + ta).view(torch.int16).numpy().view(np.uint16)
    got = oracle.residual_add(h, a, "bf16")
    fin = np.isfinite(W.bf16_bits_to_f32(want))
    assert np.array_equal(got[fin], want[fin])
    assert np.array_equal(np.isnan(W.bf16_bits_to_f32(got)), np.isnan(W.bf16_bits_to_f32(want)))
    fin_h = np.isfinite(W.bf16_bits_to_f32(h[:1000]))
    assert np.all(got[:1000][fin_h] == 0)                         # x + (-x) = +0 under round to nearest


def test_f32_residual_matches_numpy_add():
    rng = np.random.default_rng(5)
    h, a = wide_f32(rng, 300000), wide_f32(rng, 300000)
    with np.errstate(over="ignore", invalid="ignore"):
        want = h + a
    got = oracle.residual_add(h, a, "f32")
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_overflow_and_infinities():
    big = (2 - 2.0 ** -7) * 2.0 ** 127                            # largest finite bf16
    half_ulp = 2.0 ** 119
    h = bf16_bits_of(np.array([big, big, -big, 2.0 ** 127, np.inf, np.inf, 1.0], np.float32))
    a = bf16_bits_of(np.array([0.0, 2.0 ** 120, -(2.0 ** 120), 2.0 ** 127, 1.0, -np.inf, -np.inf], np.float32))
    got = W.bf16_bits_to_f32(oracle.residual_add(h, a, "bf16"))
    assert got[0] == big
    assert got[1] == np.inf and got[2] == -np.inf                 # 2^120 > half ulp at the top: overflow
    assert got[3] == np.inf                                       # 2^128 is past the format
    assert got[4] == np.inf and np.isnan(got[5]) and got[6] == -np.inf
    assert half_ulp < 2.0 ** 120


def test_small_integers_are_exact():
    rng = np.random.default_rng(6)
    x, y = rng.integers(-128, 128, 5000), rng.integers(-128, 128, 5000)
    h, a = bf16_bits_of(x.astype(np.float32)), bf16_bits_of(y.astype(np.float32))
    got = W.bf16_bits_to_f32(oracle.residual_add(h, a, "bf16"))
    assert np.array_equal(got, (x + y).astype(np.float32))        # |x+y| <= 256 fits 8 bits


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_negative_zero_addend_reduces_to_select_pack(dtype):
    rng = np.random.default_rng(7)
    B, N, C = 9, 40, 24
    scores = rng.standard_normal((B, N)).astype(np.float32)
    keep = rng.integers(1, N + 1, B).astype(np.int32)
    x = wide_f32(rng, B * N * C).reshape(B, N, C)
    x[0, :4] = [0.0] * C
    x[0, 4:8] = [-0.0] * C
    h = bf16_bits_of(x) if dtype == "bf16" else x
    mz = np.full_like(h, 0x8000) if dtype == "bf16" else np.full_like(h, -0.0)
    i0, c0, p0, s0 = oracle.select_pack(scores, keep, h)
    i1, c1, p1, s1 = oracle.select_pack_residual(scores, keep, h, mz, dtype)
    assert s0 == s1 == 0
    assert np.array_equal(i0, i1) and np.array_equal(c0, c1)
    assert np.array_equal(p0.view(np.uint8), p1.view(np.uint8))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_residual_pack_is_sum_of_gathered_rows(dtype):
    """Gather-then-add equals add-then-gather row by row (the packed rows are
    the kept rows of h + a), and the sum is symmetric in h and a."""
    rng = np.random.default_rng(8)
    lens = np.array([1, 5, 17, 64, 3])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    tot, C = int(lens.sum()), 16
    scores = rng.standard_normal(tot).astype(np.float32)
    keep = np.array([1, 3, 10, 33, 3], np.int32)
    x, y = rng.standard_normal((2, tot, C)).astype(np.float32)
    h, a = (bf16_bits_of(x), bf16_bits_of(y)) if dtype == "bf16" else (x, y)
    idx, cuo, packed, st = oracle.select_pack_residual(scores, keep, h, a, dtype, cu_in=cu)
    assert st == 0
    rows = np.concatenate([cu[b] + idx[cuo[b]:cuo[b + 1]] for b in range(len(lens))])
    assert np.array_equal(packed, oracle.residual_add(h[rows], a[rows], dtype))
    _, _, swapped, _ = oracle.select_pack_residual(scores, keep, a, h, dtype, cu_in=cu)
    assert np.array_equal(packed.view(np.uint8), swapped.view(np.uint8))
