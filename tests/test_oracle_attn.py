"""Pins for the oracle's varlen attention (CPU only).

The paper fixes exact softmax attention inside each packed sequence with no
attention across images and no bias or token-size term (Sec. 3.5
"Inference"; App. E.5).  Each check computes the expected answer a different
way: a pure-Python triple loop, torch's fp64 scaled_dot_product_attention on
dense and padded+masked batches, hand-worked closed forms, and invariances.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
D = 64


def cu_of(lens):
    return np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)


def rand_qkv(rng, lens, H, scale_in=1.0):
    tot = int(np.sum(lens))
    return [(rng.standard_normal((tot, H, D)) * scale_in).astype(np.float32) for _ in range(3)]


def python_triple_loop(q, k, v, cu, scale):
    """Direct definition, no max subtraction (inputs are small)."""
    total, H, _ = q.shape
    out = np.zeros((total, H, D))
    for b in range(len(cu) - 1):
        s, e = cu[b], cu[b + 1]
        for h in range(H):
            for i in range(s, e):
                w = []
                for j in range(s, e):
                    dot = 0.0
                    for d in range(D):
                        dot += float(q[i, h, d]) * float(k[j, h, d])
                    w.append(math.exp(scale * dot))
                z = sum(w)
                for d in range(D):
                    out[i, h, d] = sum(w[j - s] * float(v[j, h, d]) for j in range(s, e)) / z
    return out


def test_triple_loop_tiny():
    rng = np.random.default_rng(21)
    lens = [1, 3, 5]
    q, k, v = rand_qkv(rng, lens, H=2)
    cu = cu_of(lens)
    got = oracle.varlen_attn(q, k, v, cu, "f32")
    want = python_triple_loop(q, k, v, cu, 1 / 8)
    assert np.max(np.abs(got - want)) <= 1e-12


def test_keep_all_equals_torch_sdpa():
    rng = np.random.default_rng(22)
    B, N, H = 5, 37, 3
    q, k, v = rand_qkv(rng, [N] * B, H)
    got = oracle.varlen_attn(q, k, v, cu_of([N] * B), "f32")
    t = lambda a: torch.from_numpy(a.astype(np.float64)).reshape(B, N, H, D).transpose(1, 2)
    want = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), scale=1 / 8)
    want = want.transpose(1, 2).reshape(B * N, H, D).numpy()
    assert np.max(np.abs(got - want)) <= 1e-12


def test_padded_masked_equals_packed():
    rng = np.random.default_rng(23)
    lens = np.array([7, 1, 40, 19, 64, 2])
    H = 2
    q, k, v = rand_qkv(rng, lens, H)
    cu = cu_of(lens)
    got = oracle.varlen_attn(q, k, v, cu, "f32")
    B, L = len(lens), int(lens.max())
    pad = lambda a: np.stack([np.pad(a[cu[b]:cu[b + 1]].astype(np.float64),
                                     ((0, L - lens[b]), (0, 0), (0, 0))) for b in range(B)])
    tq, tk, tv = (torch.from_numpy(pad(a)).transpose(1, 2) for a in (q, k, v))
    mask = torch.from_numpy(np.arange(L)[None, :] < lens[:, None])[:, None, None, :]
    want = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=1 / 8)
    want = want.transpose(1, 2).numpy()
    for b in range(B):
        assert np.max(np.abs(got[cu[b]:cu[b + 1]] - want[b, :lens[b]])) <= 1e-12


def test_softmax_rows_sum_to_one_via_one_hot_values():
    rng = np.random.default_rng(24)
    lens = np.array([5, 64, 33])
    H = 2
    q, k, _ = rand_qkv(rng, lens, H, scale_in=3.0)
    cu = cu_of(lens)
    v = np.zeros_like(q)
    for b in range(len(lens)):
        for j in range(lens[b]):
            v[cu[b] + j, :, j] = 1.0           # V = identity: output row = softmax row
    got = oracle.varlen_attn(q, k, v, cu, "f32")
    assert np.all(got >= 0)
    assert np.max(np.abs(got.sum(axis=2) - 1.0)) <= 1e-12
    for b in range(len(lens)):                # nothing leaks past the segment's own keys
        assert np.all(got[cu[b]:cu[b + 1], :, lens[b]:] == 0)


def test_segment_permutation_is_exact():
    rng = np.random.default_rng(25)
    lens = np.array([3, 17, 1, 40, 8])
    H = 3
    q, k, v = rand_qkv(rng, lens, H)
    cu = cu_of(lens)
    base = oracle.varlen_attn(q, k, v, cu, "f32")
    perm = np.array([3, 0, 4, 2, 1])
    cat = lambda a: np.concatenate([a[cu[b]:cu[b + 1]] for b in perm])
    pc = cu_of(lens[perm])
    out = oracle.varlen_attn(cat(q), cat(k), cat(v), pc, "f32")
    assert np.array_equal(out, cat(base))


def test_key_permutation_within_segment():
    rng = np.random.default_rng(26)
    lens = np.array([29, 12])
    H = 2
    q, k, v = rand_qkv(rng, lens, H)
    cu = cu_of(lens)
    base = oracle.varlen_attn(q, k, v, cu, "f32")
    p = np.concatenate([rng.permutation(lens[0]), lens[0] + rng.permutation(lens[1])])
    out = oracle.varlen_attn(q, k[p], v[p], cu, "f32")
    assert np.max(np.abs(out - base)) <= 1e-12


def test_closed_forms():
    rng = np.random.default_rng(27)
    lens = np.array([1, 1, 6])
    H = 2
    q, k, v = rand_qkv(rng, lens, H)
    cu = cu_of(lens)
    k[2:8] = k[2]                                # identical keys in the third segment
    out = oracle.varlen_attn(q, k, v, cu, "f32")
    assert np.array_equal(out[0:2], v[0:2].astype(np.float64))            # single token: O = V
    assert np.max(np.abs(out[2:8] - v[2:8].astype(np.float64).mean(axis=0))) <= 1e-12


def test_scale_parameter():
    rng = np.random.default_rng(28)
    lens = np.array([9])
    q, k, v = rand_qkv(rng, lens, 1)
    cu = cu_of(lens)
    a = oracle.varlen_attn(q, k, v, cu, "f32", scale=0.3)
    b = oracle.varlen_attn(q * np.float32(0.5), k, v, cu, "f32", scale=0.6)
    assert np.max(np.abs(a - b)) <= 1e-12


def test_bf16_widening_is_exact():
    bits = np.array([0x3F80, 0xC000, 0x0001, 0x7F80, 0xFF80, 0x8000], np.uint16)
    got = oracle.widen(bits, "bf16")
    want = np.array([1.0, -2.0, 2.0 ** -133, np.inf, -np.inf, -0.0])
    assert np.array_equal(got, want) and np.signbit(got[5])
    x = np.random.default_rng(1).standard_normal(1000).astype(np.float32)
    b = workloads.f32_to_bf16_bits(x)
    assert np.array_equal(oracle.widen(b, "bf16"), workloads.bf16_bits_to_f32(b).astype(np.float64))
    assert np.max(np.abs(oracle.widen(b, "bf16") - x) / np.abs(x)) <= 2.0 ** -8          # unit roundoff of an 8-bit significand


def test_golden_hand_cases():
    for c in json.load(open(os.path.join(GOLDEN, "attn_hand.json")))["cases"]:
        n = c["len"]
        arr = {}
        for name in "qkv":
            a = np.zeros((n, 1, D), np.float32)
            for row, entries in c[name].items():
                for dim, val in entries:
                    a[int(row), 0, dim] = val
            arr[name] = a
        out = oracle.varlen_attn(arr["q"], arr["k"], arr["v"], np.array([0, n], np.int32), "f32")
        for row, dim, val in c["expect"]:
            assert abs(out[row, 0, dim] - val) <= c["tol"], c["why"]


def test_bf16_inputs_decode_then_attend():
    rng = np.random.default_rng(29)
    lens = np.array([11, 4])
    qf, kf, vf = rand_qkv(rng, lens, 2)
    qb, kb, vb = (workloads.f32_to_bf16_bits(a) for a in (qf, kf, vf))
    cu = cu_of(lens)
    got = oracle.varlen_attn(qb, kb, vb, cu, "bf16")
    dec = lambda a: workloads.bf16_bits_to_f32(a)
    want = oracle.varlen_attn(dec(qb), dec(kb), dec(vb), cu, "f32")
    assert np.array_equal(got, want)


def test_selected_rows_equal_the_full_oracle():
    """varlen_attn_rows evaluates the same definition for chosen query rows."""
    rng = np.random.default_rng(77)
    lens = np.array([5, 1, 37, 12])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    q, k, v = (rng.standard_normal((int(lens.sum()), 3, 64)).astype(np.float32) for _ in range(3))
    full = oracle.varlen_attn(q, k, v, cu, "f32")
    rows = np.array([0, 4, 5, 6, 20, 42, 54])
    assert np.array_equal(oracle.varlen_attn_rows(q, k, v, cu, rows, "f32"), full[rows])
