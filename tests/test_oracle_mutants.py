"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake (a flipped comparison, a wrong index, a dropped
term) into a copy of the oracle's C source, builds it on the CPU, and checks
that the brute-force / library pins reject the mutant while the unmodified
source passes the same battery.
"""
import itertools
import os
import subprocess

import numpy as np
import pytest
import torch

import oracle
from test_oracle_select import brute_keep_masks, masks_from_idx

SRC = os.path.join(os.path.dirname(oracle.__file__), "dora_oracle.c")

MUTANTS = {
    "score_direction": ("if (x > y) return -1;\n    if (x < y) return 1;\n  }\n  return (a->pos < b->pos)",
                        "if (x < y) return -1;\n    if (x > y) return 1;\n  }\n  return (a->pos < b->pos)"),
    "tie_direction": ("return (a->pos < b->pos) ? -1 : (a->pos > b->pos) ? 1 : 0;",
                      "return (a->pos > b->pos) ? -1 : (a->pos < b->pos) ? 1 : 0;"),
    "nan_on_top": ("if (an != bn) return an ? 1 : -1;", "if (an != bn) return an ? -1 : 1;"),
    "cls_not_pinned": ("kept[0] = 0;", "kept[0] = cand[0].pos;"),
    "order_not_preserved": ("qsort(kept, (size_t)keep[b], sizeof(int32_t), ascending_int);", ""),
    "one_short": ("for (int32_t r = 0; r < keep[b] - 1; ++r) kept[r + 1] = cand[r].pos;",
                  "for (int32_t r = 0; r < keep[b] - 2; ++r) kept[r + 1] = cand[r].pos;\n"
                  "    kept[keep[b] - 1] = kept[keep[b] > 1 ? keep[b] - 2 : 0];"),
    "cu_not_running": ("cu_out[b + 1] = cu_out[b] + keep[b];", "cu_out[b + 1] = keep[b] + (b > 0 ? cu_out[b - 1] : 0);"),
    "pack_wrong_segment": ("tokens + (size_t)(off_in[b] + kept[r])", "tokens + (size_t)(kept[r])"),
    "no_scale": ("logits[j] = scale * dot;", "logits[j] = dot;"),
    "query_for_key": ("const double* kj = k + ((start + j) * H + h) * D;",
                      "const double* kj = q + ((start + j) * H + h) * D;"),
    "wrong_head_stride": ("const double* vj = v + ((start + j) * H + h) * D;",
                          "const double* vj = v + ((start + j) * H + 0) * D;"),
    "unnormalised": ("const double p = logits[j] / z;", "const double p = logits[j];"),
    "key_index_is_query": ("for (int32_t d = 0; d < D; ++d) dot += qi[d] * kj[d];",
                           "for (int32_t d = 0; d < D; ++d) dot += qi[d] * k[(i * H + h) * D + d];"),
    "ties_away_from_zero": ("if (frac > 0.5 || (frac == 0.5 && fmod(n, 2.0) != 0.0)) n += 1.0;",
                            "if (frac >= 0.5) n += 1.0;"),
    "truncating_round": ("if (frac > 0.5 || (frac == 0.5 && fmod(n, 2.0) != 0.0)) n += 1.0;", ""),
    "no_subnormal_quantum": ("const int lead = (e - 1 < emin) ? emin : e - 1;", "const int lead = e - 1;"),
    "bf16_one_bit_too_many": ("is_bf16 ? 8 : 24", "is_bf16 ? 9 : 24"),
    "sign_dropped": ("return copysign(r, x);", "return r;"),
    "addend_dropped": ("stored_value(h, i, is_bf16) + stored_value(a, i, is_bf16)",
                       "stored_value(h, i, is_bf16) + stored_value(h, i, is_bf16)"),
    "addend_row_shifted": ("stored_value(h, i, is_bf16) + stored_value(a, i, is_bf16)",
                           "stored_value(h, i, is_bf16) + stored_value(a, i > 0 ? i - 1 : 0, is_bf16)"),
    "bf16_widened_wrong": ("bits = (uint32_t)((const uint16_t*)v)[i] << 16;",
                           "bits = (uint32_t)((const uint16_t*)v)[i] << 15;"),
    "gate_strict_threshold": ("p_gate[b] >= 0.5f", "p_gate[b] > 0.5f"),
    "legal_off_by_one": ("if (2 * (m + 1) <= (n_tok - 1) - 4) ++count;", "if (2 * (m + 1) < (n_tok - 1) - 4) ++count;"),
    "cls_counted_as_visual": ("if (2 * (m + 1) <= (n_tok - 1) - 4) ++count;", "if (2 * (m + 1) <= n_tok - 4) ++count;"),
    "argmax_last_tie": ("if (isnan(x) || x > y) best = m;", "if (isnan(x) || x >= y) best = m;"),
    "argmax_skips_nan": ("if (isnan(x) || x > y) best = m;", "if (x > y) best = m;"),
    "odd_budget": ("keep[b] = n_tok[b] - 2 * (best + 1);", "keep[b] = n_tok[b] - (2 * best + 1);"),
    "keep_counts_visual_only": ("keep[b] = n_tok[b] - 2 * (best + 1);", "keep[b] = n_tok[b] - 1 - 2 * (best + 1);"),
    "rank_not_compacted": ("on_rank[b] = open ? r : -1;", "on_rank[b] = open ? b : -1;"),
    "gate_off_drops_one": ("keep[b] = n_tok[b];\n      continue;", "keep[b] = n_tok[b] - 1;\n      continue;"),
    "negate_magnitude": ("out[i] = -s[i];", "out[i] = -fabsf(s[i]);"),
    "gumbel_subtracted": ("const float key = sb[j] + gb[j];", "const float key = sb[j] - gb[j];"),
    "draw_smallest_key_first": ("if (x > y) return -1;\n    if (x < y) return 1;\n  }\n  return (a->pos > b->pos)",
                                "if (x < y) return -1;\n    if (x > y) return 1;\n  }\n  return (a->pos > b->pos)"),
    "draw_ties_by_lower_position": ("return (a->pos > b->pos) ? -1 : (a->pos < b->pos) ? 1 : 0;",
                                    "return (a->pos < b->pos) ? -1 : (a->pos > b->pos) ? 1 : 0;"),
    "draw_nan_last": ("if (an != bn) return an ? -1 : 1;", "if (an != bn) return an ? 1 : -1;"),
    "cls_in_denominator": ("for (int64_t j = 1; j < n; ++j)\n      if (!drawn[j])",
                           "for (int64_t j = 0; j < n; ++j)\n      if (!drawn[j])"),
    "denominator_keeps_drawn": ("if (!drawn[j]) z += exp((double)s[j] - m);", "z += exp((double)s[j] - m);"),
    "denominator_without_log": ("lp += ((double)s[order[t]] - m) - log(z);", "lp += ((double)s[order[t]] - m) - z;"),
    "drawn_never_marked": ("drawn[order[t]] = 1;", ""),
    "variance_unbiased": ("  var /= C;", "  var /= (C - 1);"),
    "eps_outside_root": ("const double r = 1.0 / sqrt(var + eps);", "const double r = 1.0 / (sqrt(var) + eps);"),
    "variance_not_centred": ("var += (x[c] - mu) * (x[c] - mu);", "var += x[c] * x[c];"),
    "mean_includes_cls": ("for (int64_t r = r0 + 1; r < r1; ++r) {", "for (int64_t r = r0; r < r1; ++r) {"),
    "mean_over_all_rows": ("ob[C + c] /= (double)(r1 - r0 - 1);", "ob[C + c] /= (double)(r1 - r0);"),
    "gamma_beta_swapped": ("y[c] = (x[c] - mu) * r * gamma[c] + beta[c];", "y[c] = (x[c] - mu) * r * beta[c] + gamma[c];"),
}


def lc1_battery(lib, rng):
    """LC1 readout pin: torch layer_norm + mean in fp64."""
    lens = np.array([2, 7, 40])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    C = 48
    x = (rng.standard_normal((int(cu[-1]), C)) * 2 + 1).astype(np.float32)
    gamma = rng.uniform(0.5, 1.5, C).astype(np.float32)
    beta = rng.standard_normal(C).astype(np.float32)
    got = oracle.lc1_readout(x, cu, gamma, beta, 1e-6, "f32", lib=lib)
    g, bt = torch.from_numpy(gamma.astype(np.float64)), torch.from_numpy(beta.astype(np.float64))
    want = []
    for i in range(len(lens)):
        y = torch.nn.functional.layer_norm(torch.from_numpy(x[cu[i]:cu[i + 1]].astype(np.float64)), (C,), g, bt,
                                           1e-6)
        want.append(torch.cat([y[0], y[1:].mean(dim=0)]).numpy())
    return [] if np.allclose(got, np.stack(want), rtol=0, atol=1e-12) else ["lc1"]


def pl_battery(lib, rng):
    """Plackett-Luce pins: all orders sum to one, k = 1 is log_softmax, lexsort order,
    select/pack consistency, sampled frequencies."""
    failed = []
    s5 = np.array([0.0, 1.0, -0.5, 0.3, 2.0], np.float32)
    orders = list(itertools.permutations(range(1, 5), 3))
    lp, st = oracle.pl_logprob(np.tile(s5, (len(orders), 1)), np.array(orders, np.int32).reshape(-1),
                               (np.arange(len(orders) + 1) * 3).astype(np.int32), lib=lib)
    if st or abs(np.exp(lp).sum() - 1.0) > 1e-12:
        failed.append("pl mass")
    B, n = 200, 30
    s = (rng.standard_normal((B, n)) * 2).astype(np.float32)
    o1 = rng.integers(1, n, B).astype(np.int32)
    lp1, _ = oracle.pl_logprob(s, o1, np.arange(B + 1, dtype=np.int32), lib=lib)
    ls = torch.log_softmax(torch.from_numpy(s[:, 1:].astype(np.float64)), dim=1).numpy()
    if not np.allclose(lp1, ls[np.arange(B), o1 - 1], rtol=0, atol=1e-12):
        failed.append("pl log_softmax")
    g = rng.choice(np.array([0.0, 0.5, -0.0, 1.5], np.float32), (B, n))
    s[::7, 4] = np.nan
    s[::5] = np.round(s[::5])
    k = rng.integers(0, n, B).astype(np.int32)
    order, cu, _, st = oracle.pl_sample(s, g, k, lib=lib)
    if st:
        return failed + ["pl status"]
    key = s + g
    pos = np.arange(1, n)
    for b in range(B):
        kb = key[b, 1:]
        nan_first = np.lexsort((-pos, np.where(np.isnan(kb), 0.0, -kb), ~np.isnan(kb)))
        if not np.array_equal(order[cu[b]:cu[b + 1]], pos[nan_first][:k[b]]):
            failed.append("pl order")
            break
    # frequencies of the first draw against softmax
    Bs = 60000
    gs = rng.gumbel(size=(Bs, 5)).astype(np.float32)
    o, c, _, _ = oracle.pl_sample(np.tile(s5, (Bs, 1)), gs, np.ones(Bs, np.int32), lib=lib)
    p = np.exp(s5[1:]) / np.exp(s5[1:]).sum()
    freq = np.bincount(o, minlength=5)[1:] / Bs
    if np.any(np.abs(freq - p) > 5 * np.sqrt(p * (1 - p) / Bs)):
        failed.append("pl frequencies")
    return failed


def actor_battery(lib, rng):
    """Actor-decode pins: Table 3 grids, the set definitions, torch's argmax, NumPy compaction / negation."""
    failed = []
    for N0, M in ((196, 96), (256, 126)):
        n_tok = np.full(M, N0 + 1, np.int32)
        on_rank, _, n_on = oracle.actor_gate(np.ones(M, np.float32), n_tok, M, lib=lib)
        keep = oracle.actor_budget(np.eye(M, dtype=np.float32), n_tok, on_rank, lib=lib)
        if n_on != M or list(n_tok - keep) != list(range(2, N0 - 4 + 1, 2)):
            failed.append("table 3")
    B, M = 3000, 96
    n_tok = rng.integers(1, 198, B).astype(np.int32)
    p = rng.choice(np.array([0.5, np.nextafter(np.float32(0.5), np.float32(0)), 0.9, 0.1, np.nan], np.float32), B)
    on_rank, on_list, n_on = oracle.actor_gate(p, n_tok, M, lib=lib)
    n_legal = np.array([len([k for k in range(2, 2 * M + 1, 2) if k <= n - 5]) for n in n_tok])
    on = (p >= 0.5) & (n_legal > 0)
    if n_on != on.sum() or not np.array_equal(on_list[:n_on], np.flatnonzero(on)) or \
            not np.array_equal(on_rank[on], np.arange(n_on)) or not np.all(on_rank[~on] == -1):
        failed.append("gate")
        return failed
    logits = rng.choice(np.array([-1.0, 0.0, 2.0, np.nan], np.float32), (B, M), p=[0.3, 0.3, 0.38, 0.02])
    keep = oracle.actor_budget(logits, n_tok, on_rank, lib=lib)
    t = torch.from_numpy(logits[np.maximum(on_rank, 0)])
    m = torch.argmax(t.masked_fill(torch.arange(M)[None, :] >= torch.from_numpy(n_legal)[:, None], -np.inf),
                     dim=1).numpy()
    if not np.array_equal(np.where(on, n_tok - 2 * (m + 1), n_tok), keep):
        failed.append("budget")
    s = rng.standard_normal(1000).astype(np.float32)
    if not np.array_equal(oracle.negate(s, lib=lib).view(np.uint32), np.negative(s).view(np.uint32)):
        failed.append("negate")
    return failed


def residual_battery(lib, rng):
    """Residual pins: torch bf16 addition, NumPy fp32 addition, hand-worked roundings."""
    failed = []
    n = 20000
    bits = lambda x: torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    wide = lambda: ((rng.integers(0, 2, n, dtype=np.uint32) << 31) | (rng.integers(0, 255, n, dtype=np.uint32) << 23)
                    | rng.integers(0, 1 << 23, n, dtype=np.uint32)).view(np.float32)
    h, a = bits(wide()), bits(np.concatenate([wide()[: n // 2], rng.standard_normal(n - n // 2)]))
    want = (torch.from_numpy(h.view(np.int16)).view(torch.bfloat16)
            + torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)).view(torch.int16).numpy().view(np.uint16)
    got = oracle.residual_add(h, a, "bf16", lib=lib)
    fin = (want & 0x7F80) != 0x7F80
    if not np.array_equal(got[fin], want[fin]):
        failed.append("bf16 add")
    x, y = wide(), wide()
    with np.errstate(over="ignore", invalid="ignore"):
        if not np.array_equal(oracle.residual_add(x, y, "f32", lib=lib).view(np.uint32), (x + y).view(np.uint32)):
            failed.append("f32 add")
    ties = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, 1.5 * 2.0 ** -133, (2 - 2.0 ** -8) * 2.0 ** 127])
    want_t = np.array([1.0, 1 + 2.0 ** -6, 2.0 ** -132, np.inf], np.float32)
    if not np.array_equal(oracle.round_to_format(ties, "bf16", lib=lib), (want_t.view(np.uint32) >> 16).astype(np.uint16)):
        failed.append("ties")
    return failed


def build_variant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path_c = tmp_path / f"{name}.c"
    path_c.write_text(src.replace(old, new))
    path_so = tmp_path / f"lib{name}.so"
    subprocess.run(["gcc", "-O1", "-std=c99", "-fopenmp", "-fPIC", "-shared", str(path_c),
                    "-o", str(path_so), "-lm"], check=True)
    return oracle.load_library(str(path_so))


def battery(lib):
    """Return the list of pins the library fails."""
    failed = []
    rng = np.random.default_rng(101)
    # selection vs counting definition, heavy ties and NaNs
    n, B = 7, 3000
    s = rng.choice(np.array([-2.0, -0.0, 0.0, 0.5, 3.0, np.nan], np.float32), size=(B, n))
    keep = rng.integers(1, n + 1, size=B).astype(np.int32)
    tok = rng.standard_normal((B, n, 4)).astype(np.float32)
    idx, cu, packed, st = oracle.select_pack(s, keep, tok, lib=lib)
    if st or not np.array_equal(masks_from_idx(idx, cu, B, n), brute_keep_masks(s, keep)):
        failed.append("select")
    if st == 0:
        if not (cu[0] == 0 and np.array_equal(cu[1:], np.cumsum(keep))):
            failed.append("cu")
        elif not all(np.array_equal(packed[cu[b] + r], tok[b, idx[cu[b] + r]])
                     for b in range(B) for r in range(keep[b])):
            failed.append("pack")
        elif not all(np.all(np.diff(idx[cu[b]:cu[b + 1]]) > 0) for b in range(B)):
            failed.append("order")
    # attention vs torch fp64 SDPA, padded + masked
    lens = np.array([5, 1, 23, 12])
    H, D = 3, 64
    cuq = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    q, k, v = (rng.standard_normal((int(lens.sum()), H, D)).astype(np.float32) for _ in range(3))
    got = oracle.varlen_attn(q, k, v, cuq, "f32", lib=lib)
    L = int(lens.max())
    pad = lambda a: np.stack([np.pad(a[cuq[b]:cuq[b + 1]].astype(np.float64),
                                     ((0, L - lens[b]), (0, 0), (0, 0))) for b in range(len(lens))])
    tq, tk, tv = (torch.from_numpy(pad(a)).transpose(1, 2) for a in (q, k, v))
    mask = torch.from_numpy(np.arange(L)[None, :] < lens[:, None])[:, None, None, :]
    want = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=1 / 8)
    want = want.transpose(1, 2).numpy()
    if any(np.max(np.abs(got[cuq[b]:cuq[b + 1]] - want[b, :lens[b]])) > 1e-12 for b in range(len(lens))):
        failed.append("attention")
    return failed + residual_battery(lib, rng) + actor_battery(lib, rng) + pl_battery(lib, rng) + \
        lc1_battery(lib, rng)


def test_unmodified_source_passes(tmp_path):
    lib = build_variant(tmp_path, "original", "int oracle_max_threads(void) {", "int oracle_max_threads(void) {")
    assert battery(lib) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    lib = build_variant(tmp_path, name, old, new)
    assert battery(lib), f"planted mistake '{name}' passed every pin"
