"""GPU parity for dora_pl_sample / dora_pl_logprob against the oracle.

The drawing orders and offsets are integer results of FP32 key comparisons
that both sides make on the same FP32 keys: compared exactly.  The ordered
log-probability is computed in fp32 on the GPU and in fp64 by the oracle;
the bound it must meet is derived per image from the fp32 steps (see
`fp32_bound`).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import to_dev

pytestmark = pytest.mark.gpu

U = 2.0 ** -24   # unit roundoff of fp32


def geometry(s, cu):
    if cu is None:
        B, n = s.shape
        return [(b * n, n) for b in range(B)], s.reshape(-1)
    return [(int(cu[b]), int(cu[b + 1] - cu[b])) for b in range(len(cu) - 1)], s


def fp32_bound(s, order, cu_order, cu=None):
    """Error bound of the fp32 log-probability, per image, from its steps:
    s - m (one rounding), exp (2 ulp), suffix sums of up to n positive terms
    (n + 16 roundings), log (2 ulp), and the sum of the k terms."""
    segs, flat = geometry(s, cu)
    out = []
    for b, (o, n) in enumerate(segs):
        sv = flat[o + 1:o + n].astype(np.float64)
        ob = order[cu_order[b]:cu_order[b + 1]]
        k = len(ob)
        if k == 0:
            out.append(0.0)
            continue
        m = sv.max()
        e = np.exp(sv - m)
        drawn = np.zeros(n - 1, bool)
        drawn[ob - 1] = True
        surv = e[~drawn].sum()
        de = e[ob - 1]
        S = np.cumsum(de[::-1])[::-1] + surv
        terms = (sv[ob - 1] - m) - np.log(S)
        d = np.abs(sv[ob - 1] - m)
        per = 3 * d + 3 * np.max(np.abs(sv - m)) + 2 * np.abs(np.log(S)) + n + 16
        out.append(U * (per.sum() + k * np.abs(terms).sum()))
    return np.array(out)


def run_sample(dora, s, g, k, cu=None, N=None, cap=None):
    o, c, lp, st = dora.dora_pl_sample(to_dev(s), to_dev(g), to_dev(k.astype(np.int32)),
                                       cu_in=None if cu is None else to_dev(cu), N=N, cap=cap)
    torch.cuda.synchronize()
    c = c.cpu().numpy()
    return o.cpu().numpy()[:int(c[-1])], c, lp.cpu().numpy().astype(np.float64), int(st.item())


def check(dora, s, g, k, cu=None, N=None):
    o_o, c_o, lp_o, st_o = oracle.pl_sample(s, g, k, cu_in=cu, N=N)
    assert st_o == 0
    o_g, c_g, lp_g, st_g = run_sample(dora, s, g, k, cu, N)
    assert st_g == 0
    assert np.array_equal(c_g, c_o) and np.array_equal(o_g, o_o)
    fin = np.isfinite(lp_o)
    assert np.array_equal(np.isfinite(lp_g), fin)
    tol = fp32_bound(s, o_o, c_o, cu)
    err = np.abs(lp_g - lp_o)
    assert np.all(err[fin] <= tol[fin]), (err[fin].max(), tol[fin][np.argmax(err[fin])])
    return o_g, c_g, lp_g, err[fin].max() if fin.any() else 0.0


@pytest.mark.parametrize("N", [2, 3, 17, 197, 257, 577, 2048])
def test_dense_sizes(gpu, N):
    rng = np.random.default_rng(N)
    B = 37
    s = (rng.standard_normal((B, N)) * 2).astype(np.float32)
    g = rng.gumbel(size=(B, N)).astype(np.float32)
    k = rng.integers(0, N, B).astype(np.int32)
    k[0], k[1] = 0, N - 1
    _, _, _, err = check(gpu, s, g, k)
    print(f"[pl] N={N} max |logprob err| {err:.2e}", flush=True)


def test_deit_b_batch(gpu):
    """The DeiT-B shape: 256 images of 197 tokens, budgets from the grid 2..192."""
    rng = np.random.default_rng(5)
    B, N = 256, 197
    s = rng.standard_normal((B, N)).astype(np.float32)
    g = rng.gumbel(size=(B, N)).astype(np.float32)
    k = (2 * rng.integers(1, 97, B)).astype(np.int32)
    _, _, _, err = check(gpu, s, g, k)
    print(f"[pl] DeiT-B max |logprob err| {err:.2e}", flush=True)


def test_ties_nan_and_signed_zero_keys(gpu):
    rng = np.random.default_rng(6)
    B, N = 64, 90
    s = rng.choice(np.array([-1.0, 0.0, -0.0, 1.0, 2.5], np.float32), (B, N))
    g = rng.choice(np.array([0.0, -0.0, 0.5], np.float32), (B, N))
    s[::5, 7] = np.nan
    g[::7, 11] = np.nan
    k = rng.integers(0, N, B).astype(np.int32)
    check(gpu, s, g, k)


def test_packed_segments(gpu):
    rng = np.random.default_rng(7)
    lens = rng.integers(1, 198, 150)
    lens[:3] = [1, 2, 6]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    s = rng.standard_normal(int(cu[-1])).astype(np.float32)
    g = rng.gumbel(size=int(cu[-1])).astype(np.float32)
    k = np.array([rng.integers(0, n) for n in lens], np.int32)
    check(gpu, s, g, k, cu=cu, N=197)


def test_drawn_set_is_what_select_pack_deletes_on_the_gpu(gpu):
    rng = np.random.default_rng(8)
    B, N = 40, 197
    s = rng.standard_normal((B, N)).astype(np.float32)
    g = rng.gumbel(size=(B, N)).astype(np.float32)
    k = rng.integers(0, N, B).astype(np.int32)
    o, c, _, _ = run_sample(gpu, s, g, k)
    idx, cuk, _, st = gpu.dora_select_pack(to_dev(-(s + g)), to_dev(N - k), to_dev(np.zeros((B, N, 4), np.float32)))
    torch.cuda.synchronize()
    idx, cuk = idx.cpu().numpy(), cuk.cpu().numpy()
    for b in range(B):
        kept = set(idx[cuk[b]:cuk[b + 1]].tolist())
        drawn = set(o[c[b]:c[b + 1]].tolist())
        assert kept.isdisjoint(drawn) and len(kept) + len(drawn) == N


def test_logprob_of_given_orders_under_new_scores(gpu):
    rng = np.random.default_rng(9)
    B, N = 100, 197
    s_old = rng.standard_normal((B, N)).astype(np.float32)
    g = rng.gumbel(size=(B, N)).astype(np.float32)
    k = rng.integers(0, N, B).astype(np.int32)
    o, c, lp_sample, _ = run_sample(gpu, s_old, g, k)
    s_new = (s_old + 0.3 * rng.standard_normal((B, N))).astype(np.float32)
    for s in (s_old, s_new):
        lp, st = gpu.dora_pl_logprob(to_dev(s), to_dev(o), to_dev(c))
        torch.cuda.synchronize()
        want, st_o = oracle.pl_logprob(s, o, c)
        assert int(st.item()) == 0 and st_o == 0
        err = np.abs(lp.cpu().numpy() - want)
        assert np.all(err <= fp32_bound(s, o, c)), err.max()
    # same scores: the two GPU paths agree within the bound too
    lp_eval, _ = gpu.dora_pl_logprob(to_dev(s_old), to_dev(o), to_dev(c))
    assert np.all(np.abs(lp_eval.cpu().numpy() - lp_sample) <= 2 * fp32_bound(s_old, o, c))


def test_invalid_draw_counts_and_orders_set_status(gpu):
    rng = np.random.default_rng(10)
    B, N = 6, 30
    s = rng.standard_normal((B, N)).astype(np.float32)
    g = rng.gumbel(size=(B, N)).astype(np.float32)
    k = np.full(B, 5, np.int32)
    k[2] = N                                                          # more than the visual tokens
    k[4] = -1
    o, c, lp, st = run_sample(gpu, s, g, k)
    assert st & gpu.DORA_DEV_KEEP_RANGE
    assert np.isnan(lp[2]) and np.isnan(lp[4]) and np.all(np.isfinite(lp[[0, 1, 3, 5]]))
    good = np.full(B, 5, np.int32)
    o, c, lp, st = run_sample(gpu, s, g, good)
    assert st == 0
    for bad_order in (lambda a: a.__setitem__(1, a[0]),               # repeated position
                      lambda a: a.__setitem__(0, 0),                  # CLS
                      lambda a: a.__setitem__(3, N)):                 # past the segment
        ob = o.copy()
        bad_order(ob)
        lpb, stb = gpu.dora_pl_logprob(to_dev(s), to_dev(ob), to_dev(c))
        torch.cuda.synchronize()
        lpb = lpb.cpu().numpy()
        assert int(stb.item()) & gpu.DORA_DEV_KEEP_RANGE and np.isnan(lpb[0]) and np.all(np.isfinite(lpb[1:]))


def test_invalid_order_offsets_are_rejected_without_reading(gpu):
    rng = np.random.default_rng(12)
    B, N = 4, 30
    s = rng.standard_normal((B, N)).astype(np.float32)
    # every list stays inside the order array (cu_order[B] entries), as the
    # contract requires; the offsets themselves are what is wrong
    short = np.array([3, 4, 5, 6, 7, 8, 9, 10], np.int32)
    long_ = (np.arange(36) % (N - 1) + 1).astype(np.int32)
    for order, cu, bad in ((short, [0, 2, 1, 5, 8], [1]),         # decreasing
                           (short, [0, -5, 4, 6, 8], [0, 1]),     # negative
                           (long_, [0, 30, 32, 34, 36], [0])):    # 30 draws from 29 visual tokens
        lp, st = gpu.dora_pl_logprob(to_dev(s), to_dev(order), to_dev(np.array(cu, np.int32)))
        torch.cuda.synchronize()
        lp = lp.cpu().numpy()
        assert int(st.item()) & gpu.DORA_DEV_KEEP_RANGE, cu
        good = [i for i in range(B) if i not in bad]
        assert np.all(np.isnan(lp[bad])) and np.all(np.isfinite(lp[good])), (cu, lp)


def test_capacity_overflow(gpu):
    rng = np.random.default_rng(11)
    B, N = 8, 50
    s = rng.standard_normal((B, N)).astype(np.float32)
    g = rng.gumbel(size=(B, N)).astype(np.float32)
    k = np.full(B, 40, np.int32)
    order = torch.full((300 + 16,), -7, dtype=torch.int32, device="cuda")
    _, c, lp, st = gpu.dora_pl_sample(to_dev(s), to_dev(g), to_dev(k), order_out=order, cap=300)
    torch.cuda.synchronize()
    assert int(st.item()) & gpu.DORA_DEV_CAPACITY
    assert torch.all(order[300:] == -7).item()
    o_o, c_o, _, _ = oracle.pl_sample(s, g, k)
    assert np.array_equal(order[:300].cpu().numpy(), o_o[:300]) and np.array_equal(c.cpu().numpy(), c_o)
