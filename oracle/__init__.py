"""CPU oracle for the DORA deployment hot path (select -> pack -> varlen attention).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by ``__graft_entry__.smoke()``
and by the CPU-baseline leg of ``bench.py``; never by the product package.
It shares no code with the GPU path.

The arithmetic lives in ``dora_oracle.c`` (plain C, fp64 for attention):

* ``select_pack`` follows the deployment keep rule (Sec. 3.2 "Sampling and
  deployment"; App. A.3): CLS (position 0) is always kept and, of the visual
  tokens, the ``keep-1`` highest keep-scores survive; survivors keep their
  original order (Sec. 3.1, Eq. (1)); images are compacted into one packed
  buffer with explicit boundaries (Sec. 3.5 "Inference").  Implemented as a
  full sort of (score, position) per image.
* ``select_pack_residual`` applies the same deletion to H + A, the
  attention residual (Sec. 3.1, Eq. (1): rows are removed after the
  residual add and before the MLP): each element is the exact sum rounded
  once, to nearest even, into bf16 or fp32 (``round_to_format``).
* ``actor_gate`` / ``actor_budget`` / ``negate`` decode the deterministic
  actor's outputs into the path's inputs (Sec. 3.2 "Sampling and
  deployment"; App. A.2 legal budgets; App. A.3): gate at p >= 0.5 with a
  legal budget, gate-on images numbered in image order, the legal budget of
  the largest logit, keep = tokens - budget, keep-scores = -removal scores.
* ``pl_sample`` / ``pl_logprob``: Plackett-Luce deletion by Gumbel-top-k
  (keys = removal score + Gumbel noise in FP32, the k largest drawn in
  decreasing key order) and the ordered log-probability of Eq.
  (app-actor-pl) in fp64 (App. A.3), written as the definition reads.
* ``lc1_readout``: the DINOv2 LC1 readout input on pruned tokens (App. E.3):
  LayerNorm of CLS next to the mean of the LayerNorms of the surviving
  visual tokens, per packed sequence, in fp64.
* ``trajectory_flops``: FLOPs of the complete forward along each image's
  realised token trajectory (App. E.4): two per multiply-accumulate of the
  patch embedding, every linear layer and the attention products, with the
  actor's gate and controller where they run (App. A.1), in exact integers.
* ``varlen_attn`` is exact softmax attention inside each boundary
  (Sec. 3.5; App. E.5), computed as a dense fp64 score matrix per
  (image, head) from the exact values of the bf16 / fp32 inputs.

Pins (tests/test_oracle_*.py): brute-force counting definition of the keep
set over exhaustive tiny inputs, NumPy's stable argsort on NaN-free inputs,
closed forms (keep-all, keep-one, constant scores, monotone scores), a
hand-worked fixture; for attention a pure-Python triple loop, torch fp64
``scaled_dot_product_attention`` on keep-all and padded+masked batches,
one-hot V (softmax rows sum to 1), segment-permutation and key-permutation
invariance, keep-one (O = V) and identical keys (O = mean of V); for the
residual, torch's fp32 -> bf16 conversion and bf16 addition, NumPy's fp64 ->
fp32 cast and fp32 addition, hand-worked ties, overflow and subnormal cases,
and the -0 addend reducing to ``select_pack``.
"""
from __future__ import annotations

import ctypes
from typing import Optional, Tuple

import numpy as np

from . import build as _build

BAD_KEEP = 1
OVERFLOW = 2
BAD_SEGMENTS = 4

_lib = None


def load_library(path: str):
    """Open an oracle shared library and declare its signatures."""
    lib = ctypes.CDLL(path)
    lib.oracle_select_pack.restype = ctypes.c_int
    lib.oracle_select_pack.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
    lib.oracle_varlen_attn.restype = None
    lib.oracle_varlen_attn.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
        ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_double,
        ctypes.c_void_p, ctypes.c_int32]
    lib.oracle_max_threads.restype = ctypes.c_int
    lib.oracle_actor_gate.restype = None
    lib.oracle_actor_gate.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.oracle_actor_budget.restype = None
    lib.oracle_actor_budget.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int32, ctypes.c_void_p]
    lib.oracle_negate.restype = None
    lib.oracle_negate.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    lib.oracle_pl_sample.restype = ctypes.c_int
    lib.oracle_pl_sample.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
    lib.oracle_pl_logprob.restype = ctypes.c_int
    lib.oracle_pl_logprob.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p]
    lib.oracle_lc1_readout.restype = None
    lib.oracle_lc1_readout.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_double, ctypes.c_void_p]
    lib.oracle_varlen_attn_rows.restype = None
    lib.oracle_varlen_attn_rows.argtypes = [
        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
        ctypes.c_int32, ctypes.c_double, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    lib.oracle_round_to_format.restype = None
    lib.oracle_round_to_format.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p]
    lib.oracle_residual_add.restype = None
    lib.oracle_residual_add.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_void_p]
    return lib


def _load(lib=None):
    global _lib
    if lib is not None:
        return lib
    if _lib is None:
        _lib = load_library(_build.build(force=False))
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def select_pack(scores: np.ndarray, keep: np.ndarray, tokens: np.ndarray,
                cu_in: Optional[np.ndarray] = None, N: Optional[int] = None, lib=None
                ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, int]:
    """Keep CLS + top-(keep-1) visual tokens per image and pack them.

    scores: float32 [B,N] (dense) or [total_in] with ``cu_in`` [B+1].
    keep:   int32 [B] (counts CLS).
    tokens: [B,N,C] or [total_in,C] of any fixed-size dtype (rows copied as bytes).
    Returns (idx [sum keep] int32, cu [B+1] int32, packed [sum keep, C], status).
    On a nonzero status nothing was computed and the arrays are empty.
    """
    scores = np.ascontiguousarray(scores, dtype=np.float32)
    keep = np.ascontiguousarray(keep, dtype=np.int32)
    tokens = np.ascontiguousarray(tokens)
    B = int(keep.shape[0])
    if cu_in is None:
        if N is None:
            N = int(scores.shape[1]) if scores.ndim == 2 else int(scores.shape[0]) // max(B, 1)
        cu_arr = None
    else:
        cu_arr = np.ascontiguousarray(cu_in, dtype=np.int32)
        if N is None:
            N = int(np.max(np.diff(cu_arr))) if B else 0
    C = int(np.prod(tokens.shape[1:])) if cu_in is not None else int(np.prod(tokens.shape[2:]))
    tok2 = tokens.reshape(-1, C)
    total_in = tok2.shape[0]
    if cu_in is not None and scores.shape[0] < total_in:
        raise ValueError("packed scores shorter than the packed token rows")
    row_bytes = C * tok2.dtype.itemsize
    cap = int(keep.astype(np.int64).clip(min=0).sum())
    idx = np.zeros(max(cap, 1), dtype=np.int32)
    cu = np.zeros(B + 1, dtype=np.int32)
    packed = np.zeros((max(cap, 1), C), dtype=tok2.dtype)
    st = _load(lib).oracle_select_pack(_ptr(scores), _ptr(keep), _ptr(tok2), _ptr(cu_arr),
                                       total_in, B, int(N), row_bytes, _ptr(idx), _ptr(cu), _ptr(packed), cap)
    if st:
        return (np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros((0, C), tok2.dtype), int(st))
    return idx[:cap], cu, packed[:cap], 0


def round_to_format(x: np.ndarray, dtype: str, lib=None) -> np.ndarray:
    """fp64 values rounded to nearest-even bf16 (uint16 bits) or fp32."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16 if dtype == "bf16" else np.float32)
    _load(lib).oracle_round_to_format(_ptr(x), x.size, int(dtype == "bf16"), _ptr(out))
    return out


def residual_add(h: np.ndarray, a: np.ndarray, dtype: str, lib=None) -> np.ndarray:
    """h + a, correctly rounded to the storage type: bf16 bit patterns (uint16)
    or fp32 values, any shape (Sec. 3.1, Eq. (1): H + Attention(LayerNorm(H)))."""
    st = np.uint16 if dtype == "bf16" else np.float32
    h = np.ascontiguousarray(h, dtype=st)
    a = np.ascontiguousarray(a, dtype=st)
    if h.shape != a.shape:
        raise ValueError("h and a must have the same shape")
    out = np.empty(h.shape, dtype=st)
    _load(lib).oracle_residual_add(_ptr(h), _ptr(a), h.size, int(dtype == "bf16"), _ptr(out))
    return out


def select_pack_residual(scores: np.ndarray, keep: np.ndarray, h: np.ndarray, a: np.ndarray, dtype: str,
                         cu_in: Optional[np.ndarray] = None, N: Optional[int] = None, lib=None
                         ) -> Tuple[np.ndarray, np.ndarray, np.ndarray, int]:
    """Deletion after the attention residual (Sec. 3.1, Eq. (1)): the kept
    rows of H + A, where A is the attention branch's output in H's layout.
    Computed as the definition reads: the whole sum first, then
    ``select_pack`` of it."""
    return select_pack(scores, keep, residual_add(h, a, dtype, lib=lib), cu_in=cu_in, N=N, lib=lib)


def actor_gate(p_gate: np.ndarray, n_tok: np.ndarray, M: int, lib=None) -> Tuple[np.ndarray, np.ndarray, int]:
    """Gate of the deterministic actor (Sec. 3.2; App. A.2-A.3): image b opens
    when p_gate[b] >= 0.5 and some even budget 2..2M leaves >= 4 visual
    tokens.  n_tok counts CLS.  Returns (on_rank [B], on_list [B], n_on)."""
    p_gate = np.ascontiguousarray(p_gate, dtype=np.float32)
    n_tok = np.ascontiguousarray(n_tok, dtype=np.int32)
    B = int(n_tok.shape[0])
    on_rank = np.empty(B, np.int32)
    on_list = np.empty(B, np.int32)
    n_on = np.zeros(1, np.int32)
    _load(lib).oracle_actor_gate(_ptr(p_gate), _ptr(n_tok), B, int(M), _ptr(on_rank), _ptr(on_list), _ptr(n_on))
    return on_rank, on_list, int(n_on[0])


def actor_budget(logits: np.ndarray, n_tok: np.ndarray, on_rank: np.ndarray, lib=None) -> np.ndarray:
    """Keep counts: n_tok - k for gate-on images, k the legal budget with the
    largest logit (row on_rank[b] of logits [rows, M]); n_tok otherwise."""
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    n_tok = np.ascontiguousarray(n_tok, dtype=np.int32)
    on_rank = np.ascontiguousarray(on_rank, dtype=np.int32)
    B = int(n_tok.shape[0])
    keep = np.empty(B, np.int32)
    _load(lib).oracle_actor_budget(_ptr(logits), int(logits.shape[1]), _ptr(n_tok), _ptr(on_rank), B, _ptr(keep))
    return keep


def negate(s: np.ndarray, lib=None) -> np.ndarray:
    """Keep-scores from removal scores: -s."""
    s = np.ascontiguousarray(s, dtype=np.float32)
    out = np.empty_like(s)
    _load(lib).oracle_negate(_ptr(s), s.size, _ptr(out))
    return out


def _pl_geometry(s, cu_in, B, N):
    s = np.ascontiguousarray(s, dtype=np.float32)
    if cu_in is None:
        N = int(s.shape[1]) if N is None else N
        return s, None, B * N, N
    cu = np.ascontiguousarray(cu_in, dtype=np.int32)
    if N is None:
        N = int(np.max(np.diff(cu))) if B else 1
    return s, cu, int(s.shape[0]), N


def pl_sample(s: np.ndarray, g: np.ndarray, k: np.ndarray, cu_in: Optional[np.ndarray] = None,
              N: Optional[int] = None, lib=None) -> Tuple[np.ndarray, np.ndarray, np.ndarray, int]:
    """Plackett-Luce deletion by Gumbel-top-k: removal scores s and noise g
    ([B,N] dense or [total_in] with cu_in), k [B] draws per image.  Returns
    (order [sum k], cu_order [B+1], logprob [B] fp64, status)."""
    k = np.ascontiguousarray(k, dtype=np.int32)
    B = int(k.shape[0])
    s, cu, total_in, N = _pl_geometry(s, cu_in, B, N)
    g = np.ascontiguousarray(g, dtype=np.float32)
    cap = int(np.clip(k.astype(np.int64), 0, None).sum())
    order = np.zeros(max(cap, 1), np.int32)
    cu_order = np.zeros(B + 1, np.int32)
    lp = np.zeros(B, np.float64)
    st = _load(lib).oracle_pl_sample(_ptr(s), _ptr(g), _ptr(k), _ptr(cu), total_in, B, int(N), _ptr(order),
                                     _ptr(cu_order), _ptr(lp), cap)
    if st:
        return np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0), int(st)
    return order[:cap], cu_order, lp, 0


def pl_logprob(s: np.ndarray, order: np.ndarray, cu_order: np.ndarray, cu_in: Optional[np.ndarray] = None,
               N: Optional[int] = None, lib=None) -> Tuple[np.ndarray, int]:
    """Ordered Plackett-Luce log-probability (Eq. (app-actor-pl)) of given
    drawing orders under removal scores s.  Returns (logprob [B], status)."""
    cu_order = np.ascontiguousarray(cu_order, dtype=np.int32)
    B = int(cu_order.shape[0]) - 1
    s, cu, total_in, N = _pl_geometry(s, cu_in, B, N)
    order = np.ascontiguousarray(order, dtype=np.int32)
    if order.size == 0:
        order = np.zeros(1, np.int32)
    lp = np.zeros(B, np.float64)
    st = _load(lib).oracle_pl_logprob(_ptr(s), _ptr(order), _ptr(cu_order), _ptr(cu), total_in, B, int(N), _ptr(lp))
    return lp, int(st)


def lc1_readout(x: np.ndarray, cu: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float, dtype: str,
                lib=None) -> np.ndarray:
    """[B, 2C] fp64: LayerNorm of each image's CLS row next to the mean of the
    LayerNorms of its other rows (App. E.3, DINOv2 LC1 readout).  x: packed
    [total, C] bf16 bits or fp32; gamma, beta: fp32 [C]."""
    xd = np.ascontiguousarray(widen(x, dtype))
    total, C = xd.shape
    cu = np.ascontiguousarray(cu, dtype=np.int32)
    B = int(cu.shape[0]) - 1
    g = np.ascontiguousarray(np.asarray(gamma, np.float32).astype(np.float64))
    bt = np.ascontiguousarray(np.asarray(beta, np.float32).astype(np.float64))
    out = np.zeros((B, 2 * C))
    with np.errstate(invalid="ignore"):
        _load(lib).oracle_lc1_readout(_ptr(xd), _ptr(cu), B, C, _ptr(g), _ptr(bt), float(eps), _ptr(out))
    return out


# --- FLOP accounting of a realised token trajectory (App. E.4) -------------
#
# One multiply-accumulate counts as two FLOPs; counted are the products of
# the linear layers, the patch-embedding convolution and the two attention
# products (the paper's accounting also lists no other operation kind; see
# the tests for how close this comes to its Native figures).

def _attention_block_macs(n: int, d: int, r: int) -> Tuple[int, int]:
    """MACs of one pre-LN Transformer block of width d over n tokens, split
    into the attention part (QKV, Q K^T, P V, output projection) and the MLP
    part (d -> r d -> d) per token."""
    attn = n * d * 3 * d + n * n * d + n * n * d + n * d * d
    mlp_per_token = d * r * d + r * d * d
    return attn, mlp_per_token


def actor_gate_macs(d: int, gate_hidden: int = 64, embed: int = 16, hist: int = 3) -> int:
    """Gate MLP (d + 16 + 3) -> 64 -> 1 on the CLS key (App. A.1)."""
    return (d + embed + hist) * gate_hidden + gate_hidden * 1


def actor_controller_macs(n: int, d: int, M: int, width: int = 128, heads: int = 4, ffn: int = 256,
                          budget_hidden: int = 128, sel_hidden: int = 64, hist: int = 3) -> int:
    """Controller of a gate-on block over n tokens (CLS included; App. A.1):
    input projection d -> 128 of every key and 3 -> 128 of the history into
    CLS; one width-128 Transformer block (QKV, Q K^T, P V, projection, FFN
    128 -> 256 -> 128); budget head 128 -> 128 -> M on CLS; the 1 -> 128
    projection of k / N; selector 128 -> 64 -> 1 on the n - 1 visual tokens."""
    enc_in = n * d * width + hist * width
    attn, mlp_tok = _attention_block_macs(n, width, ffn // width)
    block = attn + n * mlp_tok
    budget = width * budget_hidden + budget_hidden * M
    selector = 1 * width + (n - 1) * (width * sel_hidden + sel_hidden * 1)
    return enc_in + block + budget + selector


def trajectory_flops(tokens: np.ndarray, d: int, L: int, N0: int, patch: int, M: int, mlp_ratio: int = 4,
                     in_chans: int = 3, classes: int = 1000, head_inputs: int = 1, actor: bool = True
                     ) -> np.ndarray:
    """FLOPs per image of the complete forward along its realised token
    trajectory (App. E.4, Eq. (app-experiments-flops) before averaging).
    tokens: int [L+1, B]; tokens[l] enters block l (N_l + 1, CLS included) and
    tokens[l+1] is what its MLP keeps (N_l - k_l + 1); tokens[0] = N0 + 1.
    Block l: attention over tokens[l], MLP over tokens[l+1]; with the actor,
    the gate runs at every block with a legal budget (N_l >= 6) and the
    controller wherever tokens were removed.  Plus the patch embedding
    (in_chans * patch^2 -> d per patch) and the classifier
    (head_inputs * d -> classes)."""
    T = np.asarray(tokens, dtype=np.int64)
    if T.shape[0] != L + 1:
        raise ValueError("tokens must be [L+1, B]")
    out = np.zeros(T.shape[1], dtype=np.int64)
    for b in range(T.shape[1]):
        macs = N0 * (in_chans * patch * patch) * d + head_inputs * d * classes
        for l in range(L):
            n, m = int(T[l, b]), int(T[l + 1, b])
            attn, mlp_tok = _attention_block_macs(n, d, mlp_ratio)
            macs += attn + m * mlp_tok
            if actor:
                if n - 1 >= 6:
                    macs += actor_gate_macs(d)
                if m < n:
                    macs += actor_controller_macs(n, d, M)
        out[b] = 2 * macs
    return out


def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 value of bf16 bit patterns (uint16) or fp32 values."""
    if dtype == "bf16":
        return (np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def varlen_attn(q: np.ndarray, k: np.ndarray, v: np.ndarray, cu: np.ndarray, dtype: str,
                scale: Optional[float] = None, threads: int = 0, lib=None) -> np.ndarray:
    """Exact fp64 softmax attention per sequence of the packed [total, H, D] inputs."""
    qd, kd, vd = (np.ascontiguousarray(widen(a, dtype)) for a in (q, k, v))
    total, H, D = qd.shape
    cu = np.ascontiguousarray(cu, dtype=np.int32)
    B = int(cu.shape[0]) - 1
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    out = np.zeros_like(qd)
    _load(lib).oracle_varlen_attn(_ptr(qd), _ptr(kd), _ptr(vd), _ptr(cu), B, H, D, float(scale),
                               _ptr(out), int(threads))
    return out


def varlen_attn_rows(q, k, v, cu, rows, dtype: str, scale: Optional[float] = None, lib=None) -> np.ndarray:
    """Oracle outputs of selected packed query rows only: [len(rows), H, D] fp64
    (each row attends to every key of its own sequence)."""
    qd, kd, vd = (np.ascontiguousarray(widen(a, dtype)) for a in (q, k, v))
    total, H, D = qd.shape
    cu = np.ascontiguousarray(cu, dtype=np.int32)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    out = np.zeros((len(rows), H, D))
    _load(lib).oracle_varlen_attn_rows(_ptr(qd), _ptr(kd), _ptr(vd), _ptr(cu), int(cu.shape[0]) - 1, H, D,
                                       float(scale), _ptr(rows), len(rows), _ptr(out))
    return out


def varlen_attn_segments(q, k, v, cu, segments, dtype: str, scale: Optional[float] = None,
                         threads: int = 0):
    """Oracle outputs for a subset of sequences only: {b: [len_b, H, D] fp64}."""
    res = {}
    for b in segments:
        s, e = int(cu[b]), int(cu[b + 1])
        sub_cu = np.array([0, e - s], dtype=np.int32)
        res[b] = varlen_attn(q[s:e], k[s:e], v[s:e], sub_cu, dtype, scale, threads)
    return res
