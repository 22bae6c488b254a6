"""Seeded synthetic inputs for the DORA deployment hot path.

This module only draws random inputs.  It holds none of the method's
arithmetic (no selection, packing or attention) and is shared by the tests,
the benchmark and the oracle checks so that both sides of every parity
comparison see the same bytes.

The six workloads mirror the shapes of the paper's backbones (Sec. 4.1 and
Table 3: patch-16 ViTs with 196 visual tokens plus CLS, d = 768 for DeiT-B /
ViT-B, d = 1024 for ViT-L) and the ragged, per-image keep counts that an
input-adaptive pruning policy produces (Sec. 3.1, Fig. 3).  ImageNet images,
trained backbones and a trained actor are not available, so keep counts,
scores, tokens and Q/K/V are drawn from the stated distributions instead.

Conventions
-----------
* Every quantity of every round draws from its own PCG64 stream,
  ``numpy.random.default_rng([seed, round, part])`` with part 0..5 for
  keep, scores, tokens (first round only), Q, K, V, and part 6 for the
  attention branch's output that the residual variant adds to the tokens,
  parts 7-9 for the actor's gate probabilities, budget logits and removal
  scores, part 10 for Gumbel noise and part 11 for the readout rows, so
  any subset can be drawn without changing the others.
* Keep counts derived from a ratio r use ``clip(rint(r * n), 1, n)``.
* bf16 values are the round-to-nearest-even truncation of the float32 draw,
  stored as raw ``uint16`` bit patterns.
* ``keep`` counts CLS (position 0 of every image segment).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np

HEAD_DIM = 64


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round-to-nearest-even); return uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    if nan.any():
        out[nan] = ((u[nan] >> 16) | 0x0040).astype(np.uint16)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    B: int
    N: int
    H: int
    dtype: str            # "f32" or "bf16"
    keep_rule: str
    rounds: int = 1
    description: str = ""

    @property
    def C(self) -> int:
        return self.H * HEAD_DIM

    @property
    def elt(self) -> int:
        return 4 if self.dtype == "f32" else 2


WORKLOADS = {
    w.name: w
    for w in [
        Workload("deit_tiny_fp32", 1, 4, 197, 3, "f32", "uniform_int_20_197",
                 description="DeiT-Tiny shape, fp32: B=4, N=197, H=3, C=192, keep ~ U{20..197}"),
        Workload("deit_s_bf16", 2, 64, 197, 6, "bf16", "ratio_uniform_0.4_1.0",
                 description="DeiT-Small shape, bf16: B=64, N=197, H=6, C=384, keep ratio ~ U[0.4,1.0]"),
        Workload("deit_b_bf16", 3, 256, 197, 12, "bf16", "ratio_beta43_0.3_1.0",
                 description="DeiT-Base shape, bf16: B=256, N=197, H=12, C=768, keep ratio 0.3+0.7*Beta(4,3)"),
        Workload("vit_l_cascade_bf16", 4, 256, 197, 16, "bf16", "cascade_uniform_0.6_0.95", rounds=3,
                 description="ViT-Large shape, bf16, 3 cascaded rounds: B=256, N=197, H=16, C=1024, "
                             "each round keeps ~U[0.6,0.95] of the current tokens"),
        Workload("vit_b384_skew_bf16", 5, 64, 577, 12, "bf16", "bimodal_skew",
                 description="ViT-Base/384 shape, bf16, skewed: B=64, N=577, H=12, C=768, "
                             "half keep 90-100%, half keep 8-15%, scores with a spatial bump"),
        Workload("dinov2_b14_bf16", 6, 256, 257, 12, "bf16", "ratio_beta43_0.3_1.0",
                 description="DINOv2-B/14 shape, bf16: B=256, N=257 (256 patches + CLS), H=12, C=768, "
                             "keep ratio 0.3+0.7*Beta(4,3)"),
    ]
}

HEADLINE = "deit_b_bf16"


@dataclass
class RoundInputs:
    """Inputs of one select -> pack -> attention pass."""
    keep: np.ndarray                 # int32 [B]
    scores: Optional[np.ndarray]     # float32 [B,N] (dense) or [sum n_in] (packed, later rounds)
    n_in: np.ndarray                 # int32 [B] segment lengths of the input
    tokens: Optional[np.ndarray]     # [B,N,C] or None (later cascade rounds use the previous packed output)
    q: Optional[np.ndarray]          # [sum keep, H, 64]
    k: Optional[np.ndarray]
    v: Optional[np.ndarray]
    attn_out: Optional[np.ndarray] = None  # [B,N,C] (first round) or [sum n_in, C]: attention branch output

    @property
    def total_keep(self) -> int:
        return int(self.keep.astype(np.int64).sum())


def _normal(rng: np.random.Generator, shape, dtype: str) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    return x if dtype == "f32" else f32_to_bf16_bits(x)


def _ratio_keep(r: np.ndarray, n: np.ndarray) -> np.ndarray:
    return np.clip(np.rint(r * n), 1, n).astype(np.int32)


def _draw_keep(w: Workload, rng: np.random.Generator, n: np.ndarray) -> np.ndarray:
    B = w.B
    if w.keep_rule == "uniform_int_20_197":
        return rng.integers(20, 198, size=B).astype(np.int32)
    if w.keep_rule == "ratio_uniform_0.4_1.0":
        return _ratio_keep(rng.uniform(0.4, 1.0, size=B), n)
    if w.keep_rule == "ratio_beta43_0.3_1.0":
        return _ratio_keep(0.3 + 0.7 * rng.beta(4.0, 3.0, size=B), n)
    if w.keep_rule == "cascade_uniform_0.6_0.95":
        return _ratio_keep(rng.uniform(0.6, 0.95, size=B), n)
    if w.keep_rule == "bimodal_skew":
        high = np.zeros(B, dtype=bool)
        high[rng.permutation(B)[: B // 2]] = True
        r = np.where(high, rng.uniform(0.90, 1.00, size=B), rng.uniform(0.08, 0.15, size=B))
        return _ratio_keep(r, n)
    raise ValueError(w.keep_rule)


def _draw_scores(w: Workload, rng: np.random.Generator, n: np.ndarray) -> np.ndarray:
    total = int(n.sum())
    s = rng.standard_normal(size=total, dtype=np.float32)
    if w.keep_rule == "bimodal_skew":
        # Salient-region bump on the 24x24 patch grid; CLS (position 0) gets none.
        side = int(round(np.sqrt(w.N - 1)))
        A = rng.uniform(1.0, 3.0, size=w.B)
        sigma = rng.uniform(1.5, 4.0, size=w.B)
        centre = rng.uniform(0.0, float(side), size=(w.B, 2))
        pos = np.arange(1, w.N) - 1
        row, col = pos // side, pos % side
        s = s.reshape(w.B, w.N).astype(np.float64)
        d2 = (row[None, :] - centre[:, 0:1]) ** 2 + (col[None, :] - centre[:, 1:2]) ** 2
        s[:, 1:] += A[:, None] * np.exp(-d2 / (2.0 * sigma[:, None] ** 2))
        s = s.astype(np.float32).reshape(-1)
    return s


PARTS = ("keep", "scores", "tokens", "qkv")
ATTN_OUT_STD = 0.5   # attention-branch output relative to the unit-variance residual stream


def _rng(seed: int, rnd: int, part: int) -> np.random.Generator:
    return np.random.default_rng([seed, rnd, part])


def generate(w: Workload, seed: Optional[int] = None, batch: Optional[int] = None,
             parts=PARTS) -> List[RoundInputs]:
    """Draw all rounds of workload ``w``.

    ``batch`` optionally overrides B (used for reduced-size parity cases); the
    seed then still fixes every draw.  ``parts`` limits what is drawn (keep
    counts are always drawn; missing parts are None).  Later cascade rounds
    take their segment lengths from the previous round's keep counts; their
    token input is the previous round's packed output and their segment
    offsets are the previous round's ``cu_seqlens``, both produced by
    whichever side (oracle or GPU) ran that round, so ``tokens`` is None there.
    """
    if batch is not None:
        w = Workload(w.name, w.seed, batch, w.N, w.H, w.dtype, w.keep_rule, w.rounds, w.description)
    sd = w.seed if seed is None else seed
    n = np.full(w.B, w.N, dtype=np.int32)
    rounds: List[RoundInputs] = []
    for r in range(w.rounds):
        keep = _draw_keep(w, _rng(sd, r, 0), n)
        scores = _draw_scores(w, _rng(sd, r, 1), n) if "scores" in parts else None
        tokens = None
        if r == 0:
            if scores is not None:
                scores = scores.reshape(w.B, w.N)
            if "tokens" in parts:
                tokens = _normal(_rng(sd, r, 2), (w.B, w.N, w.C), w.dtype)
        tot = int(keep.astype(np.int64).sum())
        q = k = v = None
        if "qkv" in parts:
            q, k, v = (_normal(_rng(sd, r, 3 + i), (tot, w.H, HEAD_DIM), w.dtype) for i in range(3))
        attn_out = None
        if "attn_out" in parts:
            shape = (w.B, w.N, w.C) if r == 0 else (int(n.astype(np.int64).sum()), w.C)
            x = _rng(sd, r, 6).standard_normal(size=shape, dtype=np.float32) * np.float32(ATTN_OUT_STD)
            attn_out = x if w.dtype == "f32" else f32_to_bf16_bits(x)
        rounds.append(RoundInputs(keep=keep, scores=scores, n_in=n.copy(), tokens=tokens, q=q, k=k, v=v,
                                  attn_out=attn_out))
        n = keep.copy()
    return rounds


def budget_outputs(w: Workload) -> int:
    """Budget-head outputs M = (N0 - 4) / 2 for N0 = N - 1 visual tokens (App. A.2, Table 3)."""
    return (w.N - 1 - 4) // 2


def actor_outputs(w: Workload, seed: Optional[int] = None):
    """Stand-ins for the trained actor's outputs on the first round of ``w``:
    gate probabilities U[0, 1] [B], budget logits N(0, 1) [B, M] (one row per
    image, enough for any number of gate-on images) and removal scores N(0, 1)
    [B, N]; parts 7, 8, 9 of round 0's streams."""
    sd = w.seed if seed is None else seed
    M = budget_outputs(w)
    p_gate = _rng(sd, 0, 7).uniform(0.0, 1.0, size=w.B).astype(np.float32)
    logits = _rng(sd, 0, 8).standard_normal(size=(w.B, M), dtype=np.float32)
    removal = _rng(sd, 0, 9).standard_normal(size=(w.B, w.N), dtype=np.float32)
    return p_gate, logits, removal


def gumbel_noise(w: Workload, seed: Optional[int] = None) -> np.ndarray:
    """Standard Gumbel noise [B, N] for a Plackett-Luce draw over the first
    round's scores (part 10 of round 0's streams)."""
    sd = w.seed if seed is None else seed
    return _rng(sd, 0, 10).gumbel(size=(w.B, w.N)).astype(np.float32)


def readout_rows(w: Workload, keep: np.ndarray, seed: Optional[int] = None):
    """Packed final-block token rows [sum keep, C] for the LC1 readout, with a
    per-channel offset N(0, 1) and scale U[0.5, 2] on N(0, 1) rows (residual
    streams carry channel-wise biases), and LayerNorm gamma U[0.5, 1.5], beta
    N(0, 0.1^2); part 11 of round 0's streams."""
    sd = w.seed if seed is None else seed
    rng = _rng(sd, 0, 11)
    off = rng.standard_normal(w.C).astype(np.float32)
    scale = rng.uniform(0.5, 2.0, w.C).astype(np.float32)
    rows = rng.standard_normal((int(keep.astype(np.int64).sum()), w.C), dtype=np.float32) * scale + off
    gamma = rng.uniform(0.5, 1.5, w.C).astype(np.float32)
    beta = (0.1 * rng.standard_normal(w.C)).astype(np.float32)
    x = rows.astype(np.float32)
    return (x if w.dtype == "f32" else f32_to_bf16_bits(x)), gamma, beta


def random_qkv(rng: np.random.Generator, lens, H: int, dtype: str):
    """Q, K, V of shape [sum(lens), H, 64] for ad-hoc attention cases."""
    tot = int(np.sum(lens))
    return tuple(_normal(rng, (tot, H, HEAD_DIM), dtype) for _ in range(3))
