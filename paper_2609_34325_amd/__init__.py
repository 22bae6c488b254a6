"""DORA deployment hot path on AMD Instinct MI355X (gfx950).

Thin ctypes binding over ``libdora.so`` (C ABI in ``include/dora.h``).  Every
step of the path runs in the library's HIP kernels; this module only checks
tensor arguments, allocates outputs with torch when the caller does not pass
them, and forwards raw device pointers and the current HIP stream.

DORA (arXiv 2609.34325): hard deletion keeps CLS and the survivors' order
(Sec. 3.1, Eq. (1)); deployment removes the highest-scoring visual tokens
(Sec. 3.2 "Sampling and deployment"; App. A.3); survivors are packed with
explicit sequence boundaries and run through variable-length attention that
never attends across images (Sec. 3.5 "Inference"; App. E.5).

There is no fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdora.so")

DORA_F32 = 0
DORA_BF16 = 1

DORA_OK = 0
DORA_ERR_NULL = -1
DORA_ERR_SHAPE = -2
DORA_ERR_DTYPE = -3
DORA_ERR_ALIGN = -4
DORA_ERR_UNSUPPORTED = -5
DORA_ERR_CAPACITY = -6
DORA_ERR_HIP = -7
DORA_ERR_WORKSPACE = -8
DORA_ERR_STATIC_LIMIT = -9

DORA_DEV_KEEP_RANGE = 0x1
DORA_DEV_CAPACITY = 0x2
DORA_DEV_CU_IN = 0x4
DORA_DEV_CU_SEQLENS = 0x8
DORA_DEV_PLAN = 0x10

DORA_DEV_ACTOR = 0x20
DORA_MAX_ROW_TOKENS = 2048
DORA_MAX_SEQLEN = 16384
DORA_HEAD_DIM = 64
DORA_NOALLOC_WORKSPACE_BYTES = 4 << 20

EXPORTS = (
    "dora_select_pack",
    "dora_select_pack_plan",
    "dora_select_pack_residual",
    "dora_actor_gate",
    "dora_actor_decode",
    "dora_pl_sample",
    "dora_pl_logprob",
    "dora_lc1_readout_workspace_size",
    "dora_lc1_readout",
    "dora_trajectory_flops",
    "dora_varlen_attn_workspace_size",
    "dora_varlen_attn_plan",
    "dora_varlen_attn_execute",
    "dora_varlen_attn",
    "dora_varlen_attn_noalloc",
    "dora_status_string",
)

_lib = None


class FlopsConfig(ctypes.Structure):
    """dora_flops_config of include/dora.h."""
    _fields_ = [(name, ctypes.c_int32) for name in
                ("d", "L", "N0", "patch", "in_chans", "classes", "head_inputs", "mlp_ratio", "M", "actor")]


class DoraError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {dora_status_string(code)} ({code})")
        self.code = code


def load_library(path: Optional[str] = None) -> ctypes.CDLL:
    """Load libdora.so (built in-tree by ``paper_2609_34325_amd.build``)."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"libdora.so not found at {p}; build it with "
                           "`python -m paper_2609_34325_amd.build` (no fallback path exists)")
    lib = ctypes.CDLL(p)
    vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.dora_select_pack.restype = ctypes.c_int
    lib.dora_select_pack.argtypes = [vp, vp, vp, vp, i64, i32, i32, i32, ctypes.c_int,
                                     vp, vp, vp, i64, vp, vp]
    lib.dora_select_pack_plan.restype = ctypes.c_int
    lib.dora_select_pack_plan.argtypes = lib.dora_select_pack.argtypes[:13] + [i32, i32, i64, vp, sz,
                                                                               vp, vp]
    lib.dora_select_pack_residual.restype = ctypes.c_int
    lib.dora_select_pack_residual.argtypes = lib.dora_select_pack.argtypes[:3] + [vp] + \
        lib.dora_select_pack.argtypes[3:]
    lib.dora_actor_gate.restype = ctypes.c_int
    lib.dora_actor_gate.argtypes = [vp, vp, i32, i32, i32, vp, vp, vp, vp, vp]
    lib.dora_actor_decode.restype = ctypes.c_int
    lib.dora_actor_decode.argtypes = [vp, i64, i32, vp, vp, i64, i32, i32, vp, vp, vp, vp, vp]
    lib.dora_pl_sample.restype = ctypes.c_int
    lib.dora_pl_sample.argtypes = [vp, vp, vp, vp, i64, i32, i32, vp, vp, vp, i64, vp, vp]
    lib.dora_pl_logprob.restype = ctypes.c_int
    lib.dora_pl_logprob.argtypes = [vp, vp, vp, vp, i64, i32, i32, vp, vp, vp]
    lib.dora_lc1_readout.restype = ctypes.c_int
    lib.dora_lc1_readout.argtypes = [vp, vp, i64, i32, i32, ctypes.c_int, vp, vp, ctypes.c_float, vp, vp, sz, vp,
                                     vp]
    lib.dora_lc1_readout_workspace_size.restype = sz
    lib.dora_lc1_readout_workspace_size.argtypes = [i32, i32]
    lib.dora_trajectory_flops.restype = ctypes.c_int
    lib.dora_trajectory_flops.argtypes = [vp, i32, ctypes.POINTER(FlopsConfig), vp, vp, vp, vp]
    lib.dora_varlen_attn_workspace_size.restype = sz
    lib.dora_varlen_attn_workspace_size.argtypes = [i32, i32, i32]
    lib.dora_varlen_attn_plan.restype = ctypes.c_int
    lib.dora_varlen_attn_plan.argtypes = [vp, i32, i32, i32, i64, vp, sz, vp, vp]
    lib.dora_varlen_attn_execute.restype = ctypes.c_int
    lib.dora_varlen_attn_execute.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i64,
                                             ctypes.c_float, ctypes.c_int, vp, vp, sz, vp, vp]
    lib.dora_varlen_attn.restype = ctypes.c_int
    lib.dora_varlen_attn.argtypes = lib.dora_varlen_attn_execute.argtypes
    lib.dora_varlen_attn_noalloc.restype = ctypes.c_int
    lib.dora_varlen_attn_noalloc.argtypes = lib.dora_varlen_attn_execute.argtypes[:12] + [vp, vp]
    lib.dora_status_string.restype = ctypes.c_char_p
    lib.dora_status_string.argtypes = [ctypes.c_int]
    if path is None:
        _lib = lib
    return lib


def dora_status_string(code: int) -> str:
    return load_library().dora_status_string(int(code)).decode()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return DORA_BF16
    if t.dtype == torch.float32:
        return DORA_F32
    raise TypeError(f"unsupported dtype {t.dtype}; expected bfloat16 or float32")


def _dev(t: torch.Tensor, name: str, dtype=None) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


def _check(fn: str, code: int) -> None:
    if code != DORA_OK:
        raise DoraError(fn, code)


def new_status(device=None) -> torch.Tensor:
    """A zeroed int32 device status word."""
    return torch.zeros(1, dtype=torch.int32, device=device or "cuda")


def _select_pack_args(scores, keep, tokens, cu_in, N, idx_out, cu_out, packed_out, cap_rows, dev_status):
    B = int(keep.shape[0])
    if cu_in is None:
        if tokens.dim() != 3:
            raise ValueError("dense tokens must be [B,N,C]")
        N = int(tokens.shape[1])
        C = int(tokens.shape[2])
        total_in = B * N
        if tuple(scores.shape) != (B, N):
            raise ValueError("scores must be [B,N]")
    else:
        if tokens.dim() != 2:
            raise ValueError("packed tokens must be [total_in,C]")
        if N is None:
            raise ValueError("packed input needs N (an upper bound on segment lengths)")
        C = int(tokens.shape[1])
        total_in = int(tokens.shape[0])
        if scores.dim() != 1 or int(scores.shape[0]) < total_in:
            raise ValueError("packed scores must be [total_in]")
        if tuple(cu_in.shape) != (B + 1,):
            raise ValueError("cu_in must be [B+1]")
    dev = tokens.device
    if cap_rows is None:
        cap_rows = int(packed_out.shape[0]) if packed_out is not None else B * int(N)
    if idx_out is None:
        idx_out = torch.empty(cap_rows, dtype=torch.int32, device=dev)
    if cu_out is None:
        cu_out = torch.empty(B + 1, dtype=torch.int32, device=dev)
    if packed_out is None:
        packed_out = torch.empty((cap_rows, C), dtype=tokens.dtype, device=dev)
    if dev_status is None:
        dev_status = new_status(dev)
    if packed_out.dtype != tokens.dtype or int(packed_out.shape[-1]) != C:
        raise ValueError("packed_out must match the tokens' dtype and C")
    if int(idx_out.numel()) < cap_rows or int(packed_out.shape[0]) < cap_rows:
        raise ValueError("outputs smaller than cap_rows")
    args = [_dev(scores, "scores", torch.float32), _dev(keep, "keep", torch.int32),
            _dev(tokens, "tokens"), None if cu_in is None else _dev(cu_in, "cu_in", torch.int32),
            total_in, B, int(N), C, _dtype_code(tokens),
            _dev(idx_out, "idx_out", torch.int32), _dev(cu_out, "cu_out", torch.int32),
            _dev(packed_out, "packed_out"), int(cap_rows)]
    return args, (idx_out, cu_out, packed_out, dev_status)


def dora_select_pack(scores: torch.Tensor, keep: torch.Tensor, tokens: torch.Tensor,
                     cu_in: Optional[torch.Tensor] = None, N: Optional[int] = None,
                     idx_out: Optional[torch.Tensor] = None,
                     cu_out: Optional[torch.Tensor] = None,
                     packed_out: Optional[torch.Tensor] = None,
                     cap_rows: Optional[int] = None,
                     dev_status: Optional[torch.Tensor] = None,
                     stream=None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]:
    """Keep CLS + the keep-1 highest keep-scores per image, pack the kept rows.

    Dense input: scores [B,N] fp32, tokens [B,N,C].  Packed input (a cascaded
    round): scores [total_in], tokens [total_in,C], cu_in [B+1] and N = an
    upper bound on the segment lengths.  keep: int32 [B] (counts CLS).
    Outputs (allocated if not given; capacity defaults to B*N rows so no
    host synchronisation is needed): idx [cap], cu [B+1], packed [cap,C],
    dev_status [1].  Returns (idx_out, cu_out, packed_out, dev_status).
    """
    lib = load_library()
    args, outs = _select_pack_args(scores, keep, tokens, cu_in, N, idx_out, cu_out, packed_out,
                                   cap_rows, dev_status)
    rc = lib.dora_select_pack(*args, _dev(outs[3], "dev_status", torch.int32), _stream(stream))
    _check("dora_select_pack", rc)
    return outs


def dora_select_pack_plan(scores: torch.Tensor, keep: torch.Tensor, tokens: torch.Tensor,
                          H: int, max_seqlen: int, total: int, workspace: torch.Tensor,
                          cu_in: Optional[torch.Tensor] = None, N: Optional[int] = None,
                          idx_out: Optional[torch.Tensor] = None,
                          cu_out: Optional[torch.Tensor] = None,
                          packed_out: Optional[torch.Tensor] = None,
                          cap_rows: Optional[int] = None,
                          dev_status: Optional[torch.Tensor] = None,
                          stream=None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]:
    """dora_select_pack plus the attention plan of the packed output in `workspace`
    (for dora_varlen_attn_execute with cu_seqlens = cu_out, H heads, max_seqlen
    and total Q/K/V rows)."""
    lib = load_library()
    args, outs = _select_pack_args(scores, keep, tokens, cu_in, N, idx_out, cu_out, packed_out,
                                   cap_rows, dev_status)
    rc = lib.dora_select_pack_plan(*args, int(H), int(max_seqlen), int(total),
                                   _dev(workspace, "workspace"),
                                   workspace.numel() * workspace.element_size(),
                                   _dev(outs[3], "dev_status", torch.int32), _stream(stream))
    _check("dora_select_pack_plan", rc)
    return outs


def dora_select_pack_residual(scores: torch.Tensor, keep: torch.Tensor, h: torch.Tensor, a: torch.Tensor,
                              cu_in: Optional[torch.Tensor] = None, N: Optional[int] = None,
                              idx_out: Optional[torch.Tensor] = None,
                              cu_out: Optional[torch.Tensor] = None,
                              packed_out: Optional[torch.Tensor] = None,
                              cap_rows: Optional[int] = None,
                              dev_status: Optional[torch.Tensor] = None,
                              stream=None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]:
    """dora_select_pack of the attention residual h + a: the kept rows of the
    sum, each element rounded once to h's dtype.  a has h's shape and dtype."""
    if a.shape != h.shape or a.dtype != h.dtype:
        raise ValueError("a must have h's shape and dtype")
    lib = load_library()
    args, outs = _select_pack_args(scores, keep, h, cu_in, N, idx_out, cu_out, packed_out,
                                   cap_rows, dev_status)
    args.insert(3, _dev(a, "a", h.dtype))
    rc = lib.dora_select_pack_residual(*args, _dev(outs[3], "dev_status", torch.int32), _stream(stream))
    _check("dora_select_pack_residual", rc)
    return outs


def dora_actor_gate(p_gate: torch.Tensor, M: int, N: int, cu_in: Optional[torch.Tensor] = None,
                    on_rank: Optional[torch.Tensor] = None, on_list: Optional[torch.Tensor] = None,
                    n_on: Optional[torch.Tensor] = None, dev_status: Optional[torch.Tensor] = None,
                    stream=None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor, torch.Tensor]:
    """Gate decisions and the ordered list of gate-on images.  p_gate: fp32 [B];
    N tokens per image (CLS included) or cu_in [B+1]; M budget-head outputs.
    Returns (on_rank [B], on_list [B], n_on [1], dev_status)."""
    B = int(p_gate.shape[0])
    dev = p_gate.device
    if cu_in is not None and tuple(cu_in.shape) != (B + 1,):
        raise ValueError("cu_in must be [B+1]")
    on_rank = torch.empty(B, dtype=torch.int32, device=dev) if on_rank is None else on_rank
    on_list = torch.empty(B, dtype=torch.int32, device=dev) if on_list is None else on_list
    n_on = torch.empty(1, dtype=torch.int32, device=dev) if n_on is None else n_on
    dev_status = new_status(dev) if dev_status is None else dev_status
    for t, name in ((on_rank, "on_rank"), (on_list, "on_list")):
        if t.numel() < B:
            raise ValueError(f"{name} needs {B} entries")
    rc = load_library().dora_actor_gate(
        _dev(p_gate, "p_gate", torch.float32), None if cu_in is None else _dev(cu_in, "cu_in", torch.int32),
        B, int(N), int(M), _dev(on_rank, "on_rank", torch.int32), _dev(on_list, "on_list", torch.int32),
        _dev(n_on, "n_on", torch.int32), _dev(dev_status, "dev_status", torch.int32), _stream(stream))
    _check("dora_actor_gate", rc)
    return on_rank, on_list, n_on, dev_status


def dora_actor_decode(budget_logits: torch.Tensor, on_rank: torch.Tensor, N: int,
                      removal_scores: Optional[torch.Tensor] = None, cu_in: Optional[torch.Tensor] = None,
                      keep_out: Optional[torch.Tensor] = None, scores_out: Optional[torch.Tensor] = None,
                      dev_status: Optional[torch.Tensor] = None,
                      stream=None) -> Tuple[torch.Tensor, Optional[torch.Tensor], torch.Tensor]:
    """Keep counts from the budget logits [rows, M] (row r = gate-on image r)
    and, if removal_scores is given, keep-scores = -removal_scores in the same
    layout.  Returns (keep [B], keep-scores or None, dev_status)."""
    B = int(on_rank.shape[0])
    dev = on_rank.device
    if budget_logits.dim() != 2:
        raise ValueError("budget_logits must be [rows, M]")
    rows, M = int(budget_logits.shape[0]), int(budget_logits.shape[1])
    keep_out = torch.empty(B, dtype=torch.int32, device=dev) if keep_out is None else keep_out
    if removal_scores is not None and scores_out is None:
        scores_out = torch.empty_like(removal_scores)
    if (removal_scores is None) != (scores_out is None):
        raise ValueError("removal_scores and scores_out go together")
    if removal_scores is not None and scores_out.shape != removal_scores.shape:
        raise ValueError("scores_out must have removal_scores' shape")
    if cu_in is None:
        total_in = B * int(N)
        if removal_scores is not None and tuple(removal_scores.shape) != (B, int(N)):
            raise ValueError("dense removal_scores must be [B,N]")
    else:
        if tuple(cu_in.shape) != (B + 1,):
            raise ValueError("cu_in must be [B+1]")
        total_in = int(removal_scores.shape[0]) if removal_scores is not None else 0
    dev_status = new_status(dev) if dev_status is None else dev_status
    rc = load_library().dora_actor_decode(
        _dev(budget_logits, "budget_logits", torch.float32) if rows > 0 else None, rows, M,
        None if removal_scores is None else _dev(removal_scores, "removal_scores", torch.float32),
        None if cu_in is None else _dev(cu_in, "cu_in", torch.int32), total_in, B, int(N),
        _dev(on_rank, "on_rank", torch.int32), _dev(keep_out, "keep_out", torch.int32),
        None if scores_out is None else _dev(scores_out, "scores_out", torch.float32),
        _dev(dev_status, "dev_status", torch.int32), _stream(stream))
    _check("dora_actor_decode", rc)
    return keep_out, scores_out, dev_status


def _pl_geometry(scores, B, cu_in, N):
    if cu_in is None:
        if scores.dim() != 2 or int(scores.shape[0]) != B:
            raise ValueError("dense scores must be [B,N]")
        return int(scores.shape[1]), B * int(scores.shape[1])
    if tuple(cu_in.shape) != (B + 1,) or scores.dim() != 1:
        raise ValueError("packed scores must be [total_in] with cu_in [B+1]")
    if N is None:
        raise ValueError("packed input needs N (an upper bound on segment lengths)")
    return int(N), int(scores.shape[0])


def dora_pl_sample(scores: torch.Tensor, gumbel: torch.Tensor, k: torch.Tensor,
                   cu_in: Optional[torch.Tensor] = None, N: Optional[int] = None,
                   order_out: Optional[torch.Tensor] = None, cu_order_out: Optional[torch.Tensor] = None,
                   logprob_out: Optional[torch.Tensor] = None, cap: Optional[int] = None,
                   dev_status: Optional[torch.Tensor] = None, stream=None):
    """Gumbel-top-k Plackett-Luce draws of k[b] visual tokens per image (removal
    scores + noise), in drawing order, and their ordered log-probability.
    Returns (order [cap], cu_order [B+1], logprob [B], dev_status)."""
    B = int(k.shape[0])
    N, total_in = _pl_geometry(scores, B, cu_in, N)
    if gumbel.shape != scores.shape:
        raise ValueError("gumbel must have the scores' shape")
    dev = scores.device
    cap = (int(order_out.numel()) if order_out is not None else B * max(N - 1, 1)) if cap is None else cap
    order_out = torch.empty(cap, dtype=torch.int32, device=dev) if order_out is None else order_out
    cu_order_out = torch.empty(B + 1, dtype=torch.int32, device=dev) if cu_order_out is None else cu_order_out
    logprob_out = torch.empty(B, dtype=torch.float32, device=dev) if logprob_out is None else logprob_out
    dev_status = new_status(dev) if dev_status is None else dev_status
    if order_out.numel() < cap:
        raise ValueError("order_out smaller than cap")
    rc = load_library().dora_pl_sample(
        _dev(scores, "scores", torch.float32), _dev(gumbel, "gumbel", torch.float32), _dev(k, "k", torch.int32),
        None if cu_in is None else _dev(cu_in, "cu_in", torch.int32), total_in, B, N,
        _dev(order_out, "order_out", torch.int32), _dev(cu_order_out, "cu_order_out", torch.int32),
        _dev(logprob_out, "logprob_out", torch.float32), int(cap), _dev(dev_status, "dev_status", torch.int32),
        _stream(stream))
    _check("dora_pl_sample", rc)
    return order_out, cu_order_out, logprob_out, dev_status


def dora_pl_logprob(scores: torch.Tensor, order: torch.Tensor, cu_order: torch.Tensor,
                    cu_in: Optional[torch.Tensor] = None, N: Optional[int] = None,
                    logprob_out: Optional[torch.Tensor] = None, dev_status: Optional[torch.Tensor] = None,
                    stream=None):
    """Ordered log-probability of given draws (order, cu_order) under scores.
    Returns (logprob [B], dev_status)."""
    B = int(cu_order.shape[0]) - 1
    N, total_in = _pl_geometry(scores, B, cu_in, N)
    dev = scores.device
    logprob_out = torch.empty(B, dtype=torch.float32, device=dev) if logprob_out is None else logprob_out
    dev_status = new_status(dev) if dev_status is None else dev_status
    rc = load_library().dora_pl_logprob(
        _dev(scores, "scores", torch.float32), _dev(order, "order", torch.int32),
        _dev(cu_order, "cu_order", torch.int32), None if cu_in is None else _dev(cu_in, "cu_in", torch.int32),
        total_in, B, N, _dev(logprob_out, "logprob_out", torch.float32),
        _dev(dev_status, "dev_status", torch.int32), _stream(stream))
    _check("dora_pl_logprob", rc)
    return logprob_out, dev_status


def dora_lc1_readout_workspace_size(B: int, C: int) -> int:
    return int(load_library().dora_lc1_readout_workspace_size(int(B), int(C)))


def new_lc1_workspace(B: int, C: int, device=None) -> torch.Tensor:
    """A workspace for dora_lc1_readout (no required contents)."""
    n = dora_lc1_readout_workspace_size(B, C)
    if n == 0:
        raise DoraError("dora_lc1_readout_workspace_size", DORA_ERR_SHAPE)
    return torch.empty(n, dtype=torch.uint8, device=device or "cuda")


def dora_lc1_readout(x: torch.Tensor, cu_seqlens: torch.Tensor, gamma: torch.Tensor, beta: torch.Tensor,
                     eps: float = 1e-6, out: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, single: bool = False,
                     dev_status: Optional[torch.Tensor] = None, stream=None):
    """LayerNorm of each packed sequence's CLS row next to the mean LayerNorm of
    its other rows: x [total, C] bf16/fp32, cu_seqlens [B+1] -> out fp32 [B, 2C].
    With a workspace (a new one when None) a sequence's rows may be
    split over several workgroups; single=True passes none (one workgroup per
    sequence).  Returns (out, dev_status)."""
    if x.dim() != 2:
        raise ValueError("x must be [total, C]")
    B = int(cu_seqlens.shape[0]) - 1
    total, C = int(x.shape[0]), int(x.shape[1])
    out = torch.empty((B, 2 * C), dtype=torch.float32, device=x.device) if out is None else out
    dev_status = new_status(x.device) if dev_status is None else dev_status
    if tuple(out.shape) != (B, 2 * C):
        raise ValueError("out must be [B, 2C]")
    if not single and workspace is None:
        workspace = new_lc1_workspace(B, C, x.device)
    ws, ws_bytes = (None, 0) if single else (_dev(workspace, "workspace"), workspace.numel() * workspace.element_size())
    rc = load_library().dora_lc1_readout(
        _dev(x, "x"), _dev(cu_seqlens, "cu_seqlens", torch.int32), total, B, C, _dtype_code(x),
        _dev(gamma, "gamma", torch.float32), _dev(beta, "beta", torch.float32), float(eps),
        _dev(out, "out", torch.float32), ws, ws_bytes, _dev(dev_status, "dev_status", torch.int32),
        _stream(stream))
    _check("dora_lc1_readout", rc)
    return out, dev_status


def dora_trajectory_flops(tokens: torch.Tensor, d: int, N0: int, patch: int, M: Optional[int] = None,
                          mlp_ratio: int = 4, in_chans: int = 3, classes: int = 1000, head_inputs: int = 1,
                          actor: bool = True, flops_out: Optional[torch.Tensor] = None,
                          total_out: Optional[torch.Tensor] = None, dev_status: Optional[torch.Tensor] = None,
                          stream=None):
    """FLOPs per image along realised token trajectories tokens [L+1, B] (int32).
    Returns (flops [B] int64, total [1] int64, dev_status)."""
    if tokens.dim() != 2:
        raise ValueError("tokens must be [L+1, B]")
    L, B = int(tokens.shape[0]) - 1, int(tokens.shape[1])
    cfg = FlopsConfig(int(d), L, int(N0), int(patch), int(in_chans), int(classes), int(head_inputs),
                      int(mlp_ratio), int((N0 - 4) // 2 if M is None else M), int(bool(actor)))
    dev = tokens.device
    flops_out = torch.empty(B, dtype=torch.int64, device=dev) if flops_out is None else flops_out
    total_out = torch.empty(1, dtype=torch.int64, device=dev) if total_out is None else total_out
    dev_status = new_status(dev) if dev_status is None else dev_status
    rc = load_library().dora_trajectory_flops(
        _dev(tokens, "tokens", torch.int32), B, ctypes.byref(cfg), _dev(flops_out, "flops_out", torch.int64),
        _dev(total_out, "total_out", torch.int64), _dev(dev_status, "dev_status", torch.int32), _stream(stream))
    _check("dora_trajectory_flops", rc)
    return flops_out, total_out, dev_status


def dora_varlen_attn_workspace_size(B: int, H: int, max_seqlen: int) -> int:
    return int(load_library().dora_varlen_attn_workspace_size(int(B), int(H), int(max_seqlen)))


def new_workspace(B: int, H: int, max_seqlen: int, device=None) -> torch.Tensor:
    n = dora_varlen_attn_workspace_size(B, H, max_seqlen)
    if n == 0:
        raise DoraError("dora_varlen_attn_workspace_size", DORA_ERR_SHAPE)
    return torch.empty(n, dtype=torch.uint8, device=device or "cuda")


def dora_varlen_attn_plan(cu_seqlens: torch.Tensor, H: int, max_seqlen: int, total: int,
                          workspace: torch.Tensor, dev_status: torch.Tensor, stream=None) -> None:
    lib = load_library()
    B = int(cu_seqlens.shape[0]) - 1
    rc = lib.dora_varlen_attn_plan(_dev(cu_seqlens, "cu_seqlens", torch.int32), B, int(H),
                                   int(max_seqlen), int(total), _dev(workspace, "workspace"),
                                   workspace.numel() * workspace.element_size(),
                                   _dev(dev_status, "dev_status", torch.int32), _stream(stream))
    _check("dora_varlen_attn_plan", rc)


def _attn_args(q, k, v, cu_seqlens, out):
    if q.dim() != 3 or q.shape != k.shape or q.shape != v.shape:
        raise ValueError("q, k, v must share the shape [total, H, 64]")
    if q.dtype != k.dtype or q.dtype != v.dtype:
        raise TypeError("q, k, v must share one dtype")
    total, H, D = (int(x) for x in q.shape)
    if out is None:
        out = torch.empty_like(q)
    if out.shape != q.shape or out.dtype != q.dtype:
        raise ValueError("out must match q")
    return total, H, D, out


def dora_varlen_attn_execute(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor,
                             cu_seqlens: torch.Tensor, max_seqlen: int, workspace: torch.Tensor,
                             out: Optional[torch.Tensor] = None, softmax_scale: float = 0.0,
                             dev_status: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    lib = load_library()
    total, H, D, out = _attn_args(q, k, v, cu_seqlens, out)
    if dev_status is None:
        dev_status = new_status(q.device)
    B = int(cu_seqlens.shape[0]) - 1
    rc = lib.dora_varlen_attn_execute(
        _dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(cu_seqlens, "cu_seqlens", torch.int32),
        B, H, D, int(max_seqlen), total, float(softmax_scale), _dtype_code(q), _dev(out, "out"),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        _dev(dev_status, "dev_status", torch.int32), _stream(stream))
    _check("dora_varlen_attn_execute", rc)
    return out


def dora_varlen_attn(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, cu_seqlens: torch.Tensor,
                     max_seqlen: int, out: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, softmax_scale: float = 0.0,
                     dev_status: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """softmax(scale * Q K^T) V inside each packed sequence; q/k/v/out [total, H, 64]."""
    lib = load_library()
    total, H, D, out = _attn_args(q, k, v, cu_seqlens, out)
    B = int(cu_seqlens.shape[0]) - 1
    if workspace is None:
        workspace = new_workspace(B, H, max_seqlen, q.device)
    if dev_status is None:
        dev_status = new_status(q.device)
    rc = lib.dora_varlen_attn(
        _dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(cu_seqlens, "cu_seqlens", torch.int32),
        B, H, D, int(max_seqlen), total, float(softmax_scale), _dtype_code(q), _dev(out, "out"),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        _dev(dev_status, "dev_status", torch.int32), _stream(stream))
    _check("dora_varlen_attn", rc)
    return out


def dora_varlen_attn_noalloc(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, cu_seqlens: torch.Tensor,
                             max_seqlen: int, out: torch.Tensor, softmax_scale: float = 0.0,
                             dev_status: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """dora_varlen_attn with the library's static per-GPU workspace: no device
    allocation in the call (out and dev_status must be given).  Calls that
    overlap in time on one GPU race on that workspace."""
    if out is None or dev_status is None:
        raise ValueError("dora_varlen_attn_noalloc allocates nothing: pass out and dev_status")
    lib = load_library()
    total, H, D, out = _attn_args(q, k, v, cu_seqlens, out)
    B = int(cu_seqlens.shape[0]) - 1
    rc = lib.dora_varlen_attn_noalloc(
        _dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(cu_seqlens, "cu_seqlens", torch.int32),
        B, H, D, int(max_seqlen), total, float(softmax_scale), _dtype_code(q), _dev(out, "out"),
        _dev(dev_status, "dev_status", torch.int32), _stream(stream))
    _check("dora_varlen_attn_noalloc", rc)
    return out
