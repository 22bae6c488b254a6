"""The C ABI library loads, exports every declared symbol, and rejects bad
arguments on the host before touching the GPU (CPU only; no compute calls)."""
import ctypes
import os
import re

import pytest

import paper_2609_34325_amd as dora

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dora.h")
FAKE = 0x100000  # never dereferenced: every call below fails validation first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dora_[a-z_0-9]+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_functions() == sorted(dora.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = dora.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_constants_match_header():
    text = open(HEADER).read()
    for name in ["DORA_DEV_KEEP_RANGE", "DORA_DEV_CAPACITY", "DORA_DEV_CU_IN", "DORA_DEV_CU_SEQLENS",
                 "DORA_DEV_PLAN", "DORA_DEV_ACTOR", "DORA_MAX_ROW_TOKENS", "DORA_MAX_SEQLEN", "DORA_HEAD_DIM"]:
        m = re.search(r"#define\s+%s\s+(0x[0-9a-fA-F]+|\d+)" % name, text)
        assert m and int(m.group(1), 0) == getattr(dora, name), name
    for name, val in re.findall(r"(DORA_(?:OK|ERR_[A-Z_]+))\s*=\s*(-?\d+)", text):
        assert getattr(dora, name) == int(val), name


def test_status_strings():
    assert dora.dora_status_string(0) == "DORA_OK"
    for code in range(-9, 0):
        assert dora.dora_status_string(code).startswith("DORA_ERR_")
    assert "unknown" in dora.dora_status_string(-99)


def call_select(lib, **kw):
    a = dict(scores=FAKE, keep=FAKE, tokens=FAKE, cu_in=None, total_in=0, B=4, N=197, C=768, dtype=1,
             idx=FAKE, cu=FAKE, packed=FAKE, cap=100, status=FAKE, stream=None)
    a.update(kw)
    return lib.dora_select_pack(a["scores"], a["keep"], a["tokens"], a["cu_in"], a["total_in"], a["B"],
                                a["N"], a["C"], a["dtype"], a["idx"], a["cu"], a["packed"], a["cap"],
                                a["status"], a["stream"])


def test_select_pack_host_validation():
    lib = dora.load_library()
    assert call_select(lib, scores=None) == dora.DORA_ERR_NULL
    assert call_select(lib, status=None) == dora.DORA_ERR_NULL
    assert call_select(lib, dtype=7) == dora.DORA_ERR_DTYPE
    assert call_select(lib, B=0) == dora.DORA_ERR_SHAPE
    assert call_select(lib, N=0) == dora.DORA_ERR_SHAPE
    assert call_select(lib, N=dora.DORA_MAX_ROW_TOKENS + 1) == dora.DORA_ERR_SHAPE
    assert call_select(lib, C=3) == dora.DORA_ERR_ALIGN            # 6-byte bf16 rows
    assert call_select(lib, C=6, dtype=0) == dora.DORA_ERR_ALIGN    # 24-byte fp32 rows
    assert call_select(lib, tokens=FAKE + 8) == dora.DORA_ERR_ALIGN
    assert call_select(lib, packed=FAKE + 2) == dora.DORA_ERR_ALIGN
    assert call_select(lib, cap=0) == dora.DORA_ERR_CAPACITY
    assert call_select(lib, cap=2 ** 31) == dora.DORA_ERR_CAPACITY
    assert call_select(lib, cu_in=FAKE, total_in=-1) == dora.DORA_ERR_SHAPE


def test_select_pack_residual_host_validation():
    lib = dora.load_library()

    def call(a=FAKE, **kw):
        args = dict(scores=FAKE, keep=FAKE, tokens=FAKE, cu_in=None, total_in=0, B=4, N=197, C=768, dtype=1,
                    idx=FAKE, cu=FAKE, packed=FAKE, cap=100, status=FAKE, stream=None)
        args.update(kw)
        return lib.dora_select_pack_residual(args["scores"], args["keep"], args["tokens"], a, args["cu_in"],
                                             args["total_in"], args["B"], args["N"], args["C"], args["dtype"],
                                             args["idx"], args["cu"], args["packed"], args["cap"],
                                             args["status"], args["stream"])

    assert call(a=None) == dora.DORA_ERR_NULL
    assert call(a=FAKE + 8) == dora.DORA_ERR_ALIGN
    assert call(tokens=None) == dora.DORA_ERR_NULL
    assert call(C=3) == dora.DORA_ERR_ALIGN
    assert call(dtype=7) == dora.DORA_ERR_DTYPE
    assert call(cap=0) == dora.DORA_ERR_CAPACITY
    assert call(N=dora.DORA_MAX_ROW_TOKENS + 1) == dora.DORA_ERR_SHAPE


def test_actor_host_validation():
    lib = dora.load_library()
    def gate(**kw):
        a = dict(p=FAKE, cu=None, B=4, N=197, M=96, rank=FAKE, lst=FAKE, n=FAKE, st=FAKE, s=None)
        a.update(kw)
        return lib.dora_actor_gate(*a.values())

    assert gate(p=None) == dora.DORA_ERR_NULL
    assert gate(n=None) == dora.DORA_ERR_NULL
    assert gate(B=0) == dora.DORA_ERR_SHAPE
    assert gate(B=(1 << 24) + 1) == dora.DORA_ERR_SHAPE
    assert gate(M=0) == dora.DORA_ERR_SHAPE
    assert gate(N=dora.DORA_MAX_ROW_TOKENS + 1) == dora.DORA_ERR_SHAPE

    def dec(**kw):
        a = dict(logits=FAKE, rows=4, M=96, rem=FAKE, cu=None, total=0, B=4, N=197, rank=FAKE, keep=FAKE,
                 out=FAKE, st=FAKE, s=None)
        a.update(kw)
        return lib.dora_actor_decode(*a.values())

    assert dec(rank=None) == dora.DORA_ERR_NULL
    assert dec(keep=None) == dora.DORA_ERR_NULL
    assert dec(out=None) == dora.DORA_ERR_NULL                       # scores in, no scores out
    assert dec(logits=None) == dora.DORA_ERR_NULL                    # rows > 0 need logits
    assert dec(rows=-1) == dora.DORA_ERR_SHAPE
    assert dec(M=0) == dora.DORA_ERR_SHAPE
    assert dec(B=0) == dora.DORA_ERR_SHAPE
    assert dec(cu=FAKE, total=-1) == dora.DORA_ERR_SHAPE


def test_pl_host_validation():
    lib = dora.load_library()

    def smp(**kw):
        a = dict(s=FAKE, g=FAKE, k=FAKE, cu=None, total=0, B=4, N=197, order=FAKE, cuo=FAKE, lp=FAKE, cap=100,
                 st=FAKE, stream=None)
        a.update(kw)
        return lib.dora_pl_sample(*a.values())

    def lpr(**kw):
        a = dict(s=FAKE, order=FAKE, cuo=FAKE, cu=None, total=0, B=4, N=197, lp=FAKE, st=FAKE, stream=None)
        a.update(kw)
        return lib.dora_pl_logprob(*a.values())

    assert smp(s=None) == dora.DORA_ERR_NULL
    assert smp(g=None) == dora.DORA_ERR_NULL
    assert smp(lp=None) == dora.DORA_ERR_NULL
    assert smp(B=0) == dora.DORA_ERR_SHAPE
    assert smp(B=8193) == dora.DORA_ERR_SHAPE
    assert smp(N=dora.DORA_MAX_ROW_TOKENS + 1) == dora.DORA_ERR_SHAPE
    assert smp(cu=FAKE, total=-1) == dora.DORA_ERR_SHAPE
    assert smp(cap=0) == dora.DORA_ERR_CAPACITY
    assert lpr(order=None) == dora.DORA_ERR_NULL
    assert lpr(cuo=None) == dora.DORA_ERR_NULL
    assert lpr(N=0) == dora.DORA_ERR_SHAPE


def test_lc1_host_validation():
    lib = dora.load_library()

    def call(**kw):
        a = dict(x=FAKE, cu=FAKE, total=100, B=4, C=768, dtype=1, g=FAKE, b=FAKE, eps=1e-6, out=FAKE, ws=None,
                 wsb=0, st=FAKE, stream=None)
        a.update(kw)
        return lib.dora_lc1_readout(*a.values())

    assert call(x=None) == dora.DORA_ERR_NULL
    assert call(g=None) == dora.DORA_ERR_NULL
    assert call(dtype=9) == dora.DORA_ERR_DTYPE
    assert call(C=3) == dora.DORA_ERR_ALIGN
    assert call(x=FAKE + 4) == dora.DORA_ERR_ALIGN
    assert call(C=4096) == dora.DORA_ERR_UNSUPPORTED                 # 8 KB bf16 rows
    assert call(B=0) == dora.DORA_ERR_SHAPE
    assert call(total=0) == dora.DORA_ERR_SHAPE
    assert call(eps=-1.0) == dora.DORA_ERR_SHAPE
    assert call(B=(1 << 24) + 1) == dora.DORA_ERR_SHAPE
    need = lib.dora_lc1_readout_workspace_size(4, 768)
    assert need == 4 * 8 * 768 * 4
    assert call(ws=FAKE, wsb=need - 1) == dora.DORA_ERR_WORKSPACE
    assert call(ws=FAKE + 16, wsb=need) == dora.DORA_ERR_ALIGN
    assert lib.dora_lc1_readout_workspace_size(0, 768) == 0
    assert lib.dora_lc1_readout_workspace_size(4, 0) == 0


def test_trajectory_flops_host_validation():
    lib = dora.load_library()
    good = dict(d=768, L=12, N0=196, patch=16, in_chans=3, classes=1000, head_inputs=1, mlp_ratio=4, M=96, actor=1)

    def call(B=4, tokens=FAKE, out=FAKE, **kw):
        cfg = dora.FlopsConfig(**{**good, **kw})
        return lib.dora_trajectory_flops(tokens, B, ctypes.byref(cfg), out, FAKE, FAKE, None)

    assert call(tokens=None) == dora.DORA_ERR_NULL
    assert call(out=None) == dora.DORA_ERR_NULL
    assert lib.dora_trajectory_flops(FAKE, 4, None, FAKE, FAKE, FAKE, None) == dora.DORA_ERR_NULL
    assert call(B=0) == dora.DORA_ERR_SHAPE
    assert call(d=0) == dora.DORA_ERR_SHAPE
    assert call(L=0) == dora.DORA_ERR_SHAPE
    assert call(M=0) == dora.DORA_ERR_SHAPE
    assert call(actor=2) == dora.DORA_ERR_SHAPE
    assert call(N0=dora.DORA_MAX_ROW_TOKENS + 1) == dora.DORA_ERR_SHAPE


def call_select_plan(lib, **kw):
    ws = dora.dora_varlen_attn_workspace_size(4, 3, 197)
    a = dict(scores=FAKE, keep=FAKE, tokens=FAKE, cu_in=None, total_in=0, B=4, N=197, C=768, dtype=1,
             idx=FAKE, cu=FAKE, packed=FAKE, cap=100, H=3, max_seqlen=197, total=100, ws=FAKE, ws_bytes=ws,
             status=FAKE, stream=None)
    a.update(kw)
    return lib.dora_select_pack_plan(a["scores"], a["keep"], a["tokens"], a["cu_in"], a["total_in"], a["B"],
                                     a["N"], a["C"], a["dtype"], a["idx"], a["cu"], a["packed"], a["cap"],
                                     a["H"], a["max_seqlen"], a["total"], a["ws"], a["ws_bytes"],
                                     a["status"], a["stream"])


def test_select_pack_plan_host_validation():
    """The fused call checks both argument sets before anything is enqueued."""
    lib = dora.load_library()
    assert call_select_plan(lib, scores=None) == dora.DORA_ERR_NULL
    assert call_select_plan(lib, C=3) == dora.DORA_ERR_ALIGN
    assert call_select_plan(lib, cap=0) == dora.DORA_ERR_CAPACITY
    assert call_select_plan(lib, H=0) == dora.DORA_ERR_SHAPE
    assert call_select_plan(lib, H=257) == dora.DORA_ERR_SHAPE
    assert call_select_plan(lib, max_seqlen=0) == dora.DORA_ERR_SHAPE
    assert call_select_plan(lib, max_seqlen=dora.DORA_MAX_SEQLEN + 1) == dora.DORA_ERR_SHAPE
    assert call_select_plan(lib, total=-1) == dora.DORA_ERR_SHAPE
    assert call_select_plan(lib, B=8193, cap=100) == dora.DORA_ERR_SHAPE
    assert call_select_plan(lib, ws=None) == dora.DORA_ERR_WORKSPACE
    assert call_select_plan(lib, ws=FAKE + 16) == dora.DORA_ERR_WORKSPACE
    ws = dora.dora_varlen_attn_workspace_size(4, 3, 197)
    assert call_select_plan(lib, ws_bytes=ws - 1) == dora.DORA_ERR_WORKSPACE


def test_workspace_size():
    assert dora.dora_varlen_attn_workspace_size(256, 12, 197) > 0
    assert dora.dora_varlen_attn_workspace_size(0, 12, 197) == 0
    assert dora.dora_varlen_attn_workspace_size(4, 0, 197) == 0
    assert dora.dora_varlen_attn_workspace_size(4, 3, dora.DORA_MAX_SEQLEN + 1) == 0
    a = dora.dora_varlen_attn_workspace_size(256, 12, 197)
    b = dora.dora_varlen_attn_workspace_size(256, 12, 577)
    assert b > a and a % 256 == 0


def test_attention_host_validation():
    lib = dora.load_library()
    ws = dora.dora_varlen_attn_workspace_size(4, 3, 197)

    def ex(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, cu=FAKE, B=4, H=3, D=64, max_seqlen=197, total=100, scale=0.0,
                 dtype=1, out=FAKE, ws=FAKE, ws_bytes=ws, status=FAKE, stream=None)
        a.update(kw)
        args = (a["q"], a["k"], a["v"], a["cu"], a["B"], a["H"], a["D"], a["max_seqlen"], a["total"],
                a["scale"], a["dtype"], a["out"], a["ws"], a["ws_bytes"], a["status"], a["stream"])
        return lib.dora_varlen_attn_execute(*args), lib.dora_varlen_attn(*args)

    assert ex(q=None) == (dora.DORA_ERR_NULL,) * 2
    assert ex(dtype=5) == (dora.DORA_ERR_DTYPE,) * 2
    assert ex(D=128) == (dora.DORA_ERR_SHAPE,) * 2
    assert ex(q=FAKE + 4) == (dora.DORA_ERR_ALIGN,) * 2
    assert ex(ws=FAKE + 16) == (dora.DORA_ERR_WORKSPACE,) * 2
    assert ex(ws_bytes=ws - 1) == (dora.DORA_ERR_WORKSPACE,) * 2
    assert ex(B=0) == (dora.DORA_ERR_SHAPE,) * 2
    assert ex(max_seqlen=0) == (dora.DORA_ERR_SHAPE,) * 2
    assert ex(total=-1) == (dora.DORA_ERR_SHAPE,) * 2
    assert lib.dora_varlen_attn_plan(None, 4, 3, 197, 100, FAKE, ws, FAKE, None) == dora.DORA_ERR_NULL
    assert lib.dora_varlen_attn_plan(FAKE, 4, 3, 197, 100, None, ws, FAKE, None) == dora.DORA_ERR_WORKSPACE


def test_noalloc_host_validation():
    """dora_varlen_attn_noalloc rejects bad arguments, and sizes whose plan
    would not fit the static workspace, before any device call."""
    lib = dora.load_library()
    m = re.search(r"#define\s+DORA_NOALLOC_WORKSPACE_BYTES\s+\((\d+)u\s*<<\s*(\d+)\)", open(HEADER).read())
    assert m and int(m.group(1)) << int(m.group(2)) == dora.DORA_NOALLOC_WORKSPACE_BYTES

    def na(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, cu=FAKE, B=4, H=3, D=64, max_seqlen=197, total=100, scale=0.0,
                 dtype=1, out=FAKE, status=FAKE, stream=None)
        a.update(kw)
        return lib.dora_varlen_attn_noalloc(a["q"], a["k"], a["v"], a["cu"], a["B"], a["H"], a["D"],
                                            a["max_seqlen"], a["total"], a["scale"], a["dtype"], a["out"],
                                            a["status"], a["stream"])

    assert na(q=None) == dora.DORA_ERR_NULL
    assert na(status=None) == dora.DORA_ERR_NULL
    assert na(dtype=5) == dora.DORA_ERR_DTYPE
    assert na(D=128) == dora.DORA_ERR_SHAPE
    assert na(B=0) == dora.DORA_ERR_SHAPE
    assert na(out=FAKE + 8) == dora.DORA_ERR_ALIGN
    # 4094 x 128 one-chunk items fill the 4 MiB array exactly; one more sequence does not fit
    assert dora.dora_varlen_attn_workspace_size(4094, 128, 192) == dora.DORA_NOALLOC_WORKSPACE_BYTES
    assert dora.dora_varlen_attn_workspace_size(4095, 128, 192) > dora.DORA_NOALLOC_WORKSPACE_BYTES
    assert na(B=4095, H=128, max_seqlen=192) == dora.DORA_ERR_STATIC_LIMIT
    assert na(B=8192, H=64, max_seqlen=dora.DORA_MAX_SEQLEN) == dora.DORA_ERR_STATIC_LIMIT


def test_product_package_does_not_touch_the_oracle():
    pkg = os.path.dirname(dora.__file__)
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.lower(), f
