"""The step (select/pack + plan, then attention) captured in a HIP graph.

No entry point allocates, sets memory or synchronises, so the whole step can
be captured and replayed.  Every replay is checked against the eager result,
with eager work and host synchronisation between replays.
"""
import numpy as np
import pytest
import torch

import workloads as W
from gpu_util import to_dev, to_host_bits

pytestmark = pytest.mark.gpu


def test_step_replays_match_eager(gpu):
    w = W.WORKLOADS["deit_s_bf16"]
    r = W.generate(w)[0]
    sk = r.total_keep
    ms = int(r.keep.max())
    scores, keep, tokens = to_dev(r.scores), to_dev(r.keep), to_dev(r.tokens)
    q, k, v = to_dev(r.q), to_dev(r.k), to_dev(r.v)
    idx = torch.empty(sk, dtype=torch.int32, device="cuda")
    cu = torch.empty(w.B + 1, dtype=torch.int32, device="cuda")
    packed = torch.empty((sk, w.C), dtype=tokens.dtype, device="cuda")
    out = torch.empty_like(q)
    ws = gpu.new_workspace(w.B, w.H, ms)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")

    def step():
        gpu.dora_select_pack_plan(scores, keep, tokens, w.H, ms, sk, ws, idx_out=idx, cu_out=cu,
                                  packed_out=packed, cap_rows=sk, dev_status=st)
        gpu.dora_varlen_attn_execute(q, k, v, cu, ms, ws, out=out, dev_status=st)

    step()
    torch.cuda.synchronize()
    want = [to_host_bits(t).copy() for t in (idx, cu, packed, out)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                                   # warm the side stream before capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(4):
        for t in (idx, cu, packed, out):
            t.view(torch.uint8).fill_(0xA5)      # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert int(st.item()) == 0, rep
        for got, exp in zip((idx, cu, packed, out), want):
            assert np.array_equal(to_host_bits(got), exp), rep
