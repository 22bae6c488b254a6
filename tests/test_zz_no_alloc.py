"""dora_varlen_attn_noalloc (the static-workspace entry point for callers that
cannot allocate) against dora_varlen_attn: two calls in a row through the C
ABI, the second on a smaller input, each bit-identical to the workspace
entry point and within the attention tolerance of the oracle."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W
from gpu_util import assert_attn_close, cu_of, to_dev, to_host_bits, widen

pytestmark = pytest.mark.gpu


def _case(rng, lens, H, dtype):
    q, k, v = W.random_qkv(rng, lens, H, dtype)
    return q, k, v, cu_of(lens)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_entry_point(gpu, dtype):
    rng = np.random.default_rng(71)
    big = rng.integers(1, 400, 96)
    big[0] = 577
    small = rng.integers(1, 90, 5)
    for step, (lens, H) in enumerate(((big, 12), (small, 3))):
        q, k, v, cu = _case(rng, lens, H, dtype)
        ms = int(lens.max())
        print(f"[noalloc] {dtype} call {step}: B={len(lens)} H={H} max_seqlen={ms}", flush=True)
        tq, tk, tv, tcu = to_dev(q), to_dev(k), to_dev(v), to_dev(cu)
        want = gpu.dora_varlen_attn(tq, tk, tv, tcu, ms)
        out = torch.empty_like(tq)
        out.view(torch.int16 if dtype == "bf16" else torch.int32).fill_(0x3C3C)
        st = torch.zeros(1, dtype=torch.int32, device="cuda")
        gpu.dora_varlen_attn_noalloc(tq, tk, tv, tcu, ms, out=out, dev_status=st)
        torch.cuda.synchronize()
        assert int(st.item()) == 0
        assert np.array_equal(to_host_bits(out), to_host_bits(want))
        assert_attn_close(widen(out), oracle.varlen_attn(q, k, v, cu, dtype), dtype, f"noalloc call {step}")


def test_noalloc_rejects_sizes_past_the_static_workspace(gpu):
    q = torch.zeros((4, 16, 64), dtype=torch.bfloat16, device="cuda")   # 4095 x 16 x 86 items: 44 MB of plan
    cu = torch.zeros(4096, dtype=torch.int32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    with pytest.raises(gpu.DoraError) as e:
        gpu.dora_varlen_attn_noalloc(q, q, q, cu, gpu.DORA_MAX_SEQLEN, out=torch.empty_like(q), dev_status=st)
    assert e.value.code == gpu.DORA_ERR_STATIC_LIMIT
