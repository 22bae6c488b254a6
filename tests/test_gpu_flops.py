"""GPU parity for dora_trajectory_flops: exact (int64) against the oracle,
on legal trajectories of the paper's backbones (Table 3), with and without
the actor, past the kernel's 1024-image stride, and with invalid rows."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import to_dev

pytestmark = pytest.mark.gpu

BACKBONES = {  # d, L, N0, patch, head inputs
    "DeiT-B": (768, 12, 196, 16, 1),
    "ViT-L": (1024, 24, 196, 16, 1),
    "DINOv2-B/14": (768, 12, 256, 14, 2),
}


def trajectories(rng, B, L, N0, M, p_prune=0.4):
    T = np.empty((L + 1, B), np.int32)
    T[0] = N0 + 1
    for l in range(L):
        nv = T[l] - 1
        kmax = np.minimum(2 * M, (nv - 4) // 2 * 2)
        k = np.where((kmax >= 2) & (rng.random(B) < p_prune), 2 * rng.integers(1, np.maximum(kmax // 2, 1) + 1), 0)
        T[l + 1] = T[l] - k
    return T


@pytest.mark.parametrize("name", list(BACKBONES))
@pytest.mark.parametrize("actor", [True, False])
def test_trajectories_exact(gpu, name, actor):
    d, L, N0, p, hi = BACKBONES[name]
    M = (N0 - 4) // 2
    rng = np.random.default_rng(L + N0 + actor)
    B = 5000 if name == "DeiT-B" else 256
    T = trajectories(rng, B, L, N0, M)
    f, tot, st = gpu.dora_trajectory_flops(to_dev(T), d, N0, p, head_inputs=hi, actor=actor)
    torch.cuda.synchronize()
    want = oracle.trajectory_flops(T, d, L, N0, p, M, head_inputs=hi, actor=actor)
    assert int(st.item()) == 0
    assert np.array_equal(f.cpu().numpy(), want) and int(tot.item()) == int(want.sum())
    print(f"[flops] {name} actor={actor}: {want.mean() / 1e9:.2f} GFLOPs/image", flush=True)


def test_invalid_rows(gpu):
    d, L, N0, p, hi = BACKBONES["DeiT-B"]
    M = (N0 - 4) // 2
    T = trajectories(np.random.default_rng(1), 6, L, N0, M)
    T[0, 1] = N0                      # wrong start
    T[5, 2] = T[4, 2] + 2             # grows
    T[7:, 3] = 0                      # empty
    f, tot, st = gpu.dora_trajectory_flops(to_dev(T), d, N0, p)
    torch.cuda.synchronize()
    f = f.cpu().numpy()
    want = oracle.trajectory_flops(T, d, L, N0, p, M)
    assert int(st.item()) & gpu.DORA_DEV_KEEP_RANGE
    assert np.all(f[1:4] == -1) and np.array_equal(f[[0, 4, 5]], want[[0, 4, 5]])
    assert int(tot.item()) == int(want[[0, 4, 5]].sum())
