"""Host <-> device conversions shared by the GPU tests."""
import numpy as np
import torch

import workloads

BF16_MAX_ABS, BF16_MEAN_ABS = 2e-2, 2e-3     # attention tolerance, bf16 inputs
F32_MAX_ABS = 1e-5                           # attention tolerance, fp32 inputs


def to_dev(a: np.ndarray, dtype: str = None) -> torch.Tensor:
    """numpy -> cuda tensor; uint16 arrays are bf16 bit patterns."""
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def to_host_bits(t: torch.Tensor) -> np.ndarray:
    """cuda tensor -> numpy; bf16 comes back as uint16 bit patterns."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def widen(t: torch.Tensor) -> np.ndarray:
    """Exact fp64 values of a bf16 / fp32 cuda tensor."""
    if t.dtype == torch.bfloat16:
        return workloads.bf16_bits_to_f32(to_host_bits(t)).astype(np.float64)
    return t.cpu().numpy().astype(np.float64)


def cu_of(lens) -> np.ndarray:
    return np.concatenate([[0], np.cumsum(np.asarray(lens, dtype=np.int64))]).astype(np.int32)


def attn_errors(got: np.ndarray, want: np.ndarray):
    d = np.abs(got - want)
    return float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0


def assert_attn_close(got: np.ndarray, want: np.ndarray, dtype: str, what: str = ""):
    mx, mean = attn_errors(got, want)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    if dtype == "bf16":
        assert mx <= BF16_MAX_ABS and mean <= BF16_MEAN_ABS, f"{what}: max {mx:.3e} mean {mean:.3e}"
    else:
        assert mx <= F32_MAX_ABS, f"{what}: max {mx:.3e}"
    return mx, mean
