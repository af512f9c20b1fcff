"""Shared helpers for the tests: device transfer of workload arrays and the
error metric (relative infinity norm: max|y - yref| / max|yref|)."""
import numpy as np
import torch

import workloads


def rel_err(y, ref) -> float:
    y = np.asarray(y, np.float64); ref = np.asarray(ref, np.float64)
    den = np.abs(ref).max()
    return float(np.abs(y - ref).max() / (den if den > 0 else 1.0))


def to_dev(storage: np.ndarray, dtype: str, dev="cuda") -> torch.Tensor:
    """Workload storage array (float32 / float16 / bf16 bits) -> device tensor."""
    if dtype == workloads.BF16:
        t = torch.from_numpy(np.ascontiguousarray(storage).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(storage))
    return t.to(dev)


def to_np64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def f32dev(a, dev="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)


def cplx64(a) -> np.ndarray:
    """(..., 2) float array -> complex128."""
    a = np.asarray(a, np.float64)
    return a[..., 0] + 1j * a[..., 1]


def cplx_to_f32pairs(z) -> np.ndarray:
    z = np.asarray(z)
    return np.ascontiguousarray(np.stack([z.real, z.imag], -1), dtype=np.float32)
