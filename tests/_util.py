"""Shared helpers for the tests: device transfer of workload arrays and the
error metrics.

rel_err  relative infinity norm over the whole tensor, max|y - yref| / max|yref|
         (the parity gate);
row_err  the same per row (last axis), worst row: max_r max|y_r - yref_r| /
         max|yref_r| (rows whose reference is all zero are measured against the
         tensor's max).  Two rows share one complex transform in the fused
         kernels, so a row much smaller than its partner would show up here
         and not in rel_err.

check() asserts both against the tolerance and appends the measured values
to a JSON-lines log (H3_PARITY_LOG, default gpurun_out/parity_errors.jsonl
under the repository root), so the margin under each tolerance is recorded.
"""
import json
import os

import numpy as np
import torch

import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _arr(a) -> np.ndarray:
    a = np.asarray(a)
    return a if np.iscomplexobj(a) else a.astype(np.float64, copy=False)


def rel_err(y, ref) -> float:
    y = _arr(y); ref = _arr(ref)
    den = np.abs(ref).max() if ref.size else 0.0
    return float(np.abs(y - ref).max() / (den if den > 0 else 1.0)) if ref.size else 0.0


def row_err(y, ref) -> float:
    y = _arr(y); ref = _arr(ref)
    if ref.size == 0:
        return 0.0
    n = ref.shape[-1]
    y2, r2 = y.reshape(-1, n), ref.reshape(-1, n)
    num = np.abs(y2 - r2).max(axis=1)
    den = np.abs(r2).max(axis=1)
    top = np.abs(r2).max()
    den = np.where(den > 0, den, top if top > 0 else 1.0)
    return float((num / den).max())


def _log_path() -> str:
    return os.environ.get("H3_PARITY_LOG", os.path.join(ROOT, "gpurun_out", "parity_errors.jsonl"))


def record(name: str, **fields):
    """Append one JSON line {name, **fields} to the parity log (best effort)."""
    path = _log_path()
    try:
        os.makedirs(os.path.dirname(path), exist_ok=True)
        with open(path, "a") as f:
            f.write(json.dumps({"test": name, **fields}) + "\n")
    except OSError:
        pass


def _current_test() -> str:
    return os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]


def check(y, ref, tol: float, what: str = "y", rows: bool = True) -> float:
    """Assert rel_err (and, with rows, the worst per-row error) below tol and
    record both under the running test's id and `what`; returns rel_err."""
    name = _current_test() + ":" + what
    y = y if isinstance(y, np.ndarray) else to_np64(y) if isinstance(y, torch.Tensor) else np.asarray(y)
    assert y.shape == np.shape(ref), (name, y.shape, np.shape(ref))
    e = rel_err(y, ref)
    er = row_err(y, ref) if rows else None
    rms = float(np.sqrt(np.mean(np.abs(_arr(y) - _arr(ref)) ** 2)) / max(np.sqrt(np.mean(np.abs(_arr(ref)) ** 2)), 1e-300)) \
        if np.size(ref) else 0.0
    record(name, rel_err=e, worst_row_err=er, rms_rel_err=rms, tol=tol, shape=list(np.shape(ref)))
    msg = f"{name}: rel_err {e:.3e}" + (f", worst row {er:.3e}" if er is not None else "") + f", tol {tol:g}"
    assert np.isfinite(e) and e < tol, msg
    if er is not None:
        assert er < tol, msg
    return e


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
