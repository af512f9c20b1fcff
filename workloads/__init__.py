"""Seeded synthetic inputs shaped like the paper's FlashConv workloads.

This module draws random numbers and rounds them to the I/O dtypes.  It holds
none of the method's arithmetic (no discretisation, no kernel, no convolution):
both the float64 oracle and the HIP path consume exactly the arrays it returns.

Draw order (fixed so that every consumer sees the same values), all in float64
from ``numpy.random.default_rng(seed)``:
    u, then the per-channel step size dt, then C (real parts, then imaginary
    parts), then D, then the shift-SSM taps, then the projection weights
    W_Q, W_K, W_V, W_O.
Each array is rounded once to the dtype the kernel reads (fp32 parameters,
fp16/bf16/fp32 activations); the float64 view of the rounded values is what the
oracle sees.

Diagonal SSM modes follow the S4D-Lin initialisation: A_n = -1/2 + i*pi*n,
B_n = 1, C_n ~ CN(0, 1) (real and imaginary parts iid N(0, 1/2)), dt
log-uniform per channel.  Shift-SSM taps are N(0, 1/64).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import numpy as np

F32, F16, BF16 = "f32", "f16", "bf16"


# ---------------------------------------------------------------- rounding ---
def round_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float values to bfloat16 (round to nearest, ties to even) and
    return the raw uint16 bit patterns.  Rounds float64 -> float32 first."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    b = x32.view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    r = (b + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    nan = np.isnan(x32)
    out = r.astype(np.uint16)
    out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def round_to(x: np.ndarray, dtype: str) -> tuple[np.ndarray, np.ndarray]:
    """Round ``x`` to ``dtype``.  Returns (storage array, float64 view of the
    rounded values).  Storage is float32 / float16 / uint16 (bf16 bits)."""
    if dtype == F32:
        s = np.ascontiguousarray(x, dtype=np.float32)
        return s, s.astype(np.float64)
    if dtype == F16:
        s = np.ascontiguousarray(x, dtype=np.float32).astype(np.float16)
        return s, s.astype(np.float64)
    if dtype == BF16:
        s = round_bf16_bits(x)
        return s, bf16_bits_to_f64(s)
    raise ValueError(f"unknown dtype {dtype}")


def f32(x: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(x, dtype=np.float32)


# ------------------------------------------------------------- parameters ---
@dataclasses.dataclass
class DiagSSM:
    """Continuous-time diagonal SSM parameters, one set of m modes per channel,
    stored as fp32 (complex values as interleaved (re, im) pairs)."""
    A: np.ndarray   # (H, m, 2) float32
    B: np.ndarray   # (H, m, 2) float32
    C: np.ndarray   # (H, m, 2) float32
    dt: np.ndarray  # (H,) float32

    @property
    def H(self) -> int:
        return self.A.shape[0]

    @property
    def m(self) -> int:
        return self.A.shape[1]

    def complex64(self):
        """float64 complex views of the fp32-rounded parameters."""
        c = lambda a: a[..., 0].astype(np.float64) + 1j * a[..., 1].astype(np.float64)
        return c(self.A), c(self.B), c(self.C), self.dt.astype(np.float64)


def s4d_lin_A(H: int, m: int) -> np.ndarray:
    n = np.arange(m, dtype=np.float64)
    A = np.empty((H, m, 2), np.float32)
    A[..., 0] = -0.5
    A[..., 1] = (math.pi * n)[None, :]
    return A


def draw_dt(rng: np.random.Generator, H: int, lo: float, hi: float) -> np.ndarray:
    return f32(np.exp(rng.uniform(math.log(lo), math.log(hi), size=H)))


def draw_C(rng: np.random.Generator, H: int, m: int) -> np.ndarray:
    re = rng.standard_normal((H, m)) * math.sqrt(0.5)
    im = rng.standard_normal((H, m)) * math.sqrt(0.5)
    return f32(np.stack([re, im], axis=-1))


def make_diag_ssm(rng: np.random.Generator, H: int, m: int, dt_lo: float, dt_hi: float) -> DiagSSM:
    dt = draw_dt(rng, H, dt_lo, dt_hi)
    C = draw_C(rng, H, m)
    B = np.zeros((H, m, 2), np.float32)
    B[..., 0] = 1.0
    return DiagSSM(A=s4d_lin_A(H, m), B=B, C=C, dt=dt)


# ---------------------------------------------------------------- configs ---
@dataclasses.dataclass
class ConvWorkload:
    name: str
    B: int
    H: int
    L: int
    dtype: str
    u: np.ndarray          # storage (B, H, L) in dtype
    u64: np.ndarray        # float64 view of the rounded u
    ssm: DiagSSM
    D: np.ndarray          # (H,) float32
    shift_C: Optional[np.ndarray] = None   # (H, 64) float32: shift-SSM taps


@dataclasses.dataclass
class StatePassWorkload:
    name: str
    B: int
    H: int
    L: int
    m: int
    chunk: int
    dtype: str
    u: np.ndarray
    u64: np.ndarray
    ssm: DiagSSM
    D: np.ndarray
    x0: Optional[np.ndarray]  # (B, H, m, 2) float32 or None (zero state)


@dataclasses.dataclass
class LayerWorkload:
    name: str
    B: int
    L: int
    d: int
    m_shift: int
    dtype: str
    x: np.ndarray          # (B, L, d) storage
    x64: np.ndarray
    W: dict                # name -> (storage (d, d), float64 view); Q = x @ W["q"]
    shift_C: np.ndarray    # (d, m_shift) float32
    diag: DiagSSM          # diagonal SSM (d channels)
    diag_D: np.ndarray     # (d,) float32


def conv_workload(name: str, B: int, H: int, L: int, dtype: str, seed: int,
                  m: int = 64, dt_lo: float = 1e-3, dt_hi: float = 1e-1,
                  with_shift: bool = False) -> ConvWorkload:
    rng = np.random.default_rng(seed)
    u_s, u64 = round_to(rng.standard_normal((B, H, L)), dtype)
    ssm = make_diag_ssm(rng, H, m, dt_lo, dt_hi)
    D = f32(rng.standard_normal(H))
    shift_C = f32(rng.standard_normal((H, 64)) / 8.0) if with_shift else None
    return ConvWorkload(name, B, H, L, dtype, u_s, u64, ssm, D, shift_C)


def statepass_workload(name: str, B: int, H: int, L: int, chunk: int, dtype: str, seed: int,
                       m: int = 64, dt_lo: float = 1e-4, dt_hi: float = 1e-2,
                       x0_scale: float = 0.0) -> StatePassWorkload:
    rng = np.random.default_rng(seed)
    u_s, u64 = round_to(rng.standard_normal((B, H, L)), dtype)
    ssm = make_diag_ssm(rng, H, m, dt_lo, dt_hi)
    D = f32(rng.standard_normal(H))
    x0 = None
    if x0_scale:
        x0 = f32(rng.standard_normal((B, H, m, 2)) * x0_scale)
    return StatePassWorkload(name, B, H, L, m, chunk, dtype, u_s, u64, ssm, D, x0)


def layer_workload(name: str, B: int, L: int, d: int, dtype: str, seed: int,
                   m: int = 64, m_shift: int = 64, dt_lo: float = 1e-3,
                   dt_hi: float = 1e-1) -> LayerWorkload:
    rng = np.random.default_rng(seed)
    x_s, x64 = round_to(rng.standard_normal((B, L, d)), dtype)
    diag = make_diag_ssm(rng, d, m, dt_lo, dt_hi)
    diag_D = f32(rng.standard_normal(d))
    shift_C = f32(rng.standard_normal((d, m_shift)) / math.sqrt(m_shift))
    W = {}
    for key in ("q", "k", "v", "o"):
        W[key] = round_to(rng.standard_normal((d, d)) / math.sqrt(d), dtype)
    return LayerWorkload(name, B, L, d, m_shift, dtype, x_s, x64, W, shift_C, diag, diag_D)


# The five workloads of the headline measurement, by index.
#   0: one long conv, fp32, B=1 H=64 L=1024, dt in [1e-3, 1e-1]
#   1: 125M-layer shape, fp16 I/O, B=8 H=768 L=2048 (diagonal + shift kernels)
#   2: fused-block limit, bf16 I/O, B=16 H=256 L=8192, dt in [1e-4, 1e-1]
#   3: state passing, fp16 I/O, B=2 H=1024 L=131072, chunk 8192, dt in [1e-4, 1e-2]
#   4: H3 layer forward at 2.7B width, bf16, B=4 L=2048 d=2560
def config(idx: int, **over):
    if idx == 0:
        kw = dict(B=1, H=64, L=1024, dtype=F32, seed=0, dt_lo=1e-3, dt_hi=1e-1)
        kw.update(over)
        return conv_workload("cfg0_long_conv_f32", **kw)
    if idx == 1:
        kw = dict(B=8, H=768, L=2048, dtype=F16, seed=1, dt_lo=1e-3, dt_hi=1e-1, with_shift=True)
        kw.update(over)
        return conv_workload("cfg1_h3_125m_f16", **kw)
    if idx == 2:
        kw = dict(B=16, H=256, L=8192, dtype=BF16, seed=2, dt_lo=1e-4, dt_hi=1e-1)
        kw.update(over)
        return conv_workload("cfg2_fused_limit_bf16", **kw)
    if idx == 3:
        kw = dict(B=2, H=1024, L=131072, chunk=8192, dtype=F16, seed=3, dt_lo=1e-4, dt_hi=1e-2)
        kw.update(over)
        return statepass_workload("cfg3_statepass_f16", **kw)
    if idx == 4:
        kw = dict(B=4, L=2048, d=2560, dtype=BF16, seed=4)
        kw.update(over)
        return layer_workload("cfg4_h3_layer_2p7b_bf16", **kw)
    raise ValueError(idx)
