"""Float64 CPU oracle for the FlashConv hot path (H3, arXiv 2212.14052).

TEST INFRASTRUCTURE ONLY.  The product package never imports this module;
only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` do.  It shares no code with the HIP path.

The numerical routines live in ``oracle.c`` (plain C, float64, OpenMP over
rows) and are reached through ctypes.  The layer composition (Algorithm 1)
is written here with numpy float64 matrix products as library steps.

Complex parameters are numpy complex128 arrays at this level; the C side sees
them as interleaved (re, im) float64 pairs.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

from . import build as _build

_lib = None
_dp = ctypes.POINTER(ctypes.c_double)


def lib():
    global _lib
    if _lib is None:
        path = _build.build()
        L = ctypes.CDLL(path)
        i = ctypes.c_int
        L.oracle_zoh.argtypes = [_dp, _dp, _dp, i, i, _dp, _dp]
        L.oracle_ssm_kernel.argtypes = [_dp, _dp, _dp, _dp, i, i, i, _dp]
        L.oracle_ssm_kernel_discrete.argtypes = [_dp, _dp, _dp, i, i, i, _dp]
        L.oracle_causal_conv.argtypes = [_dp, _dp, _dp, i, i, i, _dp]
        L.oracle_causal_conv_bwd.argtypes = [_dp, _dp, _dp, _dp, i, i, i, _dp, _dp, _dp]
        L.oracle_ssm_recurrence.argtypes = [_dp, _dp, _dp, _dp, _dp, _dp, i, i, i, i, _dp, _dp]
        L.oracle_statepass.argtypes = [_dp, _dp, _dp, _dp, _dp, _dp, i, i, i, i, i, _dp, _dp]
        L.oracle_shift_ssm.argtypes = [_dp, _dp, _dp, i, i, i, i, _dp]
        L.oracle_num_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _r(a) -> np.ndarray:
    """Contiguous float64 array (complex arrays become interleaved pairs)."""
    a = np.asarray(a)
    if np.iscomplexobj(a):
        a = np.ascontiguousarray(a, dtype=np.complex128)
        return a.view(np.float64)
    return np.ascontiguousarray(a, dtype=np.float64)


def _p(a: Optional[np.ndarray]):
    if a is None:
        return ctypes.cast(None, _dp)
    return a.ctypes.data_as(_dp)


def num_threads() -> int:
    return int(lib().oracle_num_threads())


# ------------------------------------------------------------- S1 pieces ---
def zoh(A, B, dt):
    """Zero-order-hold discretisation (per channel step dt): returns (Abar, Bbar)
    as complex128 (H, m)."""
    A = np.asarray(A, np.complex128); H, m = A.shape
    Ab = np.empty((H, m), np.complex128); Bb = np.empty((H, m), np.complex128)
    a, b, d = _r(A), _r(np.broadcast_to(B, (H, m))), _r(dt)
    lib().oracle_zoh(_p(a), _p(b), _p(d), H, m, _p(Ab.view(np.float64)), _p(Bb.view(np.float64)))
    return Ab, Bb


def ssm_kernel(A, B, C, dt, L: int) -> np.ndarray:
    """k[h,t] = 2 Re sum_n C Bbar exp(t dt A), (H, L) float64."""
    A = np.asarray(A, np.complex128); H, m = A.shape
    k = np.empty((H, L), np.float64)
    a, b, c, d = _r(A), _r(np.broadcast_to(B, (H, m))), _r(C), _r(dt)
    lib().oracle_ssm_kernel(_p(a), _p(b), _p(c), _p(d), H, m, L, _p(k))
    return k


def ssm_kernel_discrete(Abar, Bbar, C, L: int) -> np.ndarray:
    """k[h,t] = 2 Re sum_n C Bbar Abar^t, (H, L) float64."""
    Abar = np.asarray(Abar, np.complex128); H, m = Abar.shape
    k = np.empty((H, L), np.float64)
    a, b, c = _r(Abar), _r(Bbar), _r(C)
    lib().oracle_ssm_kernel_discrete(_p(a), _p(b), _p(c), H, m, L, _p(k))
    return k


# ------------------------------------------------------------------ S3 -----
def causal_conv(u, k, D=None) -> np.ndarray:
    """Direct O(L^2) causal convolution + skip: y[b,h,t] = sum_{j<=t} k[h,j]
    u[b,h,t-j] + D[h] u[b,h,t].  u: (..., H, L) float64; k: (H, L)."""
    u = _r(u); k = _r(k)
    H, L = k.shape
    assert u.shape[-1] == L and u.shape[-2] == H
    R = u.size // L
    y = np.empty(u.shape, np.float64)
    Dp = _r(D) if D is not None else None
    lib().oracle_causal_conv(_p(u), _p(k), _p(Dp), R, H, L, _p(y))
    return y


def causal_conv_bwd(u, k, D, dy):
    """Gradients of y = causal_conv(u, k, D) for output gradient dy, by their
    definitions (backward-pass appendix): returns (du, dk, dD) with
    du[b,h,t] = sum_{s>=t} k[h,s-t] dy[b,h,s] + D[h] dy[b,h,t],
    dk[h,j] = sum_b sum_{t>=j} dy[b,h,t] u[b,h,t-j],  dD[h] = sum_{b,t} dy u."""
    u = _r(u); k = _r(k); dy = _r(dy)
    H, L = k.shape
    assert u.shape == dy.shape and u.shape[-1] == L and u.shape[-2] == H
    R = u.size // L
    du = np.empty(u.shape, np.float64)
    dk = np.empty((H, L), np.float64)
    dD = np.empty(H, np.float64)
    Dp = _r(D) if D is not None else None
    lib().oracle_causal_conv_bwd(_p(u), _p(k), _p(Dp), _p(dy), R, H, L, _p(du), _p(dk), _p(dD))
    return du, dk, dD


# ------------------------------------------------------------------ S5 -----
def recurrence(u, Abar, Bbar, C, D, x0=None):
    """Explicit SSM recurrence.  u: (..., H, L); returns (y, x_final) with
    x_final complex128 (..., H, m)."""
    u = _r(u)
    Abar = np.asarray(Abar, np.complex128); H, m = Abar.shape
    L = u.shape[-1]; R = u.size // L
    y = np.empty(u.shape, np.float64)
    xf = np.empty(u.shape[:-1] + (m,), np.complex128)
    x0p = _r(np.asarray(x0, np.complex128).reshape(R, m)) if x0 is not None else None
    Dp = _r(D) if D is not None else None
    lib().oracle_ssm_recurrence(_p(u), _p(_r(Abar)), _p(_r(Bbar)), _p(_r(C)), _p(Dp),
                                _p(x0p), R, H, L, m, _p(y), _p(xf.view(np.float64)))
    return y, xf


def statepass(u, Abar, Bbar, C, D, chunk: int, x0=None):
    """Algorithm 2 (state passing), chunk by chunk; returns (y, x_final)."""
    u = _r(u)
    Abar = np.asarray(Abar, np.complex128); H, m = Abar.shape
    L = u.shape[-1]; R = u.size // L
    assert L % chunk == 0
    y = np.empty(u.shape, np.float64)
    xf = np.empty(u.shape[:-1] + (m,), np.complex128)
    x0p = _r(np.asarray(x0, np.complex128).reshape(R, m)) if x0 is not None else None
    Dp = _r(D) if D is not None else None
    lib().oracle_statepass(_p(u), _p(_r(Abar)), _p(_r(Bbar)), _p(_r(C)), _p(Dp),
                           _p(x0p), R, H, L, m, chunk, _p(y), _p(xf.view(np.float64)))
    return y, xf


# ------------------------------------------------------------------ S6 -----
def shift_ssm(u, Cs, Ds=None) -> np.ndarray:
    """Shift SSM as the literal shift-matrix recurrence.  u: (..., H, L);
    Cs: (H, m) real taps; Ds: (H) or None."""
    u = _r(u); Cs = _r(Cs)
    H, m = Cs.shape; L = u.shape[-1]; R = u.size // L
    y = np.empty(u.shape, np.float64)
    Dp = _r(Ds) if Ds is not None else None
    lib().oracle_shift_ssm(_p(u), _p(Cs), _p(Dp), R, H, L, m, _p(y))
    return y


def h3_layer(x, Wq, Wk, Wv, Wo, shift_C, diag_k, diag_D, shift_D=None, d_head: int = 1,
             return_O: bool = False):
    """H3 layer forward (Sec. 3.2, Algorithm 1), float64.

    x: (B, N, d) token-major.  Q = x Wq, K = x Wk, V = x Wv (row-vector
    convention).  Kbar = shift SSM of K per channel (taps shift_C (d, m_s),
    skip shift_D).  With H = d / d_head heads, per head the batched outer
    product Kbar^(h) V^(h)T (d_head x d_head per token) passes through the
    diagonal SSM given by its convolution kernel diag_k ((H*d_head*d_head, N),
    channel h*d_head^2 + i*d_head + j for entry (i, j); for d_head = 1 that is
    (d, N)) plus skip diag_D, and is multiplied on the left by Q^(h)_t.  The
    heads are concatenated and multiplied by Wo.  Returns out (B, N, d), and
    also O (before Wo) if return_O.
    """
    x = np.asarray(x, np.float64)
    Bn, N, d = x.shape
    Q = x @ np.asarray(Wq, np.float64)
    K = x @ np.asarray(Wk, np.float64)
    V = x @ np.asarray(Wv, np.float64)
    # channel-major views (B, d, N) for the sequence operators
    Kc = np.ascontiguousarray(K.transpose(0, 2, 1))
    Kbar = shift_ssm(Kc, shift_C, shift_D)                      # (B, d, N)
    Vc = V.transpose(0, 2, 1)
    Qc = Q.transpose(0, 2, 1)
    nh = d // d_head
    Kh = Kbar.reshape(Bn, nh, d_head, N)
    Vh = Vc.reshape(Bn, nh, d_head, N)
    Qh = Qc.reshape(Bn, nh, d_head, N)
    G = Kh[:, :, :, None, :] * Vh[:, :, None, :, :]            # (B, nh, i, j, N)
    G = np.ascontiguousarray(G.reshape(Bn, nh * d_head * d_head, N))
    S = causal_conv(G, diag_k, diag_D).reshape(Bn, nh, d_head, d_head, N)
    O = np.einsum("bhin,bhijn->bhjn", Qh, S).reshape(Bn, d, N)  # O_t = Q_t^(h) KV_t^(h)
    O = O.transpose(0, 2, 1)                                    # (B, N, d)
    out = O @ np.asarray(Wo, np.float64)
    if return_O:
        return out, O
    return out
