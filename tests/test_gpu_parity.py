"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded, rounded inputs.

Metric: rel_err = max|y - y_oracle| / max|y_oracle| per output tensor, and the
same per row (worst row), both below the gate: 1e-5 for float32 I/O, 2e-2 for
fp16/bf16 I/O (fp32 accumulation).  Every comparison is recorded (test id,
both errors, RMS error, tolerance) in the parity log (tests/_util.check).

The workload configurations are compared on whole tensors at full size, in
the launch configuration the benchmark times.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests._util import check, cplx64, cplx_to_f32pairs, f32dev, to_dev, to_np64

pytestmark = pytest.mark.gpu

TOL = {workloads.F32: 1e-5, workloads.F16: 2e-2, workloads.BF16: 2e-2}


@pytest.fixture(scope="module")
def h3():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2212_14052_amd as m
    m.lib()
    return m


def _diag_params(w):
    A, B, C, dt = w.ssm.complex64()
    return A, B, C, dt


# ------------------------------------------------------------ S1: kernel ---
def test_discretize(h3):
    w = workloads.config(0)
    A, B, C, dt = _diag_params(w)
    Ab, Bb = h3.ssm_discretize(f32dev(w.ssm.A), f32dev(w.ssm.B), f32dev(w.ssm.dt))
    rA, rB = oracle.zoh(A, B, dt)
    check(cplx64(to_np64(Ab)), rA, 1e-6, "Abar", rows=False)
    check(cplx64(to_np64(Bb)), rB, 1e-6, "Bbar", rows=False)


@pytest.mark.parametrize("L,dt_lo,dt_hi", [(1024, 1e-3, 1e-1), (100, 1e-3, 1e-1), (8192, 1e-4, 1e-1), (64, 1e-2, 1e-1),
                                           (192, 1e-3, 1e-1), (2049, 1e-2, 1e-1), (16, 1e-3, 1e-1)])
def test_ssm_kernel(h3, L, dt_lo, dt_hi):
    w = workloads.config(0, H=16, L=16, seed=7, dt_lo=dt_lo, dt_hi=dt_hi)
    A, B, C, dt = _diag_params(w)
    k = h3.ssm_kernel(f32dev(w.ssm.A), f32dev(w.ssm.B), f32dev(w.ssm.C), f32dev(w.ssm.dt), L)
    ref = oracle.ssm_kernel(A, B, C, dt, L)
    check(k, ref, 2e-6, "k")


# --------------------------------------------------------- S2-S4: conv ---
def _conv_case(h3, B, H, L, dtype, seed, dt_lo=1e-3, dt_hi=1e-1, with_D=True):
    w = workloads.conv_workload("t", B, H, L, dtype, seed, dt_lo=dt_lo, dt_hi=dt_hi)
    A, Bm, C, dt = _diag_params(w)
    k64 = oracle.ssm_kernel(A, Bm, C, dt, L)
    k32 = k64.astype(np.float32)
    D = w.D if with_D else None
    y = h3.fftconv(to_dev(w.u, dtype), f32dev(k32), f32dev(D) if with_D else None)
    torch.cuda.synchronize()
    ref = oracle.causal_conv(w.u64, k32.astype(np.float64), D.astype(np.float64) if with_D else None)
    return to_np64(y), ref


@pytest.mark.parametrize("L", [16, 32, 64, 128, 256, 512, 1024, 2048, 4096, 8192])
def test_fftconv_f32_all_lengths(h3, L):
    y, ref = _conv_case(h3, 3, 5, L, workloads.F32, seed=L)
    check(y, ref, TOL[workloads.F32])


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
@pytest.mark.parametrize("L", [16, 256, 2048, 8192])
def test_fftconv_16bit(h3, dtype, L):
    y, ref = _conv_case(h3, 4, 3, L, dtype, seed=L + 1, dt_lo=1e-4)
    check(y, ref, TOL[dtype])


def test_fftconv_no_skip_odd_batch(h3):
    y, ref = _conv_case(h3, 1, 7, 512, workloads.F32, seed=3, with_D=False)
    check(y, ref, 1e-5)


def test_fftconv_impulse_returns_kernel(h3):
    H, L = 4, 1024
    rng = np.random.default_rng(0)
    k = rng.standard_normal((H, L)).astype(np.float32) * np.exp(-np.arange(L) / 300).astype(np.float32)
    u = np.zeros((2, H, L), np.float32); u[:, :, 0] = 1.0
    y = to_np64(h3.fftconv(f32dev(u), f32dev(k), None))
    check(y[0], k, 1e-5, "row0")
    check(y[1], k, 1e-5, "row1")


def test_fftconv_causality(h3):
    H, L = 2, 2048
    rng = np.random.default_rng(1)
    k = rng.standard_normal((H, L)).astype(np.float32)
    u = rng.standard_normal((2, H, L)).astype(np.float32)
    y0 = to_np64(h3.fftconv(f32dev(u), f32dev(k), None))
    u2 = u.copy(); u2[:, :, 1500] += 100.0
    y1 = to_np64(h3.fftconv(f32dev(u2), f32dev(k), None))
    # outputs before the perturbation move only by rounding noise of the FFT
    assert np.abs(y1[..., :1500] - y0[..., :1500]).max() < 1e-4 * np.abs(y0).max()
    assert np.abs(y1[..., 1500:] - y0[..., 1500:]).max() > 1.0


def test_fftconv_deterministic(h3):
    w = workloads.config(1, B=4, H=16, L=2048)
    u = to_dev(w.u, w.dtype)
    k = f32dev(np.random.default_rng(2).standard_normal((16, 2048)).astype(np.float32) * 0.01)
    a = h3.fftconv(u, k, f32dev(w.D))
    b = h3.fftconv(u, k, f32dev(w.D))
    assert torch.equal(a, b)


# Two rows of one channel share one complex transform.  A row far smaller
# than its partner must keep its own relative accuracy (each row carries its
# own power-of-two scale), at every fused length and dtype.
@pytest.mark.parametrize("dtype,L", [(workloads.F16, 2048), (workloads.BF16, 2048), (workloads.F16, 8192),
                                     (workloads.BF16, 8192), (workloads.F16, 16384), (workloads.F32, 1024),
                                     (workloads.F32, 8192), (workloads.F16, 512)])
@pytest.mark.parametrize("small", [1e-3, 0.3, 7.0])
def test_fftconv_pair_with_unequal_rows(h3, dtype, L, small):
    B, H = (8, 4) if L == 2048 else (4, 3)
    w = workloads.conv_workload("t", B, H, L, workloads.F32, seed=L + 5, dt_lo=1e-4)
    A, Bm, C, dt = _diag_params(w)
    k32 = oracle.ssm_kernel(A, Bm, C, dt, L).astype(np.float32)
    u = w.u.astype(np.float64)
    u[1] *= small          # row b of pair 0 (batches 0, 1)
    u[2] *= 1.0 / small    # row a of pair 1 (batches 2, 3)
    s, u64 = workloads.round_to(u, dtype)
    y = h3.fftconv(to_dev(s, dtype), f32dev(k32), f32dev(w.D))
    torch.cuda.synchronize()
    ref = oracle.causal_conv(u64, k32.astype(np.float64), w.D.astype(np.float64))
    check(y, ref, TOL[dtype])


# The VALU convolution forms the kernel spectrum itself and shares it among a
# group of row pairs of one channel; the group size follows the launch's
# parallelism.  These shapes give one pair per group, whole groups of several
# pairs and a last group with missing pairs, with odd B (a half pair).
@pytest.mark.parametrize("B,H,L,dtype", [(64, 64, 256, workloads.F32), (9, 2048, 1024, workloads.F32),
                                         (32, 512, 512, workloads.F32), (12, 512, 4096, workloads.F16),
                                         (11, 1024, 512, workloads.BF16), (5, 4096, 1024, workloads.F32)])
def test_fftconv_shared_spectrum_groups(h3, B, H, L, dtype):
    y, ref = _conv_case(h3, B, H, L, dtype, seed=B * H + L, dt_lo=1e-4)
    check(y, ref, TOL[dtype])


def _end_to_end_conv(h3, w, k_tol, y_tol):
    """S1 -> S2/S3 on the GPU at full size, against the oracle on every row."""
    k = h3.ssm_kernel(f32dev(w.ssm.A), f32dev(w.ssm.B), f32dev(w.ssm.C), f32dev(w.ssm.dt), w.L)
    y = h3.fftconv(to_dev(w.u, w.dtype), k, f32dev(w.D))
    torch.cuda.synchronize()
    A, B, C, dt = _diag_params(w)
    k_ref = oracle.ssm_kernel(A, B, C, dt, w.L)
    check(k, k_ref, k_tol, "k")
    y_ref = oracle.causal_conv(w.u64, k_ref, w.D.astype(np.float64))
    check(y, y_ref, y_tol, "y")


def test_config0_full_f32(h3):
    _end_to_end_conv(h3, workloads.config(0), 2e-6, 1e-5)


def test_config1_full_size(h3):
    """B=8 H=768 L=2048 fp16: the benchmark's step (kernel generation + the
    one-wave fused conv) on every row."""
    _end_to_end_conv(h3, workloads.config(1), 2e-6, 2e-2)


def test_config1_shift_kernel_full_size(h3):
    """The same shape with the shift-SSM kernel (k_t = C_t for t < 64, else 0)."""
    w = workloads.config(1)
    ks = np.zeros((w.H, w.L), np.float32)
    ks[:, :64] = w.shift_C
    y = h3.fftconv(to_dev(w.u, w.dtype), f32dev(ks), None)
    torch.cuda.synchronize()
    check(y, oracle.causal_conv(w.u64, ks.astype(np.float64), None), 2e-2)


def test_config2_full_size(h3):
    """B=16 H=256 L=8192 bf16 (the four-wave conv at the paper's fused limit)."""
    _end_to_end_conv(h3, workloads.config(2), 2e-6, 2e-2)


# ------------------------------------------ S2 / S3 split: spectral entry ---
@pytest.mark.parametrize("L", [16, 128, 1024, 2048, 8192])
def test_kernel_spectrum(h3, L):
    H = 5
    rng = np.random.default_rng(L)
    k = (rng.standard_normal((H, L)) * np.exp(-np.arange(L) / (L / 4))).astype(np.float32)
    K = to_np64(h3.kernel_spectrum(f32dev(k)))
    Kc = K[..., 0] + 1j * K[..., 1]
    # definition: (1/2L) sum_t k_t exp(-2 pi i f t / 2L), f = 0..L, by a dense
    # DFT matrix product in float64
    t = np.arange(L)
    f = np.arange(L + 1)
    F = np.exp(-2j * np.pi * np.outer(f, t) / (2 * L))
    ref = (k.astype(np.float64) @ F.T) / (2 * L)
    check(Kc, ref, 1e-5)


@pytest.mark.parametrize("dtype", [workloads.F32, workloads.F16, workloads.BF16])
@pytest.mark.parametrize("L", [64, 2048, 8192])
def test_fftconv_spectral(h3, dtype, L):
    """The convolution from a spectrum computed once, reused by two calls."""
    w = workloads.conv_workload("t", 3, 4, L, dtype, seed=L + 11)
    A, Bm, C, dt = _diag_params(w)
    k32 = oracle.ssm_kernel(A, Bm, C, dt, L).astype(np.float32)
    K = h3.kernel_spectrum(f32dev(k32))
    u = to_dev(w.u, dtype)
    y1 = h3.fftconv_spectral(u, K, f32dev(w.D))
    y2 = h3.fftconv_spectral(u[:1].contiguous(), K, None)
    torch.cuda.synchronize()
    check(y1, oracle.causal_conv(w.u64, k32.astype(np.float64), w.D.astype(np.float64)), TOL[dtype], "y")
    check(y2, oracle.causal_conv(w.u64[:1], k32.astype(np.float64), None), TOL[dtype], "y_no_skip")


# --------------------------------------------------------- S5: statepass ---
def _sp_inputs(w):
    A, B, C, dt = _diag_params(w)
    Ab, Bb = oracle.zoh(A, B, dt)
    # the GPU consumes fp32 discrete parameters; the oracle the same rounded values
    Ab32, Bb32 = cplx_to_f32pairs(Ab), cplx_to_f32pairs(Bb)
    return Ab32, Bb32, cplx64(Ab32), cplx64(Bb32), C


def _sp_check(h3, w, y_tol, x_tol):
    Ab32, Bb32, Ab, Bb, C = _sp_inputs(w)
    x0 = f32dev(w.x0) if w.x0 is not None else None
    y, xf = h3.statepass_conv(to_dev(w.u, w.dtype), f32dev(Ab32), f32dev(Bb32), f32dev(w.ssm.C), f32dev(w.D),
                              w.chunk, x0=x0)
    torch.cuda.synchronize()
    ry, rx = oracle.recurrence(w.u64, Ab, Bb, C, w.D.astype(np.float64),
                               x0=cplx64(w.x0) if w.x0 is not None else None)
    check(y, ry, y_tol, "y")
    check(cplx64(to_np64(xf)), rx, x_tol, "x_final")


@pytest.mark.parametrize("dtype,L,chunk", [(workloads.F32, 1024, 128), (workloads.F32, 512, 512),
                                           (workloads.F16, 2048, 256), (workloads.BF16, 1024, 16),
                                           (workloads.F32, 256, 16), (workloads.F16, 4096, 1024),
                                           (workloads.BF16, 8192, 2048), (workloads.F16, 8192, 4096)])
def test_statepass_small(h3, dtype, L, chunk):
    w = workloads.statepass_workload("t", 3, 5, L, chunk, dtype, seed=L + chunk, dt_lo=1e-3,
                                     dt_hi=1e-1, x0_scale=0.5)
    _sp_check(h3, w, TOL[dtype], 1e-5 if dtype == workloads.F32 else 2e-2)


def test_statepass_resume(h3):
    w = workloads.statepass_workload("t", 2, 3, 1024, 128, workloads.F32, seed=5, dt_lo=1e-3, dt_hi=1e-1)
    Ab32, Bb32, Ab, Bb, C = _sp_inputs(w)
    u = f32dev(w.u)
    args = (f32dev(Ab32), f32dev(Bb32), f32dev(w.ssm.C), f32dev(w.D))
    y, xf = h3.statepass_conv(u, *args, 128)
    y1, x1 = h3.statepass_conv(u[..., :512].contiguous(), *args, 128)
    y2, x2 = h3.statepass_conv(u[..., 512:].contiguous(), *args, 256, x0=x1)
    torch.cuda.synchronize()
    check(to_np64(torch.cat([y1, y2], -1)), to_np64(y), 1e-5, "y")
    check(cplx64(to_np64(x2)), cplx64(to_np64(xf)), 1e-5, "x_final")


def test_config3_full_size(h3):
    """B=2 H=1024 L=131072, chunk 8192, fp16: every row and every final state
    against the float64 recurrence."""
    _sp_check(h3, workloads.config(3), 2e-2, 2e-2)


def test_config3_full_size_chunk16384(h3):
    """The same workload with chunk 16384, the raised fused limit: every row
    and every final state against the float64 recurrence."""
    _sp_check(h3, workloads.config(3, chunk=16384), 2e-2, 2e-2)


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_statepass_mfma_chunks(h3, dtype):
    """Chunk 8192 (the paper's fused limit) runs the matrix-core conv per chunk
    pair with the fused initial-state term."""
    w = workloads.statepass_workload("t", 2, 3, 4 * 8192, 8192, dtype, seed=77, dt_lo=1e-4,
                                     dt_hi=1e-2, x0_scale=0.3)
    _sp_check(h3, w, TOL[dtype], 2e-2)


# ------------------------------------ fused limit 16384 (32768-point) ---
@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
@pytest.mark.parametrize("B,H", [(1, 2), (3, 3)])
def test_fftconv_l16384(h3, dtype, B, H):
    y, ref = _conv_case(h3, B, H, 16384, dtype, seed=B * 10 + H, dt_lo=1e-4)
    check(y, ref, TOL[dtype])


def test_fftconv_l16384_impulse(h3):
    """u = delta returns k + D delta on every row (spectrum and skip fold)."""
    L, H = 16384, 2
    rng = np.random.default_rng(4)
    k = (rng.standard_normal((H, L)) * np.exp(-np.arange(L) / 3000.0)).astype(np.float32)
    D = rng.standard_normal(H).astype(np.float32)
    u = np.zeros((2, H, L), np.float32); u[:, :, 0] = 1.0
    y = h3.fftconv(to_dev(workloads.round_to(u, workloads.F16)[0], workloads.F16), f32dev(k), f32dev(D))
    torch.cuda.synchronize()
    ref = np.broadcast_to(k.astype(np.float64), (2, H, L)).copy(); ref[:, :, 0] += D
    check(y, ref, 2e-2)


@pytest.mark.parametrize("dtype,B,H,nchunk", [(workloads.F16, 2, 2, 2), (workloads.BF16, 2, 3, 3),
                                            (workloads.F16, 1, 4, 5)])
def test_statepass_chunk16384(h3, dtype, B, H, nchunk):
    """Chunk 16384: chunk end-states on the matrix cores (the 16384 instance
    of the chunk-state kernel), the 32768-point conv per chunk pair with the
    initial-state term computed in its read-out (odd chunk counts leave a
    last pair with one chunk)."""
    w = workloads.statepass_workload("t", B, H, nchunk * 16384, 16384, dtype, seed=8 + H, dt_lo=1e-4,
                                     dt_hi=1e-2, x0_scale=0.5)
    _sp_check(h3, w, TOL[dtype], 2e-2)


def test_fftconv_bwd_du_l16384(h3):
    """Input gradient at L = 16384: the 32768-point kernel with the conjugated
    kernel spectrum."""
    B, H, L = 2, 2, 16384
    w = workloads.conv_workload("t", B, H, L, workloads.BF16, seed=12)
    A, Bm, C, dt = _diag_params(w)
    k32 = oracle.ssm_kernel(A, Bm, C, dt, L).astype(np.float32)
    rng = np.random.default_rng(13)
    dy_s, dy64 = workloads.round_to(rng.standard_normal((B, H, L)), workloads.BF16)
    du, _, _ = h3.fftconv_bwd(None, f32dev(k32), f32dev(w.D), to_dev(dy_s, workloads.BF16), want_dk=False,
                              want_dD=False)
    torch.cuda.synchronize()
    rdu, _, _ = oracle.causal_conv_bwd(w.u64, k32.astype(np.float64), w.D.astype(np.float64), dy64)
    check(du, rdu, 2e-2, "du")


# ------------------------------------------------- conv backward pass ---
def _bwd_case(h3, B, H, L, dtype, seed, with_D=True, sel=None):
    w = workloads.conv_workload("t", B, H, L, dtype, seed=seed)
    A, Bm, C, dt = _diag_params(w)
    k32 = oracle.ssm_kernel(A, Bm, C, dt, L).astype(np.float32)
    rng = np.random.default_rng(seed + 1)
    dy_s, dy64 = workloads.round_to(rng.standard_normal((B, H, L)), dtype)
    D = w.D if with_D else None
    du, dk, dD = h3.fftconv_bwd(to_dev(w.u, dtype), f32dev(k32), f32dev(D) if with_D else None,
                                to_dev(dy_s, dtype))
    torch.cuda.synchronize()
    du, dk, dD = to_np64(du), to_np64(dk), to_np64(dD)
    h = np.arange(H) if sel is None else np.asarray(sel)
    rdu, rdk, rdD = oracle.causal_conv_bwd(w.u64[:, h], k32[h].astype(np.float64),
                                           D[h].astype(np.float64) if with_D else None, dy64[:, h])
    return (du[:, h], rdu), (dk[h], rdk), (dD[h], rdD)


# L = 16 .. 8192 covers every transform length of the kernel-gradient kernel
# and, for 16-bit I/O at L = 2048 and 8192, the wave kernels with the
# conjugated spectrum for du; odd batches leave the last row pair half empty;
# B = 19 at L = 2048 gives three workgroup groups per channel on the matrix
# cores (partial sums and their reduction).
@pytest.mark.parametrize("dtype", [workloads.F32, workloads.F16, workloads.BF16])
@pytest.mark.parametrize("B,H,L", [(1, 3, 16), (3, 5, 256), (2, 4, 1024), (5, 3, 2048), (9, 4, 2048), (4, 2, 8192),
                                   (19, 3, 2048)])
def test_fftconv_bwd(h3, dtype, B, H, L):
    (du, rdu), (dk, rdk), (dD, rdD) = _bwd_case(h3, B, H, L, dtype, seed=B * 7 + L)
    check(du, rdu, TOL[dtype], "du")
    # dk, dD: float32 outputs; on the matrix cores (16-bit I/O at L = 2048) the
    # transforms run on fp16 operands, so the 16-bit tolerance applies there
    tol_k = TOL[dtype] if (L == 2048 and dtype != workloads.F32) else 1e-5
    check(dk, rdk, tol_k, "dk")
    check(dD, rdD, tol_k, "dD", rows=False)


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_fftconv_bwd_valu_kernel_gradient_at_2048(h3, monkeypatch, dtype):
    """The float32 VALU kernel-gradient kernel forced where the matrix-core one
    runs by default (L = 2048, 16-bit I/O)."""
    monkeypatch.setenv("H3FLASH_WGRAD", "valu")
    (du, rdu), (dk, rdk), (dD, rdD) = _bwd_case(h3, 3, 4, 2048, dtype, seed=77)
    check(du, rdu, TOL[dtype], "du")
    check(dk, rdk, 1e-5, "dk")
    check(dD, rdD, 1e-5, "dD", rows=False)


def test_fftconv_bwd_no_skip_and_partial_outputs(h3):
    B, H, L = 3, 4, 512
    (du, rdu), (dk, rdk), _ = _bwd_case(h3, B, H, L, workloads.F32, seed=41, with_D=False)
    check(du, rdu, 1e-5, "du")
    check(dk, rdk, 1e-5, "dk")
    w = workloads.conv_workload("t", B, H, L, workloads.F16, seed=42)
    k = f32dev(np.random.default_rng(1).standard_normal((H, L)) / 16)
    dy = to_dev(w.u, workloads.F16)
    du_only, dk0, dD0 = h3.fftconv_bwd(None, k, None, dy, want_dk=False, want_dD=False)
    _, dk_only, dD_only = h3.fftconv_bwd(dy, k, None, dy, want_du=False)
    torch.cuda.synchronize()
    assert dk0 is None and dD0 is None
    rdu, rdk, rdD = oracle.causal_conv_bwd(w.u64, to_np64(k), None, w.u64)
    check(du_only, rdu, 2e-2, "du_only")
    check(dk_only, rdk, 1e-5, "dk_only")   # L = 512: float32 VALU kernel
    check(dD_only, rdD, 1e-5, "dD_only", rows=False)


def test_fftconv_bwd_config1_full_size(h3):
    """At the H3-125M layer shape (B=8, H=768, L=2048, fp16) on the launch
    the benchmark times; every channel against the oracle."""
    (du, rdu), (dk, rdk), (dD, rdD) = _bwd_case(h3, 8, 768, 2048, workloads.F16, seed=5)
    check(du, rdu, 2e-2, "du")
    check(dk, rdk, 2e-2, "dk")
    check(dD, rdD, 2e-2, "dD", rows=False)


def test_fftconv_bwd_adjoint_at_full_size(h3):
    """<dy, conv(u)> = <du, u> at the fused-block limit (B=16 H=256 L=8192 bf16),
    with the forward and backward both on the GPU."""
    w = workloads.config(2)
    k = h3.ssm_kernel(f32dev(w.ssm.A), f32dev(w.ssm.B), f32dev(w.ssm.C), f32dev(w.ssm.dt), w.L)
    u = to_dev(w.u, w.dtype)
    dy = to_dev(workloads.round_to(np.random.default_rng(3).standard_normal(w.u.shape), w.dtype)[0], w.dtype)
    y = h3.fftconv(u, k, f32dev(w.D))
    du, dk, dD = h3.fftconv_bwd(u, k, f32dev(w.D), dy)
    torch.cuda.synchronize()
    J1 = torch.sum(dy.double() * y.double()).item()
    J2 = torch.sum(du.double() * u.double()).item()
    J3 = (torch.sum(dk.double() * k.double()) + torch.sum(dD.double() * f32dev(w.D).double())).item()
    scale = torch.sum((dy.double() * y.double()).abs()).item()
    assert abs(J1 - J2) < 2e-2 * scale
    assert abs(J1 - J3) < 2e-2 * scale


# ------------------------------------------------- recurrent step mode ---
def _step_inputs(B, H, m, T, dtype, seed):
    rng = np.random.default_rng(seed)
    u_s, u64 = workloads.round_to(rng.standard_normal((B, H, T)), dtype)
    ssm = workloads.make_diag_ssm(rng, H, m, 1e-3, 1e-1)
    A, Bm, C, dt = ssm.complex64()
    Ab, Bb = oracle.zoh(A, Bm, dt)
    Ab32, Bb32 = cplx_to_f32pairs(Ab), cplx_to_f32pairs(Bb)
    D = workloads.f32(rng.standard_normal(H))
    x0 = cplx_to_f32pairs((rng.standard_normal((B, H, m)) + 1j * rng.standard_normal((B, H, m))) * 0.5)
    return u_s, u64, Ab32, Bb32, ssm.C, D, x0


# T = 1 is one generated token; T > 1 keeps the state in registers over
# several tokens; m = 1 and 17 leave lanes without modes; H = 33 and odd B
# leave the last workgroup partly empty.
@pytest.mark.parametrize("dtype", [workloads.F32, workloads.F16, workloads.BF16])
@pytest.mark.parametrize("B,H,m,T", [(1, 1, 1, 1), (3, 5, 17, 7), (2, 33, 64, 64), (4, 768, 64, 1)])
def test_ssm_step(h3, dtype, B, H, m, T):
    u_s, u64, Ab32, Bb32, C32, D, x0 = _step_inputs(B, H, m, T, dtype, seed=B * 1000 + H * 10 + m + T)
    x = f32dev(x0)
    y = h3.ssm_step(to_dev(u_s, dtype), f32dev(Ab32), f32dev(Bb32), f32dev(C32), f32dev(D), x)
    torch.cuda.synchronize()
    ry, rx = oracle.recurrence(u64, cplx64(Ab32), cplx64(Bb32), cplx64(C32), D.astype(np.float64), x0=cplx64(x0))
    # a single token per row: the per-row metric would compare one value
    check(y, ry, TOL[dtype], "y", rows=T > 1)
    check(cplx64(to_np64(x)), rx, 1e-5, "x")


def test_ssm_step_chained_tokens_and_no_skip(h3):
    """Eight one-token calls through the same state equal one call over eight
    tokens, and both equal the recurrence (D absent)."""
    B, H, m, T = 2, 40, 64, 8
    u_s, u64, Ab32, Bb32, C32, _, x0 = _step_inputs(B, H, m, T, workloads.F32, seed=3)
    args = (f32dev(Ab32), f32dev(Bb32), f32dev(C32), None)
    u = f32dev(u_s)
    x1 = f32dev(x0)
    y_all = h3.ssm_step(u, *args, x1)
    x2 = f32dev(x0)
    y_one = torch.cat([h3.ssm_step(u[..., t].contiguous(), *args, x2).unsqueeze(-1) for t in range(T)], -1)
    torch.cuda.synchronize()
    ry, rx = oracle.recurrence(u64, cplx64(Ab32), cplx64(Bb32), cplx64(C32), None, x0=cplx64(x0))
    check(y_all, ry, 1e-5, "y_all")
    check(y_one, ry, 1e-5, "y_one")
    check(cplx64(to_np64(x1)), cplx64(to_np64(x2)), 1e-6, "x")


def test_ssm_step_continues_statepass(h3):
    """A prompt through state passing, then generation from its final state,
    equals the recurrence over prompt + generated tokens."""
    w = workloads.statepass_workload("t", 2, 6, 2048 + 16, 2048, workloads.F16, seed=9, dt_lo=1e-3,
                                     dt_hi=1e-1)
    Ab32, Bb32, Ab, Bb, C = _sp_inputs(w)
    args = (f32dev(Ab32), f32dev(Bb32), f32dev(w.ssm.C), f32dev(w.D))
    u = to_dev(w.u, w.dtype)
    y1, xf = h3.statepass_conv(u[..., :2048].contiguous(), *args, 2048)
    y2 = h3.ssm_step(u[..., 2048:].contiguous(), *args, xf)
    torch.cuda.synchronize()
    ry, rx = oracle.recurrence(w.u64, Ab, Bb, C, w.D.astype(np.float64))
    check(to_np64(torch.cat([y1, y2], -1)), ry, 2e-2, "y")
    check(y2, ry[..., 2048:], 2e-2, "y_generated")


# ------------------------------------------------------------- S6: layer ---
def _layer_run(h3, w, k32, shift_D=None, diag_D=None, d_head=1):
    W = {n: to_dev(w.W[n][0], w.dtype) for n in "qkvo"}
    args = (to_dev(w.x, w.dtype), W["q"], W["k"], W["v"], W["o"], f32dev(w.shift_C),
            f32dev(shift_D) if shift_D is not None else None, f32dev(k32),
            f32dev(diag_D) if diag_D is not None else None)
    out = h3.layer_fwd(*args) if d_head == 1 else h3.layer_fwd_heads(*args, d_head)
    torch.cuda.synchronize()
    ref = oracle.h3_layer(w.x64, w.W["q"][1], w.W["k"][1], w.W["v"][1], w.W["o"][1],
                          w.shift_C.astype(np.float64), k32.astype(np.float64),
                          diag_D.astype(np.float64) if diag_D is not None else None,
                          shift_D=shift_D.astype(np.float64) if shift_D is not None else None, d_head=d_head)
    return out, ref


def _layer_case(h3, w):
    A, B, C, dt = w.diag.complex64()
    k32 = oracle.ssm_kernel(A, B, C, dt, w.L).astype(np.float32)
    return _layer_run(h3, w, k32, diag_D=w.diag_D)


@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
def test_layer_small(h3, dtype):
    w = workloads.layer_workload("t", 2, 256, 256, dtype, seed=21)
    y, ref = _layer_case(h3, w)
    check(y, ref, 2e-2)


# L = 2048 and 8192 take the matrix-core shift SSM, the wave FFT conv and the
# gated transpose (d = 128 is no multiple of the output GEMM's weight tiles,
# so L = 2048 keeps the transpose here too); an odd batch leaves the last row pair half empty, fewer than
# 64 shift taps leave zeros in the Toeplitz band, and a shift D adds to its
# diagonal.  L = 4096 takes the fused VALU middle kernel, L = 16384 the
# 32768-point conv.
@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
@pytest.mark.parametrize("B,L,m_s,with_D", [(3, 2048, 17, True), (1, 8192, 64, False), (2, 2048, 64, True),
                                            (1, 4096, 64, True), (1, 16384, 33, True)])
def test_layer_wave_path(h3, dtype, B, L, m_s, with_D):
    w = workloads.layer_workload("t", B, L, 128, dtype, seed=31 + B + m_s, m_shift=m_s)
    rng = np.random.default_rng(77)
    sD = rng.standard_normal(w.d).astype(np.float32) if with_D else None
    A, Bm, C, dt = w.diag.complex64()
    k32 = oracle.ssm_kernel(A, Bm, C, dt, L).astype(np.float32)
    y, ref = _layer_run(h3, w, k32, shift_D=sD, diag_D=w.diag_D)
    check(y, ref, 2e-2)


# The projections' GEMM paths: 320 x 256 tiles (d a multiple of 320),
# 256 x 256 tiles (d a multiple of 256), 128 x 128 tiles per projection
# (otherwise, or B L not a multiple of 256); Q/K/V fused or not.
@pytest.mark.parametrize("B,L,d", [(2, 256, 256), (1, 128, 256), (2, 256, 384), (1, 1024, 640), (3, 256, 1280)])
def test_layer_gemm_paths(h3, B, L, d):
    w = workloads.layer_workload("t", B, L, d, workloads.BF16, seed=23 + L + d)
    y, ref = _layer_case(h3, w)
    check(y, ref, 2e-2)


# Heads of dimension d_h > 1: d_h^2 diagonal-SSM channels per head, each
# with its own kernel; L = 2048 and 8192 take the wave conv for them, L = 256
# the VALU one, L = 16384 the 32768-point conv; with and without the skip terms.
@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
@pytest.mark.parametrize("B,L,dh,with_D", [(2, 2048, 2, True), (3, 256, 4, False), (1, 8192, 8, True),
                                           (1, 16384, 8, True)])
def test_layer_heads(h3, dtype, B, L, dh, with_D):
    d = 128
    w = workloads.layer_workload("t", B, L, d, dtype, seed=61 + dh + L, m_shift=64)
    rng = np.random.default_rng(dh * 10 + B)
    ssm = workloads.make_diag_ssm(rng, d * dh, 64, 1e-3, 1e-1)
    A, Bm, C, dt = ssm.complex64()
    k32 = oracle.ssm_kernel(A, Bm, C, dt, L).astype(np.float32)
    dD = rng.standard_normal(d * dh).astype(np.float32) if with_D else None
    sD = rng.standard_normal(d).astype(np.float32) if with_D else None
    y, ref = _layer_run(h3, w, k32, shift_D=sD, diag_D=dD, d_head=dh)
    check(y, ref, 2e-2)


# L = 2048 with d a multiple of 256 or 320: the convolution's epilogue gates
# with Q and writes O channel-major, and the output projection reads O
# K-major.  Odd batches leave a half-empty last row pair; B = 6 takes the
# one-channel-per-workgroup conv, B <= 4 the two-channel one (with and without
# the compact table); d = 256 and 768 take the 256-wide weight tiles, 1280 the
# 320-wide ones.
@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
@pytest.mark.parametrize("B,d", [(3, 256), (6, 256), (4, 768), (1, 1280)])
def test_layer_gated_conv(h3, dtype, B, d):
    # the worst rows are the first tokens, whose outputs are 20-60 times
    # smaller than the largest: the 16-bit transform's error is spread evenly
    # over a row of the convolution, so it weighs most there
    w = workloads.layer_workload("t", B, 2048, d, dtype, seed=41 + B + d)
    y, ref = _layer_case(h3, w)
    check(y, ref, 2e-2)


def test_layer_config4_full_size(h3):
    """d=2560 B=4 L=2048 bf16 (the 2.7B layer shape): every batch element."""
    w = workloads.config(4)
    y, ref = _layer_case(h3, w)
    check(y, ref, 2e-2)


# ------------------------------------------- matrix-core conv (L = 2048) ---
@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
@pytest.mark.parametrize("B,H", [(1, 3), (5, 2), (16, 4), (8, 33), (7, 1), (9, 4), (17, 5), (8, 7), (24, 2),
                                 (4, 1031), (3, 1024)])
def test_fftconv_mfma_shapes(h3, dtype, B, H):
    y, ref = _conv_case(h3, B, H, 2048, dtype, seed=B * 100 + H, dt_lo=1e-4)
    check(y, ref, TOL[dtype])


@pytest.mark.parametrize("L,B", [(2048, 4), (2048, 8), (8192, 4)])
@pytest.mark.parametrize("scale_u,scale_k", [(1e3, 1.0), (1e-3, 1.0), (1.0, 1e-5), (30.0, 10.0), (2e4, 1.0),
                                             (1e-5, 1.0), (1e-7, 1.0)])
def test_fftconv_mfma_dynamic_range(h3, scale_u, scale_k, L, B):
    """Inputs far from unit scale: the block FFT rescales by powers of two."""
    rng = np.random.default_rng(5)
    H = 6
    u = (rng.standard_normal((B, H, L)) * scale_u).astype(np.float32)
    u = np.clip(u, -60000.0, 60000.0)
    k = (rng.standard_normal((H, L)) * np.exp(-np.arange(L) / 400.0) * scale_k).astype(np.float32)
    D = rng.standard_normal(H).astype(np.float32)
    for dt in (workloads.BF16, workloads.F16):
        uu = u
        s, u64 = workloads.round_to(uu, dt)
        ref = oracle.causal_conv(u64, k.astype(np.float64), D.astype(np.float64))
        if dt == workloads.F16 and np.abs(ref).max() > 3.0e4:
            # keep the outputs representable in fp16 (the input stays large)
            uu = u * 2.0 ** -math.ceil(math.log2(np.abs(ref).max() / 3.0e4))
            s, u64 = workloads.round_to(uu, dt)
            ref = oracle.causal_conv(u64, k.astype(np.float64), D.astype(np.float64))
        y = to_np64(h3.fftconv(to_dev(s, dt), f32dev(k), f32dev(D)))
        # fp16 outputs below 2^-14 are subnormal: their spacing (2^-24) bounds
        # the absolute error, so the relative gate applies above that scale
        if dt == workloads.F16 and np.abs(ref).max() < 2.0 ** -6:
            assert np.abs(y - ref).max() < 2.0 ** -18, (dt, np.abs(y - ref).max())
        else:
            check(y, ref, TOL[dt], dt)


@pytest.mark.parametrize("L,B", [(2048, 2), (2048, 8), (8192, 2)])
def test_fftconv_mfma_zero_and_impulse(h3, L, B):
    H = 3
    rng = np.random.default_rng(6)
    k = (rng.standard_normal((H, L)) * np.exp(-np.arange(L) / 300.0)).astype(np.float32)
    u = np.zeros((B, H, L), np.float16)
    y = to_np64(h3.fftconv(to_dev(u, workloads.F16), f32dev(k), None))
    assert np.all(y == 0.0)
    u[0, :, 0] = 1.0
    u[1, :, 100] = 1.0
    y = to_np64(h3.fftconv(to_dev(u, workloads.F16), f32dev(k), None))
    check(y[0], k, 2e-2, "impulse_at_0")
    check(y[1, :, 100:], k[:, :L - 100], 2e-2, "impulse_at_100")
    assert np.abs(y[1, :, :100]).max() < 1e-3 * np.abs(k).max()
    assert np.all(y[2:] == 0.0)   # all-zero pairs stay exactly zero


# ----------------------------------------- matrix-core conv (L = 8192) ---
@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
@pytest.mark.parametrize("B,H", [(1, 2), (3, 3), (16, 2)])
def test_fftconv_mfma16k_shapes(h3, dtype, B, H):
    y, ref = _conv_case(h3, B, H, 8192, dtype, seed=B * 10 + H + 7, dt_lo=1e-4)
    check(y, ref, TOL[dtype])


# --------------------------------------------- binding argument checks ---
# The C ABI sees bare pointers; the binding rejects tensors of the wrong
# device, shape, dtype or layout before anything is launched.
def test_binding_rejects_mismatched_tensors(h3):
    dev = torch.device("cuda")
    u = torch.zeros((2, 3, 64), dtype=torch.float16, device=dev)
    k = torch.zeros((3, 64), dtype=torch.float32, device=dev)
    D = torch.zeros(3, dtype=torch.float32, device=dev)
    with pytest.raises(ValueError):
        h3.fftconv(u, k[:2], D)                                  # k too short
    with pytest.raises(ValueError):
        h3.fftconv(u, k, D[:2])                                  # D too short
    with pytest.raises(ValueError):
        h3.fftconv(u, k.cpu(), D)                                # host tensor
    with pytest.raises(ValueError):
        h3.fftconv(u, k, D, out=torch.empty((2, 3, 64), dtype=torch.bfloat16, device=dev))   # out dtype
    with pytest.raises(ValueError):
        h3.fftconv(u, k, D, out=torch.empty((2, 3, 32), dtype=torch.float16, device=dev))    # out shape
    with pytest.raises(ValueError):
        h3.fftconv(u, k, D, out=torch.empty((2, 64, 3), dtype=torch.float16, device=dev).transpose(1, 2))
    P = torch.zeros((3, 8, 2), dtype=torch.float32, device=dev)
    with pytest.raises(ValueError):
        h3.statepass_conv(u, P, P[:2], P, D, 16)                 # Bbar too short
    with pytest.raises(ValueError):
        h3.statepass_conv(u, P, P, P, D, 16, x0=torch.zeros((2, 3, 4, 2), device=dev))   # x0 modes
    x = torch.zeros((2, 3, 8, 2), dtype=torch.float32, device=dev)
    with pytest.raises(ValueError):
        h3.ssm_step(u[..., 0], P, P, P.cpu(), D, x)              # host C
    # the step result of a non-contiguous u comes back with u's shape, computed
    # from the contiguous copy
    ut = torch.randn((3, 2), dtype=torch.float32, device=dev).t()
    y = h3.ssm_step(ut, P, P, P, D, x)
    assert y.shape == ut.shape and y.is_contiguous()
