"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded, rounded inputs.

Metric: err = max|y - y_oracle| / max|y_oracle| per output tensor.  Gates:
1e-5 for float32 I/O, 2e-2 for fp16/bf16 I/O (fp32 accumulation).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests._util import cplx64, cplx_to_f32pairs, f32dev, rel_err, to_dev, to_np64

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
    assert np.abs(cplx64(to_np64(Ab)) - rA).max() < 1e-6
    assert rel_err(cplx64(to_np64(Bb)).view(np.float64), rB.view(np.float64)) < 1e-6


@pytest.mark.parametrize("L,dt_lo,dt_hi", [(1024, 1e-3, 1e-1), (100, 1e-3, 1e-1), (8192, 1e-4, 1e-1), (64, 1e-2, 1e-1), (192, 1e-3, 1e-1),
                                           (2049, 1e-2, 1e-1), (16, 1e-3, 1e-1)])
def test_ssm_kernel(h3, L, dt_lo, dt_hi):
    w = workloads.config(0, H=16, L=16, seed=7, dt_lo=dt_lo, dt_hi=dt_hi)
    A, B, C, dt = _diag_params(w)
    k = h3.ssm_kernel(f32dev(w.ssm.A), f32dev(w.ssm.B), f32dev(w.ssm.C), f32dev(w.ssm.dt), L)
    ref = oracle.ssm_kernel(A, B, C, dt, L)
    assert rel_err(to_np64(k), ref) < 2e-6


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
    assert rel_err(y, ref) < TOL[workloads.F32]


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
@pytest.mark.parametrize("L", [16, 256, 2048, 8192])
def test_fftconv_16bit(h3, dtype, L):
    y, ref = _conv_case(h3, 4, 3, L, dtype, seed=L + 1, dt_lo=1e-4)
    # compare against the oracle rounded to the output dtype as well
    assert rel_err(y, ref) < TOL[dtype]


def test_fftconv_no_skip_odd_batch(h3):
    y, ref = _conv_case(h3, 1, 7, 512, workloads.F32, seed=3, with_D=False)
    assert rel_err(y, ref) < 1e-5


def test_fftconv_impulse_returns_kernel(h3):
    H, L = 4, 1024
    rng = np.random.default_rng(0)
    k = rng.standard_normal((H, L)).astype(np.float32) * np.exp(-np.arange(L) / 300).astype(np.float32)
    u = np.zeros((2, H, L), np.float32); u[:, :, 0] = 1.0
    y = to_np64(h3.fftconv(f32dev(u), f32dev(k), None))
    assert rel_err(y[0], k) < 1e-5 and rel_err(y[1], k) < 1e-5


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


def _end_to_end_conv(h3, w, rows):
    """S1 -> S2/S3 on the GPU at full size; oracle on the sampled rows."""
    k = h3.ssm_kernel(f32dev(w.ssm.A), f32dev(w.ssm.B), f32dev(w.ssm.C), f32dev(w.ssm.dt), w.L)
    y = h3.fftconv(to_dev(w.u, w.dtype), k, f32dev(w.D))
    torch.cuda.synchronize()
    A, B, C, dt = _diag_params(w)
    y = y.view(w.B * w.H, w.L)
    errs = []
    ysel = to_np64(y[torch.tensor(rows, device=y.device)])
    for i, r in enumerate(rows):
        b, h = divmod(r, w.H)
        kh = oracle.ssm_kernel(A[h:h + 1], B[h:h + 1], C[h:h + 1], dt[h:h + 1], w.L)
        ref = oracle.causal_conv(w.u64[b, h][None, None], kh, np.array([w.D[h]], np.float64))
        errs.append((ysel[i], ref[0, 0]))
    ya = np.stack([e[0] for e in errs]); ra = np.stack([e[1] for e in errs])
    return rel_err(ya, ra)


def test_config0_end_to_end_f32(h3):
    w = workloads.config(0)
    err = _end_to_end_conv(h3, w, list(range(w.B * w.H)))
    assert err < 1e-5, err


def test_config1_full_size_sampled_rows(h3):
    w = workloads.config(1)
    rng = np.random.default_rng(11)
    rows = sorted(rng.choice(w.B * w.H, 24, replace=False).tolist()) + [0, w.B * w.H - 1]
    err = _end_to_end_conv(h3, w, rows)
    assert err < 2e-2, err


def test_config2_full_size_sampled_rows(h3):
    w = workloads.config(2)
    rng = np.random.default_rng(12)
    rows = sorted(rng.choice(w.B * w.H, 12, replace=False).tolist()) + [w.B * w.H - 1]
    err = _end_to_end_conv(h3, w, rows)
    assert err < 2e-2, err


# --------------------------------------------------------- S5: statepass ---
def _sp_inputs(w):
    A, B, C, dt = _diag_params(w)
    Ab, Bb = oracle.zoh(A, B, dt)
    # the GPU consumes fp32 discrete parameters; the oracle the same rounded values
    Ab32, Bb32 = cplx_to_f32pairs(Ab), cplx_to_f32pairs(Bb)
    return Ab32, Bb32, cplx64(Ab32), cplx64(Bb32), C


@pytest.mark.parametrize("dtype,L,chunk", [(workloads.F32, 1024, 128), (workloads.F32, 512, 512),
                                           (workloads.F16, 2048, 256), (workloads.BF16, 1024, 16),
                                           (workloads.F32, 256, 16), (workloads.F16, 4096, 1024),
                                           (workloads.BF16, 8192, 2048), (workloads.F16, 8192, 4096)])
def test_statepass_small(h3, dtype, L, chunk):
    w = workloads.statepass_workload("t", 3, 5, L, chunk, dtype, seed=L + chunk, dt_lo=1e-3,
                                     dt_hi=1e-1, x0_scale=0.5)
    Ab32, Bb32, Ab, Bb, C = _sp_inputs(w)
    x0 = cplx64(w.x0)
    y, xf = h3.statepass_conv(to_dev(w.u, dtype), f32dev(Ab32), f32dev(Bb32), f32dev(w.ssm.C),
                              f32dev(w.D), chunk, x0=f32dev(w.x0))
    torch.cuda.synchronize()
    ry, rx = oracle.recurrence(w.u64, Ab, Bb, C, w.D.astype(np.float64), x0=x0)
    assert rel_err(to_np64(y), ry) < TOL[dtype]
    xg = cplx64(to_np64(xf))
    assert np.abs(xg - rx).max() / np.abs(rx).max() < (1e-5 if dtype == workloads.F32 else 2e-2)


def test_statepass_resume(h3):
    w = workloads.statepass_workload("t", 2, 3, 1024, 128, workloads.F32, seed=5, dt_lo=1e-3, dt_hi=1e-1)
    Ab32, Bb32, Ab, Bb, C = _sp_inputs(w)
    u = f32dev(w.u)
    args = (f32dev(Ab32), f32dev(Bb32), f32dev(w.ssm.C), f32dev(w.D))
    y, xf = h3.statepass_conv(u, *args, 128)
    y1, x1 = h3.statepass_conv(u[..., :512].contiguous(), *args, 128)
    y2, x2 = h3.statepass_conv(u[..., 512:].contiguous(), *args, 256, x0=x1)
    torch.cuda.synchronize()
    assert rel_err(to_np64(torch.cat([y1, y2], -1)), to_np64(y)) < 1e-5
    assert rel_err(to_np64(x2), to_np64(xf)) < 1e-5


# ------------------------------------ fused limit 16384 (32768-point) ---
@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
@pytest.mark.parametrize("B,H", [(1, 2), (3, 3)])
def test_fftconv_l16384(h3, dtype, B, H):
    y, ref = _conv_case(h3, B, H, 16384, dtype, seed=B * 10 + H, dt_lo=1e-4)
    assert rel_err(y, ref) < TOL[dtype]


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
    assert rel_err(to_np64(y), ref) < 2e-2


@pytest.mark.parametrize("dtype,B,H,nchunk", [(workloads.F16, 2, 2, 2), (workloads.BF16, 2, 3, 3)])
def test_statepass_chunk16384(h3, dtype, B, H, nchunk):
    """Chunk 16384: chunk end-states on the matrix cores (the 16384 instance
    of the chunk-state kernel), the 32768-point conv per chunk."""
    w = workloads.statepass_workload("t", B, H, nchunk * 16384, 16384, dtype, seed=8 + H, dt_lo=1e-4,
                                     dt_hi=1e-2, x0_scale=0.5)
    Ab32, Bb32, Ab, Bb, C = _sp_inputs(w)
    y, xf = h3.statepass_conv(to_dev(w.u, w.dtype), f32dev(Ab32), f32dev(Bb32), f32dev(w.ssm.C), f32dev(w.D),
                              16384, x0=f32dev(w.x0))
    torch.cuda.synchronize()
    ry, rx = oracle.recurrence(w.u64, Ab, Bb, C, w.D.astype(np.float64), x0=cplx64(w.x0))
    assert rel_err(to_np64(y), ry) < TOL[dtype]
    xg = cplx64(to_np64(xf))
    assert np.abs(xg - rx).max() / np.abs(rx).max() < 2e-2


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
    assert rel_err(to_np64(du), rdu) < 2e-2


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
@pytest.mark.parametrize("B,H,L", [(1, 3, 16), (3, 5, 256), (2, 4, 1024), (5, 3, 2048), (4, 2, 8192),
                                   (19, 3, 2048)])
def test_fftconv_bwd(h3, dtype, B, H, L):
    (du, rdu), (dk, rdk), (dD, rdD) = _bwd_case(h3, B, H, L, dtype, seed=B * 7 + L)
    assert rel_err(du, rdu) < TOL[dtype]
    # dk, dD: float32 outputs; on the matrix cores (16-bit I/O at L = 2048) the
    # transforms run on fp16 operands, so the 16-bit tolerance applies there
    tol_k = TOL[dtype] if (L == 2048 and dtype != workloads.F32) else 1e-5
    assert rel_err(dk, rdk) < tol_k
    assert rel_err(dD, rdD) < tol_k


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_fftconv_bwd_valu_kernel_gradient_at_2048(h3, monkeypatch, dtype):
    """The float32 VALU kernel-gradient kernel forced where the matrix-core one
    runs by default (L = 2048, 16-bit I/O)."""
    monkeypatch.setenv("H3FLASH_WGRAD", "valu")
    (du, rdu), (dk, rdk), (dD, rdD) = _bwd_case(h3, 3, 4, 2048, dtype, seed=77)
    assert rel_err(du, rdu) < TOL[dtype]
    assert rel_err(dk, rdk) < 1e-5
    assert rel_err(dD, rdD) < 1e-5


def test_fftconv_bwd_no_skip_and_partial_outputs(h3):
    B, H, L = 3, 4, 512
    (du, rdu), (dk, rdk), _ = _bwd_case(h3, B, H, L, workloads.F32, seed=41, with_D=False)
    assert rel_err(du, rdu) < 1e-5 and rel_err(dk, rdk) < 1e-5
    w = workloads.conv_workload("t", B, H, L, workloads.F16, seed=42)
    k = f32dev(np.random.default_rng(1).standard_normal((H, L)) / 16)
    dy = to_dev(w.u, workloads.F16)
    du_only, dk0, dD0 = h3.fftconv_bwd(None, k, None, dy, want_dk=False, want_dD=False)
    _, dk_only, dD_only = h3.fftconv_bwd(dy, k, None, dy, want_du=False)
    torch.cuda.synchronize()
    assert dk0 is None and dD0 is None
    rdu, rdk, rdD = oracle.causal_conv_bwd(w.u64, to_np64(k), None, w.u64)
    assert rel_err(to_np64(du_only), rdu) < 2e-2
    assert rel_err(to_np64(dk_only), rdk) < 1e-5   # L = 512: float32 VALU kernel
    assert rel_err(to_np64(dD_only), rdD) < 1e-5


def test_fftconv_bwd_config1_full_size_sampled_channels(h3):
    """At the H3-125M layer shape (B=8, H=768, L=2048, fp16) on the launch
    the benchmark times; sampled channels against the oracle."""
    sel = [0, 1, 383, 500, 767]
    (du, rdu), (dk, rdk), (dD, rdD) = _bwd_case(h3, 8, 768, 2048, workloads.F16, seed=5, sel=sel)
    assert rel_err(du, rdu) < 2e-2
    assert rel_err(dk, rdk) < 2e-2
    assert rel_err(dD, rdD) < 2e-2


def test_fftconv_bwd_adjoint_at_full_size(h3):
    """<dy, conv(u)> = <du, u> at the fused-block limit (B=16 H=256 L=8192 bf16),
    with the forward and backward both on the GPU."""
    w = workloads.config(2)
    A, Bm, C, dt = _diag_params(w)
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
    assert rel_err(to_np64(y), ry) < TOL[dtype]
    xg = cplx64(to_np64(x))
    assert np.abs(xg - rx).max() / np.abs(rx).max() < 1e-5


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
    assert rel_err(to_np64(y_all), ry) < 1e-5
    assert rel_err(to_np64(y_one), ry) < 1e-5
    assert rel_err(to_np64(x1), to_np64(x2)) < 1e-6


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
    assert rel_err(to_np64(torch.cat([y1, y2], -1)), ry) < 2e-2
    assert rel_err(to_np64(y2), ry[..., 2048:]) < 2e-2


def test_config3_full_size_sampled_rows(h3):
    w = workloads.config(3)
    Ab32, Bb32, Ab, Bb, C = _sp_inputs(w)
    y, xf = h3.statepass_conv(to_dev(w.u, w.dtype), f32dev(Ab32), f32dev(Bb32), f32dev(w.ssm.C),
                              f32dev(w.D), w.chunk)
    torch.cuda.synchronize()
    rows = [0, 777, 1024 + 5, 2 * 1024 - 1]
    y = y.view(w.B * w.H, w.L)
    xf = xf.view(w.B * w.H, w.m, 2)
    ys, rs, xs, rxs = [], [], [], []
    for r in rows:
        b, h = divmod(r, w.H)
        ry, rx = oracle.recurrence(w.u64[b, h][None, None], Ab[h:h + 1], Bb[h:h + 1], C[h:h + 1],
                                   w.D[h:h + 1].astype(np.float64))
        ys.append(to_np64(y[r])); rs.append(ry[0, 0])
        xs.append(cplx64(to_np64(xf[r]))); rxs.append(rx[0, 0])
    assert rel_err(np.stack(ys), np.stack(rs)) < 2e-2
    xs, rxs = np.stack(xs), np.stack(rxs)
    assert np.abs(xs - rxs).max() / np.abs(rxs).max() < 2e-2


# ------------------------------------------------------------- S6: layer ---
def _layer_case(h3, w, b_sel=None):
    d, L = w.d, w.L
    A, B, C, dt = w.diag.complex64()
    k64 = oracle.ssm_kernel(A, B, C, dt, L)
    k32 = k64.astype(np.float32)
    W = {n: to_dev(w.weight_out_in(n), w.dtype) for n in "qkvo"}
    out = h3.layer_fwd(to_dev(w.x, w.dtype), W["q"], W["k"], W["v"], W["o"], f32dev(w.shift_C), None,
                       f32dev(k32), f32dev(w.diag_D))
    torch.cuda.synchronize()
    bs = list(range(w.B)) if b_sel is None else b_sel
    ref = oracle.h3_layer(w.x64[bs], w.W["q"][1], w.W["k"][1], w.W["v"][1], w.W["o"][1],
                          w.shift_C.astype(np.float64), k32.astype(np.float64),
                          w.diag_D.astype(np.float64))
    return to_np64(out[bs]), ref


@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
def test_layer_small(h3, dtype):
    w = workloads.layer_workload("t", 2, 256, 256, dtype, seed=21)
    y, ref = _layer_case(h3, w)
    assert rel_err(y, ref) < 2e-2


# L = 2048 and 8192 take the matrix-core shift SSM, the wave FFT conv and the
# gated transpose; an odd batch leaves the last row pair half empty, fewer than
# 64 shift taps leave zeros in the Toeplitz band, and a shift D adds to its
# diagonal.
@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
@pytest.mark.parametrize("B,L,m_s,with_D", [(3, 2048, 17, True), (1, 8192, 64, False), (2, 2048, 64, True)])
def test_layer_wave_path(h3, dtype, B, L, m_s, with_D):
    w = workloads.layer_workload("t", B, L, 128, dtype, seed=31 + B + m_s, m_shift=m_s)
    rng = np.random.default_rng(77)
    sD = rng.standard_normal(w.d).astype(np.float32) if with_D else None
    A, Bm, C, dt = w.diag.complex64()
    k32 = oracle.ssm_kernel(A, Bm, C, dt, L).astype(np.float32)
    W = {n: to_dev(w.weight_out_in(n), w.dtype) for n in "qkvo"}
    out = h3.layer_fwd(to_dev(w.x, w.dtype), W["q"], W["k"], W["v"], W["o"], f32dev(w.shift_C),
                       f32dev(sD) if with_D else None, f32dev(k32), f32dev(w.diag_D))
    torch.cuda.synchronize()
    ref = oracle.h3_layer(w.x64, w.W["q"][1], w.W["k"][1], w.W["v"][1], w.W["o"][1],
                          w.shift_C.astype(np.float64), k32.astype(np.float64), w.diag_D.astype(np.float64),
                          shift_D=sD.astype(np.float64) if with_D else None)
    assert rel_err(to_np64(out), ref) < 2e-2


# The library's own matrix-core GEMM (used where hipBLASLt rejects a shape),
# forced through the documented switch, on both mixing paths.
@pytest.mark.parametrize("L", [256, 2048])
def test_layer_native_gemm(h3, monkeypatch, L):
    monkeypatch.setenv("H3FLASH_GEMM", "native")
    w = workloads.layer_workload("t", 2, L, 256, workloads.BF16, seed=23 + L)
    y, ref = _layer_case(h3, w)
    assert rel_err(y, ref) < 2e-2


# Heads of dimension d_h > 1: d_h^2 diagonal-SSM channels per head, each
# with its own kernel; L = 2048 and 8192 take the wave conv for them, L = 256
# the VALU one; with and without the skip terms.
@pytest.mark.parametrize("dtype", [workloads.BF16, workloads.F16])
@pytest.mark.parametrize("B,L,dh,with_D", [(2, 2048, 2, True), (3, 256, 4, False), (1, 8192, 8, True)])
def test_layer_heads(h3, dtype, B, L, dh, with_D):
    d = 128
    w = workloads.layer_workload("t", B, L, d, dtype, seed=61 + dh + L, m_shift=64)
    rng = np.random.default_rng(dh * 10 + B)
    ssm = workloads.make_diag_ssm(rng, d * dh, 64, 1e-3, 1e-1)
    A, Bm, C, dt = ssm.complex64()
    k32 = oracle.ssm_kernel(A, Bm, C, dt, L).astype(np.float32)
    dD = rng.standard_normal(d * dh).astype(np.float32) if with_D else None
    sD = rng.standard_normal(d).astype(np.float32) if with_D else None
    W = {n: to_dev(w.weight_out_in(n), w.dtype) for n in "qkvo"}
    out = h3.layer_fwd_heads(to_dev(w.x, w.dtype), W["q"], W["k"], W["v"], W["o"], f32dev(w.shift_C),
                             f32dev(sD) if with_D else None, f32dev(k32), f32dev(dD) if with_D else None, dh)
    torch.cuda.synchronize()
    ref = oracle.h3_layer(w.x64, w.W["q"][1], w.W["k"][1], w.W["v"][1], w.W["o"][1],
                          w.shift_C.astype(np.float64), k32.astype(np.float64),
                          dD.astype(np.float64) if with_D else None,
                          shift_D=sD.astype(np.float64) if with_D else None, d_head=dh)
    assert rel_err(to_np64(out), ref) < 2e-2


def test_layer_config4_one_batch_element(h3):
    w = workloads.config(4)
    y, ref = _layer_case(h3, w, b_sel=[3])
    assert rel_err(y, ref) < 2e-2


# ------------------------------------------- matrix-core conv (L = 2048) ---
@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
@pytest.mark.parametrize("B,H", [(1, 3), (5, 2), (16, 4), (8, 33)])
def test_fftconv_mfma_shapes(h3, dtype, B, H):
    y, ref = _conv_case(h3, B, H, 2048, dtype, seed=B * 100 + H, dt_lo=1e-4)
    assert rel_err(y, ref) < TOL[dtype]


@pytest.mark.parametrize("L", [2048, 8192])
@pytest.mark.parametrize("scale_u,scale_k", [(1e3, 1.0), (1e-3, 1.0), (1.0, 1e-5), (30.0, 10.0), (2e4, 1.0)])
def test_fftconv_mfma_dynamic_range(h3, scale_u, scale_k, L):
    """Inputs far from unit scale: the block FFT rescales by powers of two."""
    rng = np.random.default_rng(5)
    B, H = 4, 6
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
        assert rel_err(y, ref) < TOL[dt], (dt, rel_err(y, ref))


@pytest.mark.parametrize("L", [2048, 8192])
def test_fftconv_mfma_zero_and_impulse(h3, L):
    H = 3
    rng = np.random.default_rng(6)
    k = (rng.standard_normal((H, L)) * np.exp(-np.arange(L) / 300.0)).astype(np.float32)
    u = np.zeros((2, H, L), np.float16)
    y = to_np64(h3.fftconv(to_dev(u, workloads.F16), f32dev(k), None))
    assert np.all(y == 0.0)
    u[0, :, 0] = 1.0
    u[1, :, 100] = 1.0
    y = to_np64(h3.fftconv(to_dev(u, workloads.F16), f32dev(k), None))
    kr = k.astype(np.float16).astype(np.float64)
    assert rel_err(y[0], k) < 2e-2
    assert rel_err(y[1, :, 100:], k[:, :L - 100]) < 2e-2
    assert np.abs(y[1, :, :100]).max() < 1e-3 * np.abs(k).max()


# ----------------------------------------- matrix-core conv (L = 8192) ---
@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
@pytest.mark.parametrize("B,H", [(1, 2), (3, 3), (16, 2)])
def test_fftconv_mfma16k_shapes(h3, dtype, B, H):
    y, ref = _conv_case(h3, B, H, 8192, dtype, seed=B * 10 + H + 7, dt_lo=1e-4)
    assert rel_err(y, ref) < TOL[dtype]


@pytest.mark.parametrize("dtype", [workloads.F16, workloads.BF16])
def test_statepass_mfma_chunks(h3, dtype):
    """Chunk 8192 (the fused limit) runs the matrix-core conv per chunk pair."""
    w = workloads.statepass_workload("t", 2, 3, 4 * 8192, 8192, dtype, seed=77, dt_lo=1e-4,
                                     dt_hi=1e-2, x0_scale=0.3)
    Ab32, Bb32, Ab, Bb, C = _sp_inputs(w)
    y, xf = h3.statepass_conv(to_dev(w.u, dtype), f32dev(Ab32), f32dev(Bb32), f32dev(w.ssm.C),
                              f32dev(w.D), w.chunk, x0=f32dev(w.x0))
    torch.cuda.synchronize()
    ry, rx = oracle.recurrence(w.u64, Ab, Bb, C, w.D.astype(np.float64), x0=cplx64(w.x0))
    assert rel_err(to_np64(y), ry) < TOL[dtype]
    xg = cplx64(to_np64(xf))
    assert np.abs(xg - rx).max() / np.abs(rx).max() < 2e-2
