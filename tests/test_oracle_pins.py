"""Pins for the float64 oracle (CPU only).

Each test ties an oracle routine to something other than itself: a closed
form, an invariant the paper states, a brute-force evaluation, a library
routine for a special case, or the paper's worked example.  A plausible slip
in the oracle (dropped factor 2, off-by-one power, wrong sign, transposed
operand) fails at least one of them.
"""
import math
import os

import numpy as np
import pytest
from scipy.integrate import solve_ivp

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_diag(rng, H, m, dt_lo=1e-3, dt_hi=1e-1):
    A = -0.5 + 1j * math.pi * np.arange(m)[None, :].repeat(H, 0)
    A = A + 0.2 * rng.standard_normal((H, m))          # off the S4D-Lin grid too
    B = 1.0 + 0.3 * (rng.standard_normal((H, m)) + 1j * rng.standard_normal((H, m)))
    C = (rng.standard_normal((H, m)) + 1j * rng.standard_normal((H, m))) / math.sqrt(2)
    dt = np.exp(rng.uniform(math.log(dt_lo), math.log(dt_hi), H))
    return A, B, C, dt


# ------------------------------------------------------------------ ZOH -----
def test_zoh_is_exact_solution_of_the_ode_under_held_input():
    """Abar, Bbar are the exact one-step map of x' = A x + B u with u held
    constant: integrate the ODE numerically and compare (Sec. 2.1)."""
    rng = np.random.default_rng(11)
    A, B, C, dt = _rand_diag(rng, 3, 5)
    Ab, Bb = oracle.zoh(A, B, dt)
    for h in range(3):
        for n in range(5):
            a, b = A[h, n], B[h, n]

            def f(t, y, uu):
                x = y[0] + 1j * y[1]
                dx = a * x + b * uu
                return [dx.real, dx.imag]

            s1 = solve_ivp(f, (0, dt[h]), [1.0, 0.0], args=(0.0,), rtol=1e-12, atol=1e-14)
            s2 = solve_ivp(f, (0, dt[h]), [0.0, 0.0], args=(1.0,), rtol=1e-12, atol=1e-14)
            x1 = s1.y[0, -1] + 1j * s1.y[1, -1]
            x2 = s2.y[0, -1] + 1j * s2.y[1, -1]
            assert abs(x1 - Ab[h, n]) < 1e-9
            assert abs(x2 - Bb[h, n]) < 1e-9 * max(1.0, abs(Bb[h, n]))


def test_zoh_small_step_series():
    """Bbar = dt B + dt^2 A B / 2 + O(dt^3) as dt -> 0."""
    A = np.array([[-0.5 + 3j, -2.0 - 1j]])
    B = np.array([[1.0 + 0.5j, 2.0]])
    for dt in (1e-2, 1e-3, 1e-4):
        _, Bb = oracle.zoh(A, B, np.array([dt]))
        err = np.abs(Bb - (dt * B + dt * dt * A * B / 2)).max()
        assert err < 10 * dt ** 3


# --------------------------------------------------------------- kernel -----
def test_kernel_matches_dense_state_space_powers():
    """Sec. 2.1 defines f = [CB, CAB, CA^2B, ...].  Build a real, dense
    state-space system equivalent to the diagonal complex one (conjugate pairs
    of modes, then a random similarity transform) and evaluate C A^t B by
    repeated matrix multiplication."""
    rng = np.random.default_rng(1)
    H, m, L = 2, 6, 64
    A, B, C, dt = _rand_diag(rng, H, m)
    Ab, Bb = oracle.zoh(A, B, dt)
    k = oracle.ssm_kernel_discrete(Ab, Bb, C, L)
    for h in range(H):
        Ad = np.diag(np.concatenate([Ab[h], Ab[h].conj()]))
        Bd = np.concatenate([Bb[h], Bb[h].conj()])[:, None]
        Cd = np.concatenate([C[h], C[h].conj()])[None, :]
        T = rng.standard_normal((2 * m, 2 * m)) + 1j * rng.standard_normal((2 * m, 2 * m))
        Ti = np.linalg.inv(T)
        A2, B2, C2 = T @ Ad @ Ti, T @ Bd, Cd @ Ti
        x = B2.copy()
        for t in range(L):
            f_t = (C2 @ x)[0, 0]
            assert abs(f_t.imag) < 1e-9
            assert abs(f_t.real - k[h, t]) < 1e-9 * max(1.0, np.abs(k[h]).max())
            x = A2 @ x


def test_kernel_is_impulse_response_of_recurrence():
    """With u = delta_0 the recurrence outputs k_t (+ D at t = 0).  This fixes
    the factor 2 Re in the output convention."""
    rng = np.random.default_rng(2)
    H, m, L = 3, 8, 128
    A, B, C, dt = _rand_diag(rng, H, m)
    D = rng.standard_normal(H)
    Ab, Bb = oracle.zoh(A, B, dt)
    k = oracle.ssm_kernel_discrete(Ab, Bb, C, L)
    u = np.zeros((1, H, L)); u[..., 0] = 1.0
    y, _ = oracle.recurrence(u, Ab, Bb, C, D)
    expect = k.copy(); expect[:, 0] += D
    np.testing.assert_allclose(y[0], expect, rtol=0, atol=1e-12)


def test_kernel_geometric_series_single_real_mode():
    """m = 1, Abar = 1/2, Bbar = 1, C = 1/4: k_t = 2 * (1/4) * 2^-t = 2^-(t+1)."""
    k = oracle.ssm_kernel_discrete(np.array([[0.5 + 0j]]), np.array([[1.0 + 0j]]),
                                   np.array([[0.25 + 0j]]), 20)
    np.testing.assert_allclose(k[0], 2.0 ** -(np.arange(20) + 1.0), rtol=1e-14, atol=0)


def test_kernel_continuous_equals_discrete_after_zoh():
    rng = np.random.default_rng(3)
    A, B, C, dt = _rand_diag(rng, 4, 16)
    Ab, Bb = oracle.zoh(A, B, dt)
    k1 = oracle.ssm_kernel(A, B, C, dt, 300)
    k2 = oracle.ssm_kernel_discrete(Ab, Bb, C, 300)
    np.testing.assert_allclose(k1, k2, rtol=0, atol=1e-11 * np.abs(k1).max())


def test_shift_kernel_is_its_taps():
    """Shift SSM with B = e_1: the output is a 1-D convolution whose taps are C
    (Sec. 3.2): impulse response = [C_0, ..., C_{m-1}, 0, ...]."""
    rng = np.random.default_rng(4)
    Cs = rng.standard_normal((3, 5))
    u = np.zeros((1, 3, 12)); u[..., 0] = 1.0
    y = oracle.shift_ssm(u, Cs)
    expect = np.zeros((3, 12)); expect[:, :5] = Cs
    np.testing.assert_array_equal(y[0], expect)


# ----------------------------------------------------------------- conv -----
def _dft_matrix(n):
    j = np.arange(n)
    return np.exp(-2j * np.pi * np.outer(j, j) / n)


def test_conv_impulse_returns_kernel_and_skip():
    rng = np.random.default_rng(5)
    H, L = 4, 64
    k = rng.standard_normal((H, L)); D = rng.standard_normal(H)
    u = np.zeros((1, H, L)); u[..., 0] = 1.0
    np.testing.assert_array_equal(oracle.causal_conv(u, k)[0], k)
    y = oracle.causal_conv(u, k, D)[0]
    np.testing.assert_allclose(y[:, 0], k[:, 0] + D, rtol=0, atol=1e-15)
    np.testing.assert_array_equal(y[:, 1:], k[:, 1:])


@pytest.mark.parametrize("L", [1, 2, 3, 8, 16, 32])
def test_conv_equals_bruteforce_dft_convolution(L):
    """FFT convolution (Sec. 2.1): zero-pad to 2L, multiply the DFTs, invert,
    keep the first L.  Evaluated with explicit O(N^2) DFT matrices."""
    rng = np.random.default_rng(100 + L)
    H, Bn = 3, 2
    u = rng.standard_normal((Bn, H, L)); k = rng.standard_normal((H, L)); D = rng.standard_normal(H)
    N = 2 * L
    F = _dft_matrix(N); Fi = np.conj(F) / N
    up = np.zeros((Bn, H, N)); up[..., :L] = u
    kp = np.zeros((H, N)); kp[:, :L] = k
    Y = (up @ F.T) * (kp @ F.T)[None]
    y = (Y @ Fi.T).real[..., :L] + D[None, :, None] * u
    np.testing.assert_allclose(oracle.causal_conv(u, k, D), y, rtol=0, atol=1e-12 * max(1, np.abs(y).max()))


def test_conv_equals_numpy_rfft_at_length_1024():
    rng = np.random.default_rng(6)
    H, L = 8, 1024
    u = rng.standard_normal((2, H, L)); k = rng.standard_normal((H, L)) * np.exp(-np.arange(L) / 200)
    D = rng.standard_normal(H)
    y = np.fft.irfft(np.fft.rfft(u, 2 * L) * np.fft.rfft(k, 2 * L)[None], 2 * L)[..., :L] + D[:, None] * u
    np.testing.assert_allclose(oracle.causal_conv(u, k, D), y, rtol=0, atol=1e-10)


def test_conv_linear_time_invariant_causal():
    rng = np.random.default_rng(7)
    H, L = 2, 200
    k = rng.standard_normal((H, L)); D = rng.standard_normal(H)
    u1 = rng.standard_normal((1, H, L)); u2 = rng.standard_normal((1, H, L))
    y1, y2 = oracle.causal_conv(u1, k, D), oracle.causal_conv(u2, k, D)
    np.testing.assert_allclose(oracle.causal_conv(2.5 * u1 - 0.75 * u2, k, D), 2.5 * y1 - 0.75 * y2, atol=1e-11)
    s = 37
    us = np.zeros_like(u1); us[..., s:] = u1[..., :-s]
    np.testing.assert_allclose(oracle.causal_conv(us, k, D)[..., s:], y1[..., :-s], atol=1e-11)
    up = u1.copy(); up[..., 120] += 10.0
    yp = oracle.causal_conv(up, k, D)
    np.testing.assert_array_equal(yp[..., :120], y1[..., :120])
    assert np.abs(yp[..., 120:] - y1[..., 120:]).max() > 0


# --------------------------------------------------- conv backward pass -----
def test_conv_bwd_adjoint_identity():
    """The gradients are the adjoint of the (pinned) forward convolution:
    <dy, conv(u, k, D)> = <du, u> = <dk, k> + <dD, D>  (the forward is
    bilinear in u and (k, D))."""
    rng = np.random.default_rng(31)
    Bn, H, L = 3, 4, 96
    u = rng.standard_normal((Bn, H, L)); k = rng.standard_normal((H, L)) / 8
    D = rng.standard_normal(H); dy = rng.standard_normal((Bn, H, L))
    y = oracle.causal_conv(u, k, D)
    du, dk, dD = oracle.causal_conv_bwd(u, k, D, dy)
    J = np.sum(dy * y)
    assert abs(np.sum(du * u) - J) < 1e-10 * abs(J) + 1e-9
    assert abs(np.sum(dk * k) + np.sum(dD * D) - J) < 1e-10 * abs(J) + 1e-9


def test_conv_bwd_unit_perturbations():
    """The forward is linear in each of u, k, D, so a unit change of one entry
    changes J = <dy, y> by exactly the gradient at that entry."""
    rng = np.random.default_rng(32)
    Bn, H, L = 2, 3, 40
    u = rng.standard_normal((Bn, H, L)); k = rng.standard_normal((H, L))
    D = rng.standard_normal(H); dy = rng.standard_normal((Bn, H, L))
    J0 = np.sum(dy * oracle.causal_conv(u, k, D))
    du, dk, dD = oracle.causal_conv_bwd(u, k, D, dy)
    for (b, h, t) in [(0, 0, 0), (1, 2, 39), (0, 1, 17), (1, 0, 5)]:
        u2 = u.copy(); u2[b, h, t] += 1.0
        assert abs(np.sum(dy * oracle.causal_conv(u2, k, D)) - J0 - du[b, h, t]) < 1e-9
    for (h, j) in [(0, 0), (2, 39), (1, 11)]:
        k2 = k.copy(); k2[h, j] += 1.0
        assert abs(np.sum(dy * oracle.causal_conv(u, k2, D)) - J0 - dk[h, j]) < 1e-9
    for h in range(H):
        D2 = D.copy(); D2[h] += 1.0
        assert abs(np.sum(dy * oracle.causal_conv(u, k, D2)) - J0 - dD[h]) < 1e-9
    du0, _, _ = oracle.causal_conv_bwd(u, k, None, dy)      # no D: no skip term
    np.testing.assert_allclose(du - du0, D[None, :, None] * dy, atol=1e-12)


def test_conv_bwd_matches_autograd():
    """Against reverse-mode differentiation (float64 CPU autograd) of the
    convolution written as a 1-D correlation with the flipped kernel."""
    import torch
    rng = np.random.default_rng(33)
    Bn, H, L = 2, 3, 33
    u = torch.tensor(rng.standard_normal((Bn, H, L)), requires_grad=True)
    k = torch.tensor(rng.standard_normal((H, L)), requires_grad=True)
    D = torch.tensor(rng.standard_normal(H), requires_grad=True)
    dy = rng.standard_normal((Bn, H, L))
    # y[b,h,t] = sum_j k[h,j] u[b,h,t-j]: grouped conv1d over left-padded u
    y = torch.nn.functional.conv1d(torch.nn.functional.pad(u, (L - 1, 0)), k.flip(-1).unsqueeze(1), groups=H)
    y = y + D[None, :, None] * u
    (y * torch.tensor(dy)).sum().backward()
    du, dk, dD = oracle.causal_conv_bwd(u.detach().numpy(), k.detach().numpy(), D.detach().numpy(), dy)
    np.testing.assert_allclose(du, u.grad.numpy(), atol=1e-11)
    np.testing.assert_allclose(dk, k.grad.numpy(), atol=1e-11)
    np.testing.assert_allclose(dD, D.grad.numpy(), atol=1e-11)


# ----------------------------------------------------------- recurrence -----
def test_recurrence_equals_convolution_plus_initial_state_term():
    """Sec. 2.1: from an initial state x0, y_t = (C Abar^{t+1} x0 term) +
    (f * u)_t + D u_t.  Here the state is complex diagonal, so the
    initial-state term is 2 Re sum_n C_n Abar_n^{t+1} x0_n; with x0 = 0 the
    recurrence is exactly the convolution."""
    rng = np.random.default_rng(8)
    H, m, L, Bn = 3, 8, 150, 2
    A, B, C, dt = _rand_diag(rng, H, m)
    D = rng.standard_normal(H)
    Ab, Bb = oracle.zoh(A, B, dt)
    k = oracle.ssm_kernel_discrete(Ab, Bb, C, L)
    u = rng.standard_normal((Bn, H, L))
    y0, _ = oracle.recurrence(u, Ab, Bb, C, D)
    np.testing.assert_allclose(y0, oracle.causal_conv(u, k, D), atol=1e-11)
    x0 = rng.standard_normal((Bn, H, m)) + 1j * rng.standard_normal((Bn, H, m))
    y1, _ = oracle.recurrence(u, Ab, Bb, C, D, x0=x0)
    t = np.arange(L)
    pw = Ab[None, :, :, None] ** (t + 1)[None, None, None, :]          # (1, H, m, L)
    free = 2 * np.real(np.einsum("hn,bhn,bhnt->bht", C, x0, np.broadcast_to(pw, (Bn, H, m, L))))
    np.testing.assert_allclose(y1 - y0, free, atol=1e-11)


def test_recurrence_token_by_token_and_final_state_closed_form():
    """Step mode (generation) chains one-token recurrences through the state:
    that must equal one pass over the whole sequence, and the final state must
    equal its closed form x_{L-1} = Abar^L x0 + sum_i Abar^{L-1-i} Bbar u_i
    (the unrolled recurrence of Sec. 2, written with explicit powers)."""
    rng = np.random.default_rng(19)
    H, m, L, Bn = 3, 5, 40, 2
    A, B, C, dt = _rand_diag(rng, H, m)
    D = rng.standard_normal(H)
    Ab, Bb = oracle.zoh(A, B, dt)
    u = rng.standard_normal((Bn, H, L))
    x0 = rng.standard_normal((Bn, H, m)) + 1j * rng.standard_normal((Bn, H, m))
    y, xf = oracle.recurrence(u, Ab, Bb, C, D, x0=x0)
    x, ys = x0, []
    for t in range(L):
        yt, x = oracle.recurrence(u[..., t:t + 1], Ab, Bb, C, D, x0=x)
        ys.append(yt)
    np.testing.assert_allclose(np.concatenate(ys, -1), y, atol=1e-12)
    np.testing.assert_allclose(x, xf, atol=1e-12)
    i = np.arange(L)
    pw = Ab[:, :, None] ** (L - 1 - i)[None, None, :]                  # (H, m, L)
    closed = Ab[None] ** L * x0 + Bb[None] * np.einsum("hnl,bhl->bhn", pw, u)
    np.testing.assert_allclose(xf, closed, atol=1e-11)
    # an absent D is no skip term, in the recurrence and in state passing
    y0, x0f = oracle.recurrence(u, Ab, Bb, C, None, x0=x0)
    np.testing.assert_array_equal(y0, oracle.recurrence(u, Ab, Bb, C, np.zeros(H), x0=x0)[0])
    np.testing.assert_allclose(y - y0, D[None, :, None] * u, atol=1e-12)
    np.testing.assert_allclose(oracle.statepass(u, Ab, Bb, C, None, 8, x0=x0)[0], y0, atol=1e-10)


def test_toy_diag_ssm_cumulative_sum_exact():
    """Appendix C.1 remark: a diagonal SSM with A = 1, B = 1 acts as a
    cumulative sum.  With complex-mode convention C = 1/2 gives 2 Re(C x) = x."""
    rng = np.random.default_rng(9)
    L = 500
    u = rng.integers(-50, 50, (2, 1, L)).astype(np.float64)
    y, xf = oracle.recurrence(u, np.array([[1 + 0j]]), np.array([[1 + 0j]]), np.array([[0.5 + 0j]]), np.array([3.0]))
    np.testing.assert_array_equal(y, np.cumsum(u, axis=-1) + 3.0 * u)
    np.testing.assert_array_equal(xf[..., 0].real, u.sum(-1))


def test_toy_shift_ssm_is_one_step_delay():
    """Appendix C.1 remark: shift SSM with B = e_1, C = [0 1] delays by one."""
    rng = np.random.default_rng(10)
    u = rng.standard_normal((2, 3, 40))
    y = oracle.shift_ssm(u, np.tile([0.0, 1.0], (3, 1)))
    np.testing.assert_array_equal(y[..., 1:], u[..., :-1])
    np.testing.assert_array_equal(y[..., 0], 0.0)


def test_shift_ssm_equals_fir_with_taps():
    rng = np.random.default_rng(12)
    H, L, m = 4, 300, 64
    Cs = rng.standard_normal((H, m)) / 8; Ds = rng.standard_normal(H)
    u = rng.standard_normal((2, H, L))
    k = np.zeros((H, L)); k[:, :m] = Cs
    np.testing.assert_allclose(oracle.shift_ssm(u, Cs, Ds), oracle.causal_conv(u, k, Ds), atol=1e-12)


# ------------------------------------------------------- state passing -----
def test_statepass_equals_recurrence_for_every_chunk():
    """Proposition 2: Algorithm 2 returns the SSM output for any chunk size
    dividing the length, and its last state is the recurrence's."""
    rng = np.random.default_rng(13)
    H, m, L, Bn = 2, 8, 256, 2
    A, B, C, dt = _rand_diag(rng, H, m, 1e-2, 1e-1)
    D = rng.standard_normal(H)
    Ab, Bb = oracle.zoh(A, B, dt)
    u = rng.standard_normal((Bn, H, L))
    x0 = rng.standard_normal((Bn, H, m)) + 1j * rng.standard_normal((Bn, H, m))
    for x in (None, x0):
        yr, xr = oracle.recurrence(u, Ab, Bb, C, D, x0=x)
        for chunk in (256, 128, 64, 32, 16, 8, 1):
            ys, xs = oracle.statepass(u, Ab, Bb, C, D, chunk, x0=x)
            np.testing.assert_allclose(ys, yr, atol=1e-10)
            np.testing.assert_allclose(xs, xr, atol=1e-10)


def test_statepass_resume_from_final_state():
    rng = np.random.default_rng(14)
    H, m, L = 3, 4, 192
    A, B, C, dt = _rand_diag(rng, H, m)
    D = rng.standard_normal(H)
    Ab, Bb = oracle.zoh(A, B, dt)
    u = rng.standard_normal((1, H, L))
    y, x = oracle.statepass(u, Ab, Bb, C, D, 32)
    y1, x1 = oracle.statepass(u[..., :64], Ab, Bb, C, D, 32)
    y2, x2 = oracle.statepass(u[..., 64:], Ab, Bb, C, D, 64, x0=x1)
    np.testing.assert_allclose(np.concatenate([y1, y2], -1), y, atol=1e-11)
    np.testing.assert_allclose(x2, x, atol=1e-11)


# ---------------------------------------------------------------- layer -----
def _read_golden(name):
    blocks, cur = {}, None
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("["):
                cur = line.strip("[]"); blocks[cur] = []
            else:
                blocks[cur].append([float(v) for v in line.split()])
    return {k: np.array(v) for k, v in blocks.items()}


def test_layer_associative_recall_worked_example():
    """Appendix C.1: with the printed W_Q = W_K, W_V, a one-step-delay shift SSM
    and a cumulative-sum diagonal SSM (d = 8, H = 4 heads of size 2), the output
    at the final (query) token is zero in every head but the queried key's, and
    there it is a multiple of the binary code of the associated value."""
    g = _read_golden("h3_associative_recall.txt")
    Wq, Wv, codes = g["W_Q"], g["W_V"], g["codes"]
    d, dh, nh = 8, 2, 4
    rng = np.random.default_rng(15)
    shift_C = np.tile([0.0, 1.0], (d, 1))
    for trial in range(20):
        Npairs = int(rng.integers(2, 9))
        f_map = rng.integers(0, 4, 4)                   # key i -> value f_map[i]
        keys = rng.integers(0, 4, Npairs)
        seq = []
        for kk in keys:
            seq += [kk, 4 + f_map[kk]]
        q = int(rng.choice(keys))
        seq.append(q)
        x = np.eye(8)[seq][None]                        # (1, N+1, 8) one-hot embeddings
        N1 = x.shape[1]
        diag_k = np.ones((nh * dh * dh, N1))            # A = 1, B = C = e_1: cumulative sum
        _, O = oracle.h3_layer(x, Wq, Wq, Wv, np.eye(d), shift_C, diag_k, np.zeros(nh * dh * dh),
                               d_head=dh, return_O=True)
        last = O[0, -1].reshape(nh, dh)
        for j in range(nh):
            if j != q:
                np.testing.assert_array_equal(last[j], 0.0)
        count = int((keys == q).sum())
        # sum over the two rows of the head's d_h x d_h state, times the count
        np.testing.assert_allclose(last[q], 2 * count * codes[f_map[q]], atol=1e-12)


def test_layer_head_dim_one_closed_form():
    """d_h = 1 with identity projections, a one-step-delay shift SSM and a
    cumulative-sum diagonal SSM: out_t = x_t * sum_{j<=t} x_{j-1} x_j
    (Algorithm 1 with d_h = 1: Q * SSM_diag(SSM_shift(K) * V))."""
    rng = np.random.default_rng(16)
    Bn, N, d = 2, 30, 6
    x = rng.integers(-3, 4, (Bn, N, d)).astype(np.float64)
    I = np.eye(d)
    out = oracle.h3_layer(x, I, I, I, I, np.tile([0.0, 1.0], (d, 1)), np.ones((d, N)), np.zeros(d))
    prev = np.concatenate([np.zeros((Bn, 1, d)), x[:, :-1]], 1)
    expect = x * np.cumsum(prev * x, axis=1)
    np.testing.assert_array_equal(out, expect)


def test_layer_projection_convention_row_vector():
    """Q = x W_Q (row-vector convention): a non-symmetric W must not be
    applied transposed.  Diagonal SSM = identity (k = delta, D = 0), shift =
    identity (taps [1]); then out = ((x Wq) * (x Wk) * (x Wv)) Wo."""
    rng = np.random.default_rng(17)
    Bn, N, d = 1, 5, 4
    x = rng.standard_normal((Bn, N, d))
    W = [rng.standard_normal((d, d)) for _ in range(4)]
    k = np.zeros((d, N)); k[:, 0] = 1.0
    out = oracle.h3_layer(x, *W, np.ones((d, 1)), k, np.zeros(d))
    expect = ((x @ W[0]) * (x @ W[1]) * (x @ W[2])) @ W[3]
    np.testing.assert_allclose(out, expect, atol=1e-12)


# ------------------------------------------------------------ block FFT -----
@pytest.mark.parametrize("N1,N2", [(4, 4), (4, 8), (8, 4), (2, 16), (8, 8)])
def test_block_fft_factorisation(N1, N2):
    """Sec. 4.1: F_N = P (I_{N2} x F_{N1}) P^T D (I_{N1} x F_{N2}) P, with P the
    permutation that reshapes a length-N vector row-major as N2 x N1 and
    transposes it, and D[i] = w_N^{floor(i/N2) * (i mod N2)}."""
    N = N1 * N2
    P = np.zeros((N, N))
    for i in range(N):
        v = np.zeros(N); v[i] = 1
        P[:, i] = v.reshape(N2, N1).T.reshape(-1)
    i = np.arange(N)
    D = np.diag(np.exp(-2j * np.pi * (i // N2) * (i % N2) / N))
    M = P @ np.kron(np.eye(N2), _dft_matrix(N1)) @ P.T @ D @ np.kron(np.eye(N1), _dft_matrix(N2)) @ P
    np.testing.assert_allclose(M, _dft_matrix(N), atol=1e-10)


# ------------------------------------------------------------ workloads -----
def test_workload_shapes_and_rounding():
    w = workloads.config(0)
    assert w.u.dtype == np.float32 and w.u.shape == (1, 64, 1024)
    assert w.ssm.A.shape == (64, 64, 2) and w.ssm.dt.min() >= 1e-3 * 0.999 and w.ssm.dt.max() <= 0.1 * 1.001
    w1 = workloads.config(1, B=2, H=4, L=64)
    assert w1.u.dtype == np.float16 and w1.shift_C.shape == (4, 64)
    np.testing.assert_array_equal(w1.u.astype(np.float64), w1.u64)
    bits, v = workloads.round_to(np.array([1.0, 1.00390625, 1.01171875, -3.3, 65504.0 * 3]), "bf16")
    # 1 + 2^-8 is a tie -> even (1.0); 1 + 3*2^-8 is a tie -> even (1 + 2^-6)
    np.testing.assert_array_equal(v[:3], [1.0, 1.0, 1.015625])
    assert abs(v[3] + 3.3) < 3.3 * 2 ** -8
