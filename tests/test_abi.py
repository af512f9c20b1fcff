"""C ABI checks that need no GPU: the library loads, exports every function
the header declares, sizes its workspaces, and rejects invalid arguments with
the documented status before launching anything."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "h3flash.h")

import paper_2212_14052_amd as h3

OK, EINVAL, EUNSUP, EWS = 0, -1, -2, -3
P = lambda v: ctypes.c_void_p(v)
U, K, Y, W, X = 0x100000, 0x4000000, 0x8000000, 0xC000000, 0x10000000   # fake, aligned


def declared_functions():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(h3_\w+)\s*\(", txt, re.M)))


def test_library_exports_every_declared_function():
    L = h3.lib()
    names = declared_functions()
    assert len(names) >= 7
    for n in names:
        assert hasattr(L, n), n


def test_status_strings():
    assert h3.status_string(0) == "ok"
    for s in (-1, -2, -3, -4):
        assert h3.status_string(s) not in ("ok", "unknown status")
    assert h3.status_string(7) == "unknown status"


def test_workspace_sizes():
    ws = h3.workspace_size(h3.OP_FFTCONV, 8, 768, 2048, 0, 0, h3.F16)
    assert ws >= 768 * 2049 * 8
    ws = h3.workspace_size(h3.OP_STATEPASS, 2, 1024, 131072, 64, 8192, h3.F16)
    # fused initial-state path: end-states, power tables and normalised
    # weights (the convs form the chunk kernel themselves), not a (B, H, L)
    # correction term
    assert 2 * 1024 * 16 * 64 * 8 + 1024 * 1600 * 16 <= ws < 1024 * 8192 * 4 + 2 * 1024 * 16 * 64 * 8 + 1024 * 1600 * 16 + (4 << 20)
    # float32 I/O keeps the float32 correction term (B, H, L)
    assert h3.workspace_size(h3.OP_STATEPASS, 2, 64, 16384, 64, 1024, h3.F32) >= 2 * 64 * 16384 * 4
    assert h3.workspace_size(h3.OP_STATEPASS, 2, 4, 100, 64, 64, h3.F16) == 0   # L % chunk
    assert h3.workspace_size(99, 1, 1, 16, 0, 0, 0) == 0
    assert h3.workspace_size(h3.OP_FFTCONV, 1, 1, 16, 0, 0, 7) == 0
    assert h3.workspace_size(h3.OP_LAYER, 4, 2560, 2048, 64, 0, h3.BF16) > 4 * 2560 * 2048 * 2 * 5
    # backward: at least the conv's spectrum; with more than four row pairs per
    # channel at L = 2048 (16-bit) also the kernel-gradient partial sums
    assert h3.workspace_size(h3.OP_FFTCONV_BWD, 8, 768, 2048, 0, 0, h3.F16) >= 768 * 2049 * 8
    assert h3.workspace_size(h3.OP_FFTCONV_BWD, 32, 768, 2048, 0, 0, h3.F16) >= 4 * 768 * 2048 * 4


def fftconv(u=U, k=K, D=None, y=Y, B=2, H=4, L=64, dt=0, ws=W, wsb=1 << 24):
    return h3.lib().h3_fftconv(P(u), P(k), P(D), P(y), B, H, L, dt, P(ws), wsb, None)


def test_fftconv_validation():
    assert fftconv(u=0) == EINVAL
    assert fftconv(k=0) == EINVAL
    assert fftconv(y=0) == EINVAL
    assert fftconv(B=0) == EINVAL
    assert fftconv(L=48) == EUNSUP                  # not a power of two
    assert fftconv(L=8) == EUNSUP                   # below the minimum
    assert fftconv(L=16384) == EUNSUP               # above the float32 fused limit
    assert fftconv(L=32768, dt=1) == EUNSUP         # above the 16-bit fused limit
    assert fftconv(dt=3) == EUNSUP
    assert fftconv(ws=0) == EWS
    assert fftconv(wsb=16) == EWS
    assert fftconv(u=U + 2) == EINVAL               # misaligned
    assert fftconv(y=U + 64) == EINVAL              # overlaps u
    assert fftconv(ws=U + 256) == EINVAL            # workspace overlaps u


def statepass(u=U, A=K, Bb=K + 4096, C=K + 8192, D=None, x0=None, B=2, H=4, L=256, m=64,
              chunk=64, dt=1, y=Y, xf=None, ws=W, wsb=1 << 26):
    return h3.lib().h3_statepass_conv(P(u), P(A), P(Bb), P(C), P(D), P(x0), B, H, L, m, chunk, dt,
                                      P(y), P(xf), P(ws), wsb, None)


def test_statepass_validation():
    assert statepass(u=0) == EINVAL
    assert statepass(A=0) == EINVAL
    assert statepass(L=250) == EINVAL               # chunk does not divide L
    assert statepass(chunk=48, L=96) == EUNSUP
    assert statepass(chunk=32768, L=32768) == EUNSUP
    assert statepass(chunk=16384, L=16384, dt=0) == EUNSUP   # float32 chunks stop at 8192
    assert statepass(m=65) == EUNSUP
    assert statepass(m=0) == EINVAL
    assert statepass(dt=5) == EUNSUP
    assert statepass(ws=0) == EWS
    assert statepass(wsb=100) == EWS
    assert statepass(y=U) == EINVAL                 # y aliases u
    assert statepass(xf=Y + 16) == EINVAL           # x_final inside y


def layer(x=U, B=2, L=64, d=128, m_s=64, dt=2, out=Y, ws=W, wsb=1 << 28, shift=K, diag=K + 65536):
    return h3.lib().h3_layer_fwd(P(x), P(K), P(K), P(K), P(K), P(shift), None, P(diag), None,
                                 B, L, d, m_s, dt, P(out), P(ws), wsb, None)


def test_layer_validation():
    assert layer(x=0) == EINVAL
    assert layer(shift=0) == EINVAL
    assert layer(dt=0) == EUNSUP                    # fp32 layer not built
    assert layer(d=100) == EUNSUP
    assert layer(d=64) == EUNSUP                    # d a multiple of 128 (documented)
    assert layer(d=192) == EUNSUP
    assert layer(m_s=65) == EUNSUP
    assert layer(L=100) == EUNSUP
    assert layer(B=1, L=64) == EUNSUP               # B*L not a multiple of 128
    assert layer(ws=0) == EWS
    assert layer(out=U) == EINVAL


def test_discretize_and_kernel_validation():
    L = h3.lib()
    assert L.h3_ssm_discretize(None, P(K), P(K), 4, 8, P(Y), P(Y), None) == EINVAL
    assert L.h3_ssm_discretize(P(K), P(K), P(K), 4, 65, P(Y), P(Y), None) == EUNSUP
    assert L.h3_ssm_kernel(P(K), P(K), P(K), P(K), 4, 8, 0, P(Y), None) == EINVAL
    assert L.h3_ssm_kernel(P(K), P(K), P(K), P(K), 4, 70, 16, P(Y), None) == EUNSUP


def test_spectral_validation():
    L = h3.lib()
    assert L.h3_kernel_spectrum(None, 4, 64, P(Y), None) == EINVAL
    assert L.h3_kernel_spectrum(P(K), 4, 100, P(Y), None) == EUNSUP
    assert L.h3_kernel_spectrum(P(K), 4, 64, P(K + 64), None) == EINVAL      # overlap
    assert L.h3_fftconv_spectral(P(U), P(K), None, P(U), 2, 4, 64, 0, None) == EINVAL
    assert L.h3_fftconv_spectral(P(U), P(K), None, P(Y), 2, 4, 64, 9, None) == EUNSUP
    assert L.h3_fftconv_spectral(P(U), P(K), None, P(Y), 2, 4, 32768, 1, None) == EUNSUP
    assert L.h3_fftconv_spectral(P(U), P(K), None, P(Y), 2, 4, 16384, 1, None) == EUNSUP
    assert L.h3_kernel_spectrum(P(K), 4, 16384, P(Y), None) == EUNSUP


def step(u=U, A=K, Bb=K + 4096, C=K + 8192, D=None, B=2, H=4, m=64, T=1, dt=1, x=X, y=Y):
    return h3.lib().h3_ssm_step(P(u), P(A), P(Bb), P(C), P(D), B, H, m, T, dt, P(x), P(y), None)


def test_step_validation():
    assert step(u=0) == EINVAL
    assert step(x=0) == EINVAL
    assert step(T=0) == EINVAL
    assert step(m=0) == EINVAL
    assert step(m=65) == EUNSUP
    assert step(dt=3) == EUNSUP
    assert step(x=X + 4) == EINVAL                   # complex state not 8-byte aligned
    assert step(u=U + 1) == EINVAL                   # 16-bit tokens misaligned
    assert step(y=U) == EINVAL                       # y aliases u
    assert step(y=X + 64) == EINVAL                  # y inside the state
    assert step(x=K + 256) == EINVAL                 # state overlaps Abar


def bwd(u=U, k=K, D=None, dy=X, B=2, H=4, L=64, dt=1, du=Y, dk=K + 0x100000, dD=None, ws=W, wsb=1 << 24):
    return h3.lib().h3_fftconv_bwd(P(u), P(k), P(D), P(dy), B, H, L, dt, P(du), P(dk), P(dD), P(ws), wsb, None)


def test_bwd_validation():
    assert bwd(dy=0) == EINVAL
    assert bwd(k=0) == EINVAL
    assert bwd(du=0, dk=0, dD=0) == EINVAL            # nothing asked
    assert bwd(u=0) == EINVAL                         # dk needs u
    assert bwd(L=48) == EUNSUP
    assert bwd(L=16384) == EUNSUP                     # kernel gradient stops at 8192
    assert bwd(L=32768, dk=0) == EUNSUP
    assert bwd(dt=3) == EUNSUP
    assert bwd(ws=0) == EWS
    assert bwd(du=X) == EINVAL                        # du aliases dy
    assert bwd(dk=K + 64) == EINVAL                   # dk overlaps k
    assert bwd(dD=Y + 8) == EINVAL                    # dD inside du
    assert bwd(dD=K + 0x100000 + 2) == EINVAL         # dD misaligned
    assert bwd(du=U + 0x100000, ws=U + 0x100000 - 256) == EINVAL   # workspace overlaps du


def heads(x=U, B=2, L=64, d=128, dh=2, m_s=64, dt=2, out=Y, ws=W, wsb=1 << 28, diag=K + 65536):
    return h3.lib().h3_layer_fwd_heads(P(x), P(K), P(K), P(K), P(K), P(K), None, P(diag), None,
                                       B, L, d, dh, m_s, dt, P(out), P(ws), wsb, None)


def test_layer_heads_validation():
    assert heads(x=0) == EINVAL
    assert heads(dh=3) == EUNSUP
    assert heads(dh=16) == EUNSUP
    assert heads(L=32) == EUNSUP                     # heads need L >= 64
    assert heads(dt=1, d=100) == EUNSUP
    assert heads(ws=0) == EWS
    assert heads(wsb=h3.workspace_size(h3.OP_LAYER_HEADS, 2, 128, 64, 64, 2, h3.BF16) - 1) == EWS
    assert heads(out=U) == EINVAL
    assert h3.workspace_size(h3.OP_LAYER_HEADS, 4, 2560, 2048, 64, 8, h3.BF16) > 4 * 2560 * 2048 * 2 * 16
    assert h3.workspace_size(h3.OP_LAYER_HEADS, 4, 2560, 2048, 64, 3, h3.BF16) == 0
    assert (h3.workspace_size(h3.OP_LAYER_HEADS, 4, 2560, 2048, 64, 1, h3.BF16)
            == h3.workspace_size(h3.OP_LAYER, 4, 2560, 2048, 64, 0, h3.BF16))


def test_binding_rejects_host_tensors():
    """The binding refuses CPU tensors before reaching the library (no GPU
    needed: nothing is launched)."""
    import torch
    u = torch.zeros((2, 3, 64), dtype=torch.float16)
    k = torch.zeros((3, 64))
    with pytest.raises(ValueError):
        h3.fftconv(u, k)
    with pytest.raises(ValueError):
        h3.kernel_spectrum(k)
    P = torch.zeros((3, 8, 2))
    with pytest.raises(ValueError):
        h3.statepass_conv(u, P, P, P, None, 16)
    with pytest.raises(ValueError):
        h3.ssm_step(u[..., 0], P, P, P, None, torch.zeros((2, 3, 8, 2)))
    x = torch.zeros((2, 128, 128), dtype=torch.bfloat16)
    W = torch.zeros((128, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        h3.layer_fwd(x, W, W, W, W, torch.zeros((128, 4)), None, torch.zeros((128, 128)), None)


def test_statepass_noalloc_validation():
    """The no-allocation variant validates like h3_statepass_conv and rejects
    a call whose scratch would exceed its static array, before touching the
    GPU."""
    L = h3.lib()

    def call(u=U, A=K, B=2, H=4, Ln=256, m=64, chunk=64, dt=1, y=Y, xf=None):
        return L.h3_statepass_conv_noalloc(P(u), P(A), P(K + 4096), P(K + 8192), None, None, B, H, Ln, m, chunk,
                                           dt, P(y), P(xf), None)

    assert call(u=0) == EINVAL
    assert call(Ln=250) == EINVAL
    assert call(m=65) == EUNSUP
    assert call(y=U) == EINVAL
    # float32, chunk 1024 at B=2 H=1024 L=131072: a 1 GiB correction term
    assert h3.workspace_size(h3.OP_STATEPASS, 2, 1024, 131072, 64, 1024, h3.F32) > (128 << 20)
    assert call(u=1 << 40, y=2 << 40, B=2, H=1024, Ln=131072, chunk=1024, dt=0) == EWS
