"""MI355X-native FlashConv hot path of "Hungry Hungry Hippos" (arXiv 2212.14052).

Thin Python binding over the C ABI of ``libh3flash.so`` (declared in
``include/h3flash.h``).  Every function here only marshals arguments: tensors
are PyTorch device tensors (PyTorch supplies device memory and the stream),
and all arithmetic runs in the library's HIP kernels.  There is no fallback:
if the library is missing, importing the ops raises.

Complex parameters are accepted either as complex64 tensors or as float32
tensors with a trailing dimension of 2 (re, im).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

__all__ = [
    "H3Error", "lib", "ssm_discretize", "ssm_kernel", "fftconv", "statepass_conv",
    "statepass_conv_noalloc", "layer_fwd", "layer_fwd_heads", "ssm_step", "fftconv_bwd", "kernel_spectrum", "fftconv_spectral", "workspace_size", "status_string", "F32", "F16", "BF16",
    "OP_FFTCONV", "OP_STATEPASS", "OP_LAYER", "OP_FFTCONV_BWD", "OP_LAYER_HEADS", "FUSED_LIMIT", "FUSED_LIMIT_F32", "MAX_MODES",
]

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libh3flash.so")

F32, F16, BF16 = 0, 1, 2
OP_FFTCONV, OP_STATEPASS, OP_LAYER, OP_FFTCONV_BWD, OP_LAYER_HEADS = 1, 2, 3, 4, 5
FUSED_LIMIT = 16384       # 16-bit I/O
FUSED_LIMIT_F32 = 8192    # float32 I/O, spectral entry points, kernel gradient
MAX_MODES = 64

_DTYPES = {torch.float32: F32, torch.float16: F16, torch.bfloat16: BF16}

_lib = None


class H3Error(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: {status_string(status)} (status {status})")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libh3flash.so (built by ``paper_2212_14052_amd.build``)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2212_14052_amd.build` "
                "(there is no non-HIP fallback)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        L.h3_ssm_discretize.argtypes = [vp, vp, vp, i, i, vp, vp, vp]
        L.h3_ssm_kernel.argtypes = [vp, vp, vp, vp, i, i, i, vp, vp]
        L.h3_fftconv.argtypes = [vp, vp, vp, vp, i, i, i, i, vp, sz, vp]
        L.h3_kernel_spectrum.argtypes = [vp, i, i, vp, vp]
        L.h3_fftconv_spectral.argtypes = [vp, vp, vp, vp, i, i, i, i, vp]
        L.h3_statepass_conv.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, vp, vp, vp, sz, vp]
        L.h3_statepass_conv_noalloc.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, vp, vp, vp]
        L.h3_layer_fwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, vp, vp, sz, vp]
        L.h3_ssm_step.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, vp, vp, vp]
        L.h3_fftconv_bwd.argtypes = [vp, vp, vp, vp, i, i, i, i, vp, vp, vp, vp, sz, vp]
        L.h3_layer_fwd_heads.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, vp, vp, sz, vp]
        L.h3_workspace_size.argtypes = [i, i, i, i, i, i, i]
        L.h3_workspace_size.restype = sz
        L.h3_status_string.argtypes = [i]
        L.h3_status_string.restype = ctypes.c_char_p
        for fn in ("h3_ssm_discretize", "h3_ssm_kernel", "h3_fftconv", "h3_statepass_conv", "h3_statepass_conv_noalloc",
                   "h3_layer_fwd", "h3_kernel_spectrum", "h3_fftconv_spectral", "h3_ssm_step", "h3_fftconv_bwd",
                   "h3_layer_fwd_heads"):
            getattr(L, fn).restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().h3_status_string(int(status)).decode()


def workspace_size(op: int, B: int, H_or_d: int, L: int, m: int = 0, chunk: int = 0,
                   dtype: int = F32) -> int:
    return int(lib().h3_workspace_size(op, B, H_or_d, L, m, chunk, dtype))


# ------------------------------------------------------------- helpers -----
def _ptr(t: Optional[torch.Tensor]):
    # a plain int: the c_void_p argtypes convert it
    return None if t is None else t.data_ptr()


_raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None)


def _stream(dev: torch.device):
    """The current HIP stream of `dev` as an int (the raw-stream accessor is
    the cheap path: this runs on every call)."""
    idx = dev.index if dev.index is not None else torch.cuda.current_device()
    if _raw_stream is not None:
        return _raw_stream(idx)
    return torch.cuda.current_stream(idx).cuda_stream


def _check(fn: str, status: int):
    if status != 0:
        raise H3Error(fn, status)


def _cplx(t: torch.Tensor) -> torch.Tensor:
    """complex64 or (..., 2) float32 -> contiguous (..., 2) float32."""
    if t.is_complex():
        t = torch.view_as_real(t.to(torch.complex64).contiguous())
    if t.dtype != torch.float32 or t.shape[-1] != 2:
        raise ValueError("complex parameters must be complex64 or float32 (..., 2)")
    return t.contiguous()


def _f32(t: Optional[torch.Tensor]) -> Optional[torch.Tensor]:
    if t is None:
        return None
    return t.to(torch.float32).contiguous()


def _dtype(t: torch.Tensor) -> int:
    if t.dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {t.dtype}")
    return _DTYPES[t.dtype]


def _workspace(nbytes: int, dev: torch.device, workspace: Optional[torch.Tensor]) -> torch.Tensor:
    if workspace is not None:
        _on(dev, workspace=workspace)
        if not workspace.is_contiguous():
            raise ValueError("workspace must be contiguous")
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError("workspace too small")
        return workspace
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=dev)


# ----------------------------------------------------------- validation ----
# The C ABI receives bare pointers and cannot see sizes, devices or strides:
# every tensor is checked here before anything is launched.
def _gpu(name: str, t: torch.Tensor) -> torch.device:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device})")
    return t.device


def _on(dev: torch.device, **ts):
    for name, t in ts.items():
        if t is None:
            continue
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch.Tensor")
        if t.device != dev:
            raise ValueError(f"{name} must be on {dev} (got {t.device})")


def _shape(name: str, t: Optional[torch.Tensor], shape):
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")


def _out(name: str, t: Optional[torch.Tensor], shape, dtype, dev):
    """A caller-supplied output: exact shape, dtype, device, contiguous."""
    if t is None:
        return
    _on(dev, **{name: t})
    _shape(name, t, shape)
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


# ----------------------------------------------------------------- ops -----
def ssm_discretize(A: torch.Tensor, B: torch.Tensor, dt: torch.Tensor):
    """ZOH: Abar = exp(dt A), Bbar = (exp(dt A) - 1)/A * B.  Returns (Abar, Bbar)
    as float32 (H, m, 2)."""
    dev = _gpu("A", A)
    A, B, dt = _cplx(A), _cplx(B), _f32(dt)
    _on(dev, B=B, dt=dt)
    H, m = A.shape[0], A.shape[1]
    _shape("A", A, (H, m, 2)); _shape("B", B, (H, m, 2)); _shape("dt", dt, (H,))
    Ab = torch.empty_like(A); Bb = torch.empty_like(A)
    _check("h3_ssm_discretize", lib().h3_ssm_discretize(
        _ptr(A), _ptr(B), _ptr(dt), H, m, _ptr(Ab), _ptr(Bb), _stream(A.device)))
    return Ab, Bb


def ssm_kernel(A: torch.Tensor, B: torch.Tensor, C: torch.Tensor, dt: torch.Tensor, L: int,
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """k[h, t] = 2 Re sum_n C Bbar exp(t dt A), (H, L) float32."""
    dev = _gpu("A", A)
    A, B, C, dt = _cplx(A), _cplx(B), _cplx(C), _f32(dt)
    _on(dev, B=B, C=C, dt=dt)
    H, m = A.shape[0], A.shape[1]
    for n, t in (("A", A), ("B", B), ("C", C)):
        _shape(n, t, (H, m, 2))
    _shape("dt", dt, (H,))
    _out("out", out, (H, L), torch.float32, dev)
    k = out if out is not None else torch.empty((H, L), dtype=torch.float32, device=A.device)
    _check("h3_ssm_kernel", lib().h3_ssm_kernel(
        _ptr(A), _ptr(B), _ptr(C), _ptr(dt), H, m, L, _ptr(k), _stream(A.device)))
    return k


def fftconv(u: torch.Tensor, k: torch.Tensor, D: Optional[torch.Tensor] = None,
            out: Optional[torch.Tensor] = None,
            workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """y = causal_conv(u, k) + D u over (B, H, L) rows, fused FFT."""
    dev = _gpu("u", u)
    u = u.contiguous()
    if u.dim() != 3:
        raise ValueError("u must be (B, H, L)")
    Bn, H, L = u.shape
    k, D = _f32(k), _f32(D)
    dt = _dtype(u)
    _on(dev, k=k, D=D)
    _shape("k", k, (H, L)); _shape("D", D, (H,))
    _out("out", out, u.shape, u.dtype, dev)
    y = out if out is not None else torch.empty_like(u)
    ws = _workspace(workspace_size(OP_FFTCONV, Bn, H, L, 0, 0, dt), u.device, workspace)
    _check("h3_fftconv", lib().h3_fftconv(
        _ptr(u), _ptr(k), _ptr(D), _ptr(y), Bn, H, L, dt, _ptr(ws),
        ws.numel() * ws.element_size(), _stream(u.device)))
    return y


def kernel_spectrum(k: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Kspec[h, f] = DFT_{2L}(k[h] zero-padded)[f] / 2L for f = 0..L; returns
    float32 (H, L+1, 2)."""
    dev = _gpu("k", k)
    k = _f32(k)
    if k.dim() != 2:
        raise ValueError("k must be (H, L)")
    H, L = k.shape
    _out("out", out, (H, L + 1, 2), torch.float32, dev)
    K = out if out is not None else torch.empty((H, L + 1, 2), dtype=torch.float32, device=k.device)
    _check("h3_kernel_spectrum", lib().h3_kernel_spectrum(_ptr(k), H, L, _ptr(K), _stream(k.device)))
    return K


def fftconv_spectral(u: torch.Tensor, Kspec: torch.Tensor, D: Optional[torch.Tensor] = None,
                     out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Fused convolution given the kernel spectrum from kernel_spectrum."""
    dev = _gpu("u", u)
    u = u.contiguous()
    if u.dim() != 3:
        raise ValueError("u must be (B, H, L)")
    Bn, H, L = u.shape
    D = _f32(D)
    Kspec = _cplx(Kspec)
    _on(dev, Kspec=Kspec, D=D)
    _shape("Kspec", Kspec, (H, L + 1, 2)); _shape("D", D, (H,))
    _out("out", out, u.shape, u.dtype, dev)
    y = out if out is not None else torch.empty_like(u)
    _check("h3_fftconv_spectral", lib().h3_fftconv_spectral(
        _ptr(u), _ptr(Kspec), _ptr(D), _ptr(y), Bn, H, L, _dtype(u), _stream(u.device)))
    return y


def statepass_conv(u: torch.Tensor, Abar: torch.Tensor, Bbar: torch.Tensor, C: torch.Tensor,
                   D: Optional[torch.Tensor], chunk: int, x0: Optional[torch.Tensor] = None,
                   out: Optional[torch.Tensor] = None,
                   workspace: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """State passing (Algorithm 2) for the diagonal SSM (Abar, Bbar, C, D).
    Returns (y, x_final) with x_final float32 (B, H, m, 2)."""
    dev = _gpu("u", u)
    u = u.contiguous()
    if u.dim() != 3:
        raise ValueError("u must be (B, H, L)")
    Bn, H, L = u.shape
    Abar, Bbar, C, D = _cplx(Abar), _cplx(Bbar), _cplx(C), _f32(D)
    m = Abar.shape[1]
    x0 = _cplx(x0) if x0 is not None else None
    _on(dev, Abar=Abar, Bbar=Bbar, C=C, D=D, x0=x0)
    for n, t in (("Abar", Abar), ("Bbar", Bbar), ("C", C)):
        _shape(n, t, (H, m, 2))
    _shape("D", D, (H,)); _shape("x0", x0, (Bn, H, m, 2))
    dt = _dtype(u)
    _out("out", out, u.shape, u.dtype, dev)
    y = out if out is not None else torch.empty_like(u)
    xf = torch.empty((Bn, H, m, 2), dtype=torch.float32, device=u.device)
    ws = _workspace(workspace_size(OP_STATEPASS, Bn, H, L, m, chunk, dt), u.device, workspace)
    _check("h3_statepass_conv", lib().h3_statepass_conv(
        _ptr(u), _ptr(Abar), _ptr(Bbar), _ptr(C), _ptr(D), _ptr(x0), Bn, H, L, m, chunk, dt,
        _ptr(y), _ptr(xf), _ptr(ws), ws.numel() * ws.element_size(), _stream(u.device)))
    return y, xf


def statepass_conv_noalloc(u: torch.Tensor, Abar: torch.Tensor, Bbar: torch.Tensor, C: torch.Tensor,
                           D: Optional[torch.Tensor], chunk: int, x0: Optional[torch.Tensor] = None,
                           out: Optional[torch.Tensor] = None,
                           x_final: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """statepass_conv through h3_statepass_conv_noalloc: the library's static
    scratch instead of a workspace (the library allocates nothing; the outputs
    are allocated here unless given)."""
    dev = _gpu("u", u)
    u = u.contiguous()
    if u.dim() != 3:
        raise ValueError("u must be (B, H, L)")
    Bn, H, L = u.shape
    Abar, Bbar, C, D = _cplx(Abar), _cplx(Bbar), _cplx(C), _f32(D)
    m = Abar.shape[1]
    x0 = _cplx(x0) if x0 is not None else None
    _on(dev, Abar=Abar, Bbar=Bbar, C=C, D=D, x0=x0)
    for n, t in (("Abar", Abar), ("Bbar", Bbar), ("C", C)):
        _shape(n, t, (H, m, 2))
    _shape("D", D, (H,)); _shape("x0", x0, (Bn, H, m, 2))
    _out("out", out, u.shape, u.dtype, dev)
    _out("x_final", x_final, (Bn, H, m, 2), torch.float32, dev)
    y = out if out is not None else torch.empty_like(u)
    xf = x_final if x_final is not None else torch.empty((Bn, H, m, 2), dtype=torch.float32, device=u.device)
    _check("h3_statepass_conv_noalloc", lib().h3_statepass_conv_noalloc(
        _ptr(u), _ptr(Abar), _ptr(Bbar), _ptr(C), _ptr(D), _ptr(x0), Bn, H, L, m, chunk, _dtype(u),
        _ptr(y), _ptr(xf), _stream(u.device)))
    return y, xf


def fftconv_bwd(u: Optional[torch.Tensor], k: torch.Tensor, D: Optional[torch.Tensor], dy: torch.Tensor,
                want_du: bool = True, want_dk: bool = True, want_dD: bool = True,
                workspace: Optional[torch.Tensor] = None):
    """Backward pass of fftconv for output gradient dy (B, H, L).  Returns
    (du, dk, dD); an output not asked for is None."""
    dev = _gpu("dy", dy)
    dy = dy.contiguous()
    if dy.dim() != 3:
        raise ValueError("dy must be (B, H, L)")
    Bn, H, L = dy.shape
    dt = _dtype(dy)
    if u is not None:
        _on(dev, u=u)
        u = u.contiguous()
        if u.shape != dy.shape or u.dtype != dy.dtype:
            raise ValueError("u must match dy in shape and dtype")
    k, D = _f32(k), _f32(D)
    _on(dev, k=k, D=D)
    _shape("k", k, (H, L)); _shape("D", D, (H,))
    du = torch.empty_like(dy) if want_du else None
    dk = torch.empty((H, L), dtype=torch.float32, device=dy.device) if want_dk else None
    dD = torch.empty((H,), dtype=torch.float32, device=dy.device) if want_dD else None
    ws = _workspace(workspace_size(OP_FFTCONV_BWD, Bn, H, L, 0, 0, dt), dy.device, workspace)
    _check("h3_fftconv_bwd", lib().h3_fftconv_bwd(
        _ptr(u), _ptr(k), _ptr(D), _ptr(dy), Bn, H, L, dt, _ptr(du), _ptr(dk), _ptr(dD), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(dy.device)))
    return du, dk, dD


def _layer_args(x, Wq, Wk, Wv, Wo, shift_C, shift_D, diag_k, diag_D, d_head):
    dev = _gpu("x", x)
    x = x.contiguous()
    if x.dim() != 3:
        raise ValueError("x must be (B, L, d)")
    Bn, L, d = x.shape
    dt = _dtype(x)
    _on(dev, Wq=Wq, Wk=Wk, Wv=Wv, Wo=Wo)
    Ws = [w.to(x.dtype).contiguous() for w in (Wq, Wk, Wv, Wo)]
    for n, w in zip(("Wq", "Wk", "Wv", "Wo"), Ws):
        _shape(n, w, (d, d))
    shift_C = _f32(shift_C)
    if shift_C.dim() != 2:
        raise ValueError("shift_C must be (d, m_s)")
    m_s = shift_C.shape[1]
    shift_D, diag_k, diag_D = _f32(shift_D), _f32(diag_k), _f32(diag_D)
    _on(dev, shift_C=shift_C, shift_D=shift_D, diag_k=diag_k, diag_D=diag_D)
    _shape("shift_C", shift_C, (d, m_s)); _shape("shift_D", shift_D, (d,))
    _shape("diag_k", diag_k, (d * d_head, L)); _shape("diag_D", diag_D, (d * d_head,))
    return Bn, L, d, dt, Ws, shift_C, m_s, shift_D, diag_k, diag_D, x


def layer_fwd_heads(x: torch.Tensor, Wq: torch.Tensor, Wk: torch.Tensor, Wv: torch.Tensor,
                    Wo: torch.Tensor, shift_C: torch.Tensor, shift_D: Optional[torch.Tensor],
                    diag_k: torch.Tensor, diag_D: Optional[torch.Tensor], d_head: int,
                    out: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """H3 layer forward with heads of dimension d_head (Algorithm 1).  x: (B, L, d);
    weights (d, d) with Q = x Wq; diag_k (d d_head, L), diag_D (d d_head)."""
    Bn, L, d, dt, Ws, shift_C, m_s, shift_D, diag_k, diag_D, x = _layer_args(
        x, Wq, Wk, Wv, Wo, shift_C, shift_D, diag_k, diag_D, d_head)
    _out("out", out, x.shape, x.dtype, x.device)
    o = out if out is not None else torch.empty_like(x)
    ws = _workspace(workspace_size(OP_LAYER_HEADS, Bn, d, L, m_s, d_head, dt), x.device, workspace)
    _check("h3_layer_fwd_heads", lib().h3_layer_fwd_heads(
        _ptr(x), *[_ptr(w) for w in Ws], _ptr(shift_C), _ptr(shift_D), _ptr(diag_k),
        _ptr(diag_D), Bn, L, d, d_head, m_s, dt, _ptr(o), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(x.device)))
    return o


def ssm_step(u: torch.Tensor, Abar: torch.Tensor, Bbar: torch.Tensor, C: torch.Tensor,
             D: Optional[torch.Tensor], x: torch.Tensor,
             out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Recurrent step mode: advance the state ``x`` (B, H, m, 2) float32, in
    place, over the tokens ``u`` (B, H) or (B, H, T); returns y shaped like u."""
    dev = _gpu("x", x)
    if x.dtype != torch.float32 or x.dim() != 4 or x.shape[-1] != 2 or not x.is_contiguous():
        raise ValueError("x must be a contiguous float32 (B, H, m, 2) tensor (it is updated in place)")
    Bn, H, m = x.shape[0], x.shape[1], x.shape[2]
    _on(dev, u=u)
    uu = u.contiguous()
    if uu.dim() == 2:
        uu = uu.unsqueeze(-1)
    if uu.dim() != 3 or uu.shape[0] != Bn or uu.shape[1] != H:
        raise ValueError("u must be (B, H) or (B, H, T) with the state's B and H")
    T = uu.shape[2]
    Abar, Bbar, C, D = _cplx(Abar), _cplx(Bbar), _cplx(C), _f32(D)
    _on(dev, Abar=Abar, Bbar=Bbar, C=C, D=D)
    for n, t in (("Abar", Abar), ("Bbar", Bbar), ("C", C)):
        _shape(n, t, (H, m, 2))
    _shape("D", D, (H,))
    _out("out", out, u.shape, uu.dtype, dev)
    y = out.view(uu.shape) if out is not None else torch.empty_like(uu)
    _check("h3_ssm_step", lib().h3_ssm_step(
        _ptr(uu), _ptr(Abar), _ptr(Bbar), _ptr(C), _ptr(D), Bn, H, m, T, _dtype(uu), _ptr(x), _ptr(y),
        _stream(x.device)))
    return y.view(u.shape)


def layer_fwd(x: torch.Tensor, Wq: torch.Tensor, Wk: torch.Tensor, Wv: torch.Tensor,
              Wo: torch.Tensor, shift_C: torch.Tensor, shift_D: Optional[torch.Tensor],
              diag_k: torch.Tensor, diag_D: Optional[torch.Tensor],
              out: Optional[torch.Tensor] = None,
              workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """H3 layer forward (Algorithm 1, head dimension 1).  x: (B, L, d); the
    weights are (d, d) as Algorithm 1 writes them: Q = x Wq."""
    Bn, L, d, dt, Ws, shift_C, m_s, shift_D, diag_k, diag_D, x = _layer_args(
        x, Wq, Wk, Wv, Wo, shift_C, shift_D, diag_k, diag_D, 1)
    _out("out", out, x.shape, x.dtype, x.device)
    o = out if out is not None else torch.empty_like(x)
    ws = _workspace(workspace_size(OP_LAYER, Bn, d, L, m_s, 0, dt), x.device, workspace)
    _check("h3_layer_fwd", lib().h3_layer_fwd(
        _ptr(x), *[_ptr(w) for w in Ws], _ptr(shift_C), _ptr(shift_D), _ptr(diag_k),
        _ptr(diag_D), Bn, L, d, m_s, dt, _ptr(o), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(x.device)))
    return o
