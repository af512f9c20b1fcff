/*
 * h3flash: MI355X (gfx950) FlashConv hot path of "Hungry Hungry Hippos"
 * (Fu, Dao et al., arXiv 2212.14052).  C ABI of libh3flash.so.
 *
 * General conventions
 *  - Every tensor pointer is a DEVICE pointer owned by the caller.  Scratch
 *    space is passed in as `workspace` (size it with h3_workspace_size) and
 *    must not alias any other argument.  The library allocates no device
 *    memory (h3_statepass_conv_noalloc uses a static device array instead of
 *    a workspace).
 *  - Complex values are interleaved (re, im) float32 pairs.
 *  - Tensors are dense, row-major, with the last dimension contiguous.
 *    Sequence tensors are (B, H, L): row (b, h) is L contiguous elements.
 *  - 16-bit I/O (H3_F16, H3_BF16) is read and written as IEEE half / bfloat16;
 *    all arithmetic is float32 (matrix-core operands may be rounded to 16 bit,
 *    accumulation is float32).  Stores round to nearest, ties to even.
 *  - `stream` is a hipStream_t (NULL = the legacy default stream).  Every call
 *    validates its arguments on the host, enqueues its kernels on `stream` and
 *    returns without synchronising.  On a validation error nothing is launched.
 *  - NaN and Inf in the inputs propagate to the outputs; they are not masked.
 *  - Return value: H3_OK (0) or a negative h3_status.  No C++ exception crosses
 *    this boundary.
 *  - The library keeps no state between calls apart from values looked up
 *    once and cached (a kernel's resident workgroups per CU; the device
 *    address of h3_statepass_conv_noalloc's array, per device).  Every entry
 *    point may be called from several host threads.
 */
#ifndef H3FLASH_H
#define H3FLASH_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    H3_OK = 0,
    H3_EINVAL = -1,        /* null pointer, bad size, misaligned or aliased buffers    */
    H3_EUNSUPPORTED = -2,  /* length / chunk / mode count / dtype outside what is built */
    H3_EWORKSPACE = -3,    /* workspace missing or smaller than h3_workspace_size       */
    H3_EDEVICE = -4        /* a kernel launch failed (hipGetLastError after launching)  */
} h3_status;

typedef enum { H3_F32 = 0, H3_F16 = 1, H3_BF16 = 2 } h3_dtype;

/* Operation codes for h3_workspace_size. */
enum { H3_OP_FFTCONV = 1, H3_OP_STATEPASS = 2, H3_OP_LAYER = 3, H3_OP_FFTCONV_BWD = 4, H3_OP_LAYER_HEADS = 5 };

/* Limits of this build. */
#define H3_MAX_MODES 64     /* m: complex modes per channel of a diagonal SSM      */
#define H3_MIN_LEN 16       /* smallest fused convolution length (and chunk)       */
#define H3_FUSED_LIMIT 16384     /* longest fused convolution length (and chunk), 16-bit I/O */
#define H3_FUSED_LIMIT_F32 8192  /* the same for float32 I/O, the spectral entry points and
                                    the kernel gradient of h3_fftconv_bwd                    */
#define H3_MAX_SHIFT 64     /* longest shift-SSM filter in h3_layer_fwd            */

/*
 * h3_ssm_discretize — zero-order-hold discretisation of H diagonal SSMs of m
 * complex modes (the continuous SSM x' = Ax + Bu of Sec. 2.1, diagonal A as in
 * Sec. 3.2):  Abar = exp(dt_h A),  Bbar = (exp(dt_h A) - 1) / A * B.
 *   A, B       (H, m) complex, read.     dt (H) float32 > 0, read.
 *   Abar, Bbar (H, m) complex, written.  Computed in float64, stored float32.
 * Errors: EINVAL (null, H < 1, m < 1), EUNSUPPORTED (m > H3_MAX_MODES).
 */
int h3_ssm_discretize(const float *A, const float *B, const float *dt, int H, int m,
                      float *Abar, float *Bbar, void *stream);

/*
 * h3_ssm_kernel — the SSM convolution kernel f = [CB, CAB, CA^2B, ...] of
 * Sec. 2.1 for a diagonal SSM, from continuous parameters and step dt:
 *   k[h, t] = 2 Re sum_{n<m} C[h,n] Bbar[h,n] exp(t dt_h A[h,n]),  t < L,
 * with Bbar the ZOH input matrix above.  Each complex mode stands for a
 * conjugate pair (hence 2 Re), so k is the impulse response of the recurrence
 * y_t = 2 Re(C x_t) + D u_t.  Phases t*dt*Im(A) are reduced in float64.
 *   A, B, C (H, m) complex; dt (H); k (H, L) float32, written.
 * Errors: EINVAL (null, H, m or L < 1), EUNSUPPORTED (m > H3_MAX_MODES).
 */
int h3_ssm_kernel(const float *A, const float *B, const float *C, const float *dt,
                  int H, int m, int L, float *k, void *stream);

/*
 * h3_fftconv — fused FFT convolution (Sec. 4.1; the convolution of Sec. 2.1):
 *   y[b,h,:] = irfft(rfft(u[b,h,:], 2L) * rfft(k[h,:], 2L))[:L] + D[h] u[b,h,:]
 * i.e. the causal linear convolution y_t = sum_{j<=t} k[h,j] u[b,h,t-j] + D u_t.
 *   u, y  (B, H, L) of `dtype`; must not overlap.
 *   k     (H, L) float32.   D (H) float32, or NULL for no skip term.
 *   L     power of two in [H3_MIN_LEN, H3_FUSED_LIMIT].
 *   workspace >= h3_workspace_size(H3_OP_FFTCONV, B, H, L, 0, 0, dtype) bytes
 *   (holds the kernel spectra, H * (L + 1) complex).
 * Errors: EINVAL, EUNSUPPORTED (L, dtype), EWORKSPACE, EDEVICE.
 */
int h3_fftconv(const void *u, const float *k, const float *D, void *y,
               int B, int H, int L, int dtype,
               void *workspace, size_t ws_bytes, void *stream);

/*
 * h3_kernel_spectrum — the kernel half of the fused convolution, split out so a
 * spectrum can be reused across calls that share k (e.g. every batch row, or
 * repeated inputs):  Kspec[h, f] = (1/2L) sum_{t<L} k[h,t] exp(-2 pi i f t / 2L),
 * f = 0..L (the non-redundant half of the length-2L DFT of the zero-padded
 * kernel, with the inverse transform's 1/2L folded in).
 *   k (H, L) float32.  Kspec (H, L+1) complex, written.
 *   L power of two in [H3_MIN_LEN, H3_FUSED_LIMIT_F32].
 * Errors: EINVAL, EUNSUPPORTED (L), EDEVICE.
 */
int h3_kernel_spectrum(const float *k, int H, int L, float *Kspec, void *stream);

/*
 * h3_fftconv_spectral — the fused convolution of h3_fftconv given the kernel
 * spectrum from h3_kernel_spectrum (no workspace needed).
 *   u, y (B, H, L) of `dtype`, not overlapping.  Kspec (H, L+1) complex.
 *   D (H) float32 or NULL.  L as for h3_kernel_spectrum (the float32-VALU
 *   convolution runs, for every dtype).
 * Errors: EINVAL, EUNSUPPORTED (L, dtype), EDEVICE.
 */
int h3_fftconv_spectral(const void *u, const float *Kspec, const float *D, void *y,
                        int B, int H, int L, int dtype, void *stream);

/*
 * h3_statepass_conv — state passing (Sec. 4.2, Algorithm 2) for a diagonal
 * SSM given in discrete form, over sequences longer than the fused limit:
 * the sequence is cut into L/chunk chunks; each chunk is a fused FFT
 * convolution with the length-`chunk` kernel plus the contribution of the
 * state carried in, and the state is advanced chunk to chunk.  The result is
 * that of the recurrence (Proposition 2):
 *   x_t = Abar x_{t-1} + Bbar u_t (per mode),  y_t = 2 Re(C . x_t) + D u_t,
 *   x_{-1} = x0,  x_final = x_{L-1}.
 *   u, y        (B, H, L) of `dtype`; must not overlap.
 *   Abar, Bbar, C (H, m) complex.  D (H) float32 (NULL: no skip term).
 *   x0          (B, H, m) complex, or NULL for the zero state.
 *   x_final     (B, H, m) complex written, or NULL.
 *   chunk       power of two in [H3_MIN_LEN, H3_FUSED_LIMIT] dividing L.
 *   workspace >= h3_workspace_size(H3_OP_STATEPASS, B, H, L, m, chunk, dtype)
 *   (the chunk kernel, the chunk end-states and the initial-state term's
 *   inputs; its contents on entry do not matter).
 * Errors: EINVAL (null, sizes, L % chunk), EUNSUPPORTED (chunk, m, dtype),
 *         EWORKSPACE, EDEVICE.
 */
int h3_statepass_conv(const void *u, const float *Abar, const float *Bbar,
                      const float *C, const float *D, const float *x0,
                      int B, int H, int L, int m, int chunk, int dtype,
                      void *y, float *x_final,
                      void *workspace, size_t ws_bytes, void *stream);

/*
 * h3_statepass_conv_noalloc — h3_statepass_conv without a workspace argument,
 * for callers that cannot allocate device memory (code under graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  Arguments, result
 * and errors as for h3_statepass_conv; it calls no allocating routine.  The
 * scratch lives in a static device array of H3_NOALLOC_SCRATCH_BYTES per GPU,
 * held from the library's first use on that GPU until the process ends;
 * `stream` must belong to the current device.  Calls on one GPU share that
 * array: calls that overlap in time on one GPU race (serialise them, e.g. on
 * one stream).  Every scratch region is written before it is read, so the
 * previous call's contents do not matter.
 * Errors: as h3_statepass_conv; EWORKSPACE when the scratch this call needs
 * (h3_workspace_size(H3_OP_STATEPASS, ...)) exceeds H3_NOALLOC_SCRATCH_BYTES;
 * EDEVICE if the array's device address cannot be looked up.
 */
#define H3_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
int h3_statepass_conv_noalloc(const void *u, const float *Abar, const float *Bbar,
                              const float *C, const float *D, const float *x0,
                              int B, int H, int L, int m, int chunk, int dtype,
                              void *y, float *x_final, void *stream);

/*
 * h3_fftconv_bwd — backward pass of the fused convolution (the appendix on
 * FlashConv's backward pass): for y = h3_fftconv(u, k, D) and an output
 * gradient dy,
 *   du[b,h,t] = sum_{s>=t} k[h,s-t] dy[b,h,s] + D[h] dy[b,h,t]
 *               (the same fused kernel with the conjugated kernel spectrum),
 *   dk[h,j]   = sum_b sum_{t>=j} dy[b,h,t] u[b,h,t-j]
 *               (Re IFFT of sum_b conj(F u_b) . F dy_b, one transform pair per
 *               row pair and one inverse per channel),
 *   dD[h]     = sum_{b,t} dy[b,h,t] u[b,h,t].
 *   u, dy, du   (B, H, L) of `dtype`; u may be NULL when only du is asked.
 *   k (H, L) float32; D (H) float32 or NULL (then du has no skip term).
 *   dk (H, L) float32, dD (H) float32.  Each of du, dk, dD may be NULL (not
 *   computed), not all three.  Outputs overlap no input, output or the
 *   workspace.  L as for h3_fftconv.
 *   workspace >= h3_workspace_size(H3_OP_FFTCONV_BWD, B, H, L, 0, 0, dtype).
 * Errors: EINVAL, EUNSUPPORTED (L, dtype), EWORKSPACE, EDEVICE.
 */
int h3_fftconv_bwd(const void *u, const float *k, const float *D, const void *dy,
                   int B, int H, int L, int dtype, void *du, float *dk, float *dD,
                   void *workspace, size_t ws_bytes, void *stream);

/*
 * h3_ssm_step — recurrent (step) mode of a diagonal SSM, for generation
 * (Sec. 2, the recurrent view; Sec. 5 generation): advances the carried state
 * over T new tokens per (b, h) row,
 *   x_n <- Abar_n x_n + Bbar_n u_t,   y_t = 2 Re(C . x) + D u_t,  t = 0..T-1,
 * which is the recurrence whose impulse response is k, so a state written by
 * h3_statepass_conv (x_final) continues that sequence.
 *   u, y        (B, H, T) of `dtype` (T = 1: one token per row); must not
 *               overlap each other or the state.
 *   Abar, Bbar, C (H, m) complex (e.g. from h3_ssm_discretize).  D (H)
 *               float32 or NULL.
 *   x           (B, H, m) complex, read and overwritten with the state after
 *               the last token (the caller owns it between calls).
 *   m in [1, H3_MAX_MODES].  Arithmetic in float32.  Pointers aligned to
 *   their element size (8 bytes for complex).
 * Errors: EINVAL (null, sizes, alignment, overlap), EUNSUPPORTED (m, dtype),
 *         EDEVICE.
 */
int h3_ssm_step(const void *u, const float *Abar, const float *Bbar, const float *C,
                const float *D, int B, int H, int m, int T, int dtype,
                float *x, void *y, void *stream);

/*
 * h3_layer_fwd — H3 layer forward with head dimension 1 (Sec. 3.2,
 * Algorithm 1):
 *   Q = x Wq, K = x Wk, V = x Wv           (Q[b,t,c] = sum_j x[b,t,j] Wq[j,c])
 *   Kbar = SSM_shift(K): Kbar_t = sum_{j<m_s} shift_C[c,j] K_{t-j} + shift_D[c] K_t
 *   G = Kbar * V;  S = SSM_diag(G) = diag_k[c] (*) G + diag_D[c] G   (causal conv)
 *   out = (Q * S) Wo
 *   x, out   (B, L, d) of `dtype` (H3_F16 or H3_BF16); must not overlap.
 *   Wq, Wk, Wv, Wo  (d, d) of `dtype`, row-major as Algorithm 1 writes the
 *   projections (rows index the input features, columns the output
 *   features).  Must not overlap out or the workspace.
 *   shift_C  (d, m_s) float32, m_s in [1, H3_MAX_SHIFT].  shift_D (d) or NULL.
 *   diag_k   (d, L) float32 (e.g. from h3_ssm_kernel).  diag_D (d) or NULL.
 *   L power of two in [H3_MIN_LEN, H3_FUSED_LIMIT]; d a multiple of 128;
 *   B * L a multiple of 128 (the tiles of the library's own GEMM).
 *   workspace >= h3_workspace_size(H3_OP_LAYER, B, d, L, m_s, 0, dtype).
 * The four projections run on the library's own matrix-core GEMM: when d is
 * a multiple of 320 (or 256) and B * L of 256 it reads the weights as stored,
 * Q, K and V in one launch of 320 x 256 (256 x 256) tiles; other shapes take
 * one 128 x 128-tile launch per projection on transposed copies of the
 * weights made in the workspace.
 * Errors: EINVAL, EUNSUPPORTED (L, d, B * L, m_s, dtype), EWORKSPACE, EDEVICE.
 */
int h3_layer_fwd(const void *x, const void *Wq, const void *Wk, const void *Wv,
                 const void *Wo, const float *shift_C, const float *shift_D,
                 const float *diag_k, const float *diag_D,
                 int B, int L, int d, int m_s, int dtype, void *out,
                 void *workspace, size_t ws_bytes, void *stream);

/*
 * h3_layer_fwd_heads — H3 layer forward with heads of dimension d_head
 * (Sec. 3.2, Algorithm 1; pure H3 uses d_head = 8): Q, K, V, Kbar as for
 * h3_layer_fwd; per head h (channels h d_head .. h d_head + d_head - 1) and
 * token t the outer product KV_t[i][j] = Kbar_t[h d_head + i] V_t[h d_head + j]
 * passes through the diagonal SSM of channel c = (h d_head + i) d_head + j,
 *   S[c] = diag_k[c] (*) KV[i][j] + diag_D[c] KV[i][j]   (causal conv),
 * the head's output is O_t[h d_head + j] = sum_i Q_t[h d_head + i] S_t[c], and
 * out = O Wo^T.
 *   Arguments as for h3_layer_fwd, except diag_k (d d_head, L) float32 and
 *   diag_D (d d_head) or NULL.  d_head in {1, 2, 4, 8} (1 is h3_layer_fwd);
 *   for d_head > 1, L is a power of two in [64, H3_FUSED_LIMIT].  d and B * L
 *   multiples of 128 as for h3_layer_fwd.
 *   workspace >= h3_workspace_size(H3_OP_LAYER_HEADS, B, d, L, m_s, d_head, dtype).
 * Errors: EINVAL, EUNSUPPORTED (L, d, d_head, m_s, dtype), EWORKSPACE, EDEVICE.
 */
int h3_layer_fwd_heads(const void *x, const void *Wq, const void *Wk, const void *Wv,
                       const void *Wo, const float *shift_C, const float *shift_D,
                       const float *diag_k, const float *diag_D,
                       int B, int L, int d, int d_head, int m_s, int dtype, void *out,
                       void *workspace, size_t ws_bytes, void *stream);

/*
 * h3_workspace_size — bytes of workspace an operation needs (0 if the
 * arguments are invalid).  H_or_d is H for the convolutions, d for the layer;
 * m is the mode count (state passing) or the shift length (layer); chunk is
 * the chunk length (state passing) or the head dimension (H3_OP_LAYER_HEADS).
 */
size_t h3_workspace_size(int op, int B, int H_or_d, int L, int m, int chunk, int dtype);

/* Human-readable name of a status code (static string). */
const char *h3_status_string(int status);

#ifdef __cplusplus
}
#endif
#endif /* H3FLASH_H */
