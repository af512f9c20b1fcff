// Internal launcher declarations of libh3flash (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>

#define H3_MAX_MODES_DEV 64

namespace h3 {

hipError_t launch_discretize(const float *A, const float *B, const float *dt, int H, int m,
                             float *Abar, float *Bbar, hipStream_t s);
// mode 0: P0 = A, P1 = B, dt used (continuous, ZOH).  mode 1: P0 = Abar, P1 = Bbar.
hipError_t launch_kernel_gen(int mode, const float *P0, const float *P1, const float *C,
                             const float *dt, int H, int m, int L, float *k, hipStream_t s);

// Recurrent step mode: T tokens per (b, h) row from the carried state x
// (B, H, m) complex, updated in place; u, y (B, H, T).
hipError_t launch_ssm_step(const void *u, const float *Abar, const float *Bbar, const float *C, const float *D,
                           int B, int H, int m, int T, int dtype, float *x, void *y, hipStream_t s);

// Kernel spectra: Kspec[h][f] = (1/N) sum_{t<L} k[h][t] exp(-2 pi i f t / N),
// f = 0..L, N = 2L.  Kspec: (H, L+1) float2.
hipError_t launch_spectrum(const float *k, int H, int L, float2 *Kspec, hipStream_t s);

// Fused FFT convolution over pairs of rows that share a channel.
//   pair_mode 0: rows (b, h) of a (B, H, L) tensor, pairs (2j, 2j+1) along b.
//   pair_mode 1: chunk rows of a (B, H, nchunk*L) tensor, pairs of
//                consecutive chunks of one (b, h) row; corr (optional) holds the
//                per-chunk initial-state correction inputs (see statepass).
struct ConvArgs {
    const void *u;
    void *y;
    const float2 *Kspec;   // (H, L+1)
    const float *D;        // (H) or null
    int B, H, L;           // L = convolution length (chunk length in mode 1)
    int nchunk;            // mode 1: chunks per row
    int pair_mode;
    int dtype;
    // state-passing initial-state term (mode 1 only, may be null):
    // (B, H, nchunk * L) added to the output; float32, or the I/O dtype if corr16
    const void *corr;
    int corr16;
    // fused initial-state term (mode 1, L = 8192 and 16384 convs): when corr_tab is
    // set, corr holds the normalised weights (B, H, nchunk, 64) fp16 complex
    // and corr_e their exponents (B, H, nchunk), as written by
    // launch_state_scan_w16, and corr_tab the per-channel tables written by
    // launch_corr_tables
    const uint4 *corr_tab;
    const int *corr_e;
    // conj_k: convolve with the conjugated kernel spectrum, i.e. correlate:
    // y[t] = sum_{s>=t} k[s-t] u[s] (+ D u[t]), the input gradient of the
    // convolution.  Supported by the wave kernels and the VALU kernel.
    int conj_k;
    // gate (mode 0, L = 2048 wave kernel only; may be null): y = gate * (the
    // convolution + D u), elementwise, gate in the I/O dtype and layout of y
    // (the output gating of the H3 layer, O = Q * S)
    const void *gate;
    // gen_C, gen_Bbar (the L = 8192 and 16384 convs with the fused state term;
    // may be null): the convolution kernel k_t = 2 Re sum_n C_n Bbar_n
    // Abar_n^t (the state-passing f of length L) is formed in the kernel
    // from them and the channel's power tables instead of read from k
    const float *gen_C, *gen_Bbar;
    int m_gen;   // their modes per channel (<= 64)
};
hipError_t launch_fftconv(const ConvArgs &a, hipStream_t s);
// The VALU convolution of plain (B, H, L) rows (pair_mode 0, no correction
// term) with each channel's spectrum computed in the kernel from k (skip term
// folded into k[0]); L a power of two in [16, 4096].
bool fftconv_kgen_supported(int L);
hipError_t launch_fftconv_kgen(const ConvArgs &a, const float *k, hipStream_t s);
// The eight-wave register-resident convolution at L = 16384 (16-bit I/O):
// plain rows or chunk pairs, with an optional correction term (float32, I/O
// dtype, or the fused state term from corr_tab as at L = 8192).
bool fftconv_wave32k_supported(int L, int dtype);
hipError_t launch_fftconv_wave32k(const ConvArgs &a, const float *k, hipStream_t s);
// Matrix-core block-FFT convolution (16-bit I/O, L = 2048, 8192 or 16384),
// the kernel spectrum computed from k inside; hipErrorInvalidValue for other
// shapes.
hipError_t launch_fftconv_mfma(const ConvArgs &a, const float *k, hipStream_t s);
bool fftconv_mfma_supported(int L, int dtype);
// One-wavefront-per-transform variant for L = 2048 (16-bit I/O); used by
// launch_fftconv_mfma for that length.
hipError_t launch_fftconv_wave(const ConvArgs &a, const float *k, hipStream_t s);
bool fftconv_wave_supported(int L, int dtype);
// Four-wavefronts-per-pair variant for L = 8192 (16-bit I/O); used by
// launch_fftconv_mfma for that length.
hipError_t launch_fftconv_wave16k(const ConvArgs &a, const float *k, hipStream_t s);
bool fftconv_wave16k_supported(int L, int dtype);

size_t fftconv_workspace(int B, int H, int L);

// Kernel and skip gradients of the convolution: dk[h, j] = sum_b sum_{t>=j}
// dy[b,h,t] u[b,h,t-j] (float32 (H, L)), dD[h] = sum_{b,t} dy u (either may be
// null).  u, dy (B, H, L) of dtype.
hipError_t launch_conv_wgrad(const void *u, const void *dy, int B, int H, int L, int dtype, float *dk, float *dD,
                             hipStream_t s);
// The same on the matrix cores at L = 2048, 16-bit I/O (fftconv_wave_supported):
// one workgroup per channel and group of four row pairs; with more than one
// group per channel the partial sums go to ws (wgrad_wave_workspace bytes)
// and a reduction kernel writes dk, dD.
hipError_t launch_wgrad_wave(const void *u, const void *dy, int B, int H, int dtype, float *dk, float *dD,
                             void *ws, hipStream_t s);
size_t wgrad_wave_workspace(int B, int H);

// State passing pieces.
// Optional tail of the matrix-core chunk-state kernel (chunk 8192 or 16384):
// when one workgroup covers a channel it also writes the channel's table of
// the fused state term (ctab, as launch_corr_tables) and the scan of its rows
// (w16, wexp, x_final, as launch_state_scan_w16); *fused tells whether it did.
struct StateTail {
    const float *C;
    const float *x0;
    uint32_t *w16;
    int *wexp;
    float *x_final;
    uint4 *ctab;
    int fuse;
};
hipError_t launch_chunk_states(const void *u, const float *Abar, const float *Bbar, int B, int H,
                               int L, int m, int chunk, int dtype, float2 *states, hipStream_t s,
                               const StateTail *tail = nullptr, bool *fused = nullptr);
hipError_t launch_state_scan(const float *Abar, const float *C, const float *x0,
                             const float2 *states, int B, int H, int m, int chunk, int nchunk,
                             float2 *corr_W, float *x_final, hipStream_t s);
// corr[row, c*chunk + t] = 2 Re sum_n corr_W[row, c, n] Abar_n^t  (row = b*H + h)
hipError_t launch_state_correction(const float *Abar, const float2 *corr_W, int B, int H, int m,
                                   int chunk, int nchunk, float *corr, hipStream_t s);
bool state_correction_mfma_ok(int chunk, int dtype);
// Per-channel tables for the fused initial-state term of the L = 8192 and
// L = 16384 convs (CORR_TAB_U4 uint4 per channel, the last 32 unused; m <= 64).
constexpr int CORR_TAB_U4 = 1600;
hipError_t launch_corr_tables(const float *Abar, int H, int m, uint4 *tab, hipStream_t s);
// Scan variant for the fused term: normalised fp16 weights and exponents.
hipError_t launch_state_scan_w16(const float *Abar, const float *C, const float *x0, const float2 *states,
                                 int B, int H, int m, int chunk, int nchunk, uint32_t *w16, int *wexp,
                                 float *x_final, hipStream_t s);
hipError_t launch_state_correction_mfma(const float *Abar, const float2 *corr_W, int B, int H, int m,
                                        int chunk, int nchunk, int dtype, void *corr, hipStream_t s);

// State passing (the C ABI entry points validate, then run it).
size_t statepass_workspace(int B, int H, int L, int m, int chunk, int dtype);
int statepass_check(const void *u, const float *Abar, const float *Bbar, const float *C, const void *y,
                    const float *x_final, int B, int H, int L, int m, int chunk, int dtype);
int statepass_run(const void *u, const float *Abar, const float *Bbar, const float *C, const float *D,
                  const float *x0, int B, int H, int L, int m, int chunk, int dtype, void *y, float *x_final,
                  char *ws, hipStream_t s);

// Layer pieces.
hipError_t launch_transpose_batched(const void *in, void *out, int nb, int R, int C, hipStream_t s);
// O (B, L, d) token-major = (Q * S)^T per batch slice, Q and S (B, d, L); R = d, C = L.
hipError_t launch_gate_transpose(const void *q, const void *sv, void *out, int nb, int R, int C, int dtype,
                                 hipStream_t s);
// G = (shift FIR of K + shift_D K) * V over (B, d, L) rows (m_s <= 64, L % 16 == 0);
// v null: G = the shift FIR of K alone.
hipError_t launch_shift_gate(const void *k, const void *v, const float *shift_C, const float *shift_D, int m_s,
                             int B, int d, int L, int dtype, void *g, hipStream_t s);
// Heads of dimension dh in {2, 4, 8} (d % 64 == 0, L % 64 == 0): the outer
// products G (B, d dh, L) of Kbar and V, and their contraction with Q into
// O (B, L, d) token-major.
hipError_t launch_heads_expand(int dh, const void *kbar, const void *v, void *g, int B, int d, int L, int dtype,
                               hipStream_t s);
hipError_t launch_heads_contract(int dh, const void *q, const void *sv, void *o, int B, int d, int L, int dtype,
                                 hipStream_t s);
// The layer's projections on TW x 256 tiles (TW = 320 or 256) with the
// weights as stored, (K, d) row-major (Q = x W): out_mode 1: W[0..2] = W_Q,
// W_K, W_V into the channel-major [Q;K;V] layout as launch_gemm_nt
// (out_mode 1); out_mode 0: W[0] = W_O, C = X W_O row-major (Nx, d).  X is
// (Nx, K) row-major; out_mode 2: as out_mode 0 with X stored K-major,
// (Nx / L, K, L) (needs L % 256 == 0).  gemm_w_tile gives the tile height (0: not supported:
// needs Nx % 256 == 0, K % 32 == 0, d a multiple of 320 or 256).
int gemm_w_tile(int d, int Nx, int K);
hipError_t launch_gemm_w(const void *const *W, const void *X, void *C, int Nx, int K, int dtype, int out_mode, int d,
                         int L, hipStream_t s);
hipError_t launch_gemm_nt(const void *A, const void *Bt, void *C, int M, int N, int K, int dtype,
                          int out_mode, int d, int L, hipStream_t s);
hipError_t launch_layer_mid(const void *q, const void *k, const void *v, const float *shift_C,
                            const float *shift_D, int m_s, const float2 *Kspec,
                            const float *diag_D, int B, int d, int L, int dtype, void *o,
                            hipStream_t s);

}  // namespace h3
