// C ABI of libh3flash: argument validation and kernel dispatch.
// Every check runs on the host before anything is enqueued.
#include <stdint.h>
#include <algorithm>
#include <stdlib.h>
#include <string.h>

#include "../../include/h3flash.h"
#include "internal.h"

using namespace h3;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool pow2_in(int x, int lo, int hi) { return x >= lo && x <= hi && (x & (x - 1)) == 0; }

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

size_t esize(int dtype) { return dtype == H3_F32 ? 4 : 2; }

bool dtype_ok(int dtype) { return dtype == H3_F32 || dtype == H3_F16 || dtype == H3_BF16; }

// [p, p + n) and [q, q + m) overlap?
bool overlap(const void *p, size_t n, const void *q, size_t m) {
    if (!p || !q || n == 0 || m == 0) return false;
    uintptr_t a = (uintptr_t)p, b = (uintptr_t)q;
    return a < b + m && b < a + n;
}

int launched(hipError_t e) { return e == hipSuccess ? H3_OK : H3_EDEVICE; }

// fused length / chunk: a power of two in [H3_MIN_LEN, H3_FUSED_LIMIT]; above
// H3_FUSED_LIMIT_F32 only where the matrix-core kernels take it (16-bit I/O)
bool fused_len_ok(int L, int dtype) {
    return pow2_in(L, H3_MIN_LEN, H3_FUSED_LIMIT) && (L <= H3_FUSED_LIMIT_F32 || fftconv_mfma_supported(L, dtype));
}

// Workspace layouts (each region 256-byte aligned).
//
// State passing, by path (a region a path does not use has size 0):
//   k       (H, chunk) float32            the chunk kernel f
//   kspec   (H, chunk + 1) complex        its spectrum (VALU conv only)
//   states  (B, H, nchunk, m) complex     chunk end-states s_c = M_ux u^(c)
//   fused initial-state term (16-bit, chunk 8192 or 16384): per-channel power
//   tables ctab, normalised weights w16 (B, H, nchunk, 64) fp16 complex and
//   their exponents wexp (B, H, nchunk);
//   otherwise: weights corr_w (B, H, nchunk, m) complex and the term itself,
//   corr (B, H, L), in the I/O dtype on the matrix-core paths, else float32.
struct StatepassWs {
    size_t k, kspec, states, corr_w, corr, ctab, w16, wexp, total;
    bool fused, mfma, corr16;
};
StatepassWs statepass_ws(int B, int H, int L, int m, int chunk, int dtype) {
    StatepassWs w{};
    const size_t nchunk = (size_t)(L / chunk);
    w.fused = fftconv_wave16k_supported(chunk, dtype) || fftconv_wave32k_supported(chunk, dtype);
    w.mfma = fftconv_mfma_supported(chunk, dtype);
    w.corr16 = w.mfma && state_correction_mfma_ok(chunk, dtype);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align_up(bytes);
        return at;
    };
    // the chunk kernel f: the fused-term convs form it themselves
    if (!w.fused) w.k = take((size_t)H * chunk * sizeof(float));
    if (!w.mfma) w.kspec = take((size_t)H * (chunk + 1) * sizeof(float2));
    w.states = take((size_t)B * H * nchunk * m * sizeof(float2));
    if (w.fused) {
        w.ctab = take((size_t)H * CORR_TAB_U4 * sizeof(uint4));
        w.w16 = take((size_t)B * H * nchunk * 64 * sizeof(uint32_t));
        w.wexp = take((size_t)B * H * nchunk * sizeof(int));
    } else {
        w.corr_w = take((size_t)B * H * nchunk * m * sizeof(float2));
        w.corr = take((size_t)B * H * L * (w.corr16 ? 2 : sizeof(float)));
    }
    w.total = off;
    return w;
}

struct LayerWs {
    size_t qkv, o_cm, o_tm, kspec, wt, total;
};
// wt: the four weights transposed to (out, in), only for shapes the
// weight-tiled GEMM does not take (the 128 x 128-tile GEMM reads both operands
// reduction-contiguous)
LayerWs layer_ws(int B, int d, int L) {
    LayerWs w;
    const size_t act = (size_t)B * d * L * 2;
    w.qkv = 0;
    w.o_cm = w.qkv + align_up(3 * act);
    w.o_tm = w.o_cm + align_up(act);
    w.kspec = w.o_tm + align_up(act);
    w.wt = w.kspec + align_up((size_t)d * (L + 1) * sizeof(float2));
    w.total = w.wt + (gemm_w_tile(d, B * L, d) ? 0 : align_up((size_t)4 * d * d * 2));
    return w;
}

// Layer heads with d_h > 1: Q, K, V, Kbar, the outer products G and their
// convolutions S (d_h rows per channel), O token-major, the spectra for the
// VALU convolution, the transposed weights.
struct HeadsWs {
    size_t qkv, kbar, g, sv, o_tm, kspec, wt, total;
};
HeadsWs heads_ws(int B, int d, int L, int dh) {
    HeadsWs w;
    const size_t act = (size_t)B * d * L * 2;
    w.qkv = 0;
    w.kbar = w.qkv + align_up(3 * act);
    w.g = w.kbar + align_up(act);
    w.sv = w.g + align_up((size_t)dh * act);
    w.o_tm = w.sv + align_up((size_t)dh * act);
    w.kspec = w.o_tm + align_up(act);
    w.wt = w.kspec + align_up((size_t)d * dh * (L + 1) * sizeof(float2));
    w.total = w.wt + (gemm_w_tile(d, B * L, d) ? 0 : align_up((size_t)4 * d * d * 2));
    return w;
}

// [Q;K;V] channel-major: per projection j and batch b the (d, L) block
// j B d L + b d L is (x_b W_j)^T.  The weights come as Algorithm 1 writes
// them, (in, out) with Q = x W_Q, and the weight-tiled GEMM reads them so:
// one launch for Q, K and V (d a multiple of 320 or 256, B L of 256).  Other
// shapes take the 128 x 128-tile GEMM per projection, which reads both
// operands reduction-contiguous: the weights are transposed into wt first.
hipError_t layer_qkv(const void *x, const void *Wq, const void *Wk, const void *Wv, char *qkv, int B, int L, int d,
                     int dtype, void *wt, hipStream_t s) {
    const void *Wqkv[3] = {Wq, Wk, Wv};
    if (gemm_w_tile(d, B * L, d)) return launch_gemm_w(Wqkv, x, qkv, B * L, d, dtype, 1, d, L, s);
    const size_t act = (size_t)B * L * d * 2, wb = (size_t)d * d * 2;
    for (int j = 0; j < 3; ++j) {
        char *wj = (char *)wt + j * wb;
        hipError_t e = launch_transpose_batched(Wqkv[j], wj, 1, d, d, s);
        if (e == hipSuccess) e = launch_gemm_nt(wj, x, qkv + j * act, d, B * L, d, dtype, 1, d, L, s);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// out = O (B L, d) . Wo (d, d), O token-major
hipError_t layer_out(const void *o_tm, const void *Wo, void *out, int B, int L, int d, int dtype, void *wt,
                     hipStream_t s) {
    if (gemm_w_tile(d, B * L, d)) return launch_gemm_w(&Wo, o_tm, out, B * L, d, dtype, 0, d, L, s);
    char *wo = (char *)wt + 3 * (size_t)d * d * 2;
    hipError_t e = launch_transpose_batched(Wo, wo, 1, d, d, s);
    if (e != hipSuccess) return e;
    return launch_gemm_nt(o_tm, wo, out, B * L, d, d, dtype, 0, d, L, s);
}

}  // namespace

namespace h3 {

size_t statepass_workspace(int B, int H, int L, int m, int chunk, int dtype) {
    return statepass_ws(B, H, L, m, chunk, dtype).total;
}

// Argument checks of h3_statepass_conv that do not involve the workspace.
int statepass_check(const void *u, const float *Abar, const float *Bbar, const float *C, const void *y,
                    const float *x_final, int B, int H, int L, int m, int chunk, int dtype) {
    if (!u || !Abar || !Bbar || !C || !y || B < 1 || H < 1 || L < 1 || m < 1 || chunk < 1) return H3_EINVAL;
    if (L % chunk) return H3_EINVAL;
    if (!dtype_ok(dtype) || m > H3_MAX_MODES || !fused_len_ok(chunk, dtype)) return H3_EUNSUPPORTED;
    if (!aligned16(u) || !aligned16(y)) return H3_EINVAL;
    const size_t io = (size_t)B * H * L * esize(dtype), xs = (size_t)B * H * m * 8;
    if (overlap(u, io, y, io) || overlap(x_final, xs, y, io) || overlap(x_final, xs, u, io)) return H3_EINVAL;
    return H3_OK;
}

// State passing on validated arguments, scratch at ws (statepass_workspace
// bytes, 256-byte aligned).  Every scratch region is written before it is
// read, so its prior contents do not matter.
int statepass_run(const void *u, const float *Abar, const float *Bbar, const float *C, const float *D,
                  const float *x0, int B, int H, int L, int m, int chunk, int dtype, void *y, float *x_final,
                  char *ws, hipStream_t s) {
    const int nchunk = L / chunk;
    const StatepassWs w = statepass_ws(B, H, L, m, chunk, dtype);
    float *kbuf = (float *)(ws + w.k);
    float2 *Kspec = w.mfma ? nullptr : (float2 *)(ws + w.kspec);
    float2 *states = (float2 *)(ws + w.states);
    hipError_t e;
    // f = [C Bbar, C Abar Bbar, ...] of length chunk, and its spectrum (the
    // L = 8192 and 16384 convs with the fused state term form f themselves)
    const bool gen_f = w.fused;
    if (!gen_f && (e = launch_kernel_gen(1, Abar, Bbar, C, nullptr, H, m, chunk, kbuf, s)) != hipSuccess)
        return H3_EDEVICE;
    if (!w.mfma && (e = launch_spectrum(kbuf, H, chunk, Kspec, s)) != hipSuccess) return H3_EDEVICE;
    // s_c = M_ux u^(c) for every chunk, then the scan over chunks (for the
    // fused term, inside the chunk-state kernel when it covers each channel
    // with one workgroup)
    StateTail tail{C, x0, (uint32_t *)(ws + w.w16), (int *)(ws + w.wexp), x_final, (uint4 *)(ws + w.ctab), 0};
    bool fused_tail = false;
    if ((e = launch_chunk_states(u, Abar, Bbar, B, H, L, m, chunk, dtype, states, s, w.fused ? &tail : nullptr,
                                 &fused_tail)) != hipSuccess)
        return H3_EDEVICE;
    ConvArgs a{};
    a.u = u; a.y = y; a.Kspec = Kspec; a.D = D;
    a.B = B; a.H = H; a.L = chunk; a.nchunk = nchunk; a.pair_mode = 1; a.dtype = dtype;
    if (w.fused) {
        // chunk 8192 or 16384: the conv computes M_xy x^(c) itself from normalised
        // weights (scan output) and per-channel power tables
        uint4 *ctab = (uint4 *)(ws + w.ctab);
        uint32_t *w16 = (uint32_t *)(ws + w.w16);
        int *wexp = (int *)(ws + w.wexp);
        if (!fused_tail) {
            if ((e = launch_state_scan_w16(Abar, C, x0, states, B, H, m, chunk, nchunk, w16, wexp, x_final, s)) !=
                hipSuccess)
                return H3_EDEVICE;
            if ((e = launch_corr_tables(Abar, H, m, ctab, s)) != hipSuccess) return H3_EDEVICE;
        }
        a.corr = w16;
        a.corr_tab = ctab;
        a.corr_e = wexp;
        if (gen_f) {
            a.gen_C = C;
            a.gen_Bbar = Bbar;
            a.m_gen = m;
        }
        return launched(launch_fftconv_mfma(a, gen_f ? nullptr : kbuf, s));
    }
    float2 *corr_W = (float2 *)(ws + w.corr_w);
    void *corr = ws + w.corr;
    if ((e = launch_state_scan(Abar, C, x0, states, B, H, m, chunk, nchunk, corr_W, x_final, s)) != hipSuccess)
        return H3_EDEVICE;
    // M_xy x^(c) for every chunk (in the I/O dtype when the matrix-core paths apply)
    if (w.corr16)
        e = launch_state_correction_mfma(Abar, corr_W, B, H, m, chunk, nchunk, dtype, corr, s);
    else
        e = launch_state_correction(Abar, corr_W, B, H, m, chunk, nchunk, (float *)corr, s);
    if (e != hipSuccess) return H3_EDEVICE;
    a.corr = corr;
    a.corr16 = w.corr16 ? 1 : 0;
    if (w.mfma) return launched(launch_fftconv_mfma(a, kbuf, s));
    return launched(launch_fftconv(a, s));
}

}  // namespace h3

namespace {
}  // namespace

extern "C" {

const char *h3_status_string(int status) {
    switch (status) {
        case H3_OK: return "ok";
        case H3_EINVAL: return "invalid argument";
        case H3_EUNSUPPORTED: return "unsupported size, mode count or dtype";
        case H3_EWORKSPACE: return "workspace missing or too small";
        case H3_EDEVICE: return "kernel launch failed";
    }
    return "unknown status";
}

size_t h3_workspace_size(int op, int B, int H, int L, int m, int chunk, int dtype) {
    if (B < 1 || H < 1 || L < 1 || !dtype_ok(dtype)) return 0;
    switch (op) {
        case H3_OP_FFTCONV:
            return align_up(fftconv_workspace(B, H, L));
        case H3_OP_STATEPASS:
            if (m < 1 || chunk < 1 || L % chunk) return 0;
            return statepass_ws(B, H, L, m, chunk, dtype).total;
        case H3_OP_LAYER:
            return layer_ws(B, H, L).total;
        case H3_OP_LAYER_HEADS:   // chunk = head dimension
            if (chunk == 1) return layer_ws(B, H, L).total;
            if (chunk != 2 && chunk != 4 && chunk != 8) return 0;
            return heads_ws(B, H, L, chunk).total;
        case H3_OP_FFTCONV_BWD: {
            // the spectrum of the du pass, then (same bytes, later in stream
            // order) the kernel-gradient partial sums
            size_t n = align_up(fftconv_workspace(B, H, L));
            if (fftconv_wave_supported(L, dtype)) n = std::max(n, align_up(wgrad_wave_workspace(B, H)));
            return n;
        }
    }
    return 0;
}

int h3_ssm_discretize(const float *A, const float *B, const float *dt, int H, int m, float *Abar,
                      float *Bbar, void *stream) {
    if (!A || !B || !dt || !Abar || !Bbar || H < 1 || m < 1) return H3_EINVAL;
    if (m > H3_MAX_MODES) return H3_EUNSUPPORTED;
    return launched(launch_discretize(A, B, dt, H, m, Abar, Bbar, (hipStream_t)stream));
}

int h3_ssm_step(const void *u, const float *Abar, const float *Bbar, const float *C, const float *D, int B, int H,
                int m, int T, int dtype, float *x, void *y, void *stream) {
    if (!u || !Abar || !Bbar || !C || !x || !y || B < 1 || H < 1 || m < 1 || T < 1) return H3_EINVAL;
    if (!dtype_ok(dtype) || m > H3_MAX_MODES) return H3_EUNSUPPORTED;
    const size_t io = (size_t)B * H * T * esize(dtype), xs = (size_t)B * H * m * 8, ps = (size_t)H * m * 8;
    const uintptr_t ea = esize(dtype) - 1;
    if (((uintptr_t)u & ea) || ((uintptr_t)y & ea) || ((uintptr_t)x & 7) || ((uintptr_t)Abar & 7) ||
        ((uintptr_t)Bbar & 7) || ((uintptr_t)C & 7) || ((uintptr_t)D & 3))
        return H3_EINVAL;
    if (overlap(u, io, y, io) || overlap(x, xs, u, io) || overlap(x, xs, y, io) || overlap(x, xs, Abar, ps) ||
        overlap(x, xs, Bbar, ps) || overlap(x, xs, C, ps) || overlap(x, xs, D, (size_t)H * 4) ||
        overlap(y, io, Abar, ps) || overlap(y, io, Bbar, ps) || overlap(y, io, C, ps) || overlap(y, io, D, (size_t)H * 4))
        return H3_EINVAL;
    return launched(launch_ssm_step(u, Abar, Bbar, C, D, B, H, m, T, dtype, x, y, (hipStream_t)stream));
}

int h3_ssm_kernel(const float *A, const float *B, const float *C, const float *dt, int H, int m,
                  int L, float *k, void *stream) {
    if (!A || !B || !C || !dt || !k || H < 1 || m < 1 || L < 1) return H3_EINVAL;
    if (m > H3_MAX_MODES) return H3_EUNSUPPORTED;
    return launched(launch_kernel_gen(0, A, B, C, dt, H, m, L, k, (hipStream_t)stream));
}

int h3_fftconv(const void *u, const float *k, const float *D, void *y, int B, int H, int L,
               int dtype, void *workspace, size_t ws_bytes, void *stream) {
    if (!u || !k || !y || B < 1 || H < 1 || L < 1) return H3_EINVAL;
    if (!dtype_ok(dtype) || !fused_len_ok(L, dtype)) return H3_EUNSUPPORTED;
    const size_t io = (size_t)B * H * L * esize(dtype);
    const size_t need = h3_workspace_size(H3_OP_FFTCONV, B, H, L, 0, 0, dtype);
    if (!workspace || ws_bytes < need) return H3_EWORKSPACE;
    if (!aligned16(u) || !aligned16(y) || !aligned16(k) || !aligned16(workspace)) return H3_EINVAL;
    if (overlap(u, io, y, io) || overlap(workspace, need, u, io) || overlap(workspace, need, y, io) ||
        overlap(workspace, need, k, (size_t)H * L * 4))
        return H3_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    ConvArgs a{};
    a.u = u; a.y = y; a.D = D;
    a.B = B; a.H = H; a.L = L; a.nchunk = 1; a.pair_mode = 0; a.dtype = dtype;
    a.corr = nullptr;
    a.corr16 = 0;
    if (fftconv_mfma_supported(L, dtype)) return launched(launch_fftconv_mfma(a, k, s));
    if (fftconv_kgen_supported(L)) return launched(launch_fftconv_kgen(a, k, s));
    float2 *Kspec = (float2 *)workspace;
    hipError_t e = launch_spectrum(k, H, L, Kspec, s);
    if (e != hipSuccess) return H3_EDEVICE;
    a.Kspec = Kspec;
    return launched(launch_fftconv(a, s));
}

int h3_fftconv_bwd(const void *u, const float *k, const float *D, const void *dy, int B, int H, int L, int dtype,
                   void *du, float *dk, float *dD, void *workspace, size_t ws_bytes, void *stream) {
    if (!dy || !k || B < 1 || H < 1 || L < 1 || (!du && !dk && !dD)) return H3_EINVAL;
    if ((dk || dD) && !u) return H3_EINVAL;
    if (!dtype_ok(dtype) || !fused_len_ok(L, dtype) || ((dk || dD) && L > H3_FUSED_LIMIT_F32)) return H3_EUNSUPPORTED;
    const size_t io = (size_t)B * H * L * esize(dtype), kb = (size_t)H * L * 4, db = (size_t)H * 4;
    const size_t need = h3_workspace_size(H3_OP_FFTCONV_BWD, B, H, L, 0, 0, dtype);
    if (!workspace || ws_bytes < need) return H3_EWORKSPACE;
    if ((u && !aligned16(u)) || !aligned16(dy) || (du && !aligned16(du)) || !aligned16(k) || (dk && !aligned16(dk)) ||
        ((uintptr_t)dD & 3) || !aligned16(workspace))
        return H3_EINVAL;
    // outputs overlap no input, no other output and not the workspace
    const void *outs[3] = {du, dk, dD};
    const size_t osz[3] = {io, kb, db};
    for (int i = 0; i < 3; ++i) {
        if (!outs[i]) continue;
        if (overlap(outs[i], osz[i], u, io) || overlap(outs[i], osz[i], dy, io) || overlap(outs[i], osz[i], k, kb) ||
            overlap(outs[i], osz[i], D, db) || overlap(outs[i], osz[i], workspace, need))
            return H3_EINVAL;
        for (int j = i + 1; j < 3; ++j)
            if (outs[j] && overlap(outs[i], osz[i], outs[j], osz[j])) return H3_EINVAL;
    }
    if (overlap(workspace, need, u, io) || overlap(workspace, need, dy, io) || overlap(workspace, need, k, kb))
        return H3_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    if (du) {
        // du = dy correlated with k (+ D dy): the forward convolution with the
        // conjugated kernel spectrum
        ConvArgs a{};
        a.u = dy; a.y = du; a.D = D;
        a.B = B; a.H = H; a.L = L; a.nchunk = 1; a.pair_mode = 0; a.dtype = dtype;
        a.conj_k = 1;
        if (fftconv_mfma_supported(L, dtype)) {   // the wave kernels (2048, 8192) or the 32768-point one
            e = launch_fftconv_mfma(a, k, s);
        } else if (fftconv_kgen_supported(L)) {
            e = launch_fftconv_kgen(a, k, s);
        } else {
            float2 *Kspec = (float2 *)workspace;
            e = launch_spectrum(k, H, L, Kspec, s);
            if (e == hipSuccess) {
                a.Kspec = Kspec;
                e = launch_fftconv(a, s);
            }
        }
        if (e != hipSuccess) return H3_EDEVICE;
    }
    if (dk || dD) {
        const char *sel = getenv("H3FLASH_WGRAD");   // "valu": the float32 VALU kernel at every length
        const bool valu = sel && strcmp(sel, "valu") == 0;
        if (!valu && fftconv_wave_supported(L, dtype))
            return launched(launch_wgrad_wave(u, dy, B, H, dtype, dk, dD, workspace, s));
        return launched(launch_conv_wgrad(u, dy, B, H, L, dtype, dk, dD, s));
    }
    return launched(hipSuccess);
}

int h3_kernel_spectrum(const float *k, int H, int L, float *Kspec, void *stream) {
    if (!k || !Kspec || H < 1 || L < 1) return H3_EINVAL;
    if (!pow2_in(L, H3_MIN_LEN, H3_FUSED_LIMIT_F32)) return H3_EUNSUPPORTED;
    if (!aligned16(k) || !aligned16(Kspec)) return H3_EINVAL;
    if (overlap(k, (size_t)H * L * 4, Kspec, (size_t)H * (L + 1) * 8)) return H3_EINVAL;
    return launched(launch_spectrum(k, H, L, (float2 *)Kspec, (hipStream_t)stream));
}

int h3_fftconv_spectral(const void *u, const float *Kspec, const float *D, void *y, int B, int H,
                        int L, int dtype, void *stream) {
    if (!u || !Kspec || !y || B < 1 || H < 1 || L < 1) return H3_EINVAL;
    if (!dtype_ok(dtype) || !pow2_in(L, H3_MIN_LEN, H3_FUSED_LIMIT_F32)) return H3_EUNSUPPORTED;
    if (!aligned16(u) || !aligned16(y) || !aligned16(Kspec)) return H3_EINVAL;
    const size_t io = (size_t)B * H * L * esize(dtype);
    if (overlap(u, io, y, io) || overlap(Kspec, (size_t)H * (L + 1) * 8, y, io)) return H3_EINVAL;
    ConvArgs a{};
    a.u = u; a.y = y; a.Kspec = (const float2 *)Kspec; a.D = D;
    a.B = B; a.H = H; a.L = L; a.nchunk = 1; a.pair_mode = 0; a.dtype = dtype;
    a.corr = nullptr;
    a.corr16 = 0;
    return launched(launch_fftconv(a, (hipStream_t)stream));
}

int h3_statepass_conv(const void *u, const float *Abar, const float *Bbar, const float *C,
                      const float *D, const float *x0, int B, int H, int L, int m, int chunk,
                      int dtype, void *y, float *x_final, void *workspace, size_t ws_bytes,
                      void *stream) {
    const int st = statepass_check(u, Abar, Bbar, C, y, x_final, B, H, L, m, chunk, dtype);
    if (st != H3_OK) return st;
    const size_t io = (size_t)B * H * L * esize(dtype), xs = (size_t)B * H * m * 8;
    const size_t need = statepass_workspace(B, H, L, m, chunk, dtype);
    if (!workspace || ws_bytes < need) return H3_EWORKSPACE;
    if (!aligned16(workspace)) return H3_EINVAL;
    if (overlap(workspace, need, u, io) || overlap(workspace, need, y, io) || overlap(x_final, xs, workspace, need))
        return H3_EINVAL;
    return statepass_run(u, Abar, Bbar, C, D, x0, B, H, L, m, chunk, dtype, y, x_final, (char *)workspace,
                         (hipStream_t)stream);
}

int h3_layer_fwd(const void *x, const void *Wq, const void *Wk, const void *Wv, const void *Wo,
                 const float *shift_C, const float *shift_D, const float *diag_k,
                 const float *diag_D, int B, int L, int d, int m_s, int dtype, void *out,
                 void *workspace, size_t ws_bytes, void *stream) {
    if (!x || !Wq || !Wk || !Wv || !Wo || !shift_C || !diag_k || !out || B < 1 || L < 1 || d < 1 ||
        m_s < 1)
        return H3_EINVAL;
    if ((dtype != H3_F16 && dtype != H3_BF16) || !pow2_in(L, H3_MIN_LEN, H3_FUSED_LIMIT) ||
        d % 128 != 0 || ((long)B * L) % 128 != 0 || m_s > H3_MAX_SHIFT)
        return H3_EUNSUPPORTED;
    const size_t need = h3_workspace_size(H3_OP_LAYER, B, d, L, m_s, 0, dtype);
    if (!workspace || ws_bytes < need) return H3_EWORKSPACE;
    if (!aligned16(x) || !aligned16(out) || !aligned16(Wq) || !aligned16(Wk) || !aligned16(Wv) ||
        !aligned16(Wo) || !aligned16(workspace))
        return H3_EINVAL;
    const size_t act = (size_t)B * L * d * 2;
    if (overlap(x, act, out, act) || overlap(workspace, need, x, act) || overlap(workspace, need, out, act))
        return H3_EINVAL;
    const size_t wbytes = (size_t)d * d * 2;
    for (const void *W : {Wq, Wk, Wv, Wo})
        if (overlap(W, wbytes, out, act) || overlap(W, wbytes, workspace, need)) return H3_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    const LayerWs w = layer_ws(B, d, L);
    char *ws = (char *)workspace;
    char *qkv = ws + w.qkv;
    void *o_cm = ws + w.o_cm;
    void *o_tm = ws + w.o_tm;
    float2 *Kspec = (float2 *)(ws + w.kspec);
    hipError_t e;
    void *wt = ws + w.wt;
    if ((e = layer_qkv(x, Wq, Wk, Wv, qkv, B, L, d, dtype, wt, s)) != hipSuccess) return H3_EDEVICE;
    const char *q = qkv, *kk = qkv + act, *v = qkv + 2 * act;
    if (fftconv_mfma_supported(L, dtype) && L % 64 == 0) {
        // G = (shift SSM of K) * V  ->  o_cm;  S = diag conv of G (+ D G)  ->  K's slot (K is dead);
        // O (B, L, d) = (Q * S)^T  ->  o_tm
        if ((e = launch_shift_gate(kk, v, shift_C, shift_D, m_s, B, d, L, dtype, o_cm, s)) != hipSuccess)
            return H3_EDEVICE;
        ConvArgs ca{};
        ca.u = o_cm; ca.y = (void *)kk; ca.D = diag_D;
        ca.B = B; ca.H = d; ca.L = L; ca.nchunk = 1; ca.pair_mode = 0; ca.dtype = dtype;
        if (fftconv_wave_supported(L, dtype) && gemm_w_tile(d, B * L, d)) {
            // L = 2048: the convolution's epilogue gates with Q and writes
            // O = Q * S channel-major into K's slot; the output projection
            // reads it K-major
            ca.gate = q;
            if ((e = launch_fftconv_mfma(ca, diag_k, s)) != hipSuccess) return H3_EDEVICE;
            return launched(launch_gemm_w(&Wo, kk, out, B * L, d, dtype, 2, d, L, s));
        }
        if ((e = launch_fftconv_mfma(ca, diag_k, s)) != hipSuccess) return H3_EDEVICE;
        if ((e = launch_gate_transpose(q, kk, o_tm, B, d, L, dtype, s)) != hipSuccess) return H3_EDEVICE;
    } else {
        if ((e = launch_spectrum(diag_k, d, L, Kspec, s)) != hipSuccess) return H3_EDEVICE;
        if ((e = launch_layer_mid(q, kk, v, shift_C, shift_D, m_s, Kspec, diag_D, B, d, L, dtype, o_cm,
                                  s)) != hipSuccess)
            return H3_EDEVICE;
        // O (B, d, L) -> (B, L, d)
        if ((e = launch_transpose_batched(o_cm, o_tm, B, d, L, s)) != hipSuccess) return H3_EDEVICE;
    }
    return launched(layer_out(o_tm, Wo, out, B, L, d, dtype, wt, s));
}

int h3_layer_fwd_heads(const void *x, const void *Wq, const void *Wk, const void *Wv, const void *Wo,
                       const float *shift_C, const float *shift_D, const float *diag_k, const float *diag_D, int B,
                       int L, int d, int d_head, int m_s, int dtype, void *out, void *workspace, size_t ws_bytes,
                       void *stream) {
    if (d_head == 1)
        return h3_layer_fwd(x, Wq, Wk, Wv, Wo, shift_C, shift_D, diag_k, diag_D, B, L, d, m_s, dtype, out, workspace,
                            ws_bytes, stream);
    if (!x || !Wq || !Wk || !Wv || !Wo || !shift_C || !diag_k || !out || B < 1 || L < 1 || d < 1 || m_s < 1 ||
        d_head < 1)
        return H3_EINVAL;
    if ((dtype != H3_F16 && dtype != H3_BF16) || !pow2_in(L, 64, H3_FUSED_LIMIT) || d % 128 != 0 ||
        ((long)B * L) % 128 != 0 || m_s > H3_MAX_SHIFT || (d_head != 2 && d_head != 4 && d_head != 8))
        return H3_EUNSUPPORTED;
    const size_t need = h3_workspace_size(H3_OP_LAYER_HEADS, B, d, L, m_s, d_head, dtype);
    if (!workspace || ws_bytes < need) return H3_EWORKSPACE;
    if (!aligned16(x) || !aligned16(out) || !aligned16(Wq) || !aligned16(Wk) || !aligned16(Wv) ||
        !aligned16(Wo) || !aligned16(workspace))
        return H3_EINVAL;
    const size_t act = (size_t)B * L * d * 2;
    if (overlap(x, act, out, act) || overlap(workspace, need, x, act) || overlap(workspace, need, out, act))
        return H3_EINVAL;
    const size_t wbytes = (size_t)d * d * 2;
    for (const void *W : {Wq, Wk, Wv, Wo})
        if (overlap(W, wbytes, out, act) || overlap(W, wbytes, workspace, need)) return H3_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    const HeadsWs w = heads_ws(B, d, L, d_head);
    char *ws = (char *)workspace;
    char *qkv = ws + w.qkv;
    void *kbar = ws + w.kbar, *g = ws + w.g, *sv = ws + w.sv, *o_tm = ws + w.o_tm, *wt = ws + w.wt;
    float2 *Kspec = (float2 *)(ws + w.kspec);
    const char *q = qkv, *kk = qkv + act, *v = qkv + 2 * act;
    hipError_t e;
    if ((e = layer_qkv(x, Wq, Wk, Wv, qkv, B, L, d, dtype, wt, s)) != hipSuccess) return H3_EDEVICE;
    // Kbar = shift SSM of K (no gating); G = per-head outer products of Kbar and V
    if ((e = launch_shift_gate(kk, nullptr, shift_C, shift_D, m_s, B, d, L, dtype, kbar, s)) != hipSuccess)
        return H3_EDEVICE;
    if ((e = launch_heads_expand(d_head, kbar, v, g, B, d, L, dtype, s)) != hipSuccess) return H3_EDEVICE;
    // S = diagonal SSM of every (h, i, j) row: the fused convolution over d d_h channels
    ConvArgs ca{};
    ca.u = g; ca.y = sv; ca.D = diag_D;
    ca.B = B; ca.H = d * d_head; ca.L = L; ca.nchunk = 1; ca.pair_mode = 0; ca.dtype = dtype;
    if (fftconv_mfma_supported(L, dtype)) {
        if ((e = launch_fftconv_mfma(ca, diag_k, s)) != hipSuccess) return H3_EDEVICE;
    } else {
        if ((e = launch_spectrum(diag_k, d * d_head, L, Kspec, s)) != hipSuccess) return H3_EDEVICE;
        ca.Kspec = Kspec;
        if ((e = launch_fftconv(ca, s)) != hipSuccess) return H3_EDEVICE;
    }
    // O_t[j] = sum_i Q_t[i] S_t[i][j], token-major; out = O Wo^T
    if ((e = launch_heads_contract(d_head, q, sv, o_tm, B, d, L, dtype, s)) != hipSuccess) return H3_EDEVICE;
    return launched(layer_out(o_tm, Wo, out, B, L, d, dtype, wt, s));
}

}  // extern "C"
