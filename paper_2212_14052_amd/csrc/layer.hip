// H3 layer forward pieces (Sec. 3.2, Algorithm 1 with head dimension 1), gfx950.
//
//   [Q;K;V] channel-major  = Wt_qkv . x^T          (MFMA GEMM, bf16/fp16 in, fp32 acc)
//   O = Q * (diag_k (*) (Kbar * V) + D (Kbar * V)),  Kbar = shift FIR of K
//                                                  (one fused kernel per row pair)
//   out = O . Wo                                    (MFMA GEMM)
// The projections are the layer's dense contractions (O(d^2 N), Proposition 1)
// and run on the matrix cores; the sequence mixing is the fused FFT conv.
#include "common.h"
#include "fft_valu.h"
#include "internal.h"

namespace h3 {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

template <int DT> struct Mfma;
template <> struct Mfma<F16> {
    static __device__ __forceinline__ f32x16_t run(uint4 a, uint4 b, f32x16_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(*(half8_t *)&a, *(half8_t *)&b, c, 0, 0, 0);
    }
};
template <> struct Mfma<BF16> {
    static __device__ __forceinline__ f32x16_t run(uint4 a, uint4 b, f32x16_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(bf16x8_t *)&a, *(bf16x8_t *)&b, c, 0, 0, 0);
    }
};

// ------------------------------------------------------------------ GEMM ---
// C = A . Bt^T with A (M, K) and Bt (N, K) both K-contiguous (16-bit), fp32
// accumulation, 16-bit result.  Tile 128 x 128 x 32, 4 waves of 64 x 64, each
// a 2 x 2 grid of 32x32x16 MFMAs.  Requires M, N % 128 == 0 and K % 32 == 0.
// out_mode 0: C row-major (M, N).
// out_mode 1: rows are channels of [Q;K;V] (M = 3 d), columns tokens
//             (N = B L); element (m, n) goes to
//             [(m / d)][(n / L)][(m % d)][(n % L)]  (three (B, d, L) tensors).
constexpr int GB_M = 128, GB_N = 128, GB_K = 32, GB_LDK = GB_K + 8;

template <int DT>
__global__ __launch_bounds__(256) void gemm_nt_kernel(const uint16_t *A, const uint16_t *Bt,
                                                      uint16_t *C, int M, int N, int K,
                                                      int out_mode, int d, int L) {
    __shared__ __attribute__((aligned(16))) uint16_t As[GB_M * GB_LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[GB_N * GB_LDK];
    const int nbn = N / GB_N;
    const int blk = xcd_logical_block(blockIdx.x, gridDim.x);
    const int m0 = (blk / nbn) * GB_M, n0 = (blk % nbn) * GB_N;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int wm = w >> 1, wn = w & 1;
    // global -> register staging: 2 x 16 B of A and of B per thread
    const int lr = t >> 2, lk = (t & 3) * 8;
    uint4 ra[2], rb[2];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            ra[i] = *(const uint4 *)(A + (long)(m0 + lr + 64 * i) * K + k0 + lk);
            rb[i] = *(const uint4 *)(Bt + (long)(n0 + lr + 64 * i) * K + k0 + lk);
        }
    };
    auto lstore = [&]() {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            *(uint4 *)(As + (lr + 64 * i) * GB_LDK + lk) = ra[i];
            *(uint4 *)(Bs + (lr + 64 * i) * GB_LDK + lk) = rb[i];
        }
    };
    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    gload(0);
    lstore();
    __syncthreads();
    for (int k0 = 0; k0 < K; k0 += GB_K) {
        const bool more = k0 + GB_K < K;
        if (more) gload(k0 + GB_K);
#pragma unroll
        for (int ks = 0; ks < GB_K / 16; ++ks) {
            uint4 af[2], bf[2];
            const int kk = ks * 16 + 8 * (lane >> 5);
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                af[i] = *(const uint4 *)(As + (wm * 64 + i * 32 + (lane & 31)) * GB_LDK + kk);
                bf[i] = *(const uint4 *)(Bs + (wn * 64 + i * 32 + (lane & 31)) * GB_LDK + kk);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = Mfma<DT>::run(af[i], bf[j], acc[i][j]);
        }
        __syncthreads();
        if (more) {
            lstore();
            __syncthreads();
        }
    }
    // epilogue: lane holds column (lane & 31) and rows 8(e/4) + 4(lane/32) + e%4
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int m = m0 + wm * 64 + i * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
                const int n = n0 + wn * 64 + j * 32 + (lane & 31);
                const uint16_t v = (DT == BF16) ? f32_to_bf16(acc[i][j][e]) : f32_to_f16(acc[i][j][e]);
                long dst;
                if (out_mode == 0) {
                    dst = (long)m * N + n;
                } else {
                    dst = (long)(m / d) * ((long)N * d) + (long)(n / L) * ((long)d * L) +
                          (long)(m % d) * L + (n % L);
                }
                C[dst] = v;
            }
}

// --------------------------------------------------------- transposes ------
// out[b][c][r] = in[b][r][c] for batch of (R, C) matrices of 16-bit values.
__global__ __launch_bounds__(256) void transpose16_kernel(const uint16_t *in, uint16_t *out, int R,
                                                          int Cc) {
    __shared__ uint16_t tile[64][66];
    const int tr = (R + 63) / 64, tc = (Cc + 63) / 64;
    const int b = blockIdx.x / (tr * tc), rem = blockIdx.x % (tr * tc);
    const int r0 = (rem / tc) * 64, c0 = (rem % tc) * 64;
    const long off = (long)b * R * Cc;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int r = r0 + i, c = c0 + tx;
        if (r < R && c < Cc) tile[i][tx] = in[off + (long)r * Cc + c];
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int c = c0 + i, r = r0 + tx;
        if (r < R && c < Cc) out[off + (long)c * R + r] = tile[tx][i];
    }
}

// ------------------------------------------------------- fused middle ------
// Per pair of rows (batches 2j, 2j+1) of channel c, all (B, d, L):
//   G = (sum_{j<m_s} shift_C[c,j] K_{t-j} + shift_D[c] K_t) * V_t
//   S = diag_k (*) G + diag_D G      (FFT conv, packed as G_a + i G_b)
//   O = Q * S
template <int N, int DT>
__global__ __launch_bounds__(N / 16 >= 64 ? N / 16 : 64) void layer_mid_kernel(
    const uint16_t *q, const uint16_t *k, const uint16_t *v, const float *shift_C,
    const float *shift_D, int m_s, const float2 *Kspec, const float *diag_D, int B, int d,
    uint16_t *o, int npairs) {
    using P = FFTPlan<N>;
    using io = IO<DT>;
    constexpr int T = P::T, R1 = P::R1, Q = 16 / R1, HALF = R1 / 2;
    constexpr int S = (T >= 64) ? 1 : 64 / T;
    constexpr int L = N / 2;
    extern __shared__ float2 lds[];
    const int sig = threadIdx.x / T, tid = threadIdx.x % T;
    float2 *X = lds + sig * P::LDS;
    const int blk = xcd_logical_block(blockIdx.x, gridDim.x);
    const int p = blk * S + sig;
    const bool active = p < npairs;
    const int nbp = (B + 1) / 2;
    const int pp = active ? p : 0;
    const int c = pp / nbp, bp = pp % nbp;
    const long oa = ((long)(2 * bp) * d + c) * L;
    const bool hb = active && (2 * bp + 1 < B);
    const long ob = hb ? ((long)(2 * bp + 1) * d + c) * L : 0;

    // stage K of both rows in LDS (unpadded, index t)
    for (int t = tid; t < L; t += T) {
        const float ka = active ? io::ld(k, oa + t) : 0.f;
        const float kb = hb ? io::ld(k, ob + t) : 0.f;
        X[t] = make_float2(ka, kb);
    }
    __syncthreads();
    const float *cs = shift_C + (long)c * m_s;
    const float ds = shift_D ? shift_D[c] : 0.f;
    float2 vv[16];
    float ga[8], gb[8];
#pragma unroll
    for (int qq = 0; qq < Q; ++qq) {
        const int j = tid + qq * T;
#pragma unroll
        for (int r = 0; r < R1; ++r) {
            if (r < HALF) {
                const int n = j + r * (N / R1);
                float2 kb = cscale(X[n], ds);
                const int jmax = n < m_s - 1 ? n : m_s - 1;
                for (int jj = 0; jj <= jmax; ++jj) {
                    const float2 x = X[n - jj];
                    kb.x = fmaf(cs[jj], x.x, kb.x);
                    kb.y = fmaf(cs[jj], x.y, kb.y);
                }
                const float va = active ? io::ld(v, oa + n) : 0.f;
                const float vb = hb ? io::ld(v, ob + n) : 0.f;
                ga[qq * HALF + r] = kb.x * va;
                gb[qq * HALF + r] = kb.y * vb;
                vv[qq * R1 + r] = make_float2(kb.x * va, kb.y * vb);
            } else {
                vv[qq * R1 + r] = make_float2(0.f, 0.f);
            }
        }
    }
    __syncthreads();
    fft_forward_from_regs<N>(X, tid, vv);
    const float2 *K = Kspec + (long)c * (L + 1);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int f = tid + r * T;
        const float2 kf = (f <= L) ? K[f] : cconj(K[N - f]);
        vv[r] = cconj(cmul(vv[r], kf));
    }
    fft_second_from_regs<N>(X, tid, vv);
    const float dd = diag_D ? diag_D[c] : 0.f;
    if (!active) return;
#pragma unroll
    for (int qq = 0; qq < Q; ++qq) {
        const int j = tid + qq * T;
#pragma unroll
        for (int r = 0; r < HALF; ++r) {
            const int n = j + r * (N / R1);
            const float2 w = vv[qq * R1 + r];
            const float sa = w.x + dd * ga[qq * HALF + r];
            io::st(o, oa + n, io::ld(q, oa + n) * sa);
            if (hb) {
                const float sb = -w.y + dd * gb[qq * HALF + r];
                io::st(o, ob + n, io::ld(q, ob + n) * sb);
            }
        }
    }
}

// --------------------------------------------------------------- launch ----
hipError_t launch_transpose_w(const void *W, int d, int dtype, void *Wt, hipStream_t s) {
    (void)dtype;
    const int tiles = ((d + 63) / 64) * ((d + 63) / 64);
    hipLaunchKernelGGL(transpose16_kernel, dim3(tiles), dim3(256), 0, s, (const uint16_t *)W,
                       (uint16_t *)Wt, d, d);
    return hipGetLastError();
}

hipError_t launch_transpose_batched(const void *in, void *out, int nb, int R, int C, hipStream_t s) {
    const int tiles = ((R + 63) / 64) * ((C + 63) / 64);
    hipLaunchKernelGGL(transpose16_kernel, dim3(nb * tiles), dim3(256), 0, s, (const uint16_t *)in,
                       (uint16_t *)out, R, C);
    return hipGetLastError();
}

hipError_t launch_gemm_nt(const void *A, const void *Bt, void *C, int M, int N, int K, int dtype,
                          int out_mode, int d, int L, hipStream_t s) {
    const int nblk = (M / GB_M) * (N / GB_N);
    if (dtype == BF16)
        hipLaunchKernelGGL(gemm_nt_kernel<BF16>, dim3(nblk), dim3(256), 0, s, (const uint16_t *)A,
                           (const uint16_t *)Bt, (uint16_t *)C, M, N, K, out_mode, d, L);
    else
        hipLaunchKernelGGL(gemm_nt_kernel<F16>, dim3(nblk), dim3(256), 0, s, (const uint16_t *)A,
                           (const uint16_t *)Bt, (uint16_t *)C, M, N, K, out_mode, d, L);
    return hipGetLastError();
}

template <int N, int DT>
static hipError_t launch_mid_n(const void *q, const void *k, const void *v, const float *shift_C,
                               const float *shift_D, int m_s, const float2 *Kspec,
                               const float *diag_D, int B, int d, void *o, hipStream_t s) {
    using P = FFTPlan<N>;
    constexpr int T = P::T, S = (T >= 64) ? 1 : 64 / T;
    const int npairs = ((B + 1) / 2) * d;
    const size_t lds = (size_t)S * P::LDS * sizeof(float2);
    auto fn = layer_mid_kernel<N, DT>;
    if (lds > 65536) (void)hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(fn, dim3((npairs + S - 1) / S), dim3(S * T), lds, s, (const uint16_t *)q,
                       (const uint16_t *)k, (const uint16_t *)v, shift_C, shift_D, m_s, Kspec,
                       diag_D, B, d, (uint16_t *)o, npairs);
    return hipGetLastError();
}

template <int N>
static hipError_t launch_mid_dt(int dtype, const void *q, const void *k, const void *v,
                                const float *shift_C, const float *shift_D, int m_s,
                                const float2 *Kspec, const float *diag_D, int B, int d, void *o,
                                hipStream_t s) {
    if (dtype == BF16) return launch_mid_n<N, BF16>(q, k, v, shift_C, shift_D, m_s, Kspec, diag_D, B, d, o, s);
    return launch_mid_n<N, F16>(q, k, v, shift_C, shift_D, m_s, Kspec, diag_D, B, d, o, s);
}

hipError_t launch_layer_mid(const void *q, const void *k, const void *v, const float *shift_C,
                            const float *shift_D, int m_s, const float2 *Kspec,
                            const float *diag_D, int B, int d, int L, int dtype, void *o,
                            hipStream_t s) {
#define H3_MID_CASE(LL)                                                                         \
    case LL:                                                                                    \
        return launch_mid_dt<2 * LL>(dtype, q, k, v, shift_C, shift_D, m_s, Kspec, diag_D, B, d, \
                                     o, s);
    switch (L) {
        H3_MID_CASE(16)
        H3_MID_CASE(32)
        H3_MID_CASE(64)
        H3_MID_CASE(128)
        H3_MID_CASE(256)
        H3_MID_CASE(512)
        H3_MID_CASE(1024)
        H3_MID_CASE(2048)
        H3_MID_CASE(4096)
        H3_MID_CASE(8192)
    }
#undef H3_MID_CASE
    return hipErrorInvalidValue;
}

}  // namespace h3
