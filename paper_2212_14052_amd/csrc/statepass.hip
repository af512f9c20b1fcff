// State passing (Sec. 4.2, Algorithm 2) pieces, gfx950.
//
// With chunk length N' and the state x^(c) carried into chunk c (the state
// after the previous chunk's last input):
//   end-of-chunk contribution  s_c = M_ux u^(c),  M_ux[n, i] = Abar_n^{N'-1-i} Bbar_n
//   state update               x^(c+1) = Abar^{N'} x^(c) + s_c
//   output                     y^(c)_t = (f * u^(c))_t + D u^(c)_t
//                                        + 2 Re sum_n C_n Abar_n^{t+1} x^(c)_n
// The chunk-local sums s_c of all chunks are independent (one workgroup per
// chunk row); only the short scan over chunks is sequential.
#include "common.h"
#include "internal.h"

namespace h3 {

// ----------------------------------------------------------- chunk sums ----
// s_c[n] = Bbar_n sum_i Abar_n^{N'-1-i} u_i, factorised with i = T a + b:
//   s_c[n] = Bbar_n sum_a Abar_n^{N' - T(a+1)} R[a][n],
//   R[a][n] = sum_{b<T} Abar_n^{T-1-b} u_{T a + b}.
constexpr int CS_T = 64;
constexpr int CS_THREADS = 256;

template <int DT>
__global__ __launch_bounds__(CS_THREADS) void chunk_states_kernel(const void *u_, const float *Abar,
                                                                  const float *Bbar, int H, int L,
                                                                  int m, int chunk, float2 *states) {
    using io = IO<DT>;
    typedef typename io::T T_;
    const T_ *u = (const T_ *)u_;
    extern __shared__ float smem[];
    float *us = smem;                                   // chunk of u, float32
    float2 *Qs = (float2 *)(smem + chunk);              // [b][n] Abar_n^{T-1-b}
    float2 *red = Qs + CS_T * H3_MAX_MODES_DEV;         // [4][n] partial sums
    const int nchunk = L / chunk;
    const int crow = blockIdx.x;                        // (b*H + h) * nchunk + c
    const int row = crow / nchunk, c = crow % nchunk;
    const int h = row % H;
    const int tid = threadIdx.x;
    const long base = (long)row * L + (long)c * chunk;
    for (int i = tid; i < chunk; i += CS_THREADS) us[i] = io::ld(u, base + i);
    const int T = chunk < CS_T ? chunk : CS_T;
    const int NA = chunk / T;
    const int n = tid % H3_MAX_MODES_DEV, g = tid / H3_MAX_MODES_DEV;
    double lr = 0, li = 0;
    if (n < m) {
        const long i = (long)h * m + n;
        const double ar = Abar[2 * i], ai = Abar[2 * i + 1];
        lr = 0.5 * log(ar * ar + ai * ai);
        li = atan2(ai, ar);
        for (int b = g; b < T; b += CS_THREADS / H3_MAX_MODES_DEV)
            Qs[b * H3_MAX_MODES_DEV + n] = cexp_scaled((double)(T - 1 - b), lr, li);
    }
    __syncthreads();
    float2 acc = make_float2(0.f, 0.f);
    if (n < m) {
        constexpr int G = CS_THREADS / H3_MAX_MODES_DEV;     // 4 groups over a
        // a = g + G i, i descending, so the anchor power grows in magnitude:
        // exponent N' - T(a+1) increases by G T per step.
        int alast = g + G * ((NA - 1 - g) / G);
        if (g < NA) {
            float2 pw = cexp_scaled((double)(chunk - T * (alast + 1)), lr, li);
            const float2 step = cexp_scaled((double)(G * T), lr, li);
            for (int a = alast; a >= 0; a -= G) {
                float rr = 0.f, ri = 0.f;
                const float *ua = us + T * a;
                for (int b = 0; b < T; ++b) {
                    const float2 q = Qs[b * H3_MAX_MODES_DEV + n];
                    const float x = ua[b];
                    rr = fmaf(q.x, x, rr);
                    ri = fmaf(q.y, x, ri);
                }
                acc = cadd(acc, cmul(pw, make_float2(rr, ri)));
                pw = cmul(pw, step);
            }
        }
    }
    red[g * H3_MAX_MODES_DEV + n] = acc;
    __syncthreads();
    if (g == 0 && n < m) {
        float2 s = red[n];
        for (int k = 1; k < CS_THREADS / H3_MAX_MODES_DEV; ++k) s = cadd(s, red[k * H3_MAX_MODES_DEV + n]);
        const long i = (long)h * m + n;
        const float2 bb = make_float2(Bbar[2 * i], Bbar[2 * i + 1]);
        states[(long)crow * m + n] = cmul(bb, s);
    }
}

// ------------------------------------------------------------------ scan ---
// One thread per (row, mode): x <- Abar^{N'} x + s_c across the chunks.
// Writes corr_W[row, c, n] = C_n x^(c)_n Abar_n (so that the initial-state
// term of chunk c is 2 Re sum_n corr_W Abar_n^t) and x_final = x^(nchunk).
__global__ void state_scan_kernel(const float *Abar, const float *C, const float *x0,
                                  const float2 *states, int B, int H, int m, int chunk, int nchunk,
                                  float2 *corr_W, float *x_final) {
    const long gid = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (long)B * H * m) return;
    const int n = (int)(gid % m);
    const long row = gid / m;
    const int h = (int)(row % H);
    const long i = (long)h * m + n;
    const double ar = Abar[2 * i], ai = Abar[2 * i + 1];
    const float2 ab = make_float2((float)ar, (float)ai);
    const float2 cc = make_float2(C[2 * i], C[2 * i + 1]);
    const float2 cab = cmul(cc, ab);
    const float2 AN = cexp_scaled((double)chunk, 0.5 * log(ar * ar + ai * ai), atan2(ai, ar));
    float2 x = x0 ? make_float2(x0[2 * gid], x0[2 * gid + 1]) : make_float2(0.f, 0.f);
    for (int c = 0; c < nchunk; ++c) {
        const long ci = (row * nchunk + c) * m + n;
        corr_W[ci] = cmul(cab, x);
        x = cadd(cmul(AN, x), states[ci]);
    }
    if (x_final) {
        x_final[2 * gid] = x.x;
        x_final[2 * gid + 1] = x.y;
    }
}

hipError_t launch_chunk_states(const void *u, const float *Abar, const float *Bbar, int B, int H,
                               int L, int m, int chunk, int dtype, float2 *states, hipStream_t s) {
    const int nchunk = L / chunk;
    const long ncr = (long)B * H * nchunk;
    const size_t lds = (size_t)chunk * sizeof(float) +
                       (size_t)(CS_T + CS_THREADS / H3_MAX_MODES_DEV) * H3_MAX_MODES_DEV * sizeof(float2);
    dim3 grid((unsigned)ncr), block(CS_THREADS);
    if (lds > 65536) {
        (void)hipFuncSetAttribute((const void *)chunk_states_kernel<F32>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        (void)hipFuncSetAttribute((const void *)chunk_states_kernel<F16>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        (void)hipFuncSetAttribute((const void *)chunk_states_kernel<BF16>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    }
    switch (dtype) {
        case F32:
            hipLaunchKernelGGL(chunk_states_kernel<F32>, grid, block, lds, s, u, Abar, Bbar, H, L, m, chunk, states);
            break;
        case F16:
            hipLaunchKernelGGL(chunk_states_kernel<F16>, grid, block, lds, s, u, Abar, Bbar, H, L, m, chunk, states);
            break;
        case BF16:
            hipLaunchKernelGGL(chunk_states_kernel<BF16>, grid, block, lds, s, u, Abar, Bbar, H, L, m, chunk, states);
            break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_state_scan(const float *Abar, const float *C, const float *x0,
                             const float2 *states, int B, int H, int m, int chunk, int nchunk,
                             float2 *corr_W, float *x_final, hipStream_t s) {
    const long n = (long)B * H * m;
    hipLaunchKernelGGL(state_scan_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, Abar, C,
                       x0, states, B, H, m, chunk, nchunk, corr_W, x_final);
    return hipGetLastError();
}

}  // namespace h3
