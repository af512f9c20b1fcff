// Recurrent (step) mode of a diagonal SSM, the generation path of Sec. 2:
// from a carried state x (B, H, m) complex, for each of T new tokens
//     x_n <- Abar_n x_n + Bbar_n u_t,      y_t = 2 Re sum_n C_n x_n + D u_t,
// the same recurrence whose impulse response is the convolution kernel k, so a
// state left by state passing (x_final) continues the sequence exactly.
//
// Layout: 16 lanes per channel h, walking NB batch rows (b, h) of that
// channel with the channel's Abar, Bbar, C held in registers; lane s owns
// modes 2s, 2s + 1, 2s + 32, 2s + 33 (16-byte loads, 256 contiguous bytes per
// instruction and row) when m is even, else s, s + 16, s + 32, s + 48 (8-byte
// loads).  The state stays in registers across the T tokens of one call and
// is written back once; the NB rows' loads are all issued before the first
// update.  The sum over modes is a 16-lane butterfly.  Each call reads and
// writes the state once: the kernel is bound by HBM bandwidth (512 B per row
// and direction at m = 64).
#include "common.h"
#include "internal.h"

namespace h3 {
namespace {

constexpr int SL = 16;                       // lanes per channel
constexpr int MPL = H3_MAX_MODES_DEV / SL;   // modes per lane
constexpr int NB = 2;                        // batch rows per lane group

// Lane s's modes of one row (slot i of v): VEC 2: 2s + (i & 1) + 32 (i >> 1);
// VEC 1: s + 16 i.  Modes at or past m read as zero and are not stored.
template <int VEC>
__device__ __forceinline__ void load_modes(const float2 *__restrict__ p, int s, int m, float2 (&v)[MPL]) {
    if constexpr (VEC == 2) {
#pragma unroll
        for (int q = 0; q < MPL / 2; ++q) {
            const int n = 2 * s + 32 * q;   // m even: n < m implies n + 1 < m
            float4 t = make_float4(0.f, 0.f, 0.f, 0.f);
            if (n < m) t = *(const float4 *)(p + n);
            v[2 * q] = make_float2(t.x, t.y);
            v[2 * q + 1] = make_float2(t.z, t.w);
        }
    } else {
#pragma unroll
        for (int i = 0; i < MPL; ++i) {
            const int n = s + SL * i;
            v[i] = n < m ? p[n] : make_float2(0.f, 0.f);
        }
    }
}

template <int VEC>
__device__ __forceinline__ void store_modes(float2 *__restrict__ p, int s, int m, const float2 (&v)[MPL]) {
    if constexpr (VEC == 2) {
#pragma unroll
        for (int q = 0; q < MPL / 2; ++q) {
            const int n = 2 * s + 32 * q;
            if (n < m) *(float4 *)(p + n) = make_float4(v[2 * q].x, v[2 * q].y, v[2 * q + 1].x, v[2 * q + 1].y);
        }
    } else {
#pragma unroll
        for (int i = 0; i < MPL; ++i) {
            const int n = s + SL * i;
            if (n < m) p[n] = v[i];
        }
    }
}

template <int DT, int VEC>
__global__ __launch_bounds__(64) void ssm_step_kernel(const float2 *__restrict__ Abar, const float2 *__restrict__ Bbar,
                                                       const float2 *__restrict__ C, const float *__restrict__ D,
                                                       const typename IO<DT>::T *__restrict__ u,
                                                       float2 *__restrict__ x, typename IO<DT>::T *__restrict__ y,
                                                       int B, int H, int m, int T) {
    const long tid = (long)blockIdx.x * blockDim.x + threadIdx.x;
    const long grp = tid / SL;
    const int s = (int)(tid % SL);
    const int h = (int)(grp % H), b0 = (int)(grp / H) * NB;
    if (b0 >= B) return;   // whole 16-lane groups leave together
    float2 a[MPL], bb[MPL], c[MPL], st[NB][MPL];
#pragma unroll
    for (int r = 0; r < NB; ++r) {
        if (b0 + r < B) load_modes<VEC>(x + ((long)(b0 + r) * H + h) * m, s, m, st[r]);
    }
    load_modes<VEC>(Abar + (long)h * m, s, m, a);
    load_modes<VEC>(Bbar + (long)h * m, s, m, bb);
    load_modes<VEC>(C + (long)h * m, s, m, c);
    const float dd = D ? D[h] : 0.f;
#pragma unroll
    for (int r = 0; r < NB; ++r) {
        if (b0 + r >= B) break;
        const long row = (long)(b0 + r) * H + h;
        for (int t = 0; t < T; ++t) {
            const float ut = IO<DT>::ld(u, row * T + t);
            float acc = 0.f;
#pragma unroll
            for (int i = 0; i < MPL; ++i) {
                const float2 p = st[r][i];
                st[r][i] = make_float2(a[i].x * p.x - a[i].y * p.y + bb[i].x * ut,
                                       a[i].x * p.y + a[i].y * p.x + bb[i].y * ut);
                acc += c[i].x * st[r][i].x - c[i].y * st[r][i].y;
            }
            acc += __shfl_xor(acc, 8, SL);
            acc += __shfl_xor(acc, 4, SL);
            acc += __shfl_xor(acc, 2, SL);
            acc += __shfl_xor(acc, 1, SL);
            if (s == 0) IO<DT>::st(y, row * T + t, 2.f * acc + dd * ut);
        }
        store_modes<VEC>(x + row * m, s, m, st[r]);
    }
}

}  // namespace

hipError_t launch_ssm_step(const void *u, const float *Abar, const float *Bbar, const float *C, const float *D,
                           int B, int H, int m, int T, int dtype, float *x, void *y, hipStream_t s) {
    if (m < 1 || m > H3_MAX_MODES_DEV) return hipErrorInvalidValue;
    const long groups = (long)H * ((B + NB - 1) / NB);
    const dim3 grid((unsigned)((groups * SL + 63) / 64)), block(64);   // one wave per workgroup
    const float2 *A2 = (const float2 *)Abar, *B2 = (const float2 *)Bbar, *C2 = (const float2 *)C;
    float2 *x2 = (float2 *)x;
    const bool v2 = m % 2 == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)Abar & 15) == 0 &&
                    ((uintptr_t)Bbar & 15) == 0 && ((uintptr_t)C & 15) == 0;
#define H3_STEP(DTV, TT)                                                                                          \
    do {                                                                                                          \
        if (v2)                                                                                                   \
            hipLaunchKernelGGL((ssm_step_kernel<DTV, 2>), grid, block, 0, s, A2, B2, C2, D, (const TT *)u, x2,   \
                               (TT *)y, B, H, m, T);                                                              \
        else                                                                                                      \
            hipLaunchKernelGGL((ssm_step_kernel<DTV, 1>), grid, block, 0, s, A2, B2, C2, D, (const TT *)u, x2,   \
                               (TT *)y, B, H, m, T);                                                              \
    } while (0)
    if (dtype == F32) H3_STEP(F32, float);
    else if (dtype == F16) H3_STEP(F16, uint16_t);
    else H3_STEP(BF16, uint16_t);
#undef H3_STEP
    return hipGetLastError();
}

}  // namespace h3
