// H3 layer with heads of dimension d_h > 1 (Sec. 3.2, Algorithm 1): per head
// h (channels h d_h .. h d_h + d_h - 1) and token t the d_h x d_h outer
// product  KV_t[i][j] = Kbar_t[i] V_t[j]  passes through the diagonal SSM (one
// kernel per entry (h, i, j)), and the head's output is  O_t[j] =
// sum_i Q_t[i] S_t[i][j].  The outer products are d_h^2 sequence rows per head,
// channel (h d_h + i) d_h + j, convolved by the fused FFT convolution like any
// other rows; the two kernels here build them and contract them with Q.
#include "common.h"
#include "internal.h"

namespace h3 {
namespace {

__device__ __forceinline__ float ld16(uint16_t v, int dt) { return dt == BF16 ? bf16_to_f32(v) : f16_to_f32(v); }
__device__ __forceinline__ uint16_t st16(float v, int dt) { return dt == BF16 ? f32_to_bf16(v) : f32_to_f16(v); }

// G[b, (h d_h + i) d_h + j, t] = Kbar[b, h d_h + i, t] V[b, h d_h + j, t], one
// rounding; Kbar, V (B, d, L) channel-major, G (B, d d_h, L).  One thread per
// (b, h, 8 consecutive t): d_h + d_h 16-byte loads, d_h^2 16-byte stores.
template <int DT, int DH>
__global__ __launch_bounds__(256) void heads_expand_kernel(const uint16_t *kbar, const uint16_t *v, int B, int d, int L,
                                                           uint16_t *g) {
    const int nh = d / DH, nt = L / 8;
    const long id = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (id >= (long)B * nh * nt) return;
    const int t = (int)(id % nt) * 8;
    const long bh = id / nt;
    const int h = (int)(bh % nh), b = (int)(bh / nh);
    float kf[DH][8], vf[DH][8];
#pragma unroll
    for (int i = 0; i < DH; ++i) {
        const long row = ((long)b * d + h * DH + i) * L + t;
        const uint4 kq = *(const uint4 *)(kbar + row), vq = *(const uint4 *)(v + row);
        const uint32_t k4[4] = {kq.x, kq.y, kq.z, kq.w}, v4[4] = {vq.x, vq.y, vq.z, vq.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            kf[i][2 * e] = ld16(k4[e] & 0xffffu, DT); kf[i][2 * e + 1] = ld16(k4[e] >> 16, DT);
            vf[i][2 * e] = ld16(v4[e] & 0xffffu, DT); vf[i][2 * e + 1] = ld16(v4[e] >> 16, DT);
        }
    }
#pragma unroll
    for (int i = 0; i < DH; ++i)
#pragma unroll
        for (int j = 0; j < DH; ++j) {
            uint32_t o4[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                o4[e] = (uint32_t)st16(kf[i][2 * e] * vf[j][2 * e], DT) |
                        ((uint32_t)st16(kf[i][2 * e + 1] * vf[j][2 * e + 1], DT) << 16);
            const long row = ((long)b * d * DH + (long)(h * DH + i) * DH + j) * L + t;
            *(uint4 *)(g + row) = make_uint4(o4[0], o4[1], o4[2], o4[3]);
        }
}

// O[b, t, h d_h + j] = sum_i Q[b, h d_h + i, t] S[b, (h d_h + i) d_h + j, t],
// one rounding, written token-major (B, L, d) for the output projection.
// Tile of 64 channels x 64 tokens per 256 threads: thread -> one channel and
// 16 consecutive tokens, then the tile goes through LDS so that the stores are
// 16 bytes along the channels.
template <int DT, int DH>
__global__ __launch_bounds__(256) void heads_contract_kernel(const uint16_t *q, const uint16_t *s, int B, int d, int L,
                                                             uint16_t *o) {
    __shared__ __attribute__((aligned(16))) uint16_t tile[64][64 + 8];   // [token][channel]
    const int ntt = L / 64, nct = d / 64;
    const int blk = blockIdx.x;
    const int tt = blk % ntt, ct = (blk / ntt) % nct, b = blk / (ntt * nct);
    const int cl = threadIdx.x >> 2, tq = (threadIdx.x & 3) * 16;
    const int c = ct * 64 + cl, h = c / DH, j = c % DH;
    const int t0 = tt * 64 + tq;
    float acc[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
    for (int i = 0; i < DH; ++i) {
        const uint16_t *qr = q + ((long)b * d + h * DH + i) * L + t0;
        const uint16_t *sr = s + ((long)b * d * DH + (long)(h * DH + i) * DH + j) * L + t0;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const uint4 qv = *(const uint4 *)(qr + 8 * hh), sv = *(const uint4 *)(sr + 8 * hh);
            const uint32_t q4[4] = {qv.x, qv.y, qv.z, qv.w}, s4[4] = {sv.x, sv.y, sv.z, sv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                acc[8 * hh + 2 * e] += ld16(q4[e] & 0xffffu, DT) * ld16(s4[e] & 0xffffu, DT);
                acc[8 * hh + 2 * e + 1] += ld16(q4[e] >> 16, DT) * ld16(s4[e] >> 16, DT);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) tile[tq + r][cl] = st16(acc[r], DT);
    __syncthreads();
    // 64 tokens x 64 channels: thread -> token tk, channels 16 (tid & 3) .. + 15
    const int tk = threadIdx.x >> 2, cq = (threadIdx.x & 3) * 16;
    uint16_t *orow = o + ((long)b * L + tt * 64 + tk) * d + ct * 64 + cq;
    *(uint4 *)orow = *(const uint4 *)&tile[tk][cq];
    *(uint4 *)(orow + 8) = *(const uint4 *)&tile[tk][cq + 8];
}

template <int DT>
hipError_t launch_heads_dt(int dh, const void *kbar, const void *v, const void *q, void *g, const void *sv, void *o,
                           int B, int d, int L, bool expand, hipStream_t st) {
    const uint16_t *k16 = (const uint16_t *)kbar, *v16 = (const uint16_t *)v, *q16 = (const uint16_t *)q;
    const uint16_t *s16 = (const uint16_t *)sv;
    uint16_t *g16 = (uint16_t *)g, *o16 = (uint16_t *)o;
    if (expand) {
        const long n = (long)B * (d / dh) * (L / 8);
        const dim3 grid((unsigned)((n + 255) / 256)), block(256);
        switch (dh) {
            case 2: hipLaunchKernelGGL((heads_expand_kernel<DT, 2>), grid, block, 0, st, k16, v16, B, d, L, g16); break;
            case 4: hipLaunchKernelGGL((heads_expand_kernel<DT, 4>), grid, block, 0, st, k16, v16, B, d, L, g16); break;
            case 8: hipLaunchKernelGGL((heads_expand_kernel<DT, 8>), grid, block, 0, st, k16, v16, B, d, L, g16); break;
            default: return hipErrorInvalidValue;
        }
    } else {
        const dim3 grid((unsigned)((long)B * (d / 64) * (L / 64))), block(256);
        switch (dh) {
            case 2: hipLaunchKernelGGL((heads_contract_kernel<DT, 2>), grid, block, 0, st, q16, s16, B, d, L, o16); break;
            case 4: hipLaunchKernelGGL((heads_contract_kernel<DT, 4>), grid, block, 0, st, q16, s16, B, d, L, o16); break;
            case 8: hipLaunchKernelGGL((heads_contract_kernel<DT, 8>), grid, block, 0, st, q16, s16, B, d, L, o16); break;
            default: return hipErrorInvalidValue;
        }
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_heads_expand(int dh, const void *kbar, const void *v, void *g, int B, int d, int L, int dtype,
                               hipStream_t s) {
    if (d % 64 || L % 64) return hipErrorInvalidValue;
    return dtype == BF16 ? launch_heads_dt<BF16>(dh, kbar, v, nullptr, g, nullptr, nullptr, B, d, L, true, s)
                         : launch_heads_dt<F16>(dh, kbar, v, nullptr, g, nullptr, nullptr, B, d, L, true, s);
}

hipError_t launch_heads_contract(int dh, const void *q, const void *sv, void *o, int B, int d, int L, int dtype,
                                 hipStream_t s) {
    if (d % 64 || L % 64) return hipErrorInvalidValue;
    return dtype == BF16 ? launch_heads_dt<BF16>(dh, nullptr, nullptr, q, nullptr, sv, o, B, d, L, false, s)
                         : launch_heads_dt<F16>(dh, nullptr, nullptr, q, nullptr, sv, o, B, d, L, false, s);
}

}  // namespace h3
