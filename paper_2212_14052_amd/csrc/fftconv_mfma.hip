// Fused block-FFT convolution at L = 16384 (Sec. 4.1: kernel fusion + block
// FFT, past the 8192 limit the paper's SRAM set; Sec. 4.2 uses it as the
// state-passing chunk), gfx950, 16-bit I/O.  Transform length N = 2L = 32768 =
// 8 x 4096, held in LDS as fp16 complex (128 KB of the 160 KB).
//
// The DFT of each 4096-point block is, as in the paper's four-step
// factorisation, three layers of length-16 DFTs (block-diagonal I (x) F_16
// products) with twiddle diagonals in between.  Each layer of 256 DFT-16s runs
// as 16 pairs of v_mfma_f32_16x16x32_f16: the 16x16 complex DFT matrix is the
// A operand (as a 16 x 32 real matrix for the real rows and one for the
// imaginary rows), 16 signal vectors are the columns of B.  Block index
// p = 256 p2 + 16 p1 + p0 (fp16 complex per dword).  Forward (decimation in
// frequency):
//   A: DFT over p2, then * w_4096^{p2 (16 p1 + p0)}
//   B: DFT over p1, then * w_256^{p1 p0}
//   C: DFT over p0            -> position p holds X[p2 + 16 p1 + 256 p0]
// The spectrum stays in this digit-reversed order; the kernel spectrum is made
// by the same pipeline, so the pointwise product needs no permutation.  The
// second transform (conj(F(conj Y)) = N IDFT(Y)) runs the layers in reverse
// and ends in natural order.
//
// Two rows of one channel travel as one complex signal (u_a + i u_b).
// Dynamic range: each row is scaled by its own power of two to max |.| in
// [1/2, 1), each DFT-16 layer carries a factor 1/4 (folded into the fp16 DFT
// matrix) and the kernel spectrum is normalised to max |K| in [1/2, 1); all
// scale factors are powers of two and are undone exactly in fp32 at the
// output.
#include "common.h"
#include "fft_valu.h"
#include "internal.h"

namespace h3 {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));

namespace mf {


__device__ __forceinline__ uint32_t pack(float re, float im) {
    h2_t h = {(_Float16)re, (_Float16)im};
    return __builtin_bit_cast(uint32_t, h);
}
__device__ __forceinline__ h2_t as_h2(uint32_t v) { return __builtin_bit_cast(h2_t, v); }
__device__ __forceinline__ uint32_t as_u32(h2_t v) { return __builtin_bit_cast(uint32_t, v); }

// (a.re + i a.im)(w.re + i w.im) in packed fp16
__device__ __forceinline__ uint32_t cmul_h(uint32_t a_, uint32_t w_) {
    const h2_t a = as_h2(a_), w = as_h2(w_);
    const h2_t t = a.xx * w;
    const h2_t ws = {-w.y, w.x};
    return as_u32(a.yy * ws + t);
}

__device__ __forceinline__ uint32_t twiddle_h(int e, int n) {
    // exp(-2 pi i e / n), e reduced mod n first (n a power of two)
    e &= n - 1;
    float s, c;
    __sincosf(-6.283185307179586f * (float)e / (float)n, &s, &c);
    return pack(c, s);
}

struct Dft16 {
    h8_t re, im;
};
// Rows r = lane % 16 (output frequency), columns 8 g .. 8 g + 7 (g = lane / 16)
// = interleaved (re, im) of input points 4g .. 4g+3; entries scaled by 1/4.
__device__ __forceinline__ Dft16 make_dft16(int lane) {
    const int r = lane & 15, g = lane >> 4;
    Dft16 F;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = (r * (4 * g + i)) & 15;
        const float c = 0.25f * kCos16[q], s = 0.25f * kSin16[q];
        // Y_re = sum c x_re + s x_im ;  Y_im = sum -s x_re + c x_im   (w = e^{-i theta})
        F.re[2 * i] = (_Float16)c;
        F.re[2 * i + 1] = (_Float16)s;
        F.im[2 * i] = (_Float16)(-s);
        F.im[2 * i + 1] = (_Float16)c;
    }
    return F;
}

__device__ __forceinline__ h8_t h8_from(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
    uint4 v = make_uint4(a, b, c, d);
    return __builtin_bit_cast(h8_t, v);
}

__device__ __forceinline__ void dft16(const Dft16 &F, h8_t x, f4_t &re, f4_t &im) {
    const f4_t z = {0.f, 0.f, 0.f, 0.f};
    re = __builtin_amdgcn_mfma_f32_16x16x32_f16(F.re, x, z, 0, 0, 0);
    im = __builtin_amdgcn_mfma_f32_16x16x32_f16(F.im, x, z, 0, 0, 0);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

// Raw 16-bit I/O values.
template <int DT> __device__ __forceinline__ float lo_f(uint32_t r);
template <int DT> __device__ __forceinline__ float hi_f(uint32_t r);
template <> __device__ __forceinline__ float lo_f<F16>(uint32_t r) { return (float)as_h2(r).x; }
template <> __device__ __forceinline__ float hi_f<F16>(uint32_t r) { return (float)as_h2(r).y; }
template <> __device__ __forceinline__ float lo_f<BF16>(uint32_t r) { return __uint_as_float(r << 16); }
template <> __device__ __forceinline__ float hi_f<BF16>(uint32_t r) { return __uint_as_float(r & 0xffff0000u); }
// (lo, hi) -> packed raw pair, round to nearest even
template <int DT> __device__ __forceinline__ uint32_t pack_io(float lo, float hi);
template <> __device__ __forceinline__ uint32_t pack_io<F16>(float lo, float hi) { return pack(lo, hi); }
template <> __device__ __forceinline__ uint32_t pack_io<BF16>(float lo, float hi) {
    typedef __bf16 b2_t __attribute__((ext_vector_type(2)));
    b2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

}  // namespace mf

namespace mf32 {
constexpr int N = 32768;
constexpr int L = 16384;
constexpr int NW = 16;
constexpr int NT = 64 * NW;
constexpr int NB = 8;   // 4096-point blocks
}  // namespace mf32

namespace mf {
// exp(-2 pi i e / n) from the hardware sine and cosine, whose argument is in
// revolutions (e / n is exact for n a power of two), packed fp16
__device__ __forceinline__ uint32_t twiddle_rev(int e, int n) {
    e &= n - 1;
    const float r = (float)e / (float)n;
    return pack(__builtin_amdgcn_cosf(r), -__builtin_amdgcn_sinf(r));
}
// exp(-2 pi i q / 8) for q = 0..7 (cos, -sin); q is a compile-time constant
// at every use (unrolled loops)
constexpr float kC8[8] = {1.f, 0.70710678118654752f, 0.f, -0.70710678118654752f,
                          -1.f, -0.70710678118654752f, 0.f, 0.70710678118654752f};
__device__ __forceinline__ float2 w8(int q) { return make_float2(kC8[q & 7], -kC8[(q + 6) & 7]); }
}  // namespace mf

template <int DT>
__global__ __launch_bounds__(mf32::NT) void fftconv_mfma32768_kernel(ConvArgs a, const float *k, int wg_per_ch,
                                                                     int pairs_per_ch) {
    using namespace mf;
    using mf32::NT;
    using mf32::NW;
    using mf32::NB;
    constexpr int NN = mf32::N, LL = mf32::L, BLK = 4096;
    __shared__ uint32_t X[NN];        // eight 4096-point blocks, fp16 complex
    __shared__ float red[2][NW];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int c = lane & 15, g = lane >> 4;
    const int blk = xcd_logical_block(blockIdx.x, gridDim.x);
    const int h = blk / wg_per_ch, part = blk % wg_per_ch;
    const int per = (pairs_per_ch + wg_per_ch - 1) / wg_per_ch;
    const int q0 = part * per, q1 = min(q0 + per, pairs_per_ch);
    int rsel = 0;
    auto bexp = [&](float v) -> int {
        v = wave_max(v);
        if (lane == 0) red[rsel][w] = v;
        __syncthreads();
        float m = red[rsel][0];
#pragma unroll
        for (int i = 1; i < NW; ++i) m = fmaxf(m, red[rsel][i]);
        rsel ^= 1;
        if (!(m > 0.f) || !(m < 3.0e38f)) return 0;
        int e;
        frexpf(m, &e);
        return e;
    };

    // lane bases inside a block (block beta adds 4096 beta); batch b = w
    const int mA = 1024 * g + 64 * (c >> 2) + (c & 3) + 4 * (w ^ ((c >> 2) | (g << 2)));
    int mB[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) mB[j] = 256 * w + 64 * (c >> 2) + (c & 3) + 16 * (g ^ (w >> 2)) + 4 * (j ^ (c >> 2));
    const int mC = 256 * w + 64 * g + 4 * (c ^ g ^ ((w >> 2) << 2));
    const int mR = 256 * (tid >> 6) + 64 * (tid & 3) + 4 * (((tid >> 2) & 15) ^ (tid & 3) ^ ((tid >> 8) << 2));

    uint32_t twA[4], twB[4], tw2[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        tw2[j] = twiddle_h((4 * g + j) * c, 256);
        twA[j] = twiddle_h((4 * g + j) * (16 * w + c), BLK);
        twB[j] = twiddle_h(w * (16 * (4 * g + j) + c), BLK);
    }
    const Dft16 F = make_dft16(lane);

    // layer R forward from x[e][n3] = values at 4096 n3 + m (n3 < 4, fp32,
    // already scaled); the zero padding is n3 = 4..7.  Factor 1/4 for range.
    int tz = 0;
    auto layer_R = [&](const float2 (&x)[4][4]) {
#pragma unroll
        for (int k3 = 0; k3 < NB; ++k3) {
            uint32_t o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                float yr = 0.f, yi = 0.f;
#pragma unroll
                for (int n3 = 0; n3 < 4; ++n3) {
                    const float2 wv = w8(n3 * k3), xv = x[e][n3];
                    yr += xv.x * wv.x - xv.y * wv.y;
                    yi += xv.x * wv.y + xv.y * wv.x;
                }
                o[e] = pack(0.25f * yr, 0.25f * yi);
                if (k3) o[e] = cmul_h(o[e], twiddle_rev((4 * tid + e) * k3 + tz, NN));
            }
            *(uint4 *)&X[mR + BLK * k3] = make_uint4(o[0], o[1], o[2], o[3]);
        }
        __syncthreads();
    };
    auto blocks_AB = [&]() {
#pragma unroll
        for (int be = 0; be < NB; ++be) {
            uint32_t v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = X[mA + 256 * j + BLK * be];
            f4_t re, im;
            dft16(F, h8_from(v[0], v[1], v[2], v[3]), re, im);
#pragma unroll
            for (int j = 0; j < 4; ++j) X[mA + 256 * j + BLK * be] = cmul_h(pack(re[j], im[j]), twA[j]);
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();
#pragma unroll
        for (int be = 0; be < NB; ++be) {
            uint32_t v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = X[mB[j] + BLK * be];
            f4_t re, im;
            dft16(F, h8_from(v[0], v[1], v[2], v[3]), re, im);
#pragma unroll
            for (int j = 0; j < 4; ++j) X[mB[j] + BLK * be] = cmul_h(pack(re[j], im[j]), tw2[j]);
            __builtin_amdgcn_sched_barrier(0);
        }
        // no barrier: layer C of batch b = p2 is read back by the same wave
    };

    // ---- kernel spectrum of channel h (k[0] += D), F(k 2^-ek) / 256 2^-e2 ----
    uint32_t K[NB][4];
    int kexp;
    {
        float4 kv[4];
#pragma unroll
        for (int n3 = 0; n3 < 4; ++n3) kv[n3] = ((const float4 *)(k + (long)h * LL + BLK * n3))[tid];
        if (tid == 0 && a.D) kv[0].x += a.D[h];
        float mx = 0.f;
#pragma unroll
        for (int n3 = 0; n3 < 4; ++n3)
            mx = fmaxf(mx, fmaxf(fmaxf(fabsf(kv[n3].x), fabsf(kv[n3].y)), fmaxf(fabsf(kv[n3].z), fabsf(kv[n3].w))));
        const int ek = bexp(mx);
        const float sk = ldexpf(1.0f, -ek);
        float2 x[4][4];
#pragma unroll
        for (int n3 = 0; n3 < 4; ++n3) {
            x[0][n3] = make_float2(kv[n3].x * sk, 0.f);
            x[1][n3] = make_float2(kv[n3].y * sk, 0.f);
            x[2][n3] = make_float2(kv[n3].z * sk, 0.f);
            x[3][n3] = make_float2(kv[n3].w * sk, 0.f);
        }
        layer_R(x);
        blocks_AB();
        // |F(k 2^-ek)| / 256 <= 64: packed unnormalised, then scaled by 2^-e2
        float km = 0.f;
#pragma unroll
        for (int be = 0; be < NB; ++be) {
            const uint4 v = *(const uint4 *)&X[mC + BLK * be];
            f4_t re, im;
            dft16(F, __builtin_bit_cast(h8_t, v), re, im);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                K[be][j] = pack(re[j], im[j]);
                km = fmaxf(km, fmaxf(fabsf(re[j]), fabsf(im[j])));
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        const int e2 = bexp(km);
        const _Float16 s2 = (_Float16)ldexpf(1.0f, -e2);
        const h2_t s22 = {s2, s2};
        const uint32_t cj = a.conj_k ? 0x80000000u : 0u;
#pragma unroll
        for (int be = 0; be < NB; ++be)
#pragma unroll
            for (int j = 0; j < 4; ++j) K[be][j] = as_u32(as_h2(K[be][j]) * s22) ^ cj;
        kexp = -ek - 8 - e2;   // forward scale 1/256 (R: 1/4, A, B, C: 1/4 each)
        __syncthreads();       // X is rewritten by the first pair's layer R
    }

    const uint16_t *u = (const uint16_t *)a.u;
    uint16_t *y = (uint16_t *)a.y;
    auto rows = [&](int qq, long &oa, long &ob) {
        if (a.pair_mode == 0) {
            oa = ((long)(2 * qq) * a.H + h) * LL;
            ob = (2 * qq + 1 < a.B) ? ((long)(2 * qq + 1) * a.H + h) * LL : -1;
        } else {
            const int ncp = (a.nchunk + 1) / 2;
            const int bb = qq / ncp, cp = qq % ncp;
            oa = (((long)bb * a.H + h) * a.nchunk + 2 * cp) * LL;
            ob = (2 * cp + 1 < a.nchunk) ? oa + LL : -1;
        }
    };
    for (int qq = q0; qq < q1; ++qq) {
        // an opaque zero added to the twiddle arguments: they are evaluated
        // where they are used instead of being hoisted out of the pair loop
        // (56 values that would stay live, and spill, across it)
        asm volatile("v_mov_b32 %0, 0" : "=v"(tz));
        long oa, ob;
        rows(qq, oa, ob);
        float mxa = 0.f, mxb = 0.f;
        float2 x[4][4];   // [e][n3]: (row a, row b) at 4096 n3 + 4 tid + e
#pragma unroll
        for (int n3 = 0; n3 < 4; ++n3) {
            const uint2 ra = *(const uint2 *)(u + oa + BLK * n3 + 4 * tid);
            const uint2 rb = (ob >= 0) ? *(const uint2 *)(u + ob + BLK * n3 + 4 * tid) : make_uint2(0, 0);
            const uint32_t pa[2] = {ra.x, ra.y}, pb[2] = {rb.x, rb.y};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t va = (e & 1) ? (pa[e >> 1] >> 16) : (pa[e >> 1] & 0xffffu);
                const uint32_t vb = (e & 1) ? (pb[e >> 1] >> 16) : (pb[e >> 1] & 0xffffu);
                x[e][n3] = make_float2(lo_f<DT>(va), lo_f<DT>(vb));
                mxa = fmaxf(mxa, fabsf(x[e][n3].x));
                mxb = fmaxf(mxb, fabsf(x[e][n3].y));
            }
        }
        // one power-of-two scale per row of the pair
        const int eua = bexp(mxa), eub = bexp(mxb);
        {
            const float sua = ldexpf(1.0f, -eua), sub = ldexpf(1.0f, -eub);
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int n3 = 0; n3 < 4; ++n3) x[e][n3] = make_float2(x[e][n3].x * sua, x[e][n3].y * sub);
            layer_R(x);
        }
        blocks_AB();
        // layer C forward, pointwise product, layer C of the second transform
#pragma unroll
        for (int be = 0; be < NB; ++be) {
            uint4 *px = (uint4 *)&X[mC + BLK * be];
            f4_t re, im;
            dft16(F, __builtin_bit_cast(h8_t, *px), re, im);
            uint32_t yv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) yv[j] = cmul_h(pack(re[j], im[j]), K[be][j]) ^ 0x80000000u;
            dft16(F, h8_from(yv[0], yv[1], yv[2], yv[3]), re, im);
            uint4 o;
            o.x = cmul_h(pack(re[0], im[0]), tw2[0]);
            o.y = cmul_h(pack(re[1], im[1]), tw2[1]);
            o.z = cmul_h(pack(re[2], im[2]), tw2[2]);
            o.w = cmul_h(pack(re[3], im[3]), tw2[3]);
            *px = o;
            __builtin_amdgcn_sched_barrier(0);
        }
        // layers B and A of the second transform (per block); B is wave-local
#pragma unroll
        for (int be = 0; be < NB; ++be) {
            uint32_t v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = X[mB[j] + BLK * be];
            f4_t re, im;
            dft16(F, h8_from(v[0], v[1], v[2], v[3]), re, im);
#pragma unroll
            for (int j = 0; j < 4; ++j) X[mB[j] + BLK * be] = cmul_h(pack(re[j], im[j]), twB[j]);
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();
#pragma unroll
        for (int be = 0; be < NB; ++be) {
            uint32_t v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = X[mA + 256 * j + BLK * be];
            f4_t re, im;
            dft16(F, h8_from(v[0], v[1], v[2], v[3]), re, im);
#pragma unroll
            for (int j = 0; j < 4; ++j) X[mA + 256 * j + BLK * be] = pack(re[j], im[j]);
            __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();
        // twiddle w_32768^{p3 m} and radix 8 over p3 -> t = 4096 t3 + m, t3 < 4
        // y = Re / -Im * 2^(eu - kexp) * 256 * 64 / N, eu of the row
        const float sca = ldexpf(256.0f * 64.0f / (float)NN, eua - kexp);
        const float scb = ldexpf(256.0f * 64.0f / (float)NN, eub - kexp);
        float ya[4][4], yb[4][4];   // [t3][e]
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float2 v[NB];
#pragma unroll
            for (int p3 = 0; p3 < NB; ++p3) {
                uint32_t xv = X[mR + BLK * p3 + e];
                if (p3) xv = cmul_h(xv, twiddle_rev((4 * tid + e) * p3 + tz, NN));
                const h2_t hx = as_h2(xv);
                v[p3] = make_float2((float)hx.x, (float)hx.y);
            }
#pragma unroll
            for (int t3 = 0; t3 < 4; ++t3) {
                float wr = 0.f, wi = 0.f;
#pragma unroll
                for (int p3 = 0; p3 < NB; ++p3) {
                    const float2 wv = w8(p3 * t3);
                    wr += v[p3].x * wv.x - v[p3].y * wv.y;
                    wi += v[p3].x * wv.y + v[p3].y * wv.x;
                }
                ya[t3][e] = wr * sca;
                yb[t3][e] = -wi * scb;
            }
        }
#pragma unroll
        for (int t3 = 0; t3 < 4; ++t3) {
            const long off = BLK * t3 + 4 * tid;
            if (a.corr) {
                if (a.corr16) {
                    const uint16_t *cr = (const uint16_t *)a.corr;
                    const uint2 ca = *(const uint2 *)(cr + oa + off);
                    ya[t3][0] += lo_f<DT>(ca.x); ya[t3][1] += hi_f<DT>(ca.x);
                    ya[t3][2] += lo_f<DT>(ca.y); ya[t3][3] += hi_f<DT>(ca.y);
                    if (ob >= 0) {
                        const uint2 cb = *(const uint2 *)(cr + ob + off);
                        yb[t3][0] += lo_f<DT>(cb.x); yb[t3][1] += hi_f<DT>(cb.x);
                        yb[t3][2] += lo_f<DT>(cb.y); yb[t3][3] += hi_f<DT>(cb.y);
                    }
                } else {
                    const float *cr = (const float *)a.corr;
                    const float4 ca = *(const float4 *)(cr + oa + off);
                    ya[t3][0] += ca.x; ya[t3][1] += ca.y; ya[t3][2] += ca.z; ya[t3][3] += ca.w;
                    if (ob >= 0) {
                        const float4 cb = *(const float4 *)(cr + ob + off);
                        yb[t3][0] += cb.x; yb[t3][1] += cb.y; yb[t3][2] += cb.z; yb[t3][3] += cb.w;
                    }
                }
            }
            *(uint2 *)(y + oa + off) = make_uint2(pack_io<DT>(ya[t3][0], ya[t3][1]), pack_io<DT>(ya[t3][2], ya[t3][3]));
            if (ob >= 0)
                *(uint2 *)(y + ob + off) =
                    make_uint2(pack_io<DT>(yb[t3][0], yb[t3][1]), pack_io<DT>(yb[t3][2], yb[t3][3]));
        }
        __syncthreads();   // X is rewritten by the next pair's layer R
    }
}

bool fftconv_mfma_supported(int L, int dtype) {
    return (fftconv_wave_supported(L, dtype) || fftconv_wave16k_supported(L, dtype) || L == mf32::L) &&
           (dtype == F16 || dtype == BF16);
}

// 16-bit I/O on the matrix cores: the one-wave kernel (L = 2048), the
// four-wave kernel (L = 8192) or the 32768-point kernel here (L = 16384);
// hipErrorInvalidValue for any other shape.
hipError_t launch_fftconv_mfma(const ConvArgs &a, const float *k, hipStream_t s) {
    if (!fftconv_mfma_supported(a.L, a.dtype)) return hipErrorInvalidValue;
    if (fftconv_wave_supported(a.L, a.dtype)) return launch_fftconv_wave(a, k, s);
    if (fftconv_wave16k_supported(a.L, a.dtype)) return launch_fftconv_wave16k(a, k, s);
    int pairs_per_ch;
    if (a.pair_mode == 0)
        pairs_per_ch = (a.B + 1) / 2;
    else
        pairs_per_ch = a.B * ((a.nchunk + 1) / 2);
    // enough workgroups to fill the chip, at least 2 pairs per kernel spectrum
    int wg32 = 1;
    while (a.H * wg32 < 512 && pairs_per_ch / (2 * wg32) >= 2) wg32 *= 2;
    dim3 g32(a.H * wg32), b32(mf32::NT);
    if (a.dtype == F16)
        hipLaunchKernelGGL(fftconv_mfma32768_kernel<F16>, g32, b32, 0, s, a, k, wg32, pairs_per_ch);
    else
        hipLaunchKernelGGL(fftconv_mfma32768_kernel<BF16>, g32, b32, 0, s, a, k, wg32, pairs_per_ch);
    return hipGetLastError();
}

}  // namespace h3
