// Fused block-FFT convolution on the matrix cores (Sec. 4.1: kernel fusion +
// block FFT), gfx950, 16-bit I/O.  Transform length N = 2L = 4096 = 16^3.
//
// The DFT of a length-4096 signal is written, as in the paper's four-step
// factorisation, as three layers of length-16 DFTs (block-diagonal I (x) F_16
// products) with twiddle diagonals in between.  Each layer of 256 DFT-16s runs
// as 16 pairs of v_mfma_f32_16x16x32_f16: the 16x16 complex DFT matrix is the
// A operand (as a 16 x 32 real matrix for the real rows and one for the
// imaginary rows), 16 signal vectors are the columns of B.
//
// Index p = 256 p2 + 16 p1 + p0 of the signal held in LDS (fp16 complex per
// dword).  Forward (decimation in frequency):
//   A: DFT over p2, then * w_4096^{p2 (16 p1 + p0)}
//   B: DFT over p1, then * w_256^{p1 p0}
//   C: DFT over p0            -> position p holds X[p2 + 16 p1 + 256 p0]
// The spectrum stays in this digit-reversed order; the kernel spectrum is made
// by the same pipeline, so the pointwise product needs no permutation.  The
// second transform (conj(F(conj Y)) = N IDFT(Y)) runs the layers in reverse,
// C, * w_256^{p1 p0}, B, * w_4096^{p2 (16 p1 + p0)}, A, and ends in natural
// order.  Layer C of the first transform, the pointwise product and layer C of
// the second are fused in registers.
//
// Two rows of one channel travel as one complex signal (u_a + i u_b).  The
// zero-padded half of the input and the discarded half of the output are the
// p2 >= 8 rows of layer A.  Dynamic range: inputs are scaled by a power of two
// to max |.| in [1/2, 1), each DFT-16 layer carries a factor 1/4 (folded into
// the fp16 DFT matrix) and the kernel spectrum is normalised to max |K| in
// [1/2, 1); all scale factors are powers of two and are undone exactly in
// fp32 at the output.
//
// One workgroup (8 waves) handles a set of row pairs of one channel: it first
// transforms the channel's kernel (so the spectrum is never stored in HBM),
// keeps it in registers, then streams the pairs through the LDS buffer.
#include "common.h"
#include "fft_valu.h"
#include "internal.h"

namespace h3 {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));

namespace mf {

constexpr int N = 4096;
constexpr int L = 2048;
constexpr int NW = 8;          // waves per workgroup
constexpr int BPW = 16 / NW;   // batches per wave and layer: wave w owns 2w, 2w+1
constexpr int NT = 64 * NW;    // threads per workgroup
static_assert(BPW == 2, "address bases below assume two batches per wave");

// LDS swizzle of signal position p (dword index): bits 4-5 ^= bits 10-11 ^ bits 6-7.
// Makes the three layer access patterns (stride 1024, 64 and 16 between lane
// groups) conflict-free.
__device__ __forceinline__ int swz(int p) { return p ^ ((((p >> 10) ^ (p >> 6)) & 3) << 4); }

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

template <int DT>
__global__ __launch_bounds__(mf::NT) __attribute__((amdgpu_waves_per_eu(4))) void fftconv_mfma4096_kernel(
    ConvArgs a, const float *k, int wg_per_ch, int pairs_per_ch) {
    using namespace mf;
    __shared__ uint32_t X[N];          // signal being transformed (fp16 complex)
    __shared__ uint32_t Ub[L];         // staged rows: (a, b) raw 16-bit pairs, or k (fp32)
    __shared__ float red[2][NW];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int c = lane & 15, g = lane >> 4;
    const int blk = xcd_logical_block(blockIdx.x, gridDim.x);
    const int h = blk / wg_per_ch, part = blk % wg_per_ch;
    const int per = (pairs_per_ch + wg_per_ch - 1) / wg_per_ch;
    const int q0 = part * per, q1 = min(q0 + per, pairs_per_ch);
    int rsel = 0;

    // workgroup max |.| -> exponent e (max = m 2^e, m in [1/2, 1)); one barrier
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

    // Per-lane LDS bases (dword index; the rest of each address is an
    // immediate).  Wave w owns batches b = 2w + ib.
    //  layer A / A' / Ub:  p = 256 (4g + j) + 16 b + c  -> mA[ib] + 256 j
    //  layer B / B':       p = 256 b + 16 (4g + j) + c  -> mB[j] + 256 ib
    //  layer C:            p = 256 b + 16 c + 4g + j    -> mC + 256 ib + j
    const int s = (g ^ (w >> 1)) & 3;
    int mA[2], mB[4];
#pragma unroll
    for (int ib = 0; ib < 2; ++ib) mA[ib] = 1024 * g + 16 * ((2 * w + ib) ^ s) + c;
#pragma unroll
    for (int j = 0; j < 4; ++j) mB[j] = 512 * w + 64 * g + 16 * (j ^ s) + c;
    const int mC = 512 * w + 16 * (c ^ (((w >> 1) ^ (c >> 2)) & 3)) + 4 * g;

    // twiddles (packed fp16), fixed per lane
    uint32_t twA[2][4], twB[2][4], tw2[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        tw2[j] = twiddle_h((4 * g + j) * c, 256);
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            const int b = 2 * w + ib;
            twA[ib][j] = twiddle_h((4 * g + j) * (16 * b + c), N);
            twB[ib][j] = twiddle_h(b * (16 * (4 * g + j) + c), N);
        }
    }
    const Dft16 F = make_dft16(lane);

    // layer A from per-batch operands; outputs scaled by `sc` then twiddled
    auto layer_A = [&](const h8_t *xa, float sc) {
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            f4_t re, im;
            dft16(F, xa[ib], re, im);
#pragma unroll
            for (int j = 0; j < 4; ++j) X[mA[ib] + 256 * j] = cmul_h(pack(re[j] * sc, im[j] * sc), twA[ib][j]);
        }
        __syncthreads();
    };
    auto layer_B = [&](const uint32_t (*tw)[4]) {
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            uint32_t v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = X[mB[j] + 256 * ib];
            f4_t re, im;
            dft16(F, h8_from(v[0], v[1], v[2], v[3]), re, im);
#pragma unroll
            for (int j = 0; j < 4; ++j) X[mB[j] + 256 * ib] = cmul_h(pack(re[j], im[j]), tw[ib][j]);
        }
        __syncthreads();
    };
    const uint32_t tw2b[2][4] = {{tw2[0], tw2[1], tw2[2], tw2[3]}, {tw2[0], tw2[1], tw2[2], tw2[3]}};

    // ---- kernel spectrum of channel h ----
    uint32_t K[2][4];  // fp16 complex, holds F(k) 2^kexp
    int kexp;
    {
        const float4 k0 = ((const float4 *)(k + (long)h * L))[tid];
        const float mx = fmaxf(fmaxf(fabsf(k0.x), fabsf(k0.y)), fmaxf(fabsf(k0.z), fabsf(k0.w)));
        *(uint4 *)&Ub[swz(4 * tid)] = make_uint4(__float_as_uint(k0.x), __float_as_uint(k0.y),
                                                 __float_as_uint(k0.z), __float_as_uint(k0.w));
        const int ek = bexp(mx);   // also publishes Ub
        h8_t xa[2];
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            if (g < 2) {
#pragma unroll
                for (int i = 0; i < 4; ++i) v[i] = pack(ldexpf(__uint_as_float(Ub[mA[ib] + 256 * i]), -ek), 0.f);
            }
            xa[ib] = h8_from(v[0], v[1], v[2], v[3]);
        }
        layer_A(xa, 1.0f);
        layer_B(tw2b);
        float Kf[2][4][2];
        float km = 0.f;
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            const uint4 v = *(const uint4 *)&X[mC + 256 * ib];
            f4_t re, im;
            dft16(F, __builtin_bit_cast(h8_t, v), re, im);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                Kf[ib][j][0] = re[j];
                Kf[ib][j][1] = im[j];
                km = fmaxf(km, fmaxf(fabsf(re[j]), fabsf(im[j])));
            }
        }
        const int e2 = bexp(km);
#pragma unroll
        for (int ib = 0; ib < 2; ++ib)
#pragma unroll
            for (int j = 0; j < 4; ++j) K[ib][j] = pack(ldexpf(Kf[ib][j][0], -e2), ldexpf(Kf[ib][j][1], -e2));
        kexp = -ek - 6 - e2;
    }

    const float d = a.D ? a.D[h] : 0.f;
    const uint16_t *u = (const uint16_t *)a.u;
    uint16_t *y = (uint16_t *)a.y;
    auto rows = [&](int qq, long &oa, long &ob) {
        if (a.pair_mode == 0) {
            oa = ((long)(2 * qq) * a.H + h) * L;
            ob = (2 * qq + 1 < a.B) ? ((long)(2 * qq + 1) * a.H + h) * L : -1;
        } else {
            const int ncp = (a.nchunk + 1) / 2;
            const int bb = qq / ncp, cp = qq % ncp;
            oa = (((long)bb * a.H + h) * a.nchunk + 2 * cp) * L;
            ob = (2 * cp + 1 < a.nchunk) ? oa + L : -1;
        }
    };
    const int ubase = swz(4 * tid);    // this thread's staged elements 4 tid .. 4 tid + 3
    // coalesced loads: thread tid owns elements 4 tid .. 4 tid + 3 of both rows
    uint2 pa = make_uint2(0, 0), pb = make_uint2(0, 0);
    if (q0 < q1) {
        long oa, ob;
        rows(q0, oa, ob);
        pa = *(const uint2 *)(u + oa + 4 * tid);
        if (ob >= 0) pb = *(const uint2 *)(u + ob + 4 * tid);
    }
    for (int qq = q0; qq < q1; ++qq) {
        long oa, ob;
        rows(qq, oa, ob);
        // stage raw (a, b) pairs in Ub, max |u|
        const uint4 st = make_uint4(__builtin_amdgcn_perm(pb.x, pa.x, 0x05040100u),
                                    __builtin_amdgcn_perm(pb.x, pa.x, 0x07060302u),
                                    __builtin_amdgcn_perm(pb.y, pa.y, 0x05040100u),
                                    __builtin_amdgcn_perm(pb.y, pa.y, 0x07060302u));
        float mx = 0.f;
        mx = fmaxf(mx, fmaxf(fabsf(lo_f<DT>(st.x)), fabsf(hi_f<DT>(st.x))));
        mx = fmaxf(mx, fmaxf(fabsf(lo_f<DT>(st.y)), fabsf(hi_f<DT>(st.y))));
        mx = fmaxf(mx, fmaxf(fabsf(lo_f<DT>(st.z)), fabsf(hi_f<DT>(st.z))));
        mx = fmaxf(mx, fmaxf(fabsf(lo_f<DT>(st.w)), fabsf(hi_f<DT>(st.w))));
        *(uint4 *)&Ub[ubase] = st;
        // prefetch the next pair
        if (qq + 1 < q1) {
            long na, nb;
            rows(qq + 1, na, nb);
            pa = *(const uint2 *)(u + na + 4 * tid);
            pb = (nb >= 0) ? *(const uint2 *)(u + nb + 4 * tid) : make_uint2(0, 0);
        }
        const int eu = bexp(mx);
        h8_t xa[2];
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            uint32_t v[4] = {0u, 0u, 0u, 0u};
            if (g < 2) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const uint32_t r = Ub[mA[ib] + 256 * i];
                    if (DT == F16)
                        v[i] = r;    // fp16 pairs are the operand as they are
                    else
                        v[i] = pack(ldexpf(lo_f<DT>(r), -eu), ldexpf(hi_f<DT>(r), -eu));
                }
            }
            xa[ib] = h8_from(v[0], v[1], v[2], v[3]);
        }
        layer_A(xa, DT == F16 ? ldexpf(1.0f, -eu) : 1.0f);
        layer_B(tw2b);
        // layer C forward, pointwise product, layer C of the second transform
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            uint4 *px = (uint4 *)&X[mC + 256 * ib];
            f4_t re, im;
            dft16(F, __builtin_bit_cast(h8_t, *px), re, im);
            uint32_t yv[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) yv[j] = cmul_h(pack(re[j], im[j]), K[ib][j]) ^ 0x80000000u;  // conj(X K)
            dft16(F, h8_from(yv[0], yv[1], yv[2], yv[3]), re, im);
            // w_256^{p1 p0} with p1 = c, p0 = 4g + j: same values as tw2
            uint4 o;
            o.x = cmul_h(pack(re[0], im[0]), tw2[0]);
            o.y = cmul_h(pack(re[1], im[1]), tw2[1]);
            o.z = cmul_h(pack(re[2], im[2]), tw2[2]);
            o.w = cmul_h(pack(re[3], im[3]), tw2[3]);
            *px = o;
        }
        __syncthreads();
        layer_B(twB);
        // layer A of the second transform -> natural order; t < L kept.
        // y = Re / -Im of w * 2^(eu - kexp) * 64^2 / N  (input scale, kernel
        // scale and the two 1/64 layer factors undone; 1/N of the inverse)
        const float sc = ldexpf(64.0f * 64.0f / (float)N, eu - kexp);
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            uint32_t v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = X[mA[ib] + 256 * j];
            f4_t re, im;
            dft16(F, h8_from(v[0], v[1], v[2], v[3]), re, im);
            if (g < 2) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint32_t r = Ub[mA[ib] + 256 * j];
                    float ya = fmaf(re[j], sc, d * lo_f<DT>(r));
                    float yb = fmaf(-im[j], sc, d * hi_f<DT>(r));
                    if (a.corr) {
                        const int t = 256 * (4 * g + j) + 16 * (2 * w + ib) + c;
                        ya += a.corr[oa + t];
                        if (ob >= 0) yb += a.corr[ob + t];
                    }
                    Ub[mA[ib] + 256 * j] = pack_io<DT>(ya, yb);
                }
            }
        }
        __syncthreads();
        {
            const uint4 v = *(const uint4 *)&Ub[ubase];
            uint2 oa2, ob2;
            oa2.x = __builtin_amdgcn_perm(v.y, v.x, 0x05040100u);
            oa2.y = __builtin_amdgcn_perm(v.w, v.z, 0x05040100u);
            ob2.x = __builtin_amdgcn_perm(v.y, v.x, 0x07060302u);
            ob2.y = __builtin_amdgcn_perm(v.w, v.z, 0x07060302u);
            *(uint2 *)(y + oa + 4 * tid) = oa2;
            if (ob >= 0) *(uint2 *)(y + ob + 4 * tid) = ob2;
        }
        // the next pair rewrites Ub only after its own barrier in bexp
    }
}

bool fftconv_mfma_supported(int L, int dtype) { return L == mf::L && (dtype == F16 || dtype == BF16); }

// Launch over all channels; returns hipErrorInvalidValue if the shape is not
// handled here (N != 4096 or 32-bit I/O).
hipError_t launch_fftconv_mfma(const ConvArgs &a, const float *k, hipStream_t s) {
    if (a.L != mf::L || (a.dtype != F16 && a.dtype != BF16)) return hipErrorInvalidValue;
    int pairs_per_ch;
    if (a.pair_mode == 0)
        pairs_per_ch = (a.B + 1) / 2;
    else
        pairs_per_ch = a.B * ((a.nchunk + 1) / 2);
    // enough workgroups to fill the chip, at least 2 pairs per kernel spectrum
    int wg_per_ch = 1;
    while (a.H * wg_per_ch < 2048 && pairs_per_ch / (2 * wg_per_ch) >= 2) wg_per_ch *= 2;
    dim3 grid(a.H * wg_per_ch), block(mf::NT);
    if (a.dtype == F16)
        hipLaunchKernelGGL(fftconv_mfma4096_kernel<F16>, grid, block, 0, s, a, k, wg_per_ch, pairs_per_ch);
    else
        hipLaunchKernelGGL(fftconv_mfma4096_kernel<BF16>, grid, block, 0, s, a, k, wg_per_ch, pairs_per_ch);
    return hipGetLastError();
}

}  // namespace h3
