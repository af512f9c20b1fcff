// Register-resident block-FFT building blocks shared by the one-wavefront-
// per-transform convolution kernels (gfx950, wave64).
//
// A wavefront holds a length-4096 complex signal (packed fp16) in registers:
// lane l = 16 g + c keeps d[4 T + j], T = 0..15, j = 0..3.  A radix-16 layer
// contracts the base-16 digit in slot G = 4 g + j with pairs of
// v_mfma_f32_16x16x32_f16 (real and imaginary rows of the DFT-16 matrix).
// With the signal as the A operand the output frequency lands in slot C = c
// and the digit that was in C moves to G; with the signal as the B operand
// the frequency stays in G.  swap_GT exchanges slot G with the tile slot T
// in registers.  The compile-time tables hold the L2 twiddles w_4096 (per
// tile and lane) and the per-lane DFT-16 rows and L1 twiddles in fp16.
#pragma once
#include "common.h"

namespace h3 {
namespace wvc {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef float f2_t __attribute__((ext_vector_type(2)));
typedef __bf16 b2_t __attribute__((ext_vector_type(2)));

constexpr int kN = 4096;   // block transform length 16^3

// ------------------------------------------------- twiddle table (constant) --
// w_4096^n = exp(-2 pi i n / 4096) for n < 4096, as float (re, im), evaluated
// at compile time: the first quadrant from Taylor series of sin and cos on
// [0, pi/4] (argument reduction by the octant symmetry), the other quadrants
// by rotation by -i.
struct Cf {
    float re, im;
};
struct TwTable {
    Cf v[kN];
};
constexpr double cx_sin_small(double x) {  // |x| <= pi/4
    double t = x, s = x;
    for (int k = 1; k < 14; ++k) {
        t *= -x * x / ((2.0 * k) * (2.0 * k + 1.0));
        s += t;
    }
    return s;
}
constexpr double cx_cos_small(double x) {
    double t = 1.0, s = 1.0;
    for (int k = 1; k < 14; ++k) {
        t *= -x * x / ((2.0 * k - 1.0) * (2.0 * k));
        s += t;
    }
    return s;
}
constexpr TwTable make_tw_table() {
    TwTable t{};
    const double step = 6.283185307179586476925286766559 / kN;
    for (int n = 0; n <= kN / 8; ++n) {  // angle in [0, pi/4]
        const double c = cx_cos_small(n * step), s = cx_sin_small(n * step);
        t.v[n] = Cf{(float)c, (float)-s};
        // angle pi/2 - x: cos <-> sin
        t.v[kN / 4 - n] = Cf{(float)s, (float)-c};
    }
    for (int n = kN / 4; n < kN; ++n) {  // w^n = -i w^(n - kN/4)
        const Cf p = t.v[n - kN / 4];
        t.v[n] = Cf{p.im, -p.re};
    }
    return t;
}
// IEEE binary16 bits of x, round to nearest even (|x| < 65504, no NaN / inf).
constexpr uint32_t h16_bits(double x) {
    uint32_t sign = x < 0 ? 0x8000u : 0u;
    double a = x < 0 ? -x : x;
    if (a < 5.9604644775390625e-08 * 0.5) return sign;   // rounds to zero
    int e = 0;
    while (a >= 2.0) { a *= 0.5; ++e; }
    while (a < 1.0) { a *= 2.0; --e; }
    if (e < -14) {   // subnormal: multiple of 2^-24
        double m = a;
        for (int i = e; i < -24; ++i) m *= 0.5;
        for (int i = -24; i < e; ++i) m *= 2.0;
        const double fl = (double)(long long)m;
        double r = m - fl;
        long long q = (long long)fl;
        if (r > 0.5 || (r == 0.5 && (q & 1))) ++q;
        return sign | (uint32_t)q;
    }
    const double m = (a - 1.0) * 1024.0;
    long long q = (long long)m;
    const double r = m - (double)q;
    if (r > 0.5 || (r == 0.5 && (q & 1))) ++q;
    if (q == 1024) { q = 0; ++e; }
    return sign | ((uint32_t)(e + 15) << 10) | (uint32_t)q;
}
constexpr uint32_t h2_bits(double re, double im) { return h16_bits(re) | (h16_bits(im) << 16); }

// The same tables in fp16 and in LDS order, staged with LDS-direct loads:
//   [0, 1024)      Ytab[T * 64 + l]: the four L2 twiddles of tile T, lane l
//   [1024, 1408)   Lc[kind * 64 + l]: DFT rows (real, imaginary), conjugate
//                  DFT rows, L1 twiddles w and (-im w, re w)
constexpr int kTabY = 1024, kTabLc = 384, kTab = kTabY + kTabLc;   // in uint4
struct HalfTable {
    uint32_t v[4 * kTab];
};
constexpr HalfTable make_half_table() {
    const TwTable t = make_tw_table();
    HalfTable h{};
    for (int T = 0; T < 16; ++T)
        for (int l = 0; l < 64; ++l)
            for (int j = 0; j < 4; ++j) {
                const Cf w = t.v[(T * ((l & 15) + 16 * (4 * (l >> 4) + j))) & (kN - 1)];
                h.v[(T * 64 + l) * 4 + j] = h2_bits(w.re, w.im);
            }
    for (int l = 0; l < 64; ++l)
        for (int i = 0; i < 4; ++i) {
            const Cf w = t.v[(256 * (4 * (l >> 4) + i) * (l & 15)) & (kN - 1)];
            const double re = 0.25 * w.re, im = 0.25 * w.im;
            // out.re = sum re(w) x.re - im(w) x.im ; out.im = sum im(w) x.re + re(w) x.im
            h.v[4 * (kTabY + 0 * 64 + l) + i] = h2_bits(re, -im);
            h.v[4 * (kTabY + 1 * 64 + l) + i] = h2_bits(im, re);
            h.v[4 * (kTabY + 2 * 64 + l) + i] = h2_bits(re, im);    // conjugate
            h.v[4 * (kTabY + 3 * 64 + l) + i] = h2_bits(-im, re);
            const Cf x = t.v[(16 * (l & 15) * (4 * (l >> 4) + i)) & (kN - 1)];
            h.v[4 * (kTabY + 4 * 64 + l) + i] = h2_bits(x.re, x.im);
            h.v[4 * (kTabY + 5 * 64 + l) + i] = h2_bits(-x.im, x.re);
        }
    return h;
}
// exp(-2 pi i n / nn) in double, any integer n (nn a multiple of 8)
struct Cd {
    double re, im;
};
constexpr Cd cwd(long n, long nn) {
    n %= nn;
    if (n < 0) n += nn;
    const long q4 = nn / 4, q = n / q4, r = n % q4;
    const double step = 6.283185307179586476925286766559 / (double)nn;
    double c = 0, s = 0;   // cos, sin of 2 pi r / nn, r < nn / 4
    if (2 * r <= q4) {
        c = cx_cos_small(r * step);
        s = cx_sin_small(r * step);
    } else {
        c = cx_sin_small((q4 - r) * step);
        s = cx_cos_small((q4 - r) * step);
    }
    Cd v{c, -s};
    for (long i = 0; i < q; ++i) v = Cd{v.im, -v.re};   // times -i
    return v;
}

typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

// ---------------------------------------------------------- small helpers ---
__device__ __forceinline__ h2_t as_h2(uint32_t v) { return __builtin_bit_cast(h2_t, v); }
__device__ __forceinline__ uint32_t as_u32(h2_t v) { return __builtin_bit_cast(uint32_t, v); }
// (re, im) fp32 -> packed fp16, round to nearest even
__device__ __forceinline__ uint32_t pk(float re, float im) {
    const f2_t v = {re, im};
    return as_u32(__builtin_convertvector(v, h2_t));
}
// a * w and a * conj(w) in packed fp16.  The empty asm makes w an opaque
// register value, so that both products take the half selections and the
// sign as VOP3P operand modifiers; otherwise the first element of a 128-bit
// LDS read has (-w.im, w.re) built by two extra VALU instructions.
__device__ __forceinline__ uint32_t cmul(uint32_t a_, uint32_t w_) {
    asm("" : "+v"(w_));
    const h2_t a = as_h2(a_), w = as_h2(w_);
    const h2_t t = a.xx * w;
    const h2_t ws = {-w.y, w.x};
    return as_u32(a.yy * ws + t);
}
// a * w with ws = (-w.im, w.re) supplied (loop-invariant twiddles)
__device__ __forceinline__ uint32_t cmul2(uint32_t a_, uint32_t w_, uint32_t ws_) {
    const h2_t a = as_h2(a_);
    const h2_t t = a.xx * as_h2(w_);
    return as_u32(a.yy * as_h2(ws_) + t);
}
// a * conj(w) with ws = (-w.im, w.re): (ar wr + ai wi, ai wr - ar wi)
__device__ __forceinline__ uint32_t cmulc2(uint32_t a_, uint32_t w_, uint32_t ws_) {
    const h2_t a = as_h2(a_), w = as_h2(w_), ws = as_h2(ws_);
    const h2_t t = a.yy * w;                 // (ai wr, ai wi)
    const h2_t u2 = {ws.y, ws.x};            // (wr, -wi)
    return as_u32(a.xx * u2 + t.yx);         // (ar wr + ai wi, -ar wi + ai wr)
}
__device__ __forceinline__ uint32_t cmulc(uint32_t a_, uint32_t w_) {
    asm("" : "+v"(w_));
    const h2_t a = as_h2(a_), w = as_h2(w_);
    const h2_t wc = {w.x, -w.y};
    const h2_t t = a.xx * wc;
    const h2_t ws = {w.y, w.x};
    return as_u32(a.yy * ws + t);
}
__device__ __forceinline__ h8_t h8_of(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
    return __builtin_bit_cast(h8_t, make_uint4(a, b, c, d));
}
__device__ __forceinline__ f4_t mfma(h8_t a, h8_t b) {
    const f4_t z = {0.f, 0.f, 0.f, 0.f};
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, z, 0, 0, 0);
}
// Maximum over the wavefront, returned wave-uniform: xor-swizzles within
// each half (immediate patterns, no lane-address registers), then the two
// halves' results read as scalars.
template <int XOR> __device__ __forceinline__ float swz_xor(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(__builtin_bit_cast(int, v), (XOR << 10) | 0x1F));
}
__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, swz_xor<1>(v));
    v = fmaxf(v, swz_xor<2>(v));
    v = fmaxf(v, swz_xor<4>(v));
    v = fmaxf(v, swz_xor<8>(v));
    v = fmaxf(v, swz_xor<16>(v));
    const float lo = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 0));
    const float hi = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), 32));
    return fmaxf(lo, hi);
}
// exponent e with max = m 2^e, m in [1/2, 1); 0 for 0 / non-finite
__device__ __forceinline__ int exp_of(float m) {
    if (!(m > 0.f) || !(m < 3.0e38f)) return 0;
    int e;
    frexpf(m, &e);
    return e;
}

// 16x16 DFT (entries / 4) as the lane's 8 halves: point i = h / 2 of the
// K range 4 g .. 4 g + 3, frequency c; the same values serve as A operand
// (rows = frequency) and as B operand (columns = frequency).
struct Dft {
    h8_t re, im;
};

// Position of tile T's output jj after L2: "P layout".  The G <-> T swap
// then leaves every L3 tile's four points in four consecutive registers.
__device__ __forceinline__ constexpr int pidx(int T, int jj) { return 16 * (T >> 2) + 4 * jj + (T & 3); }

template <bool SIG_A>
__device__ __forceinline__ void quad_mfma(const uint32_t *q, const Dft &F, f4_t &re, f4_t &im) {
    h8_t x = h8_of(q[0], q[1], q[2], q[3]);
    // The empty volatile asm keeps the MFMAs of a tile after the previous
    // tile's sched_barrier: the intrinsics themselves are pure, and the IR
    // passes would otherwise hoist a whole layer's MFMAs to its start.
    asm volatile("" : "+v"(x));
    if constexpr (SIG_A) {
        re = mfma(x, F.re);
        im = mfma(x, F.im);
    } else {
        re = mfma(F.re, x);
        im = mfma(F.im, x);
    }
}
// One radix-16 layer over slot G on the NQ register quads d[4 tau .. 4 tau + 3].
// Software-pipelined: the MFMAs of quad tau + 1 (and the LDS operand
// pre(tau + 1) of its epilogue) are issued before the epilogue of quad tau,
// and the scheduler may not hoist further (which would keep all 32 results
// live).  epi(tau, re, im, p) gets the fp32 outputs of quad tau (frequency /
// row 4 g + jj in element jj) and p = pre(tau).
struct NoPre {
    __device__ __forceinline__ uint4 operator()(int) const { return make_uint4(0, 0, 0, 0); }
};
template <bool SIG_A, int NQ = 16, class Pre, class Epi>
__device__ __forceinline__ void layer(uint32_t *d, const Dft &F, Pre &&pre, Epi &&epi) {
    f4_t re, im;
    quad_mfma<SIG_A>(d, F, re, im);
    uint4 pv = pre(0);
#pragma unroll
    for (int tau = 0; tau < NQ; ++tau) {
        f4_t re1, im1;
        uint4 pv1 = make_uint4(0, 0, 0, 0);
        if (tau + 1 < NQ) {
            quad_mfma<SIG_A>(d + 4 * (tau + 1), F, re1, im1);
            pv1 = pre(tau + 1);
        }
        epi(tau, re, im, pv);
        __builtin_amdgcn_sched_barrier(0);
        re = re1;
        im = im1;
        pv = pv1;
    }
}

// The same layer with the MFMAs of quads tau + 1 and tau + 2 in flight during
// the epilogue of quad tau.
template <bool SIG_A, int NQ = 16, class Pre, class Epi>
__device__ __forceinline__ void layer2(uint32_t *d, const Dft &F, Pre &&pre, Epi &&epi) {
    f4_t re0, im0, re1, im1;
    quad_mfma<SIG_A>(d, F, re0, im0);
    quad_mfma<SIG_A>(d + 4, F, re1, im1);
    uint4 pv0 = pre(0), pv1 = pre(1);
#pragma unroll
    for (int tau = 0; tau < NQ; ++tau) {
        f4_t re2, im2;
        uint4 pv2 = make_uint4(0, 0, 0, 0);
        if (tau + 2 < NQ) {
            quad_mfma<SIG_A>(d + 4 * (tau + 2), F, re2, im2);
            pv2 = pre(tau + 2);
        }
        epi(tau, re0, im0, pv0);
        __builtin_amdgcn_sched_barrier(0);
        re0 = re1; im0 = im1; pv0 = pv1;
        re1 = re2; im1 = im2; pv1 = pv2;
    }
}

// Exchange slot G's lane-row bits (lane bits 5, 4) with register-index bits
// 5, 4.  An involution.
__device__ __forceinline__ void swap_GT(uint32_t (&d)[64]) {
#pragma unroll
    for (int r = 0; r < 32; ++r) {
        const auto s = __builtin_amdgcn_permlane32_swap(d[r], d[r + 32], false, false);
        d[r] = s[0];
        d[r + 32] = s[1];
    }
#pragma unroll
    for (int r = 0; r < 64; ++r) {
        if (r & 16) continue;
        const auto s = __builtin_amdgcn_permlane16_swap(d[r], d[r + 16], false, false);
        d[r] = s[0];
        d[r + 16] = s[1];
    }
}

// s_waitcnt encoding (gfx9): vmcnt <= 16, lgkmcnt and expcnt unconstrained
constexpr int kWaitVm16 = 0x4F70;
constexpr int kWaitVm8 = 0x0F78;   // vmcnt <= 8
constexpr int kWaitVm0 = 0x0F70;   // vmcnt = 0

// Per-lane constants staged in LDS (Lc[kind * 64 + lane]): 0/1 DFT real /
// imaginary rows, 2/3 the conjugate DFT, 4 the L1 twiddles w_256^{c (4g+j)},
// 5 the same as (-im, re).  Read right before each layer so that they do not
// occupy registers across the pair pipeline.
__device__ __forceinline__ Dft lds_dft(const uint4 *Lc, int lane, bool conj) {
    asm volatile("" ::: "memory");   // re-read per layer, do not keep live
    Dft F;
    F.re = __builtin_bit_cast(h8_t, Lc[(conj ? 2 : 0) * 64 + lane]);
    F.im = __builtin_bit_cast(h8_t, Lc[(conj ? 3 : 1) * 64 + lane]);
    return F;
}


// 16-bit I/O helpers
template <int DT> __device__ __forceinline__ uint32_t pack_out(float lo, float hi);
template <> __device__ __forceinline__ uint32_t pack_out<F16>(float lo, float hi) { return pk(lo, hi); }
template <> __device__ __forceinline__ uint32_t pack_out<BF16>(float lo, float hi) {
    const f2_t v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, b2_t));
}
template <int DT> __device__ __forceinline__ float lo_f(uint32_t r) {
    return DT == F16 ? (float)as_h2(r).x : __uint_as_float(r << 16);
}
template <int DT> __device__ __forceinline__ float hi_f(uint32_t r) {
    return DT == F16 ? (float)as_h2(r).y : __uint_as_float(r & 0xffff0000u);
}
__device__ __forceinline__ h8_t h8_scale(h8_t v, _Float16 s) {
    const h8_t sv = {s, s, s, s, s, s, s, s};
    return v * sv;
}


// ------------------------------------------------- multi-wave kernels ---
// Shared by the kernels that split one transform over several wavefronts.
typedef __bf16 bf8_t __attribute__((ext_vector_type(8)));
typedef unsigned short us2_t __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------ derived rows --
// A DFT-row pair (R, I) from a base imaginary row b (entries (Im w, Re w))
// with every point multiplied by f[i]: I' = (Im w f, Re w f), R' = (Re w f,
// -Im w f).  Covers a scaled contraction side (f per point) and a scaled
// output row (the same f for all points).
__device__ __forceinline__ void kinds_scaled(uint4 b4, const uint32_t (&f)[4], uint32_t (&R)[4],
                                             uint32_t (&I)[4]) {
    const uint32_t b[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const h2_t bb = as_h2(b[i]), ff = as_h2(f[i]);
        const h2_t fs = {ff.y, ff.x}, fn = {ff.x, -ff.y};
        const h2_t ii = bb.yy * fs + bb.xx * fn;
        const h2_t rr = {ii.y, -ii.x};
        I[i] = as_u32(ii);
        R[i] = as_u32(rr);
    }
}
__device__ __forceinline__ Dft dft_of(const uint32_t (&R)[4], const uint32_t (&I)[4]) {
    Dft F;
    F.re = h8_of(R[0], R[1], R[2], R[3]);
    F.im = h8_of(I[0], I[1], I[2], I[3]);
    return F;
}
// (-i)^k3 times a DFT-row pair: k3 = 0: (R, I); 1: (I, -R); 2: (-R, -I); 3: (-I, R)
__device__ __forceinline__ void kinds_rot(int k3, const uint32_t (&R)[4], const uint32_t (&I)[4],
                                          uint32_t (&Rb)[4], uint32_t (&Ib)[4]) {
    const bool sw = (k3 & 1) != 0;
    const uint32_t nr = k3 >= 2 ? 0x80008000u : 0u;
    const uint32_t ni = (k3 == 1 || k3 == 2) ? 0x80008000u : 0u;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        Rb[i] = (sw ? I[i] : R[i]) ^ nr;
        Ib[i] = (sw ? R[i] : I[i]) ^ ni;
    }
}
// the same four rows as bf16, the entries that multiply the real half of a
// point (row a) times sa, those that multiply the imaginary half (row b)
// times sb
__device__ __forceinline__ void kinds_bf16(const uint32_t (&R)[4], const uint32_t (&I)[4], float sa, float sb,
                                           bf8_t &Rb, bf8_t &Ib) {
    float r[8], im[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        r[2 * i] = (float)as_h2(R[i]).x * sa;
        r[2 * i + 1] = (float)as_h2(R[i]).y * sb;
        im[2 * i] = (float)as_h2(I[i]).x * sa;
        im[2 * i + 1] = (float)as_h2(I[i]).y * sb;
    }
    typedef float f8_t __attribute__((ext_vector_type(8)));
    const f8_t vr = {r[0], r[1], r[2], r[3], r[4], r[5], r[6], r[7]};
    const f8_t vi = {im[0], im[1], im[2], im[3], im[4], im[5], im[6], im[7]};
    Rb = __builtin_convertvector(vr, bf8_t);
    Ib = __builtin_convertvector(vi, bf8_t);
}

__device__ __forceinline__ f4_t mfma_acc(h8_t a, h8_t b, f4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f4_t mfma_acc(bf8_t a, bf8_t b, f4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Second layer (signal B) + L2 twiddles into P layout, then the G <-> T swap.
template <bool P2 = false>
__device__ __forceinline__ void forward_mid(uint32_t (&d)[64], const uint4 *Lc, const uint4 *Ytab, int lane) {
    uint32_t e[64];
    const Dft F = lds_dft(Lc, lane, false);
    auto pre = [&](int tau) { return Ytab[tau * 64 + lane]; };
    auto run = [&](auto &&epi) {
        if constexpr (P2) layer2<false>(d, F, pre, epi);
        else layer<false>(d, F, pre, epi);
    };
    run(
                 [&](int tau, f4_t re, f4_t im, uint4 y) {
                     e[pidx(tau, 0)] = cmul(pk(re[0], im[0]), y.x);
                     e[pidx(tau, 1)] = cmul(pk(re[1], im[1]), y.y);
                     e[pidx(tau, 2)] = cmul(pk(re[2], im[2]), y.z);
                     e[pidx(tau, 3)] = cmul(pk(re[3], im[3]), y.w);
                 });
#pragma unroll
    for (int i = 0; i < 64; ++i) d[i] = e[i];
    swap_GT(d);
}

// Lane twiddles of the first layer (X = base w_256 times the wave's w_1024
// factor) and of the inverse second layer (conj(base) times w_1024^{-k3 c}),
// each with its (-im, re) companion for cmul2.
__device__ __forceinline__ void twiddles_fwd(uint4 X, const uint32_t (&xf)[4], uint32_t (&xw)[4],
                                             uint32_t (&xs)[4]) {
    const uint32_t b[4] = {X.x, X.y, X.z, X.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const h2_t v = as_h2(cmul(b[j], xf[j]));
        const h2_t s = {-v.y, v.x};
        xw[j] = as_u32(v);
        xs[j] = as_u32(s);
    }
}
__device__ __forceinline__ void twiddles_inv(uint4 X, uint32_t xh, uint32_t (&xw)[4], uint32_t (&xs)[4]) {
    const uint32_t b[4] = {X.x, X.y, X.z, X.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const h2_t v = as_h2(cmulc(xh, b[j]));
        const h2_t s = {-v.y, v.x};
        xw[j] = as_u32(v);
        xs[j] = as_u32(s);
    }
}

// Maximum |.| of 16-bit raw values (both halves of each dword)
template <int DT> __device__ __forceinline__ float raw_max(const uint4 (&ra)[4]);
template <> __device__ __forceinline__ float raw_max<F16>(const uint4 (&ra)[4]) {
    h2_t hmx = {0, 0}, hmn = {0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t v[4] = {ra[i].x, ra[i].y, ra[i].z, ra[i].w};
#pragma unroll
        for (int e = 0; e < 4; e += 2) {
            hmx = __builtin_elementwise_maximum(hmx, __builtin_elementwise_maximum(as_h2(v[e]), as_h2(v[e + 1])));
            hmn = __builtin_elementwise_minimum(hmn, __builtin_elementwise_minimum(as_h2(v[e]), as_h2(v[e + 1])));
        }
    }
    return fmaxf(fmaxf((float)hmx.x, (float)hmx.y), fmaxf(-(float)hmn.x, -(float)hmn.y));
}
template <> __device__ __forceinline__ float raw_max<BF16>(const uint4 (&ra)[4]) {
    us2_t mb = {0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t v[4] = {ra[i].x, ra[i].y, ra[i].z, ra[i].w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
            mb = __builtin_elementwise_max(mb, __builtin_bit_cast(us2_t, v[e] & 0x7fff7fffu));
    }
    const uint32_t m = max((uint32_t)mb.x, (uint32_t)mb.y);
    return __uint_as_float(m << 16);
}


// Fused initial-state term of state passing (Sec. 4.2: the M_xy x term of a
// chunk, chunk 8192 or 16384): for the wave's 4096 outputs t in [4096 qa,
// + 4096) of a chunk row, with
// t = 64 a + b,  corr(t) = 2 Re sum_n Abar_n^b V_n(a),  V_n(a) = W_n Abar_n^{64 a},
// as 16 tiles D[b][a] of 16 x 16 on the matrix cores (K = 64 modes as (re, im)
// pairs): the A operand Abar_n^b comes from the per-channel table in LDS, the
// B operand V from the row's weights W (normalised to max |W| in [1/2, 1),
// fp16) times Abar_n^{64 a}, stepping a by 16 with Abar_n^1024.  The table
// holds Abar_n^{64 a} for a in [0, 128); quarters qa = 2, 3 (chunk 16384)
// take them times Abar_n^8192.  A lane ends up with four consecutive t: they
// are added in fp32 to the outputs staged in U (rows of ROWU2 uint2, this
// row at index row) and stored as 8 bytes.
// The per-channel table CT (CORR_TAB_U4 uint4, written by the state-passing
// tables kernel): [0, 1024) Abar_n^b as A operands, [1024, 1536)
// Abar_n^{64 a}, [1536, 1552) Abar_n^1024, [1552, 1568) Abar_n^8192.
// The sum itself: out(t, D) receives D[jj] = Re sum_n Abar_n^b V_n(a) for the
// four consecutive t .. t + 3 of tile (jb, ib) (BIG: quarters qa = 2, 3 exist).
template <bool BIG, class Out>
__device__ __forceinline__ void state_term_core(const uint4 *CT, const uint4 (&wq)[4], int qa, int lane, Out &&out) {
    const int g = lane >> 4, c = lane & 15;
    const uint4 *CA = CT, *T64 = CT + 1024, *Zt = CT + 1536;
    // wq[kb]: normalised W of modes 16 kb + 4 g + q in dword q
    uint32_t V[16];   // [4 kb + q]: (Re V, -Im V) of mode 16 kb + 4 g + q, column a = 64 qa + c
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        uint4 tq = T64[((qa & 1) * 4 + kb) * 64 + lane];
        if (BIG && qa >= 2) {   // wave-uniform
            const uint4 z8 = Zt[16 + kb * 4 + g];
            tq = make_uint4(cmul(tq.x, z8.x), cmul(tq.y, z8.y), cmul(tq.z, z8.z), cmul(tq.w, z8.w));
        }
        // conj(V) = conj(W) conj(Abar^{64 a}), stored (Re V, -Im V)
        V[4 * kb + 0] = cmulc(wq[kb].x ^ 0x80000000u, tq.x);
        V[4 * kb + 1] = cmulc(wq[kb].y ^ 0x80000000u, tq.y);
        V[4 * kb + 2] = cmulc(wq[kb].z ^ 0x80000000u, tq.z);
        V[4 * kb + 3] = cmulc(wq[kb].w ^ 0x80000000u, tq.w);
    }
    const f4_t z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jb = 0; jb < 4; ++jb) {
        if (jb > 0) {
            // a += 16: V <- V Abar^1024, i.e. the stored conj(V) times conj(Abar^1024)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                const uint4 zq = Zt[kb * 4 + g];
                V[4 * kb + 0] = cmulc(V[4 * kb + 0], zq.x);
                V[4 * kb + 1] = cmulc(V[4 * kb + 1], zq.y);
                V[4 * kb + 2] = cmulc(V[4 * kb + 2], zq.z);
                V[4 * kb + 3] = cmulc(V[4 * kb + 3], zq.w);
            }
        }
#pragma unroll
        for (int ib = 0; ib < 4; ++ib) {
            f4_t D = z;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
                D = mfma_acc(__builtin_bit_cast(h8_t, CA[(ib * 4 + kb) * 64 + lane]),
                             h8_of(V[4 * kb], V[4 * kb + 1], V[4 * kb + 2], V[4 * kb + 3]), D);
            // rows b = 16 ib + 4 g + jj, column a = 64 qa + 16 jb + c
            out(4096 * qa + 1024 * jb + 64 * c + 16 * ib + 4 * g, D);
        }
    }
}
template <int DT, int ROWU2>
__device__ __forceinline__ void fused_state_term(const uint4 *U, const uint4 *CT, const uint4 (&wq)[4], int ew,
                                                 int row, int qa, int lane, uint16_t *yrow) {
    const float scorr = ldexpf(2.0f, ew);
    const uint2 *Uo = (const uint2 *)U;
    state_term_core<(ROWU2 > 2048)>(CT, wq, qa, lane, [&](int t, f4_t D) {
        const uint2 o = Uo[row * ROWU2 + (t >> 2)];
        const uint2 r = make_uint2(pack_out<DT>(fmaf(D[0], scorr, lo_f<DT>(o.x)), fmaf(D[1], scorr, hi_f<DT>(o.x))),
                                   pack_out<DT>(fmaf(D[2], scorr, lo_f<DT>(o.y)), fmaf(D[3], scorr, hi_f<DT>(o.y))));
        *(uint2 *)(yrow + t) = r;
    });
}

}  // namespace wvc
}  // namespace h3
