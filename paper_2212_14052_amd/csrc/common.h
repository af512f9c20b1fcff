// Device-side helpers shared by the h3flash HIP kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace h3 {

enum DType { F32 = 0, F16 = 1, BF16 = 2 };

// ------------------------------------------------------------ complex ------
__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
    return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ float2 cconj(float2 a) { return make_float2(a.x, -a.y); }
__device__ __forceinline__ float2 cscale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }
// multiply by -i and by +i
__device__ __forceinline__ float2 cmul_mi(float2 a) { return make_float2(a.y, -a.x); }
__device__ __forceinline__ float2 cmul_pi(float2 a) { return make_float2(-a.y, a.x); }

// ------------------------------------------------------------ 16-bit I/O ---
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t b = __float_as_uint(f);
    if ((b & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((b >> 16) | 0x40u);  // quiet NaN
    b += 0x7fffu + ((b >> 16) & 1u);                                            // RNE
    return (uint16_t)(b >> 16);
}
__device__ __forceinline__ float f16_to_f32(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
// float -> half conversion rounds to nearest even
__device__ __forceinline__ uint16_t f32_to_f16(float f) { return __builtin_bit_cast(uint16_t, (_Float16)f); }

template <int DT> struct IO;
template <> struct IO<F32> {
    typedef float T;
    static __device__ __forceinline__ float ld(const float *p, long i) { return p[i]; }
    static __device__ __forceinline__ void st(float *p, long i, float v) { p[i] = v; }
};
template <> struct IO<F16> {
    typedef uint16_t T;
    static __device__ __forceinline__ float ld(const uint16_t *p, long i) { return f16_to_f32(p[i]); }
    static __device__ __forceinline__ void st(uint16_t *p, long i, float v) { p[i] = f32_to_f16(v); }
};
template <> struct IO<BF16> {
    typedef uint16_t T;
    static __device__ __forceinline__ float ld(const uint16_t *p, long i) { return bf16_to_f32(p[i]); }
    static __device__ __forceinline__ void st(uint16_t *p, long i, float v) { p[i] = f32_to_bf16(v); }
};

// Exponent e with m = f 2^e, f in [1/2, 1) (frexp); 0 for 0, NaN and inf, so
// that such rows pass through unscaled.
__device__ __forceinline__ int pow2_exp(float m) {
    if (!(m > 0.f) || !(m < 3.0e38f)) return 0;
    int e;
    frexpf(m, &e);
    return e;
}

// --------------------------------------------------------- launch order ----
// Workgroups are dealt round-robin to the 8 XCDs (each with its own L2).  Remap
// the hardware block index so that consecutive logical indices run on the same
// XCD: work that shares data (e.g. rows of one channel) then shares an L2.
__device__ __forceinline__ int xcd_logical_block(int b, int nblocks) {
    constexpr int NXCD = 8;
    if (nblocks % NXCD != 0) return b;
    return (b % NXCD) * (nblocks / NXCD) + b / NXCD;
}

// exp(tau * lambda) for complex lambda given in float64, returned in float32:
// the phase tau*Im(lambda) is reduced modulo 2 pi in float64 before the
// float32 sine/cosine, so large arguments keep full accuracy.
__device__ __forceinline__ float2 cexp_scaled(double tau, double lre, double lim) {
    const double TWO_PI = 6.283185307179586476925286766559;
    double ph = tau * lim;
    ph -= TWO_PI * rint(ph / TWO_PI);
    float mag = expf((float)(tau * lre));
    float s, c;
    sincosf((float)ph, &s, &c);
    return make_float2(mag * c, mag * s);
}

}  // namespace h3
