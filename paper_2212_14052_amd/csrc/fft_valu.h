// Float32 FFT engine on the vector ALUs (gfx950): register radix-2/4/8/16
// butterflies, Stockham auto-sorting passes exchanged through LDS.
//
// A length-N signal (N = 2^k, 32 <= N <= 16384) is owned by T = N/16 threads;
// every pass each thread holds 16 complex values (one radix-16 butterfly, or
// 16/R butterflies of a smaller radix R).  Pass (R, Ns) of the Stockham
// decimation-in-time form, butterfly j in [0, N/R):
//     load    v[r] = X[j + r N/R]                          r < R
//     twiddle v[r] *= exp(-2 pi i (j mod Ns) r / (Ns R))
//     DFT_R   on v
//     store   X'[(j div Ns) Ns R + (j mod Ns) + r Ns] = v[r]
// Forward passes: R1 at Ns = 1 (R1 = N / 16^p in {2,4,8}, or 16), then
// radix 16 at Ns = R1, 16 R1, ..., N/16.  The last forward pass leaves
// X[j + r N/16] in thread j's registers, which is exactly what the first pass
// (radix 16, Ns = 1) of a second transform loads, so a pointwise product
// between two transforms needs no LDS exchange.
//
// The DFTs are Cooley-Tukey splits (Sec. 4.1: F_N = P (I (x) F_N1) P^T D
// (I (x) F_N2) P) applied recursively inside the registers; the LDS passes are
// the same factorisation one level up.
#pragma once
#include "common.h"

namespace h3 {

constexpr float kCos16[16] = {
    1.0f, 0.92387953251128674f, 0.70710678118654752f, 0.38268343236508977f,
    0.0f, -0.38268343236508977f, -0.70710678118654752f, -0.92387953251128674f,
    -1.0f, -0.92387953251128674f, -0.70710678118654752f, -0.38268343236508977f,
    0.0f, 0.38268343236508977f, 0.70710678118654752f, 0.92387953251128674f};
constexpr float kSin16[16] = {
    0.0f, 0.38268343236508977f, 0.70710678118654752f, 0.92387953251128674f,
    1.0f, 0.92387953251128674f, 0.70710678118654752f, 0.38268343236508977f,
    0.0f, -0.38268343236508977f, -0.70710678118654752f, -0.92387953251128674f,
    -1.0f, -0.92387953251128674f, -0.70710678118654752f, -0.38268343236508977f};

// a * exp(-2 pi i j / n) for compile-time-foldable j, n (n divides 16).
__device__ __forceinline__ float2 tw_const(float2 a, int j, int n) {
    int q = (j % n) * (16 / n);
    if (q == 0) return a;
    if (q == 4) return cmul_mi(a);
    if (q == 8) return make_float2(-a.x, -a.y);
    if (q == 12) return cmul_pi(a);
    const float c = kCos16[q], s = -kSin16[q];
    return make_float2(a.x * c - a.y * s, a.x * s + a.y * c);
}

// In-register forward DFT (natural order in and out).
template <int N> struct DFT {
    static __device__ __forceinline__ void run(float2 *v) {
        constexpr int N1 = (N > 4 && N % 4 == 0) ? 4 : 2;
        constexpr int N2 = N / N1;
        float2 A[N1][N2];
#pragma unroll
        for (int n2 = 0; n2 < N2; ++n2) {
            float2 t[N1];
#pragma unroll
            for (int n1 = 0; n1 < N1; ++n1) t[n1] = v[N2 * n1 + n2];
            DFT<N1>::run(t);
#pragma unroll
            for (int k1 = 0; k1 < N1; ++k1) A[k1][n2] = tw_const(t[k1], n2 * k1, N);
        }
#pragma unroll
        for (int k1 = 0; k1 < N1; ++k1) {
            float2 t[N2];
#pragma unroll
            for (int n2 = 0; n2 < N2; ++n2) t[n2] = A[k1][n2];
            DFT<N2>::run(t);
#pragma unroll
            for (int k2 = 0; k2 < N2; ++k2) v[k1 + N1 * k2] = t[k2];
        }
    }
};
template <> struct DFT<1> {
    static __device__ __forceinline__ void run(float2 *) {}
};
template <> struct DFT<2> {
    static __device__ __forceinline__ void run(float2 *v) {
        float2 a = v[0], b = v[1];
        v[0] = cadd(a, b);
        v[1] = csub(a, b);
    }
};
template <> struct DFT<4> {
    static __device__ __forceinline__ void run(float2 *v) {
        float2 t0 = cadd(v[0], v[2]), t1 = csub(v[0], v[2]);
        float2 t2 = cadd(v[1], v[3]), t3 = csub(v[1], v[3]);
        v[0] = cadd(t0, t2);
        v[2] = csub(t0, t2);
        v[1] = cadd(t1, cmul_mi(t3));
        v[3] = csub(t1, cmul_mi(t3));
    }
};

constexpr int ilog2c(int n) { return n <= 1 ? 0 : 1 + ilog2c(n / 2); }

__device__ __forceinline__ int lds_pad(int i) { return i + (i >> 4); }

template <int N> struct FFTPlan {
    static constexpr int LOGN = ilog2c(N);
    static constexpr int R1 = (LOGN % 4 == 0) ? 16 : (1 << (LOGN % 4));
    static constexpr int T = N / 16;               // threads per signal
    static constexpr int LDS = N + N / 16;         // float2 per signal (padded)
    static_assert(N >= 32 && N <= 16384, "FFT length out of range");
};

// Twiddles exp(-2 pi i jm r / M) for r = 1..R-1 (M = Ns R, a power of two).
// w1, w2, w4, w8 come from sincospi with exactly representable arguments;
// the others are products of at most two of them.
template <int R>
__device__ __forceinline__ void pass_twiddles(float2 *v, int jm, int M) {
    float2 w[16];
    const float base = -2.0f * (float)jm / (float)M;
    {
        float s, c;
        sincospif(base, &s, &c);
        w[1] = make_float2(c, s);
    }
    if (R > 2) {
        float s, c;
        sincospif(2.0f * base, &s, &c);
        w[2] = make_float2(c, s);
        w[3] = cmul(w[1], w[2]);
    }
    if (R > 4) {
        float s, c;
        sincospif(4.0f * base, &s, &c);
        w[4] = make_float2(c, s);
        w[5] = cmul(w[1], w[4]);
        w[6] = cmul(w[2], w[4]);
        w[7] = cmul(w[3], w[4]);
    }
    if (R > 8) {
        float s, c;
        sincospif(8.0f * base, &s, &c);
        w[8] = make_float2(c, s);
#pragma unroll
        for (int r = 9; r < 16; ++r) w[r] = cmul(w[r - 8], w[8]);
    }
#pragma unroll
    for (int r = 1; r < R; ++r) v[r] = cmul(v[r], w[r]);
}

// Stockham pass pieces for one signal in LDS buffer X (padded indexing).
template <int N, int R>
__device__ __forceinline__ void pass_load(const float2 *X, int tid, float2 *v) {
    constexpr int Q = 16 / R, T = N / 16;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = tid + q * T;
#pragma unroll
        for (int r = 0; r < R; ++r) v[q * R + r] = X[lds_pad(j + r * (N / R))];
    }
}

template <int N, int R, int Ns>
__device__ __forceinline__ void pass_twiddle(int tid, float2 *v) {
    if (Ns == 1) return;
    constexpr int Q = 16 / R, T = N / 16;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = tid + q * T;
        pass_twiddles<R>(v + q * R, j & (Ns - 1), Ns * R);
    }
}

template <int R>
__device__ __forceinline__ void pass_dft(float2 *v) {
#pragma unroll
    for (int q = 0; q < 16 / R; ++q) DFT<R>::run(v + q * R);
}

template <int N, int R, int Ns>
__device__ __forceinline__ void pass_store(float2 *X, int tid, const float2 *v) {
    constexpr int Q = 16 / R, T = N / 16;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = tid + q * T;
        const int jm = j & (Ns - 1);
        const int base = (j - jm) * R + jm;
#pragma unroll
        for (int r = 0; r < R; ++r) X[lds_pad(base + r * Ns)] = v[q * R + r];
    }
}

// Radix-16 passes with Ns = NS0, 16 NS0, ... while Ns < NSEND (exclusive):
// load, twiddle, DFT, store, barrier.
template <int N, int Ns, int NSEND>
struct MidPasses {
    static __device__ __forceinline__ void run(float2 *X, int tid, float2 *v) {
        if constexpr (Ns < NSEND) {
            pass_load<N, 16>(X, tid, v);
            pass_twiddle<N, 16, Ns>(tid, v);
            pass_dft<16>(v);
            __syncthreads();
            pass_store<N, 16, Ns>(X, tid, v);
            __syncthreads();
            MidPasses<N, Ns * 16, NSEND>::run(X, tid, v);
        }
    }
};

// Forward transform of the signal whose first pass input is already in v
// (thread tid holds X[j + r N/R1] for its butterflies j).  On return thread
// tid holds the spectrum  v[r] = F[tid + r N/16], r < 16.
// Every thread of the workgroup must call this (it contains barriers).
template <int N>
__device__ __forceinline__ void fft_forward_from_regs(float2 *X, int tid, float2 *v) {
    using P = FFTPlan<N>;
    constexpr int R1 = P::R1;
    pass_dft<R1>(v);                         // Ns = 1: no twiddles
    if constexpr (R1 * 16 <= N) {
        pass_store<N, R1, 1>(X, tid, v);
        __syncthreads();
        MidPasses<N, R1, N / 16>::run(X, tid, v);
        // last forward pass: radix 16 at Ns = N/16, result stays in registers
        pass_load<N, 16>(X, tid, v);
        pass_twiddle<N, 16, N / 16>(tid, v);
        pass_dft<16>(v);
    }
}

// Forward transform of a signal whose first pass input is in v laid out as
// the radix-16 pass at Ns = 1 expects (v[r] = X[tid + r N/16]), returning the
// last pass (radix R1 at Ns = N/R1) in registers: thread tid then holds
// F[j + r N/R1] in v[q R1 + r] for its butterflies j = tid + q N/16.
// Used for the second transform of a convolution (the "inverse").
template <int N>
__device__ __forceinline__ void fft_second_from_regs(float2 *X, int tid, float2 *v) {
    using P = FFTPlan<N>;
    constexpr int R1 = P::R1;
    pass_dft<16>(v);                         // radix 16 at Ns = 1
    __syncthreads();                         // LDS may still be read by the previous pass
    pass_store<N, 16, 1>(X, tid, v);
    __syncthreads();
    MidPasses<N, 16, N / R1>::run(X, tid, v);
    pass_load<N, R1>(X, tid, v);
    pass_twiddle<N, R1, N / R1>(tid, v);
    pass_dft<R1>(v);
}

}  // namespace h3
