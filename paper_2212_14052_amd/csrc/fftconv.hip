// Fused FFT convolution (Sec. 4.1, kernel fusion) on the vector ALUs, gfx950.
//
// y = irfft(rfft(u, 2L) * rfft(k, 2L))[:L] + D u per (batch, channel) row.
//
// Two real rows that share a channel (hence a kernel) are packed into one
// complex signal z = u_a + i u_b of length N = 2L (upper half zero).  Since k
// is real, conv(k, z) = conv(k, u_a) + i conv(k, u_b), so one complex
// transform pair serves two rows with no spectrum untangling:
//     Z = F z,   Y = Z K / N,   w = F conj(Y),   y_a = Re w,  y_b = -Im w
// (the inverse is taken as conj(F conj(.)) so both transforms share code).
// Zero-padding prunes the first pass (half its inputs are zero) and the last
// pass (only outputs t < L are formed).  The skip term D u reuses the u
// values the first pass loaded: the last pass of the second transform leaves
// exactly those positions in the same thread.
#include "common.h"
#include "fft_valu.h"
#include "internal.h"

namespace h3 {

// -------------------------------------------------------------- spectrum ---
// Two channels per signal: z = k_h + i k_{h+1}; K_h = (Z + conj Z(-f)) / 2,
// K_{h+1} = (Z - conj Z(-f)) / (2i); both scaled by 1/N.
template <int N>
__global__ __launch_bounds__(N / 16 >= 64 ? N / 16 : 64) void spectrum_kernel(
    const float *k, int H, float2 *Kspec) {
    using P = FFTPlan<N>;
    constexpr int T = P::T, L = N / 2, R1 = P::R1, Q = 16 / R1;
    constexpr int S = (T >= 64) ? 1 : 64 / T;
    extern __shared__ float2 lds[];
    const int sig = threadIdx.x / T, tid = threadIdx.x % T;
    float2 *X = lds + sig * P::LDS;
    const int h0 = 2 * (blockIdx.x * S + sig);
    const bool va = h0 < H, vb = h0 + 1 < H;
    float2 v[16];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = tid + q * T;
#pragma unroll
        for (int r = 0; r < R1; ++r) {
            float a = 0.f, b = 0.f;
            if (r < R1 / 2) {
                const int n = j + r * (N / R1);
                if (va) a = k[(long)h0 * L + n];
                if (vb) b = k[(long)(h0 + 1) * L + n];
            }
            v[q * R1 + r] = make_float2(a, b);
        }
    }
    fft_forward_from_regs<N>(X, tid, v);
    __syncthreads();
#pragma unroll
    for (int r = 0; r < 16; ++r) X[lds_pad(tid + r * T)] = v[r];
    __syncthreads();
    const float inv = 1.0f / (float)N;
    for (int f = tid; f <= L; f += T) {
        float2 z = X[lds_pad(f)];
        float2 zc = cconj(X[lds_pad((N - f) & (N - 1))]);
        float2 s = cadd(z, zc), d = csub(z, zc);
        if (va) Kspec[(long)h0 * (L + 1) + f] = make_float2(0.5f * s.x * inv, 0.5f * s.y * inv);
        if (vb) Kspec[(long)(h0 + 1) * (L + 1) + f] = make_float2(0.5f * d.y * inv, -0.5f * d.x * inv);
    }
}

// ---------------------------------------------------------------- conv -----
// Pair p -> element offsets of its two rows (ob < 0: no second row) and channel.
struct PairMap {
    long oa, ob;
    int h;
};
__device__ __forceinline__ PairMap map_pair(const ConvArgs &a, int p) {
    PairMap r;
    if (a.pair_mode == 0) {
        const int nbp = (a.B + 1) / 2;
        const int h = p / nbp, bp = p % nbp;
        r.h = h;
        r.oa = ((long)(2 * bp) * a.H + h) * a.L;
        r.ob = (2 * bp + 1 < a.B) ? ((long)(2 * bp + 1) * a.H + h) * a.L : -1;
    } else {
        const int ncp = (a.nchunk + 1) / 2;
        const int row = p / ncp, cp = p % ncp;   // row = b*H + h
        r.h = row % a.H;
        const long base = (long)row * a.nchunk * a.L;
        r.oa = base + (long)(2 * cp) * a.L;
        r.ob = (2 * cp + 1 < a.nchunk) ? r.oa + a.L : -1;
    }
    return r;
}

template <int N, int DT>
__global__ __launch_bounds__(N / 16 >= 64 ? N / 16 : 64) void fftconv_kernel(ConvArgs a, int npairs) {
    using P = FFTPlan<N>;
    using io = IO<DT>;
    typedef typename io::T T_;
    constexpr int T = P::T, R1 = P::R1, Q = 16 / R1, HALF = R1 / 2;
    constexpr int S = (T >= 64) ? 1 : 64 / T;
    constexpr int L = N / 2;
    extern __shared__ float2 lds[];
    __shared__ uint32_t rmx[2 * S];   // per signal: max |row a|, max |row b| (float bits)
    const int sig = threadIdx.x / T, tid = threadIdx.x % T;
    float2 *X = lds + sig * P::LDS;
    const int blk = xcd_logical_block(blockIdx.x, gridDim.x);
    const int p = blk * S + sig;
    const bool active = p < npairs;
    PairMap pm = map_pair(a, active ? p : 0);
    const bool hb = active && pm.ob >= 0;
    const T_ *u = (const T_ *)a.u;
    T_ *y = (T_ *)a.y;

    // load both rows at positions j + r N/R1 (r < R1/2); the rest is padding
    float2 v[16];
    float ua[8], ub[8];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = tid + q * T;
#pragma unroll
        for (int r = 0; r < R1; ++r) {
            if (r < HALF) {
                const int n = j + r * (N / R1);
                const float xa = active ? io::ld(u, pm.oa + n) : 0.f;
                const float xb = hb ? io::ld(u, pm.ob + n) : 0.f;
                ua[q * HALF + r] = xa;
                ub[q * HALF + r] = xb;
                v[q * R1 + r] = make_float2(xa, xb);
            } else {
                v[q * R1 + r] = make_float2(0.f, 0.f);
            }
        }
    }
    // Each row gets its own power-of-two scale (max |.| in [1/2, 1)): rounding
    // error of the shared transform then stays at each row's own scale, even
    // when one row is much smaller than the other.
    {
        float ma = 0.f, mb = 0.f;
#pragma unroll
        for (int i = 0; i < Q * HALF; ++i) {
            ma = fmaxf(ma, fabsf(ua[i]));
            mb = fmaxf(mb, fabsf(ub[i]));
        }
        if (tid == 0) {
            rmx[2 * sig] = 0u;
            rmx[2 * sig + 1] = 0u;
        }
        __syncthreads();
        atomicMax(&rmx[2 * sig], __float_as_uint(ma));
        atomicMax(&rmx[2 * sig + 1], __float_as_uint(mb));
        __syncthreads();
    }
    const int ea = pow2_exp(__uint_as_float(rmx[2 * sig])), eb = pow2_exp(__uint_as_float(rmx[2 * sig + 1]));
    {
        const float sa = ldexpf(1.0f, -ea), sb = ldexpf(1.0f, -eb);
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = make_float2(v[r].x * sa, v[r].y * sb);
    }
    fft_forward_from_regs<N>(X, tid, v);

    // pointwise product with the kernel spectrum (Hermitian: K(-f) = conj K(f)),
    // then conjugate for the second transform
    const float2 *K = a.Kspec + (long)pm.h * (L + 1);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int f = tid + r * T;
        float2 kf = (f <= L) ? K[f] : cconj(K[N - f]);
        if (a.conj_k) kf = cconj(kf);   // correlation (input gradient)
        v[r] = cconj(cmul(v[r], kf));
    }
    fft_second_from_regs<N>(X, tid, v);

    const float d = a.D ? a.D[pm.h] : 0.f;
    const float ya_s = ldexpf(1.0f, ea), yb_s = ldexpf(1.0f, eb);
    if (!active) return;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = tid + q * T;
#pragma unroll
        for (int r = 0; r < HALF; ++r) {
            const int n = j + r * (N / R1);
            const float2 w = v[q * R1 + r];
            float oa = fmaf(w.x, ya_s, d * ua[q * HALF + r]);
            float ob = fmaf(-w.y, yb_s, d * ub[q * HALF + r]);
            if (a.corr) {
                const float *cr = (const float *)a.corr;
                oa += cr[pm.oa + n];
                if (hb) ob += cr[pm.ob + n];
            }
            io::st(y, pm.oa + n, oa);
            if (hb) io::st(y, pm.ob + n, ob);
        }
    }
}

// --------------------------------------------------------------- launch ----
template <int N>
static hipError_t launch_spectrum_n(const float *k, int H, float2 *Kspec, hipStream_t s) {
    using P = FFTPlan<N>;
    constexpr int T = P::T, S = (T >= 64) ? 1 : 64 / T;
    const int nsig = (H + 1) / 2;
    dim3 grid((nsig + S - 1) / S), block(S * T);
    size_t lds = (size_t)S * P::LDS * sizeof(float2);
    if (lds > 65536)
        (void)hipFuncSetAttribute((const void *)spectrum_kernel<N>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(spectrum_kernel<N>, grid, block, lds, s, k, H, Kspec);
    return hipGetLastError();
}

template <int N, int DT>
static hipError_t launch_conv_n(const ConvArgs &a, hipStream_t s) {
    using P = FFTPlan<N>;
    constexpr int T = P::T, S = (T >= 64) ? 1 : 64 / T;
    int npairs;
    if (a.pair_mode == 0)
        npairs = ((a.B + 1) / 2) * a.H;
    else
        npairs = a.B * a.H * ((a.nchunk + 1) / 2);
    dim3 grid((npairs + S - 1) / S), block(S * T);
    size_t lds = (size_t)S * P::LDS * sizeof(float2);
    auto fn = fftconv_kernel<N, DT>;
    if (lds > 65536) (void)hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(fn, grid, block, lds, s, a, npairs);
    return hipGetLastError();
}

template <int N>
static hipError_t launch_conv_dt(const ConvArgs &a, hipStream_t s) {
    switch (a.dtype) {
        case F32: return launch_conv_n<N, F32>(a, s);
        case F16: return launch_conv_n<N, F16>(a, s);
        case BF16: return launch_conv_n<N, BF16>(a, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_spectrum(const float *k, int H, int L, float2 *Kspec, hipStream_t s) {
    switch (L) {
        case 16: return launch_spectrum_n<32>(k, H, Kspec, s);
        case 32: return launch_spectrum_n<64>(k, H, Kspec, s);
        case 64: return launch_spectrum_n<128>(k, H, Kspec, s);
        case 128: return launch_spectrum_n<256>(k, H, Kspec, s);
        case 256: return launch_spectrum_n<512>(k, H, Kspec, s);
        case 512: return launch_spectrum_n<1024>(k, H, Kspec, s);
        case 1024: return launch_spectrum_n<2048>(k, H, Kspec, s);
        case 2048: return launch_spectrum_n<4096>(k, H, Kspec, s);
        case 4096: return launch_spectrum_n<8192>(k, H, Kspec, s);
        case 8192: return launch_spectrum_n<16384>(k, H, Kspec, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_fftconv(const ConvArgs &a, hipStream_t s) {
    switch (a.L) {
        case 16: return launch_conv_dt<32>(a, s);
        case 32: return launch_conv_dt<64>(a, s);
        case 64: return launch_conv_dt<128>(a, s);
        case 128: return launch_conv_dt<256>(a, s);
        case 256: return launch_conv_dt<512>(a, s);
        case 512: return launch_conv_dt<1024>(a, s);
        case 1024: return launch_conv_dt<2048>(a, s);
        case 2048: return launch_conv_dt<4096>(a, s);
        case 4096: return launch_conv_dt<8192>(a, s);
        case 8192: return launch_conv_dt<16384>(a, s);
    }
    return hipErrorInvalidValue;
}

size_t fftconv_workspace(int B, int H, int L) {
    (void)B;
    return (size_t)H * (L + 1) * sizeof(float2);
}

}  // namespace h3
