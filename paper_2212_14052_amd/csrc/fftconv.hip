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
//
// fftconv_kgen_kernel is the same convolution with the kernel spectrum formed
// in the kernel itself, one spectrum shared by a group of row pairs.
#include <atomic>

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

// ------------------------------------------- conv with its own spectrum ----
// The same convolution for plain (B, H, L) rows, with the kernel spectrum
// computed in the kernel instead of read from a workspace: work item =
// (channel h, group of up to `ppg` row pairs of h).  The item's signal slot
// first transforms k_h + D delta (the skip term folded into the kernel: the
// circular convolution of the zero-padded row with k + D delta equals the
// causal convolution plus D u on t < L) and keeps F(.)/N in registers, in the
// layout the pointwise product reads; then it runs its row pairs.  One launch
// instead of two, and no spectrum round trip through HBM.
template <int N, int DT>
__global__ __launch_bounds__(N / 16 >= 64 ? N / 16 : 64) void fftconv_kgen_kernel(ConvArgs a, const float *k,
                                                                                 int groups, int ppg) {
    using P = FFTPlan<N>;
    using io = IO<DT>;
    typedef typename io::T T_;
    constexpr int T = P::T, R1 = P::R1, Q = 16 / R1, HALF = R1 / 2;
    constexpr int S = (T >= 64) ? 1 : 64 / T;
    constexpr int L = N / 2;
    extern __shared__ float2 lds[];
    __shared__ uint32_t rmx[2 * S];   // per signal slot: max |row a|, max |row b| (float bits)
    const int sig = threadIdx.x / T, tid = threadIdx.x % T;
    float2 *X = lds + sig * P::LDS;
    const int item = xcd_logical_block(blockIdx.x, gridDim.x) * S + sig;
    const bool act = item < a.H * groups;
    const int h = act ? item / groups : 0, grp = act ? item % groups : 0;
    const int npairs = (a.B + 1) / 2;
    const T_ *u = (const T_ *)a.u;
    T_ *y = (T_ *)a.y;

    // spectrum of k_h + D delta, scaled by 1/N (conjugated for the correlation)
    float2 kf[16];
#pragma unroll
    for (int q = 0; q < Q; ++q) {
        const int j = tid + q * T;
#pragma unroll
        for (int r = 0; r < R1; ++r) {
            float kr = 0.f;
            if (r < HALF && act) kr = k[(long)h * L + j + r * (N / R1)];
            kf[q * R1 + r] = make_float2(kr, 0.f);
        }
    }
    if (act && tid == 0 && a.D) kf[0].x += a.D[h];   // point 0: q = 0, r = 0, j = 0
    fft_forward_from_regs<N>(X, tid, kf);
    {
        const float inv = 1.0f / (float)N, sg = a.conj_k ? -inv : inv;
#pragma unroll
        for (int r = 0; r < 16; ++r) kf[r] = make_float2(kf[r].x * inv, kf[r].y * sg);
    }

    for (int i = 0; i < ppg; ++i) {
        // an opaque copy of the thread index per pair: the passes' twiddles
        // are evaluated where they are used instead of being hoisted out of
        // the loop (where they would all stay live)
        int tv = tid;
        asm volatile("" : "+v"(tv));
        const int pr = grp * ppg + i;
        const bool va = act && pr < npairs, vb = va && 2 * pr + 1 < a.B;
        const long oa = ((long)(2 * pr) * a.H + h) * L, ob = oa + (long)a.H * L;
        float2 v[16];
        float ma = 0.f, mb = 0.f;
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int j = tid + q * T;
#pragma unroll
            for (int r = 0; r < R1; ++r) {
                float xa = 0.f, xb = 0.f;
                if (r < HALF) {
                    const int n = j + r * (N / R1);
                    if (va) xa = io::ld(u, oa + n);
                    if (vb) xb = io::ld(u, ob + n);
                }
                ma = fmaxf(ma, fabsf(xa));
                mb = fmaxf(mb, fabsf(xb));
                v[q * R1 + r] = make_float2(xa, xb);
            }
        }
        // each row of the pair gets its own power-of-two scale
        __syncthreads();   // LDS: the previous transform's reads and the previous rmx reads are done
        if (tid == 0) {
            rmx[2 * sig] = 0u;
            rmx[2 * sig + 1] = 0u;
        }
        __syncthreads();
        atomicMax(&rmx[2 * sig], __float_as_uint(ma));
        atomicMax(&rmx[2 * sig + 1], __float_as_uint(mb));
        __syncthreads();
        const int ea = pow2_exp(__uint_as_float(rmx[2 * sig])), eb = pow2_exp(__uint_as_float(rmx[2 * sig + 1]));
        {
            const float sa = ldexpf(1.0f, -ea), sb = ldexpf(1.0f, -eb);
#pragma unroll
            for (int r = 0; r < 16; ++r) v[r] = make_float2(v[r].x * sa, v[r].y * sb);
        }
        fft_forward_from_regs<N>(X, tv, v);
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = cconj(cmul(v[r], kf[r]));
        fft_second_from_regs<N>(X, tv, v);
        const float ya_s = ldexpf(1.0f, ea), yb_s = -ldexpf(1.0f, eb);
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int j = tid + q * T;
#pragma unroll
            for (int r = 0; r < HALF; ++r) {
                const int n = j + r * (N / R1);
                const float2 w = v[q * R1 + r];
                if (va) io::st(y, oa + n, w.x * ya_s);
                if (vb) io::st(y, ob + n, w.y * yb_s);
            }
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

// Pairs per spectrum for the kgen kernel.  An item costs 2 ppg + 1
// transforms, run one after another; the items run in ceil(items / resident)
// rounds, `resident` being the items the whole device holds at once.  Take
// the ppg in 1..npairs that minimises rounds x (2 ppg + 1), the larger one on
// a tie (fewer transforms in all).  Small launches thus keep one spectrum per
// pair for parallelism; large ones share a spectrum among up to npairs pairs.
static int kgen_pairs_per_group(int H, int npairs, int S, long resident_blocks) {
    long best_cost = -1;
    int best = 1;
    for (int ppg = 1; ppg <= npairs; ppg = (ppg < npairs && 2 * ppg > npairs) ? npairs : 2 * ppg) {
        const long items = (long)H * ((npairs + ppg - 1) / ppg);
        const long blocks = (items + S - 1) / S;
        const long rounds = (blocks + resident_blocks - 1) / resident_blocks;
        const long cost = rounds * (2 * ppg + 1);
        if (best_cost < 0 || cost <= best_cost) {
            best_cost = cost;
            best = ppg;
        }
        if (ppg == npairs) break;
    }
    return best;
}

template <int N, int DT>
static hipError_t launch_kgen_n(const ConvArgs &a, const float *k, hipStream_t s) {
    using P = FFTPlan<N>;
    constexpr int T = P::T, S = (T >= 64) ? 1 : 64 / T;
    const size_t lds = (size_t)S * P::LDS * sizeof(float2);
    auto fn = fftconv_kgen_kernel<N, DT>;
    if (lds > 65536) (void)hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    // resident blocks per CU (fixed per instantiation) times the CUs of the current device
    static std::atomic<int> per_cu{0};
    if (per_cu.load(std::memory_order_relaxed) == 0) {
        int n = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, (const void *)fn, S * T, lds) != hipSuccess || n < 1) n = 1;
        per_cu.store(n, std::memory_order_relaxed);
    }
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 1;
    const int npairs = (a.B + 1) / 2;
    const int ppg = kgen_pairs_per_group(a.H, npairs, S, (long)per_cu.load(std::memory_order_relaxed) * cus);
    const int groups = (npairs + ppg - 1) / ppg;
    const long items = (long)a.H * groups;
    dim3 grid((unsigned)((items + S - 1) / S)), block(S * T);
    hipLaunchKernelGGL(fn, grid, block, lds, s, a, k, groups, ppg);
    return hipGetLastError();
}

template <int N>
static hipError_t launch_kgen_dt(const ConvArgs &a, const float *k, hipStream_t s) {
    switch (a.dtype) {
        case F32: return launch_kgen_n<N, F32>(a, k, s);
        case F16: return launch_kgen_n<N, F16>(a, k, s);
        case BF16: return launch_kgen_n<N, BF16>(a, k, s);
    }
    return hipErrorInvalidValue;
}

bool fftconv_kgen_supported(int L) { return L >= 16 && L <= 4096 && (L & (L - 1)) == 0; }

hipError_t launch_fftconv_kgen(const ConvArgs &a, const float *k, hipStream_t s) {
    if (a.pair_mode != 0 || a.corr) return hipErrorInvalidValue;
    switch (a.L) {
        case 16: return launch_kgen_dt<32>(a, k, s);
        case 32: return launch_kgen_dt<64>(a, k, s);
        case 64: return launch_kgen_dt<128>(a, k, s);
        case 128: return launch_kgen_dt<256>(a, k, s);
        case 256: return launch_kgen_dt<512>(a, k, s);
        case 512: return launch_kgen_dt<1024>(a, k, s);
        case 1024: return launch_kgen_dt<2048>(a, k, s);
        case 2048: return launch_kgen_dt<4096>(a, k, s);
        case 4096: return launch_kgen_dt<8192>(a, k, s);
    }
    return hipErrorInvalidValue;
}

size_t fftconv_workspace(int B, int H, int L) {
    (void)B;
    return (size_t)H * (L + 1) * sizeof(float2);
}

}  // namespace h3
