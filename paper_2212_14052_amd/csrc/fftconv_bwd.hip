// Kernel and skip gradients of the fused FFT convolution (the appendix on
// the backward pass of FlashConv).  For y = k * u + D u and output gradient
// dy, per channel h:
//     dk = Re IFFT( sum_b conj(F u_b) . F dy_b )[:L],      dD = sum_{b,t} u dy,
// with F the length-N = 2L DFT of the zero-padded rows.  Correlating through
// the spectrum is exact here: both rows are zero past L, so the circular
// lags that wrap around meet only padding.
//
// Two rows of one channel are packed into one complex signal, z_u = u_a +
// i u_b and z_g = dy_a + i dy_b.  Then conj(F z_u) . F z_g = conj(U_a) G_a +
// conj(U_b) G_b + i (conj(U_a) G_b - conj(U_b) G_a), and the inverse of the
// bracketed cross term is real, so it lands in the imaginary part:
//     Re IFFT( conj(F z_u) . F z_g ) = corr(u_a, dy_a) + corr(u_b, dy_b).
// One signal slot (N/16 threads, the VALU radix-16 engine of fft_valu.h) per
// channel walks the channel's row pairs, accumulating that product for its 16
// frequencies in float32 registers; one more transform per channel gives dk.
// (Re IFFT(P) = Re F(conj P) / N, so every transform here is the forward one.)
#include "fft_valu.h"
#include "internal.h"

namespace h3 {
namespace {

template <int N, int DT>
__global__ __launch_bounds__(N / 16 >= 64 ? N / 16 : 64) void conv_wgrad_kernel(const void *u_, const void *dy_,
                                                                               int B, int H, float *dk, float *dD) {
    using P = FFTPlan<N>;
    using io = IO<DT>;
    typedef typename io::T T_;
    constexpr int T = P::T, R1 = P::R1, Q = 16 / R1, HALF = R1 / 2;
    constexpr int S = (T >= 64) ? 1 : 64 / T;
    constexpr int L = N / 2;
    extern __shared__ float2 lds[];
    __shared__ float wsum[16];
    const int sig = threadIdx.x / T, tid = threadIdx.x % T;
    float2 *X = lds + sig * P::LDS;
    const int h = blockIdx.x * S + sig;
    const bool active = h < H;
    const T_ *u = (const T_ *)u_;
    const T_ *dy = (const T_ *)dy_;

    float2 acc[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = make_float2(0.f, 0.f);
    float dd = 0.f;
    const int nbp = (B + 1) / 2;   // uniform over the block: every thread runs every barrier
    for (int bp = 0; bp < nbp; ++bp) {
        const long oa = ((long)(2 * bp) * H + (active ? h : 0)) * L;
        const bool hb = active && 2 * bp + 1 < B;
        const long ob = oa + (long)H * L;
        float2 v[16], w[16];
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int j = tid + q * T;
#pragma unroll
            for (int r = 0; r < R1; ++r) {
                if (r < HALF) {
                    const int n = j + r * (N / R1);
                    const float ua = active ? io::ld(u, oa + n) : 0.f, ub = hb ? io::ld(u, ob + n) : 0.f;
                    const float ga = active ? io::ld(dy, oa + n) : 0.f, gb = hb ? io::ld(dy, ob + n) : 0.f;
                    dd += ua * ga + ub * gb;
                    v[q * R1 + r] = make_float2(ua, ub);
                    w[q * R1 + r] = make_float2(ga, gb);
                } else {
                    v[q * R1 + r] = make_float2(0.f, 0.f);
                    w[q * R1 + r] = make_float2(0.f, 0.f);
                }
            }
        }
        if (bp > 0) __syncthreads();   // the previous transform's last LDS reads are done
        fft_forward_from_regs<N>(X, tid, v);
        __syncthreads();
        fft_forward_from_regs<N>(X, tid, w);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float2 a = v[r], g = w[r];   // conj(a) . g
            acc[r].x += a.x * g.x + a.y * g.y;
            acc[r].y += a.x * g.y - a.y * g.x;
        }
    }
    // dk[n] = Re IFFT(acc)[n] = Re F(conj acc)[n] / N, n < L
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = cconj(acc[r]);
    fft_second_from_regs<N>(X, tid, acc);
    if (active && dk) {
        constexpr float inv = 1.0f / N;
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int j = tid + q * T;
#pragma unroll
            for (int r = 0; r < HALF; ++r) dk[(long)h * L + j + r * (N / R1)] = acc[q * R1 + r].x * inv;
        }
    }
    // dD: sum over the signal's T threads (lanes of one wave when T <= 64)
#pragma unroll
    for (int o = (T < 64 ? T : 64) / 2; o >= 1; o >>= 1) dd += __shfl_xor(dd, o, 64);
    if constexpr (T > 64) {   // one signal per block, T / 64 waves
        if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = dd;
        __syncthreads();
        if (threadIdx.x == 0) {
            float s = 0.f;
            for (int i = 0; i < T / 64; ++i) s += wsum[i];
            dd = s;
        }
    }
    if (tid == 0 && active && dD) dD[h] = dd;
}

template <int N, int DT>
hipError_t launch_wgrad_n(const void *u, const void *dy, int B, int H, float *dk, float *dD, hipStream_t s) {
    using P = FFTPlan<N>;
    constexpr int T = P::T, S = (T >= 64) ? 1 : 64 / T;
    static_assert(T / 64 <= 16, "wsum holds at most 16 waves");
    dim3 grid((H + S - 1) / S), block(S * T);
    const size_t lds = (size_t)S * P::LDS * sizeof(float2);
    auto fn = conv_wgrad_kernel<N, DT>;
    if (lds > 65536) (void)hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(fn, grid, block, lds, s, u, dy, B, H, dk, dD);
    return hipGetLastError();
}

template <int N>
hipError_t launch_wgrad_dt(const void *u, const void *dy, int B, int H, int dtype, float *dk, float *dD,
                           hipStream_t s) {
    switch (dtype) {
        case F32: return launch_wgrad_n<N, F32>(u, dy, B, H, dk, dD, s);
        case F16: return launch_wgrad_n<N, F16>(u, dy, B, H, dk, dD, s);
        case BF16: return launch_wgrad_n<N, BF16>(u, dy, B, H, dk, dD, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_conv_wgrad(const void *u, const void *dy, int B, int H, int L, int dtype, float *dk, float *dD,
                             hipStream_t s) {
    switch (L) {
        case 16: return launch_wgrad_dt<32>(u, dy, B, H, dtype, dk, dD, s);
        case 32: return launch_wgrad_dt<64>(u, dy, B, H, dtype, dk, dD, s);
        case 64: return launch_wgrad_dt<128>(u, dy, B, H, dtype, dk, dD, s);
        case 128: return launch_wgrad_dt<256>(u, dy, B, H, dtype, dk, dD, s);
        case 256: return launch_wgrad_dt<512>(u, dy, B, H, dtype, dk, dD, s);
        case 512: return launch_wgrad_dt<1024>(u, dy, B, H, dtype, dk, dD, s);
        case 1024: return launch_wgrad_dt<2048>(u, dy, B, H, dtype, dk, dD, s);
        case 2048: return launch_wgrad_dt<4096>(u, dy, B, H, dtype, dk, dD, s);
        case 4096: return launch_wgrad_dt<8192>(u, dy, B, H, dtype, dk, dD, s);
        case 8192: return launch_wgrad_dt<16384>(u, dy, B, H, dtype, dk, dD, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace h3
