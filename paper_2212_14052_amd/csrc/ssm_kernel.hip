// SSM discretisation and convolution-kernel generation (gfx950).
//
// The kernel of a diagonal SSM (Sec. 2.1, f = [CB, CAB, CA^2B, ...]; diagonal A
// as in Sec. 3.2) is evaluated as
//     k[t] = 2 Re sum_n W_n exp(t lambda_n),   W_n = C_n Bbar_n,
// with lambda_n = dt A_n (continuous parameters, ZOH) or lambda_n = log Abar_n
// (discrete parameters).  Writing t = T a + b turns the sum into a small
// complex matrix product  k[T a + b] = 2 Re sum_n P[a][n] Q[n][b]  with
// P[a][n] = W_n exp(T a lambda_n) and Q[n][b] = exp(b lambda_n): only
// (TT/T + T) * m complex exponentials per tile of TT outputs instead of TT * m,
// each with its phase reduced in float64, and 2 FMAs per (output, mode).
#include "common.h"
#include "internal.h"

namespace h3 {

// Per-mode prologue: lambda (float64 complex) and W = C * Bbar (float32).
// mode 0: continuous (A, B, dt) -> ZOH.  mode 1: discrete (Abar, Bbar).
__device__ void mode_params(int mode, const float *P0, const float *P1, const float *C,
                            const float *dt, int h, int m, int n, double2 *lam, float2 *W) {
    long i = (long)h * m + n;
    double cr = C[2 * i], ci = C[2 * i + 1];
    double lr, li, br, bi;
    if (mode == 0) {
        double ar = P0[2 * i], ai = P0[2 * i + 1];
        double bre = P1[2 * i], bim = P1[2 * i + 1];
        double d = dt[h];
        lr = d * ar; li = d * ai;
        // exp(lambda) - 1 without cancellation for small |lambda|
        double s = sin(li), hs = sin(0.5 * li);
        double em1r = expm1(lr) * cos(li) - 2.0 * hs * hs;
        double em1i = exp(lr) * s;
        // (exp(lambda) - 1) / A
        double den = ar * ar + ai * ai;
        double qr = (em1r * ar + em1i * ai) / den;
        double qi = (em1i * ar - em1r * ai) / den;
        br = qr * bre - qi * bim;
        bi = qr * bim + qi * bre;
    } else {
        double ar = P0[2 * i], ai = P0[2 * i + 1];
        lr = 0.5 * log(ar * ar + ai * ai);
        li = atan2(ai, ar);
        br = P1[2 * i]; bi = P1[2 * i + 1];
    }
    *lam = make_double2(lr, li);
    *W = make_float2((float)(cr * br - ci * bi), (float)(cr * bi + ci * br));
}

__global__ void discretize_kernel(const float *A, const float *B, const float *dt, int H, int m,
                                  float *Abar, float *Bbar) {
    int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= H * m) return;
    int h = i / m;
    double ar = A[2 * i], ai = A[2 * i + 1];
    double bre = B[2 * i], bim = B[2 * i + 1];
    double d = dt[h];
    double lr = d * ar, li = d * ai;
    double e = exp(lr);
    double s = sin(li), hs = sin(0.5 * li);
    Abar[2 * i] = (float)(e * cos(li));
    Abar[2 * i + 1] = (float)(e * s);
    double em1r = expm1(lr) * cos(li) - 2.0 * hs * hs;
    double em1i = e * s;
    double den = ar * ar + ai * ai;
    double qr = (em1r * ar + em1i * ai) / den;
    double qi = (em1i * ar - em1r * ai) / den;
    Bbar[2 * i] = (float)(qr * bre - qi * bim);
    Bbar[2 * i + 1] = (float)(qr * bim + qi * bre);
}

// One workgroup: one channel h, a tile of KG_TT outputs starting at t0.
constexpr int KG_T = 32;                  // inner factor (b < KG_T)
constexpr int KG_TT = 2048;               // outputs per workgroup
constexpr int KG_A = KG_TT / KG_T;        // 64 outer steps per tile
constexpr int KG_THREADS = 256;

// mode 0/1: output row = channel h, W and lambda from the SSM parameters.
// mode 2: output row o (o = row * div + chunk), channel (o / div) % H,
//         lambda = log Abar (P0) of that channel and W given per output row in P1.
__global__ __launch_bounds__(KG_THREADS) void kernel_gen(int mode, const float *P0, const float *P1,
                                                         const float *C, const float *dt, int H,
                                                         int m, int L, float *k, int div) {
    __shared__ double2 lam_s[H3_MAX_MODES_DEV];
    __shared__ float2 W_s[H3_MAX_MODES_DEV];
    __shared__ float2 Q_s[H3_MAX_MODES_DEV][KG_T];       // exp(b lambda_n)
    __shared__ float2 P_s[KG_A][H3_MAX_MODES_DEV + 1];   // W_n exp((t0 + T a) lambda_n)
    const int ntile = (L + KG_TT - 1) / KG_TT;
    const int orow = blockIdx.x / ntile;
    const int t0 = (blockIdx.x % ntile) * KG_TT;
    const int tid = threadIdx.x;
    if (tid < m) {
        if (mode < 2) {
            mode_params(mode, P0, P1, C, dt, orow, m, tid, &lam_s[tid], &W_s[tid]);
        } else {
            const int h = (orow / div) % H;
            const long i = (long)h * m + tid;
            const double ar = P0[2 * i], ai = P0[2 * i + 1];
            lam_s[tid] = make_double2(0.5 * log(ar * ar + ai * ai), atan2(ai, ar));
            const long w = (long)orow * m + tid;
            W_s[tid] = make_float2(P1[2 * w], P1[2 * w + 1]);
        }
    }
    __syncthreads();
    for (int i = tid; i < m * KG_T; i += KG_THREADS) {
        int n = i / KG_T, b = i % KG_T;
        double2 l = lam_s[n];
        Q_s[n][b] = cexp_scaled((double)b, l.x, l.y);
    }
    for (int i = tid; i < m * KG_A; i += KG_THREADS) {
        int a = i / m, n = i % m;
        double2 l = lam_s[n];
        P_s[a][n] = cmul(W_s[n], cexp_scaled((double)(t0 + KG_T * a), l.x, l.y));
    }
    __syncthreads();
    // thread -> (b, 8 consecutive a)
    const int b = tid % KG_T;
    const int a0 = (tid / KG_T) * 8;
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
    for (int n = 0; n < m; ++n) {
        float2 q = Q_s[n][b];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float2 p = P_s[a0 + j][n];
            acc[j] = fmaf(p.x, q.x, acc[j]);
            acc[j] = fmaf(-p.y, q.y, acc[j]);
        }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        int t = t0 + KG_T * (a0 + j) + b;
        if (t < L) k[(long)orow * L + t] = 2.f * acc[j];
    }
}

// ------------------------------------------------------ matrix-core form ---
// k[64 a + b] = 2 sum_n (Re P[a][n] Re Q[n][b] - Im P[a][n] Im Q[n][b]) is a real
// matrix product with reduction length 2m (m <= 64, zero-padded to 128):
//   Pm[a][j] = Re P[a][j] (j < 64), -Im P[a][j-64] (j >= 64)
//   Qm[j][b] = Re Q[j][b] (j < 64),  Im Q[j-64][b] (j >= 64)
// with P[a][n] = W_n z_n^{64 a}, Q[n][b] = z_n^b, z_n = exp(lambda_n), run as
// 16x16x4 fp32 MFMAs (exact fp32 products, fp32 accumulation).  A workgroup (4
// waves) produces rows a = a0 .. a0 + 16 NR - 1 (1024 NR outputs; NR = 4 once
// a row has 64 or more of them, so that the per-workgroup setup is shared by
// twice the outputs and long kernels need half the workgroups); wave w owns
// columns b = 16 w .. 16 w + 15.  The powers z^e are formed in float64 by repeated
// squaring and multiplication (relative error ~ e * 1e-16), so no phase is
// ever reduced in float32.
//
// Every wave derives z_n and W_n for mode n = lane itself (the global loads are
// issued first, the three float64 transcendentals of the ZOH run on three
// waves in parallel), so the power tables are built straight from registers:
// one barrier before the tables are complete, none around the mode setup
// beyond the exchange of the transcendentals.
//
// The reduction index is permuted so that MFMA step s of lane (r, q) uses
// j = 32 q + s: four consecutive steps read one 16-byte LDS word.
constexpr int KM_LD = 128 + 4;   // LDS row pitch in floats
typedef float f4v_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double2 zmul(double2 a, double2 b) {
    return make_double2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ double2 zpow(double2 z, int e) {
    double2 r = make_double2(1.0, 0.0);
    while (e) {
        if (e & 1) r = zmul(r, z);
        z = zmul(z, z);
        e >>= 1;
    }
    return r;
}

// mode 0: continuous (A, B, dt), ZOH.  mode 1: discrete (Abar, Bbar), W = C Bbar.
// mode 2: discrete Abar of channel (orow / div) % H, W given per output row in P1.
template <int NR>
__global__ __launch_bounds__(256) void kernel_gen_mfma(int mode, const float *P0, const float *P1,
                                                       const float *C, const float *dt, int H,
                                                       int m, int L, float *k, int div) {
    __shared__ double pre[3][H3_MAX_MODES_DEV];
    __shared__ float Qt[64][KM_LD];          // [b][j]  (Qm transposed)
    constexpr int KM_ROWS = 16 * NR;
    __shared__ float Pm[KM_ROWS][KM_LD];     // [a][j]
    const int nrt = (L / 64 + KM_ROWS - 1) / KM_ROWS;  // row tiles per output row
    const int orow = blockIdx.x / nrt;
    const int a0 = (blockIdx.x % nrt) * KM_ROWS;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int n = lane;
    const bool act = n < m;
    const int h = (mode == 2) ? (orow / div) % H : orow;
    // ---- loads first (every wave, lane n = mode n)
    double ar = 0.0, ai = 0.0, pr = 0.0, pi = 0.0, cr = 0.0, ci = 0.0, d = 0.0;
    if (act) {
        const long i = (long)h * m + n;
        const float2 a2 = *(const float2 *)(P0 + 2 * i);
        ar = a2.x; ai = a2.y;
        const long pi_ = (mode == 2) ? (long)orow * m + n : i;
        const float2 p2 = *(const float2 *)(P1 + 2 * pi_);
        pr = p2.x; pi = p2.y;
        if (mode != 2) {
            const float2 c2 = *(const float2 *)(C + 2 * i);
            cr = c2.x; ci = c2.y;
        }
        if (mode == 0) d = dt[h];
    }
    // ---- z_n = exp(lambda_n) and W_n, in every wave
    double2 z = make_double2(0.0, 0.0);
    float2 Wn = make_float2(0.f, 0.f);
    if (mode == 0) {
        const double lr = d * ar, li = d * ai;
        if (w < 3 && act) pre[w][n] = w == 0 ? expm1(lr) : w == 1 ? cos(li) : sin(li);
        __syncthreads();
        if (act) {
            const double em1 = pre[0][n], cs = pre[1][n], sn = pre[2][n];
            const double e = em1 + 1.0;
            z = make_double2(e * cs, e * sn);
            // exp(lambda) - 1 = (e cos - 1) + i e sin, with e cos - 1 = em1 cos + (cos - 1)
            const double em1r = em1 * cs + (cs - 1.0), em1i = e * sn;
            const double den = ar * ar + ai * ai;
            const double qr = (em1r * ar + em1i * ai) / den, qi = (em1i * ar - em1r * ai) / den;
            const double br = qr * pr - qi * pi, bi = qr * pi + qi * pr;   // Bbar = (e^lambda - 1)/A * B
            Wn = make_float2((float)(cr * br - ci * bi), (float)(cr * bi + ci * br));
        }
    } else if (act) {
        z = make_double2(ar, ai);
        if (mode == 1)
            Wn = make_float2((float)(cr * pr - ci * pi), (float)(cr * pi + ci * pr));
        else
            Wn = make_float2((float)pr, (float)pi);
    }
    // ---- Q rows b = 16 w .. 16 w + 15 and P rows 4 NR w .. 4 NR w + 4 NR - 1 of mode n
    {
        double2 p = zpow(z, 16 * w);
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            Qt[16 * w + j][n] = (float)p.x;
            Qt[16 * w + j][64 + n] = (float)p.y;
            p = zmul(p, z);
        }
        const double2 z64 = zpow(z, 64);
        double2 q = zpow(z64, a0 + 4 * NR * w);
#pragma unroll
        for (int j = 0; j < 4 * NR; ++j) {
            const float qr = (float)q.x, qi = (float)q.y;
            Pm[4 * NR * w + j][n] = Wn.x * qr - Wn.y * qi;
            Pm[4 * NR * w + j][64 + n] = -(Wn.x * qi + Wn.y * qr);
            q = zmul(q, z64);
        }
    }
    __syncthreads();
    // wave w: NR 16 x 16 tiles (rows a0 + 16 i .. a0 + 16 i + 15) of columns
    // 16 w .. 16 w + 15; lane (r, q) at step s uses reduction index 32 q + s
    f4v_t acc[NR];
#pragma unroll
    for (int i = 0; i < NR; ++i) acc[i] = (f4v_t){0.f, 0.f, 0.f, 0.f};
    const int r = lane & 15, kq = lane >> 4;
#pragma unroll
    for (int s4 = 0; s4 < 32; s4 += 4) {
        const float4 bv = *(const float4 *)&Qt[16 * w + r][32 * kq + s4];
        float4 pv[NR];
#pragma unroll
        for (int i = 0; i < NR; ++i) pv[i] = *(const float4 *)&Pm[16 * i + r][32 * kq + s4];
#pragma unroll
        for (int i = 0; i < NR; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i].x, bv.x, acc[i], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < NR; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i].y, bv.y, acc[i], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < NR; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i].z, bv.z, acc[i], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < NR; ++i) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(pv[i].w, bv.w, acc[i], 0, 0, 0);
    }
    // lane holds rows a0 + 16 i + 4 kq + j, column 16 w + r
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int t = 64 * (a0 + 4 * kq + j) + 16 * w + r;
#pragma unroll
        for (int i = 0; i < NR; ++i)
            if (t + 1024 * i < L) k[(long)orow * L + t + 1024 * i] = 2.f * acc[i][j];
    }
}

// Rows of 64 outputs per workgroup: 64 once the output row holds that many
// (half the workgroups, each sharing its setup among twice the outputs), else 32.
static inline int kgen_rows(int L) { return L / 64 >= 64 ? 64 : 32; }

static void launch_kgen_mfma(int mode, const float *P0, const float *P1, const float *C, const float *dt,
                             int H, int m, int L, float *k, int div, long nrows, hipStream_t s) {
    const int R = kgen_rows(L);
    const long nrt = (L / 64 + R - 1) / R;
    const dim3 grid((unsigned)(nrt * nrows)), block(256);
    if (R == 64)
        hipLaunchKernelGGL(kernel_gen_mfma<4>, grid, block, 0, s, mode, P0, P1, C, dt, H, m, L, k, div);
    else
        hipLaunchKernelGGL(kernel_gen_mfma<2>, grid, block, 0, s, mode, P0, P1, C, dt, H, m, L, k, div);
}

hipError_t launch_discretize(const float *A, const float *B, const float *dt, int H, int m,
                             float *Abar, float *Bbar, hipStream_t s) {
    int n = H * m;
    hipLaunchKernelGGL(discretize_kernel, dim3((n + 255) / 256), dim3(256), 0, s, A, B, dt, H, m,
                       Abar, Bbar);
    return hipGetLastError();
}

hipError_t launch_kernel_gen(int mode, const float *P0, const float *P1, const float *C,
                             const float *dt, int H, int m, int L, float *k, hipStream_t s) {
    if (L % 64 == 0) {
        launch_kgen_mfma(mode, P0, P1, C, dt, H, m, L, k, 1, H, s);
        return hipGetLastError();
    }
    const long ntile = (L + KG_TT - 1) / KG_TT;
    hipLaunchKernelGGL(kernel_gen, dim3((unsigned)(ntile * H)), dim3(KG_THREADS), 0, s, mode, P0, P1,
                       C, dt, H, m, L, k, 1);
    return hipGetLastError();
}

hipError_t launch_state_correction(const float *Abar, const float2 *corr_W, int B, int H, int m,
                                   int chunk, int nchunk, float *corr, hipStream_t s) {
    const long orows = (long)B * H * nchunk;
    if (chunk % 64 == 0) {
        launch_kgen_mfma(2, Abar, (const float *)corr_W, nullptr, nullptr, H, m, chunk, corr, nchunk, orows, s);
        return hipGetLastError();
    }
    const long ntile = (chunk + KG_TT - 1) / KG_TT;
    hipLaunchKernelGGL(kernel_gen, dim3((unsigned)(ntile * orows)), dim3(KG_THREADS), 0, s, 2, Abar,
                       (const float *)corr_W, (const float *)nullptr, (const float *)nullptr, H, m,
                       chunk, corr, nchunk);
    return hipGetLastError();
}

}  // namespace h3
