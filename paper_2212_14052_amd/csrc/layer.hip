// H3 layer forward pieces (Sec. 3.2, Algorithm 1 with head dimension 1), gfx950.
//
//   [Q;K;V] channel-major  = Wt_qkv . x^T          (MFMA GEMM, bf16/fp16 in, fp32 acc)
//   O = Q * (diag_k (*) (Kbar * V) + D (Kbar * V)),  Kbar = shift FIR of K
//                                                  (one fused kernel per row pair)
//   out = O . Wo                                    (MFMA GEMM)
// The projections are the layer's dense contractions (O(d^2 N), Proposition 1)
// and run on the matrix cores; the sequence mixing is the fused FFT conv.
#include "common.h"
#include "fft_valu.h"
#include "internal.h"

namespace h3 {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f4_t __attribute__((ext_vector_type(4)));

template <int DT> struct Mfma;
template <> struct Mfma<F16> {
    static __device__ __forceinline__ f32x16_t run(uint4 a, uint4 b, f32x16_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(*(half8_t *)&a, *(half8_t *)&b, c, 0, 0, 0);
    }
};
template <> struct Mfma<BF16> {
    static __device__ __forceinline__ f32x16_t run(uint4 a, uint4 b, f32x16_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(*(bf16x8_t *)&a, *(bf16x8_t *)&b, c, 0, 0, 0);
    }
};

// Store one 32x32 accumulator tile (rows mb + 8(e/4) + e%4 for the lane,
// column n) with the output layout chosen at compile time.
template <int DT, int OUT>
__device__ __forceinline__ void store_tile(uint16_t *C, const f32x16_t &acc, int mb, int n, int N, int d, int L) {
    long nofs;
    if constexpr (OUT == 0) {
        nofs = n;
    } else {
        nofs = (long)(n / L) * ((long)d * L) + (n % L);
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int m = mb + 8 * (e >> 2) + (e & 3);
        const uint16_t o = (DT == BF16) ? f32_to_bf16(acc[e]) : f32_to_f16(acc[e]);
        long dst;
        if constexpr (OUT == 0)
            dst = (long)m * N + nofs;
        else
            dst = (long)(m / d) * ((long)N * d) + (long)(m % d) * L + nofs;
        C[dst] = o;
    }
}

// Output-tile order for the GEMMs: the hardware block index is first remapped
// so that consecutive logical indices run on one XCD (its own L2), then
// logical indices walk groups of GROUP_M tile rows column by column, so the
// 32 or so tiles an XCD runs at once form a GROUP_M x 8 block that shares
// GROUP_M A panels and 8 B panels (a 1 x 32 row would share one A panel and
// no B panel).
constexpr int GEMM_GROUP_M = 4;
__device__ __forceinline__ void gemm_tile(int nbm, int nbn, int &tm, int &tn) {
    const int l = xcd_logical_block(blockIdx.x, gridDim.x);
    const int g = l / (GEMM_GROUP_M * nbn), rem = l - g * GEMM_GROUP_M * nbn;
    const int gm = min(GEMM_GROUP_M, nbm - g * GEMM_GROUP_M);
    tm = g * GEMM_GROUP_M + rem % gm;
    tn = rem / gm;
}

// ------------------------------------------------------------------ GEMM ---
// C = A . Bt^T with A (M, K) and Bt (N, K) both K-contiguous (16-bit), fp32
// accumulation, 16-bit result.  Tile 128 x 128 x 32, 4 waves of 64 x 64, each
// a 2 x 2 grid of 32x32x16 MFMAs.  Requires M, N % 128 == 0 and K % 32 == 0.
// out_mode 0: C row-major (M, N).
// out_mode 1: rows are channels of [Q;K;V] (M = 3 d), columns tokens
//             (N = B L); element (m, n) goes to
//             [(m / d)][(n / L)][(m % d)][(n % L)]  (three (B, d, L) tensors).
constexpr int GB_M = 128, GB_N = 128, GB_K = 32, GB_LDK = GB_K + 8;

template <int DT, int OUT>
__global__ __launch_bounds__(256) void gemm_nt_kernel(const uint16_t *A, const uint16_t *Bt,
                                                      uint16_t *C, int M, int N, int K, int d, int L) {
    __shared__ __attribute__((aligned(16))) uint16_t As[GB_M * GB_LDK];
    __shared__ __attribute__((aligned(16))) uint16_t Bs[GB_N * GB_LDK];
    int tm, tn;
    gemm_tile(M / GB_M, N / GB_N, tm, tn);
    const int m0 = tm * GB_M, n0 = tn * GB_N;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int wm = w >> 1, wn = w & 1;
    // global -> register staging: 2 x 16 B of A and of B per thread
    const int lr = t >> 2, lk = (t & 3) * 8;
    const uint16_t *ga = A + (long)(m0 + lr) * K + lk, *gb = Bt + (long)(n0 + lr) * K + lk;
    const long g64 = 64L * K;
    uint16_t *la = As + lr * GB_LDK + lk, *lb = Bs + lr * GB_LDK + lk;
    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    uint4 a0 = *(const uint4 *)(ga), a1 = *(const uint4 *)(ga + g64);
    uint4 b0 = *(const uint4 *)(gb), b1 = *(const uint4 *)(gb + g64);
    *(uint4 *)(la) = a0; *(uint4 *)(la + 64 * GB_LDK) = a1;
    *(uint4 *)(lb) = b0; *(uint4 *)(lb + 64 * GB_LDK) = b1;
    __syncthreads();
    for (int k0 = 0; k0 < K; k0 += GB_K) {
        const bool more = k0 + GB_K < K;
        if (more) {
            const int k1 = k0 + GB_K;
            a0 = *(const uint4 *)(ga + k1); a1 = *(const uint4 *)(ga + g64 + k1);
            b0 = *(const uint4 *)(gb + k1); b1 = *(const uint4 *)(gb + g64 + k1);
        }
#pragma unroll
        for (int ks = 0; ks < GB_K / 16; ++ks) {
            uint4 af[2], bf[2];
            const int kk = ks * 16 + 8 * (lane >> 5);
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                af[i] = *(const uint4 *)(As + (wm * 64 + i * 32 + (lane & 31)) * GB_LDK + kk);
                bf[i] = *(const uint4 *)(Bs + (wn * 64 + i * 32 + (lane & 31)) * GB_LDK + kk);
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = Mfma<DT>::run(af[i], bf[j], acc[i][j]);
        }
        __syncthreads();
        if (more) {
            *(uint4 *)(la) = a0; *(uint4 *)(la + 64 * GB_LDK) = a1;
            *(uint4 *)(lb) = b0; *(uint4 *)(lb + 64 * GB_LDK) = b1;
            __syncthreads();
        }
    }
    // epilogue: lane holds column (lane & 31) and rows 8(e/4) + 4(lane/32) + e%4
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            store_tile<DT, OUT>(C, acc[i][j], m0 + wm * 64 + i * 32 + 4 * (lane >> 5),
                                n0 + wn * 64 + j * 32 + (lane & 31), N, d, L);
}

// ------------------------------------------------------ GEMM, large tiles ---
// Same contract as gemm_nt_kernel for M, N % 256 == 0 and K % 64 == 0.
// Block tile 256 x 256 x 64, 8 waves as 2 (M) x 4 (N), each wave 128 x 64 =
// 4 x 2 tiles of 32x32x16 MFMA (fp32 accumulators, 128 per lane).  LDS holds
// two stages of A and B (rows padded to 72 elements: 16-byte fragment reads
// of 8 consecutive rows hit 8 different bank groups); the next stage is
// fetched into registers while the current one is multiplied, so one barrier
// per K step suffices.  Tiles run in the grouped order of gemm_tile.
constexpr int G2_M = 256, G2_N = 256, G2_K = 64, G2_LD = G2_K + 8, G2_T = 512;

template <int DT, int OUT>
__global__ __launch_bounds__(G2_T) void gemm_nt_256(const uint16_t *A, const uint16_t *Bt, uint16_t *C,
                                                    int M, int N, int K, int d, int L) {
    extern __shared__ __attribute__((aligned(16))) uint16_t g2_lds[];
    uint16_t *As = g2_lds;                          // [2][256][72]
    uint16_t *Bs = g2_lds + 2 * G2_M * G2_LD;       // [2][256][72]
    int tm, tn;
    gemm_tile(M / G2_M, N / G2_N, tm, tn);
    const int m0 = tm * G2_M, n0 = tn * G2_N;
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    const int wm = w >> 2, wn = w & 3;
    // loader mapping: thread -> rows t / 8 + 64 i, 16-byte column chunk (t % 8) * 8
    const int lr = t >> 3, lk = (t & 7) * 8;
    const uint16_t *ga = A + (long)(m0 + lr) * K + lk, *gb = Bt + (long)(n0 + lr) * K + lk;
    const long g64 = 64L * K;
    uint16_t *la = As + lr * G2_LD + lk, *lb = Bs + lr * G2_LD + lk;
    f32x16_t acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    uint4 a0 = *(const uint4 *)(ga), a1 = *(const uint4 *)(ga + g64), a2 = *(const uint4 *)(ga + 2 * g64),
          a3 = *(const uint4 *)(ga + 3 * g64);
    uint4 b0 = *(const uint4 *)(gb), b1 = *(const uint4 *)(gb + g64), b2 = *(const uint4 *)(gb + 2 * g64),
          b3 = *(const uint4 *)(gb + 3 * g64);
    constexpr int S64 = 64 * G2_LD, STAGE = G2_M * G2_LD;
    *(uint4 *)(la) = a0; *(uint4 *)(la + S64) = a1; *(uint4 *)(la + 2 * S64) = a2; *(uint4 *)(la + 3 * S64) = a3;
    *(uint4 *)(lb) = b0; *(uint4 *)(lb + S64) = b1; *(uint4 *)(lb + 2 * S64) = b2; *(uint4 *)(lb + 3 * S64) = b3;
    __syncthreads();
    const int nk = K / G2_K;
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) {
            const int k1 = (kt + 1) * G2_K;
            a0 = *(const uint4 *)(ga + k1); a1 = *(const uint4 *)(ga + g64 + k1);
            a2 = *(const uint4 *)(ga + 2 * g64 + k1); a3 = *(const uint4 *)(ga + 3 * g64 + k1);
            b0 = *(const uint4 *)(gb + k1); b1 = *(const uint4 *)(gb + g64 + k1);
            b2 = *(const uint4 *)(gb + 2 * g64 + k1); b3 = *(const uint4 *)(gb + 3 * g64 + k1);
        }
        const uint16_t *as = As + buf * STAGE, *bs = Bs + buf * STAGE;
#pragma unroll
        for (int ks = 0; ks < G2_K / 16; ++ks) {
            const int kk = ks * 16 + 8 * (lane >> 5);
            uint4 af[4], bf[2];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                af[i] = *(const uint4 *)(as + (wm * 128 + i * 32 + (lane & 31)) * G2_LD + kk);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bf[j] = *(const uint4 *)(bs + (wn * 64 + j * 32 + (lane & 31)) * G2_LD + kk);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) acc[i][j] = Mfma<DT>::run(af[i], bf[j], acc[i][j]);
        }
        if (more) {
            uint16_t *sa = la + (buf ^ 1) * STAGE, *sb = lb + (buf ^ 1) * STAGE;
            *(uint4 *)(sa) = a0; *(uint4 *)(sa + S64) = a1; *(uint4 *)(sa + 2 * S64) = a2; *(uint4 *)(sa + 3 * S64) = a3;
            *(uint4 *)(sb) = b0; *(uint4 *)(sb + S64) = b1; *(uint4 *)(sb + 2 * S64) = b2; *(uint4 *)(sb + 3 * S64) = b3;
        }
        __syncthreads();
    }
    // epilogue: lane holds column (lane & 31) and rows 8(e/4) + 4(lane/32) + e%4
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
            store_tile<DT, OUT>(C, acc[i][j], m0 + wm * 128 + i * 32 + 4 * (lane >> 5),
                                n0 + wn * 64 + j * 32 + (lane & 31), N, d, L);
}

// ------------------------------------------- GEMM, TW x 256 weight tiles ---
// C = W^T . X^T with the weights W (K, ldw) as stored (input features along
// the rows, output features contiguous: the projections of Algorithm 1 as
// written, Q = x W_Q) and the activations X (Nx, K) K-contiguous, 16-bit, fp32
// accumulation.  Mw output features: for OUT 1 the three projections Q, K, V
// (Mw = 3 d, weight tile rows w0 .. from W_{w0 / d}), for OUT 0 one (Mw = d).
// Block tile TW (output features: 320 or 256) x 256 (activation rows) x 32.
// At d = 2560 (a multiple of 320) the fused Q/K/V projection and the output
// projection over Nx = B L = 8192 tokens are 768 and 256 tiles of 320 x 256:
// whole rounds of the 256 CUs, where 256 x 256 tiles leave the last round a
// quarter full.  Eight waves, 2 (weight) x 4 (activation), each (TW / 2) x 64
// = (TW / 64) x 2 tiles of 32x32x16 MFMA (up to 160 fp32 accumulators per
// lane, two waves per SIMD).
// Operands reach LDS without passing through registers: each wave copies
// 1 KB slices of a stage (64 lanes x 16 bytes, lane i to byte 16 i of the
// slice) with global_load_lds_dwordx4, four stages deep (copies run three K
// steps ahead; a stage is waited for with vmcnt and one barrier per K step,
// which also orders the refill of the buffer read in the step before).
// A stage holds
//  - the weight tile as stored: 32 rows (k) of TW output features, row pitch
//    WP = 2 TW + 64 bytes (the last 64 bytes of a row are filled with
//    unused data).  A fragment (8 consecutive k of one output feature per
//    lane) is read with two transposing LDS reads (ds_read_b64_tr_b16: in a
//    group of 16 lanes, lane 4 i + q reads 4 features f0 + 4 q .. + 3 of row
//    k0 + i, and lane j receives rows k0 .. k0 + 3 of feature f0 + j).  With
//    WP = 64 or 192 (mod 256) the four rows of a read sit at distinct 64-byte
//    positions of the 256-byte bank row: no bank conflicts;
//  - the activation tile: 256 rows of 32 values (64 B, four 16-byte chunks),
//    chunk c of row r at slot c ^ ((r / 4) % 4), read with ds_read_b128 (16
//    consecutive rows, one chunk, per LDS cycle on 16 distinct bank groups).
// OUT 1: element (m, n) = (output feature of Q|K|V, activation row) goes to
//        the channel-major [Q;K;V] layout [(m / d)][(n / L)][(m % d)][(n % L)]
//        (d a multiple of TW: a tile lies in one projection), with the
//        activation rows along the MFMA columns (lanes), so 32 consecutive
//        tokens of one channel are one 64-byte run;
// OUT 0: element (n, m) of a row-major (Nx, Mw) result, with the output
//        features along the MFMA columns (lanes) for 64-byte runs.
constexpr int GW_X = 256, GW_K = 32, GW_T = 512, GW_NS = 4;

typedef __attribute__((address_space(3))) void lds_void;
typedef short gw_v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) gw_v4s lds_v4s;

__device__ __forceinline__ int gw_xoff(int row, int chunk) { return row * 64 + ((chunk ^ ((row >> 2) & 3)) << 4); }

template <int TW, int SS, bool XKM> struct GwShape {
    static constexpr int WP = 2 * TW + 64;            // weight row pitch, bytes (704 or 576)
    static constexpr int WB = GW_K * WP;              // weight part of a stage, bytes
    static constexpr int WS = WB / 1024;              // its slices (22 or 18)
    static constexpr int XP = 2 * GW_X + 64;          // K-major activation row pitch, bytes (576)
    static constexpr int XB = XKM ? GW_K * XP : GW_X * 64;   // activation part of a stage, bytes
    static constexpr int XS = XB / 1024;              // its slices (18 or 16)
    static constexpr int SLICES = WS + XS;
    static constexpr int NSL = (SLICES + 7) / 8;      // copies per wave per step (5)
    static constexpr int STAGE_B = WB + XB;           // bytes per stage
    static constexpr int TI = TW / 64;                // weight-side MFMA tiles per wave
    static_assert(WB % 1024 == 0 && (WP % 256 == 64 || WP % 256 == 192), "weight stage layout");
    // LDS bytes: the stages, and a 1 KB slot that takes the copies of waves
    // with fewer slices (never read), so every wave issues NSL per step
    static constexpr size_t LDS = (size_t)GW_NS * STAGE_B + (SLICES % 8 ? 1024 : 0);
    // SS stages are consumed per barrier (one super-step); the copies of the
    // next GW_NS / SS - 1 super-steps are in flight meanwhile.  s_waitcnt
    // immediate for vmcnt((GW_NS / SS - 2) SS NSL): the copies issued after
    // the super-step waited for may stay in flight (expcnt, lgkmcnt not waited)
    static constexpr int INFL = (GW_NS / SS - 2) * SS * NSL;
    static constexpr int WAIT = 0xf70 | (INFL & 15) | ((INFL >> 4) << 14);
};

// OUT 2: as OUT 0, with the activations stored K-major, (B, K, L) with row
// n = b L + t of X at column t of batch b (the gated O of the layer as the
// convolution writes it, channel-major): a stage then holds 32 rows (k) of
// 256 activation rows, pitch XP, and the fragments are read with transposing
// LDS reads like the weights.
template <int DT, int OUT, int TW, int SS>
__global__ __launch_bounds__(GW_T) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_w(
    const uint16_t *W0, const uint16_t *W1, const uint16_t *W2, const uint16_t *X, uint16_t *C, int Mw, int Nx,
    int K, int ldw, int d, int L) {
    constexpr bool XKM = OUT == 2;
    using S = GwShape<TW, SS, XKM>;
    extern __shared__ __attribute__((aligned(1024))) uint16_t gw_lds[];
    int tw, tx;
    gemm_tile(Mw / TW, Nx / GW_X, tw, tx);
    const int w0 = tw * TW, x0 = tx * GW_X;
    const int jq = OUT == 1 ? w0 / d : 0;   // the projection this tile row belongs to
    const uint16_t *Wj = jq == 0 ? W0 : (jq == 1 ? W1 : W2);
    const int wc = w0 - jq * d;             // first output feature of the tile within W_jq
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int ww = wv >> 2, wx = wv & 3;
    // this wave's slices q = wv + 8 s, s < NSL (a wave past the last slice
    // copies slice wv again into the never-read slot): the lane's source as an
    // element offset from the operand's base (W_jq for q < WS, X after) at
    // K step 0; a step adds 32 rows of W (32 ldw) or 32 columns of X
    const int wvu = __builtin_amdgcn_readfirstlane(wv);   // the wave index, in a scalar register
    uint32_t soff[S::NSL];
#pragma unroll
    for (int sl = 0; sl < S::NSL; ++sl) {
        const int q = wvu + 8 * sl < S::SLICES ? wvu + 8 * sl : wvu;
        if (q < S::WS) {
            const int b = 1024 * q + 16 * lane;
            const int r = b / S::WP, c = b % S::WP;
            soff[sl] = (uint32_t)(r * ldw + wc + (c < 2 * TW ? c / 2 : 0));
        } else if constexpr (XKM) {
            // rows k of the tile's 256 activation rows, which lie in batch x0 / L
            const int b = 1024 * (q - S::WS) + 16 * lane;
            const int r = b / S::XP, c = b % S::XP;
            soff[sl] = (uint32_t)((x0 / L) * K * L + (x0 % L) + r * L + (c < 2 * GW_X ? c / 2 : 0));
        } else {
            const int r = 16 * (q - S::WS) + (lane >> 2);
            const int c = (lane & 3) ^ ((r >> 2) & 3);
            soff[sl] = (uint32_t)((x0 + r) * K + 8 * c);
        }
    }
    const int nk = K / GW_K;
    // The copies are issued as inline assembly (M0 = the slice's LDS byte
    // address, then global_load_lds_dwordx4 with the operand base in SGPRs
    // and the lane's byte offset): the compiler then places no wait of its
    // own for them before LDS reads; the explicit vmcnt waits order them.
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void *)gw_lds;
    // copies of K step kt (clamped to the last step: past it they only keep
    // the count per step fixed) into stage kt % GW_NS
    auto issue = [&](int kt) {
        const uint32_t st = lds0 + (uint32_t)((kt % GW_NS) * S::STAGE_B);
        const uint32_t k0 = (uint32_t)min(kt, nk - 1) * GW_K;
#pragma unroll
        for (int sl = 0; sl < S::NSL; ++sl) {
            const int q = wvu + 8 * sl;
            const bool real = q < S::SLICES;
            const bool wside = (real ? q : wvu) < S::WS;
            const uint16_t *base = wside ? Wj : X;
            const uint32_t vo = 2 * (soff[sl] + k0 * (wside ? (uint32_t)ldw : (XKM ? (uint32_t)L : 1u)));
            const uint32_t la = real ? st + (uint32_t)q * 1024 : lds0 + (uint32_t)(GW_NS * S::STAGE_B);
            asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, %2"
                         :
                         : "v"(vo), "s"(la), "s"(base)
                         : "memory", "m0");
        }
    };
    f32x16_t acc[S::TI][2];
#pragma unroll
    for (int i = 0; i < S::TI; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

    // transposing weight reads: lane 4 i + q of each 16-lane group reads row
    // k0 + i, features f0 + 4 q .. + 3; f0 = the tile's first feature + 16
    // for the upper 16 lanes of each 32
    const int tr_row = (lane & 15) >> 2, tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const int tr_base = tr_row * S::WP + 2 * (ww * (TW / 2) + tr_col);
    const int trx_base = tr_row * S::XP + 2 * (wx * 64 + tr_col);
#pragma unroll
    for (int p = 0; p < GW_NS - SS; ++p) issue(p);
    for (int k0 = 0; k0 < nk; k0 += SS) {
        // the stages of this super-step landed for this wave (the copies of
        // later super-steps may still be in flight), then for every wave; the
        // reads of the buffers refilled next (last super-step's) are done.  A
        // bare barrier: a fenced one would also drain the copies in flight.
        __builtin_amdgcn_s_waitcnt(S::WAIT);
        asm volatile("s_barrier" ::: "memory");
#pragma unroll
        for (int p = 0; p < SS; ++p) issue(k0 + GW_NS - SS + p);
#pragma unroll
        for (int p = 0; p < SS; ++p) {
            const int kt = k0 + p;   // nk is a multiple of SS
            const char *stg = (const char *)gw_lds + (kt % GW_NS) * S::STAGE_B;
            const char *xs = stg + S::WB;
#pragma unroll
            for (int ks = 0; ks < GW_K / 16; ++ks) {
                uint4 fw[S::TI], fx[2];
                // weight rows 16 ks + 8 (lane / 32) + 4 h + (0..3)
                const char *wr = stg + (16 * ks + 8 * (lane >> 5)) * S::WP + tr_base;
#pragma unroll
                for (int i = 0; i < S::TI; ++i) {
                    const gw_v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(wr + 64 * i));
                    const gw_v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(wr + 4 * S::WP + 64 * i));
                    const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
                    fw[i] = make_uint4(l2.x, l2.y, h2.x, h2.y);
                }
                if constexpr (XKM) {
                    // activation rows wx 64 + 32 j + (lane & 31), k as for the weights
                    const char *xr = xs + (16 * ks + 8 * (lane >> 5)) * S::XP + trx_base;
#pragma unroll
                    for (int j = 0; j < 2; ++j) {
                        const gw_v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(xr + 64 * j));
                        const gw_v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(xr + 4 * S::XP + 64 * j));
                        const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
                        fx[j] = make_uint4(l2.x, l2.y, h2.x, h2.y);
                    }
                } else {
                    const int ch = 2 * ks + (lane >> 5);
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        fx[j] = *(const uint4 *)(xs + gw_xoff(wx * 64 + j * 32 + (lane & 31), ch));
                }
#pragma unroll
                for (int i = 0; i < S::TI; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = OUT == 1 ? Mfma<DT>::run(fw[i], fx[j], acc[i][j])
                                             : Mfma<DT>::run(fx[j], fw[i], acc[i][j]);
            }
        }
    }
    // no copy may land in LDS after the workgroup ends
    __builtin_amdgcn_s_waitcnt(0xf70);   // vmcnt(0)
    // epilogue: the lane holds MFMA column (lane & 31) and rows 8 (e / 4) +
    // 4 (lane / 32) + e % 4; element e of a tile lands at base + rstride x
    // (8 (e / 4) + e % 4)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int nx = x0 + wx * 64 + j * 32;
#pragma unroll
        for (int i = 0; i < S::TI; ++i) {
            const int mw = w0 + ww * (TW / 2) + i * 32;
            long base, rstride;
            if constexpr (OUT == 1) {
                const int n = nx + (lane & 31), m = mw + 4 * (lane >> 5);
                base = (long)jq * ((long)Nx * d) + (long)(n / L) * ((long)d * L) + (n % L) + (long)(m - jq * d) * L;
                rstride = L;
            } else {
                base = (long)(nx + 4 * (lane >> 5)) * Mw + mw + (lane & 31);
                rstride = Mw;
            }
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const float v = acc[i][j][e];
                uint16_t o;
                if constexpr (DT == BF16)
                    o = __builtin_bit_cast(uint16_t, (__bf16)v);
                else
                    o = __builtin_bit_cast(uint16_t, (_Float16)v);
                C[base + rstride * (8 * (e >> 2) + (e & 3))] = o;
            }
        }
    }
}

// --------------------------------------------------------- transposes ------
// out[b][c][r] = in[b][r][c] for batch of (R, C) matrices of 16-bit values.
__global__ __launch_bounds__(256) void transpose16_kernel(const uint16_t *in, uint16_t *out, int R,
                                                          int Cc) {
    __shared__ uint16_t tile[64][66];
    const int tr = (R + 63) / 64, tc = (Cc + 63) / 64;
    const int b = blockIdx.x / (tr * tc), rem = blockIdx.x % (tr * tc);
    const int r0 = (rem / tc) * 64, c0 = (rem % tc) * 64;
    const long off = (long)b * R * Cc;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int r = r0 + i, c = c0 + tx;
        if (r < R && c < Cc) tile[i][tx] = in[off + (long)r * Cc + c];
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int c = c0 + i, r = r0 + tx;
        if (r < R && c < Cc) out[off + (long)c * R + r] = tile[tx][i];
    }
}

// ------------------------------------------- transposes, 16-byte accesses ---
// out (C, R) = in (R, C)^T per batch slice (GATE = 0), or the gated transpose
// out (C, R) = (in * in2)^T with the product rounded once (GATE = 1).  A 64 x 64
// tile per workgroup; every global access moves 8 consecutive 16-bit values.
// Requires R % 8 == 0 and C % 8 == 0 (the callers' shapes are multiples of 64).
template <int DT, int GATE>
__global__ __launch_bounds__(256) void transpose_tile_kernel(const uint16_t *in, const uint16_t *in2,
                                                             uint16_t *out, int R, int Cc) {
    __shared__ uint16_t tile[64][64 + 8];   // [c][r]: stored transposed
    const int tr = (R + 63) / 64, tc = (Cc + 63) / 64;
    const int b = blockIdx.x / (tr * tc), rem = blockIdx.x % (tr * tc);
    const int r0 = (rem / tc) * 64, c0 = (rem % tc) * 64;
    const long off = (long)b * R * Cc;
    const int t = threadIdx.x;
    // read: thread -> (row r0 + t / 8 + 32 h, columns c0 + 8 (t % 8) .. + 7)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int i = t / 8 + 32 * h, cj = 8 * (t % 8);
        const int r = r0 + i, c = c0 + cj;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (r < R && c < Cc) {
            v = *(const uint4 *)(in + off + (long)r * Cc + c);
            if (GATE) {
                const uint4 g = *(const uint4 *)(in2 + off + (long)r * Cc + c);
                const uint32_t a4[4] = {v.x, v.y, v.z, v.w}, g4[4] = {g.x, g.y, g.z, g.w};
                uint32_t o4[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const float lo = (DT == BF16 ? bf16_to_f32(a4[e] & 0xffffu) : f16_to_f32(a4[e] & 0xffffu)) *
                                     (DT == BF16 ? bf16_to_f32(g4[e] & 0xffffu) : f16_to_f32(g4[e] & 0xffffu));
                    const float hi = (DT == BF16 ? bf16_to_f32(a4[e] >> 16) : f16_to_f32(a4[e] >> 16)) *
                                     (DT == BF16 ? bf16_to_f32(g4[e] >> 16) : f16_to_f32(g4[e] >> 16));
                    const uint32_t l16 = DT == BF16 ? f32_to_bf16(lo) : f32_to_f16(lo);
                    const uint32_t h16 = DT == BF16 ? f32_to_bf16(hi) : f32_to_f16(hi);
                    o4[e] = l16 | (h16 << 16);
                }
                v = make_uint4(o4[0], o4[1], o4[2], o4[3]);
            }
        }
        const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            tile[cj + 2 * e][i] = (uint16_t)(w4[e] & 0xffffu);
            tile[cj + 2 * e + 1][i] = (uint16_t)(w4[e] >> 16);
        }
    }
    __syncthreads();
    // write: thread -> (column c0 + t / 8 + 32 h, rows r0 + 8 (t % 8) .. + 7)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int i = t / 8 + 32 * h, rj = 8 * (t % 8);
        const int c = c0 + i, r = r0 + rj;
        if (c < Cc && r < R) *(uint4 *)(out + off + (long)c * R + r) = *(const uint4 *)&tile[i][rj];
    }
}

// ------------------------------------------------- shift SSM and gating ----
// G[b, c, t] = (sum_{j < m_s} shift_C[c, j] K[b, c, t - j] + shift_D[c] K[b, c, t]) V[b, c, t]
// (Sec. 3.2: the shift SSM's kernel is its taps, Algorithm 1 then gates with V),
// on (B, d, L) rows, fp32 arithmetic, one rounding to the I/O dtype.  One
// workgroup of 128 threads per row tile of 2048 outputs; thread -> 16
// consecutive outputs.  The taps are wave-uniform (scalar registers); the
// thread's window K[t0 - 63 .. t0 + 15] comes from the row staged in LDS.
constexpr int SG_T = 128, SG_R = 16, SG_TILE = SG_T * SG_R;
// GATE false: Kbar itself (no V), for heads of dimension > 1.
template <int DT, bool GATE>
__global__ __launch_bounds__(SG_T) void shift_gate_kernel(const uint16_t *k, const uint16_t *v,
                                                          const float *shift_C, const float *shift_D,
                                                          int m_s, int d, int L, uint16_t *g) {
    __shared__ __attribute__((aligned(16))) float ks[64 + SG_TILE];   // K[t_tile - 64 .. t_tile + SG_TILE - 1]
    __shared__ __attribute__((aligned(16))) float taps_s[64];
    const int ntile = (L + SG_TILE - 1) / SG_TILE;
    const long row = blockIdx.x / ntile;
    const int tt = (blockIdx.x % ntile) * SG_TILE;
    const int c = (int)(row % d);
    const uint16_t *kr = k + row * L;
    // every global load first, unconditional and in straight-line code
    // (addresses clamped into the row), so one memory round trip serves the
    // workgroup: this thread's V values, then its share of the K window
    const int t0 = SG_R * threadIdx.x;   // within the tile
    const bool act = tt + t0 < L;
    const long o = row * L + min(tt + t0, L - SG_R);
    uint4 vpre[SG_R / 8];
#pragma unroll
    for (int h = 0; h < SG_R / 8; ++h) vpre[h] = GATE ? *(const uint4 *)(v + o + 8 * h) : make_uint4(0, 0, 0, 0);
    constexpr int NKS = (64 + SG_TILE) / 8;   // 16-byte pieces of the window
    constexpr int PER = (NKS + SG_T - 1) / SG_T;
    uint4 kw[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int t = tt - 64 + 8 * (threadIdx.x + u * SG_T);
        kw[u] = *(const uint4 *)(kr + min(max(t, 0), L - 8));   // zeroed below where out of the row
    }
    const float tapv = threadIdx.x < 64 ? shift_C[(long)c * m_s + min((int)threadIdx.x, m_s - 1)] : 0.f;
    const float ds = shift_D ? shift_D[c] : 0.f;
    if (threadIdx.x < 64) taps_s[threadIdx.x] = (int)threadIdx.x < m_s ? tapv : 0.f;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int i = threadIdx.x + u * SG_T;
        const int t = tt - 64 + 8 * i;
        if (i < NKS) {
            const bool in = t >= 0 && t + 8 <= L;   // before the row start: causal zeros
            const uint32_t w4[4] = {kw[u].x, kw[u].y, kw[u].z, kw[u].w};
            float f[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                f[2 * e] = in ? (DT == BF16 ? bf16_to_f32(w4[e] & 0xffffu) : f16_to_f32(w4[e] & 0xffffu)) : 0.f;
                f[2 * e + 1] = in ? (DT == BF16 ? bf16_to_f32(w4[e] >> 16) : f16_to_f32(w4[e] >> 16)) : 0.f;
            }
            *(float4 *)&ks[8 * i] = make_float4(f[0], f[1], f[2], f[3]);
            *(float4 *)&ks[8 * i + 4] = make_float4(f[4], f[5], f[6], f[7]);
        }
    }
    __syncthreads();
    if (!act) return;
    float win[SG_R + 64];   // K[t0 - 64 .. t0 + 15]
#pragma unroll
    for (int i = 0; i < (SG_R + 64) / 4; ++i) {
        const float4 q = *(const float4 *)&ks[t0 + 4 * i];
        win[4 * i] = q.x; win[4 * i + 1] = q.y; win[4 * i + 2] = q.z; win[4 * i + 3] = q.w;
    }
    float acc[SG_R];
#pragma unroll
    for (int r = 0; r < SG_R; ++r) acc[r] = ds * win[64 + r];
    // taps 16 at a time (broadcast LDS reads), one tap across the 16 accumulators per group
#pragma unroll
    for (int jq = 0; jq < 64; jq += 16) {
        float tq[16];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float4 q = *(const float4 *)&taps_s[jq + 4 * i];
            tq[4 * i] = q.x; tq[4 * i + 1] = q.y; tq[4 * i + 2] = q.z; tq[4 * i + 3] = q.w;
        }
#pragma unroll
        for (int j = 0; j < 16; ++j) {
#pragma unroll
            for (int r = 0; r < SG_R; ++r) acc[r] = fmaf(tq[j], win[64 + r - jq - j], acc[r]);
            // keep the order tap-major: 16 independent FMAs between two uses
            // of an accumulator (the scheduler would otherwise run the 64
            // taps of one output as one dependent chain)
            asm volatile("" : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]),
                         "+v"(acc[6]), "+v"(acc[7]), "+v"(acc[8]), "+v"(acc[9]), "+v"(acc[10]), "+v"(acc[11]),
                         "+v"(acc[12]), "+v"(acc[13]), "+v"(acc[14]), "+v"(acc[15]));
        }
    }
#pragma unroll
    for (int h = 0; h < SG_R / 8; ++h) {
        const uint32_t v4[4] = {vpre[h].x, vpre[h].y, vpre[h].z, vpre[h].w};
        uint32_t o4[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            float lo = acc[8 * h + 2 * e], hi = acc[8 * h + 2 * e + 1];
            if (GATE) {
                lo *= DT == BF16 ? bf16_to_f32(v4[e] & 0xffffu) : f16_to_f32(v4[e] & 0xffffu);
                hi *= DT == BF16 ? bf16_to_f32(v4[e] >> 16) : f16_to_f32(v4[e] >> 16);
            }
            o4[e] = (uint32_t)(DT == BF16 ? f32_to_bf16(lo) : f32_to_f16(lo)) |
                    ((uint32_t)(DT == BF16 ? f32_to_bf16(hi) : f32_to_f16(hi)) << 16);
        }
        *(uint4 *)(g + o + 8 * h) = make_uint4(o4[0], o4[1], o4[2], o4[3]);
    }
}

// Matrix-core form of the same shift SSM and gating (L % 1024 == 0).  The
// 64-tap filter over 64-sample blocks is a banded Toeplitz product: with
// t = 64 a + r,
//   Kbar[64 a + r] = sum_{s < 128} T[r][s] K[64 (a - 1) + s],
//   T[r][s] = shift_C[r + 64 - s] for 0 <= r + 64 - s < 64 (+ shift_D on s = r + 64),
// so per row: a (64 x 128) . (128 x L/64) product on 16x16x32 MFMAs (fp32
// accumulation; the taps rounded to the I/O dtype).  T's band touches three of
// the four 32-wide reduction chunks of every 16-row block.  One wave per (b, c)
// row; the lane's MFMA result is four consecutive t of one block a, gated by V
// and stored as one 8-byte piece.
template <int DT>
__device__ __forceinline__ f4_t sg_mfma(uint4 a, uint4 b, f4_t c) {
    if constexpr (DT == BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, a), __builtin_bit_cast(half8_t, b), c, 0, 0, 0);
}
template <int DT>
__device__ __forceinline__ uint32_t sg_pack(float lo, float hi) {
    return (uint32_t)(DT == BF16 ? f32_to_bf16(lo) : f32_to_f16(lo)) |
           ((uint32_t)(DT == BF16 ? f32_to_bf16(hi) : f32_to_f16(hi)) << 16);
}
template <int DT>
__device__ __forceinline__ float sg_f(uint32_t h16) {
    return DT == BF16 ? bf16_to_f32(h16) : f16_to_f32(h16);
}
constexpr int SGM_W = 4;   // waves (channels) per workgroup
template <int DT, bool GATE>
__global__ __launch_bounds__(64 * SGM_W) void shift_gate_mfma_kernel(const uint16_t *k, const uint16_t *v,
                                                                      const float *shift_C, const float *shift_D,
                                                                      int m_s, int B, int d, int L, uint16_t *g) {
    __shared__ float taps[SGM_W][64 + 1];   // taps[w][j] = shift_C[c, j], [64] = shift_D[c]
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = blockIdx.x * SGM_W + w;   // this wave's channel: rows b d + c, b < B
    if (c >= d) return;                      // no barrier below: a spare wave may leave
    const int col = lane & 15, kg = lane >> 4;
    const int nab = L / 1024;                // 16-column blocks of 64-sample columns per row
    const int nit = B * nab;
    // loads of item it = (row b, column block ab): B fragments (chunk kc,
    // column a = 16 ab + col: K[64 (a - 1) + 32 kc + 8 kg .. + 7], zeros before
    // the row start) and V at the lane's outputs t = 64 a + 16 rb + 4 kg .. + 3
    uint4 Bf[4];
    uint2 Vq[4];
    auto issue = [&](int it) {
        const long ro = ((long)(it / nab) * d + c) * L;
        const int a = 16 * (it % nab) + col;
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) Bf[kc] = *(const uint4 *)(k + ro + max(64 * (a - 1) + 32 * kc + 8 * kg, 0));
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) Vq[rb] = GATE ? *(const uint2 *)(v + ro + 64 * a + 16 * rb + 4 * kg) : make_uint2(0, 0);
    };
    issue(0);   // in flight while the Toeplitz fragments are built
    taps[w][lane] = lane < m_s ? shift_C[(long)c * m_s + lane] : 0.f;
    if (lane == 0) taps[w][64] = shift_D ? shift_D[c] : 0.f;
    __builtin_amdgcn_wave_barrier();
    // A fragments: block rb, chunk kc = kc0(rb) + q; element i: r = 16 rb + col, s = 32 kc + 8 kg + i
    uint4 Af[4][3];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
        for (int q = 0; q < 3; ++q) {
            const int kc = (rb < 2 ? 0 : 1) + q;
            uint32_t e4[4];
#pragma unroll
            for (int i2 = 0; i2 < 4; ++i2) {
                float f2[2];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int r = 16 * rb + col, sidx = 32 * kc + 8 * kg + 2 * i2 + h;
                    const int j = r + 64 - sidx;
                    float val = 0.f;
                    if (j >= 0 && j < 64) val = taps[w][j] + (j == 0 ? taps[w][64] : 0.f);
                    f2[h] = val;
                }
                e4[i2] = sg_pack<DT>(f2[0], f2[1]);
            }
            Af[rb][q] = make_uint4(e4[0], e4[1], e4[2], e4[3]);
        }
    }
    for (int it = 0; it < nit; ++it) {
        const long ro = ((long)(it / nab) * d + c) * L;
        const int a = 16 * (it % nab) + col;
        uint4 B4[4];
        uint2 V4[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            B4[i] = 64 * (a - 1) + 32 * i + 8 * kg >= 0 ? Bf[i] : make_uint4(0, 0, 0, 0);
            V4[i] = Vq[i];
        }
        if (it + 1 < nit) issue(it + 1);   // the next item's loads overlap this item's products
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
            f4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < 3; ++q) acc = sg_mfma<DT>(Af[rb][q], B4[(rb < 2 ? 0 : 1) + q], acc);
            float g0 = acc[0], g1 = acc[1], g2 = acc[2], g3 = acc[3];
            if (GATE) {
                g0 *= sg_f<DT>(V4[rb].x & 0xffffu); g1 *= sg_f<DT>(V4[rb].x >> 16);
                g2 *= sg_f<DT>(V4[rb].y & 0xffffu); g3 *= sg_f<DT>(V4[rb].y >> 16);
            }
            *(uint2 *)(g + ro + 64 * a + 16 * rb + 4 * kg) = make_uint2(sg_pack<DT>(g0, g1), sg_pack<DT>(g2, g3));
        }
    }
}

// ------------------------------------------------------- fused middle ------
// Per pair of rows (batches 2j, 2j+1) of channel c, all (B, d, L):
//   G = (sum_{j<m_s} shift_C[c,j] K_{t-j} + shift_D[c] K_t) * V_t
//   S = diag_k (*) G + diag_D G      (FFT conv, packed as G_a + i G_b)
//   O = Q * S
template <int N, int DT>
__global__ __launch_bounds__(N / 16 >= 64 ? N / 16 : 64) void layer_mid_kernel(
    const uint16_t *q, const uint16_t *k, const uint16_t *v, const float *shift_C,
    const float *shift_D, int m_s, const float2 *Kspec, const float *diag_D, int B, int d,
    uint16_t *o, int npairs) {
    using P = FFTPlan<N>;
    using io = IO<DT>;
    constexpr int T = P::T, R1 = P::R1, Q = 16 / R1, HALF = R1 / 2;
    constexpr int S = (T >= 64) ? 1 : 64 / T;
    constexpr int L = N / 2;
    extern __shared__ float2 lds[];
    const int sig = threadIdx.x / T, tid = threadIdx.x % T;
    float2 *X = lds + sig * P::LDS;
    const int blk = xcd_logical_block(blockIdx.x, gridDim.x);
    const int p = blk * S + sig;
    const bool active = p < npairs;
    const int nbp = (B + 1) / 2;
    const int pp = active ? p : 0;
    const int c = pp / nbp, bp = pp % nbp;
    const long oa = ((long)(2 * bp) * d + c) * L;
    const bool hb = active && (2 * bp + 1 < B);
    const long ob = hb ? ((long)(2 * bp + 1) * d + c) * L : 0;

    // stage K of both rows in LDS (unpadded, index t)
    for (int t = tid; t < L; t += T) {
        const float ka = active ? io::ld(k, oa + t) : 0.f;
        const float kb = hb ? io::ld(k, ob + t) : 0.f;
        X[t] = make_float2(ka, kb);
    }
    __syncthreads();
    const float *cs = shift_C + (long)c * m_s;
    const float ds = shift_D ? shift_D[c] : 0.f;
    float2 vv[16];
    float ga[8], gb[8];
#pragma unroll
    for (int qq = 0; qq < Q; ++qq) {
        const int j = tid + qq * T;
#pragma unroll
        for (int r = 0; r < R1; ++r) {
            if (r < HALF) {
                const int n = j + r * (N / R1);
                float2 kb = cscale(X[n], ds);
                const int jmax = n < m_s - 1 ? n : m_s - 1;
                for (int jj = 0; jj <= jmax; ++jj) {
                    const float2 x = X[n - jj];
                    kb.x = fmaf(cs[jj], x.x, kb.x);
                    kb.y = fmaf(cs[jj], x.y, kb.y);
                }
                const float va = active ? io::ld(v, oa + n) : 0.f;
                const float vb = hb ? io::ld(v, ob + n) : 0.f;
                ga[qq * HALF + r] = kb.x * va;
                gb[qq * HALF + r] = kb.y * vb;
                vv[qq * R1 + r] = make_float2(kb.x * va, kb.y * vb);
            } else {
                vv[qq * R1 + r] = make_float2(0.f, 0.f);
            }
        }
    }
    __syncthreads();
    fft_forward_from_regs<N>(X, tid, vv);
    const float2 *K = Kspec + (long)c * (L + 1);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int f = tid + r * T;
        const float2 kf = (f <= L) ? K[f] : cconj(K[N - f]);
        vv[r] = cconj(cmul(vv[r], kf));
    }
    fft_second_from_regs<N>(X, tid, vv);
    const float dd = diag_D ? diag_D[c] : 0.f;
    if (!active) return;
#pragma unroll
    for (int qq = 0; qq < Q; ++qq) {
        const int j = tid + qq * T;
#pragma unroll
        for (int r = 0; r < HALF; ++r) {
            const int n = j + r * (N / R1);
            const float2 w = vv[qq * R1 + r];
            const float sa = w.x + dd * ga[qq * HALF + r];
            io::st(o, oa + n, io::ld(q, oa + n) * sa);
            if (hb) {
                const float sb = -w.y + dd * gb[qq * HALF + r];
                io::st(o, ob + n, io::ld(q, ob + n) * sb);
            }
        }
    }
}

// --------------------------------------------------------------- launch ----
hipError_t launch_transpose_batched(const void *in, void *out, int nb, int R, int C, hipStream_t s) {
    const int tiles = ((R + 63) / 64) * ((C + 63) / 64);
    if (R % 8 == 0 && C % 8 == 0)
        hipLaunchKernelGGL((transpose_tile_kernel<F16, 0>), dim3(nb * tiles), dim3(256), 0, s,
                           (const uint16_t *)in, (const uint16_t *)nullptr, (uint16_t *)out, R, C);
    else
        hipLaunchKernelGGL(transpose16_kernel, dim3(nb * tiles), dim3(256), 0, s, (const uint16_t *)in,
                           (uint16_t *)out, R, C);
    return hipGetLastError();
}

hipError_t launch_gate_transpose(const void *q, const void *sv, void *out, int nb, int R, int C, int dtype,
                                 hipStream_t s) {
    if (R % 8 != 0 || C % 8 != 0) return hipErrorInvalidValue;
    const int tiles = ((R + 63) / 64) * ((C + 63) / 64);
    if (dtype == BF16)
        hipLaunchKernelGGL((transpose_tile_kernel<BF16, 1>), dim3(nb * tiles), dim3(256), 0, s,
                           (const uint16_t *)q, (const uint16_t *)sv, (uint16_t *)out, R, C);
    else
        hipLaunchKernelGGL((transpose_tile_kernel<F16, 1>), dim3(nb * tiles), dim3(256), 0, s,
                           (const uint16_t *)q, (const uint16_t *)sv, (uint16_t *)out, R, C);
    return hipGetLastError();
}

hipError_t launch_shift_gate(const void *k, const void *v, const float *shift_C, const float *shift_D, int m_s,
                             int B, int d, int L, int dtype, void *g, hipStream_t s) {
    if (m_s > 64 || L % 16 != 0) return hipErrorInvalidValue;
    const long rows = (long)B * d;
    const bool gate = v != nullptr;
    const uint16_t *k16 = (const uint16_t *)k, *v16 = (const uint16_t *)v;
    uint16_t *g16 = (uint16_t *)g;
    if (L % 1024 == 0) {
        const dim3 grid((d + SGM_W - 1) / SGM_W), block(64 * SGM_W);
        auto fn = dtype == BF16 ? (gate ? shift_gate_mfma_kernel<BF16, true> : shift_gate_mfma_kernel<BF16, false>)
                                : (gate ? shift_gate_mfma_kernel<F16, true> : shift_gate_mfma_kernel<F16, false>);
        hipLaunchKernelGGL(fn, grid, block, 0, s, k16, v16, shift_C, shift_D, m_s, B, d, L, g16);
        return hipGetLastError();
    }
    const long grid = rows * ((L + SG_TILE - 1) / SG_TILE);
    auto fn = dtype == BF16 ? (gate ? shift_gate_kernel<BF16, true> : shift_gate_kernel<BF16, false>)
                            : (gate ? shift_gate_kernel<F16, true> : shift_gate_kernel<F16, false>);
    hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(SG_T), 0, s, k16, v16, shift_C, shift_D, m_s, d, L, g16);
    return hipGetLastError();
}

template <int DT, int OUT>
static hipError_t launch_gemm_t(const void *A, const void *Bt, void *C, int M, int N, int K, int d,
                                int L, hipStream_t s) {
    if (M % G2_M == 0 && N % G2_N == 0 && K % G2_K == 0) {
        const size_t lds = (size_t)2 * (G2_M + G2_N) * G2_LD * sizeof(uint16_t);
        (void)hipFuncSetAttribute((const void *)gemm_nt_256<DT, OUT>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        hipLaunchKernelGGL((gemm_nt_256<DT, OUT>), dim3((M / G2_M) * (N / G2_N)), dim3(G2_T), lds, s,
                           (const uint16_t *)A, (const uint16_t *)Bt, (uint16_t *)C, M, N, K, d, L);
    } else {
        hipLaunchKernelGGL((gemm_nt_kernel<DT, OUT>), dim3((M / GB_M) * (N / GB_N)), dim3(256), 0, s,
                           (const uint16_t *)A, (const uint16_t *)Bt, (uint16_t *)C, M, N, K, d, L);
    }
    return hipGetLastError();
}

hipError_t launch_gemm_nt(const void *A, const void *Bt, void *C, int M, int N, int K, int dtype,
                          int out_mode, int d, int L, hipStream_t s) {
    if (dtype == BF16)
        return out_mode ? launch_gemm_t<BF16, 1>(A, Bt, C, M, N, K, d, L, s)
                        : launch_gemm_t<BF16, 0>(A, Bt, C, M, N, K, d, L, s);
    return out_mode ? launch_gemm_t<F16, 1>(A, Bt, C, M, N, K, d, L, s)
                    : launch_gemm_t<F16, 0>(A, Bt, C, M, N, K, d, L, s);
}

// One stage per barrier: two (twice the MFMA work between barriers, one
// super-step of prefetch instead of three stages) measured 6 % slower at
// d = 2560, B L = 8192.
template <int DT, int OUT, int TW>
static hipError_t launch_gemm_w_t(const void *const *W, const void *X, void *C, int Mw, int Nx, int K, int ldw, int d,
                                  int L, hipStream_t s) {
    constexpr int SS = 1;
    const size_t lds = GwShape<TW, SS, OUT == 2>::LDS;
    auto fn = gemm_w<DT, OUT, TW, SS>;
    (void)hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(fn, dim3((Mw / TW) * (Nx / GW_X)), dim3(GW_T), lds, s, (const uint16_t *)W[0],
                       (const uint16_t *)W[OUT ? 1 : 0], (const uint16_t *)W[OUT ? 2 : 0], (const uint16_t *)X,
                       (uint16_t *)C, Mw, Nx, K, ldw, d, L);
    return hipGetLastError();
}

int gemm_w_tile(int d, int Nx, int K) {
    if (Nx % GW_X != 0 || K % GW_K != 0) return 0;
    for (int tw : {320, 256})
        if (d % tw == 0) return tw;
    return 0;
}

template <int DT>
static hipError_t launch_gemm_w_dt(const void *const *W, const void *X, void *C, int Mw, int Nx, int K, int ldw,
                                   int out_mode, int d, int L, int tw, hipStream_t s) {
    if (tw == 320)
        return out_mode == 1 ? launch_gemm_w_t<DT, 1, 320>(W, X, C, Mw, Nx, K, ldw, d, L, s)
               : out_mode == 2 ? launch_gemm_w_t<DT, 2, 320>(W, X, C, Mw, Nx, K, ldw, d, L, s)
                               : launch_gemm_w_t<DT, 0, 320>(W, X, C, Mw, Nx, K, ldw, d, L, s);
    return out_mode == 1 ? launch_gemm_w_t<DT, 1, 256>(W, X, C, Mw, Nx, K, ldw, d, L, s)
           : out_mode == 2 ? launch_gemm_w_t<DT, 2, 256>(W, X, C, Mw, Nx, K, ldw, d, L, s)
                           : launch_gemm_w_t<DT, 0, 256>(W, X, C, Mw, Nx, K, ldw, d, L, s);
}

hipError_t launch_gemm_w(const void *const *W, const void *X, void *C, int Nx, int K, int dtype, int out_mode, int d,
                         int L, hipStream_t s) {
    const int tw = gemm_w_tile(d, Nx, K);
    if (!tw) return hipErrorInvalidValue;
    if (out_mode == 2 && L % GW_X != 0) return hipErrorInvalidValue;
    const int Mw = out_mode == 1 ? 3 * d : d;
    return dtype == BF16 ? launch_gemm_w_dt<BF16>(W, X, C, Mw, Nx, K, d, out_mode, d, L, tw, s)
                         : launch_gemm_w_dt<F16>(W, X, C, Mw, Nx, K, d, out_mode, d, L, tw, s);
}

template <int N, int DT>
static hipError_t launch_mid_n(const void *q, const void *k, const void *v, const float *shift_C,
                               const float *shift_D, int m_s, const float2 *Kspec,
                               const float *diag_D, int B, int d, void *o, hipStream_t s) {
    using P = FFTPlan<N>;
    constexpr int T = P::T, S = (T >= 64) ? 1 : 64 / T;
    const int npairs = ((B + 1) / 2) * d;
    const size_t lds = (size_t)S * P::LDS * sizeof(float2);
    auto fn = layer_mid_kernel<N, DT>;
    if (lds > 65536) (void)hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    hipLaunchKernelGGL(fn, dim3((npairs + S - 1) / S), dim3(S * T), lds, s, (const uint16_t *)q,
                       (const uint16_t *)k, (const uint16_t *)v, shift_C, shift_D, m_s, Kspec,
                       diag_D, B, d, (uint16_t *)o, npairs);
    return hipGetLastError();
}

template <int N>
static hipError_t launch_mid_dt(int dtype, const void *q, const void *k, const void *v,
                                const float *shift_C, const float *shift_D, int m_s,
                                const float2 *Kspec, const float *diag_D, int B, int d, void *o,
                                hipStream_t s) {
    if (dtype == BF16) return launch_mid_n<N, BF16>(q, k, v, shift_C, shift_D, m_s, Kspec, diag_D, B, d, o, s);
    return launch_mid_n<N, F16>(q, k, v, shift_C, shift_D, m_s, Kspec, diag_D, B, d, o, s);
}

hipError_t launch_layer_mid(const void *q, const void *k, const void *v, const float *shift_C,
                            const float *shift_D, int m_s, const float2 *Kspec,
                            const float *diag_D, int B, int d, int L, int dtype, void *o,
                            hipStream_t s) {
#define H3_MID_CASE(LL)                                                                         \
    case LL:                                                                                    \
        return launch_mid_dt<2 * LL>(dtype, q, k, v, shift_C, shift_D, m_s, Kspec, diag_D, B, d, \
                                     o, s);
    switch (L) {
        H3_MID_CASE(16)
        H3_MID_CASE(32)
        H3_MID_CASE(64)
        H3_MID_CASE(128)
        H3_MID_CASE(256)
        H3_MID_CASE(512)
        H3_MID_CASE(1024)
        H3_MID_CASE(2048)
        H3_MID_CASE(4096)
        H3_MID_CASE(8192)
    }
#undef H3_MID_CASE
    return hipErrorInvalidValue;
}

}  // namespace h3
