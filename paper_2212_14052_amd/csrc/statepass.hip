// State passing (Sec. 4.2, Algorithm 2) pieces, gfx950.
//
// With chunk length N' and the state x^(c) carried into chunk c (the state
// after the previous chunk's last input):
//   end-of-chunk contribution  s_c = M_ux u^(c),  M_ux[n, i] = Abar_n^{N'-1-i} Bbar_n
//   state update               x^(c+1) = Abar^{N'} x^(c) + s_c
//   output                     y^(c)_t = (f * u^(c))_t + D u^(c)_t
//                                        + 2 Re sum_n C_n Abar_n^{t+1} x^(c)_n
// The chunk-local sums s_c of all chunks are independent (one workgroup per
// chunk row); only the short scan over chunks is sequential.
#include "common.h"
#include "internal.h"

namespace h3 {

// ----------------------------------------------------------- chunk sums ----
// s_c[n] = Bbar_n sum_i Abar_n^{N'-1-i} u_i, factorised with i = T a + b:
//   s_c[n] = Bbar_n sum_a Abar_n^{N' - T(a+1)} R[a][n],
//   R[a][n] = sum_{b<T} Abar_n^{T-1-b} u_{T a + b}.
constexpr int CS_T = 64;
constexpr int CS_THREADS = 256;

template <int DT>
__global__ __launch_bounds__(CS_THREADS) void chunk_states_kernel(const void *u_, const float *Abar,
                                                                  const float *Bbar, int H, int L,
                                                                  int m, int chunk, float2 *states) {
    using io = IO<DT>;
    typedef typename io::T T_;
    const T_ *u = (const T_ *)u_;
    extern __shared__ float smem[];
    float *us = smem;                                   // chunk of u, float32
    float2 *Qs = (float2 *)(smem + chunk);              // [b][n] Abar_n^{T-1-b}
    float2 *red = Qs + CS_T * H3_MAX_MODES_DEV;         // [4][n] partial sums
    const int nchunk = L / chunk;
    const int crow = blockIdx.x;                        // (b*H + h) * nchunk + c
    const int row = crow / nchunk, c = crow % nchunk;
    const int h = row % H;
    const int tid = threadIdx.x;
    const long base = (long)row * L + (long)c * chunk;
    for (int i = tid; i < chunk; i += CS_THREADS) us[i] = io::ld(u, base + i);
    const int T = chunk < CS_T ? chunk : CS_T;
    const int NA = chunk / T;
    const int n = tid % H3_MAX_MODES_DEV, g = tid / H3_MAX_MODES_DEV;
    double lr = 0, li = 0;
    if (n < m) {
        const long i = (long)h * m + n;
        const double ar = Abar[2 * i], ai = Abar[2 * i + 1];
        lr = 0.5 * log(ar * ar + ai * ai);
        li = atan2(ai, ar);
        for (int b = g; b < T; b += CS_THREADS / H3_MAX_MODES_DEV)
            Qs[b * H3_MAX_MODES_DEV + n] = cexp_scaled((double)(T - 1 - b), lr, li);
    }
    __syncthreads();
    float2 acc = make_float2(0.f, 0.f);
    if (n < m) {
        constexpr int G = CS_THREADS / H3_MAX_MODES_DEV;     // 4 groups over a
        // a = g + G i, i descending, so the anchor power grows in magnitude:
        // exponent N' - T(a+1) increases by G T per step.
        int alast = g + G * ((NA - 1 - g) / G);
        if (g < NA) {
            float2 pw = cexp_scaled((double)(chunk - T * (alast + 1)), lr, li);
            const float2 step = cexp_scaled((double)(G * T), lr, li);
            for (int a = alast; a >= 0; a -= G) {
                float rr = 0.f, ri = 0.f;
                const float *ua = us + T * a;
                for (int b = 0; b < T; ++b) {
                    const float2 q = Qs[b * H3_MAX_MODES_DEV + n];
                    const float x = ua[b];
                    rr = fmaf(q.x, x, rr);
                    ri = fmaf(q.y, x, ri);
                }
                acc = cadd(acc, cmul(pw, make_float2(rr, ri)));
                pw = cmul(pw, step);
            }
        }
    }
    red[g * H3_MAX_MODES_DEV + n] = acc;
    __syncthreads();
    if (g == 0 && n < m) {
        float2 s = red[n];
        for (int k = 1; k < CS_THREADS / H3_MAX_MODES_DEV; ++k) s = cadd(s, red[k * H3_MAX_MODES_DEV + n]);
        const long i = (long)h * m + n;
        const float2 bb = make_float2(Bbar[2 * i], Bbar[2 * i + 1]);
        states[(long)crow * m + n] = cmul(bb, s);
    }
}

// ------------------------------------------------- chunk sums, MFMA form ---
// Same sums for 16-bit input and chunk % 1024 == 0.  Per channel, with blocks
// of BW = 128 inputs (64 when chunk % 2048 != 0),
//   R[n][a] = sum_{b<BW} Abar_n^{BW-1-b} u_{BW a + b}
// is a real matrix product (rows: Re / Im of 64 modes; reduction b; columns
// a = 0 .. N'/BW - 1) on 16x16x32 MFMAs with the powers in 16-bit and the
// input as it is stored; then
//   s[n] = Bbar_n sum_a Abar_n^{N' - BW (a + 1)} R[n][a]
// in fp32 with the weights held in registers (powers in float64 first).  The
// second sum is the VALU's share (a complex multiply-add and a weight update
// per mode and column), so the wider block halves it at the same matrix-core
// work.
// Workgroup: one channel and a set of its chunk rows; wave w owns modes
// 16 w .. 16 w + 15 (row tile w of the real parts, w + 4 of the imaginary).
// Chunk rows reach LDS without passing through registers: the four waves copy
// 1 KB slices of a row (64 lanes x 16 bytes, lane i to byte 16 i of the
// slice) with global_load_lds_dwordx4 into two row buffers, one row ahead of
// the row being reduced (a three-row ring measured slower at chunk 8192, 187
// against 149 us: it leaves room for three workgroups per CU instead of
// four).  A row is staged as N'/BW LDS rows of
// BW inputs (2 BW bytes, 16-byte chunks), chunk c of LDS row a at slot
// c ^ ((a / (256 / 2 BW)) % (2 BW / 16)), so the 16 lanes of an operand read
// (16 consecutive rows a, one chunk) hit 16 distinct 16-byte bank groups.
// Each row's 64 end-state sums go to LDS; wave 0 stores them after the next
// barrier.
typedef _Float16 sp_h8 __attribute__((ext_vector_type(8)));
typedef __bf16 sp_b8 __attribute__((ext_vector_type(8)));
typedef float sp_f4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double2 sp_zmul(double2 a, double2 b) {
    return make_double2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ double2 sp_zpow(double2 z, int e) {
    double2 r = make_double2(1.0, 0.0);
    while (e) {
        if (e & 1) r = sp_zmul(r, z);
        z = sp_zmul(z, z);
        e >>= 1;
    }
    return r;
}

template <int DT>
__device__ __forceinline__ sp_f4 sp_mfma(uint4 a, uint4 b, sp_f4 c) {
    if constexpr (DT == BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(sp_b8, a), __builtin_bit_cast(sp_b8, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(sp_h8, a), __builtin_bit_cast(sp_h8, b), c, 0, 0, 0);
}
// (the empty asm keeps a float that came from a double opaque: otherwise the
// two roundings fold into one float64 -> 16-bit conversion, a long integer
// sequence instead of one instruction)
template <int DT>
__device__ __forceinline__ uint32_t sp_pack(float lo, float hi) {
    asm("" : "+v"(lo), "+v"(hi));
    if constexpr (DT == BF16) {
        typedef __bf16 b2 __attribute__((ext_vector_type(2)));
        b2 v = {(__bf16)lo, (__bf16)hi};
        return __builtin_bit_cast(uint32_t, v);
    } else {
        typedef _Float16 h2 __attribute__((ext_vector_type(2)));
        h2 v = {(_Float16)lo, (_Float16)hi};
        return __builtin_bit_cast(uint32_t, v);
    }
}

constexpr int SPM_CHUNK = 16384;   // largest chunk of the matrix-core form
constexpr int CS_NS = 2;   // row buffers in the copy ring

typedef __attribute__((address_space(3))) void cs_lds_t;

// LDS bytes for a chunk: the row ring, the results [2][64] float2 and a 1 KB
// slot for the copies of waves with one slice less
size_t chunk_states_lds(int chunk) { return (size_t)CS_NS * chunk * 2 + 2 * 64 * 8 + 1024; }

__device__ void cs_state_tail(const StateTail &t, const float *Abar, const float2 *states, int B, int H, int m,
                              int chunk, int nchunk, int h, uint4 *lds);

// tail.fuse (one workgroup per channel, chunk 8192 or 16384): the workgroup
// also writes the channel's fused-term table and scans its rows (cs_state_tail)
// FULL: chunk == CMAX, so every column tile is present and the tiles' matrix
// products are free to interleave (no per-tile branch)
template <int DT, int BW, int CMAX, bool FULL>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void chunk_states_mfma(
    const uint16_t *u, const float *Abar, const float *Bbar, int B, int H, int L, int m, int chunk, int wg_per_ch,
    float2 *states, StateTail tail) {
    constexpr int KS = BW / 32;          // 32-wide reduction steps per block
    constexpr int RB = 2 * BW;           // bytes per LDS row
    constexpr int SPR = RB / 16;         // 16-byte slots per LDS row
    constexpr int RPB = 256 / RB;        // LDS rows per 256-byte bank row
    constexpr int NA_MAX = CMAX / BW;
    extern __shared__ __attribute__((aligned(1024))) char cs_lds[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // the wave index, in a scalar register
    const int r16 = lane & 15, kg = lane >> 4;
    const int h = blockIdx.x / wg_per_ch, part = blockIdx.x % wg_per_ch;
    const int nchunk = L / chunk;
    const int NA = chunk / BW;          // columns a, multiple of 16
    const int NCT = NA / 16;            // column tiles
    const int rows_per_ch = B * nchunk;
    const int per = (rows_per_ch + wg_per_ch - 1) / wg_per_ch;
    const int r0 = part * per, r1 = min(r0 + per, rows_per_ch);
    if (r0 >= r1) return;   // uniform over the workgroup
    const int row_b = chunk * 2;                 // bytes of a staged row
    float2 *res = (float2 *)(cs_lds + CS_NS * row_b);   // [2][64]
    const uint32_t lds0 = (uint32_t)(uintptr_t)(cs_lds_t *)cs_lds;
    const uint32_t dummy = lds0 + (uint32_t)(CS_NS * row_b + 2 * 64 * 8);

    // A operand (powers, 16-bit): rows n = 16 w + r16, reduction b = 32 ks + 8 kg + i
    uint4 Are[KS], Aim[KS];
    {
        const int n = 16 * w + r16;
        double2 z = make_double2(0.0, 0.0);
        if (n < m) z = make_double2(Abar[2 * ((long)h * m + n)], Abar[2 * ((long)h * m + n) + 1]);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            // b from 32 ks + 8 kg + 7 down to 32 ks + 8 kg: exponents BW - 1 - b ascending
            double2 p = sp_zpow(z, BW - 1 - (32 * ks + 8 * kg + 7));
            float pr[8], pi[8];
#pragma unroll
            for (int i = 7; i >= 0; --i) {
                pr[i] = (float)p.x;
                pi[i] = (float)p.y;
                p = sp_zmul(p, z);
            }
            Are[ks] = make_uint4(sp_pack<DT>(pr[0], pr[1]), sp_pack<DT>(pr[2], pr[3]), sp_pack<DT>(pr[4], pr[5]), sp_pack<DT>(pr[6], pr[7]));
            Aim[ks] = make_uint4(sp_pack<DT>(pi[0], pi[1]), sp_pack<DT>(pi[2], pi[3]), sp_pack<DT>(pi[4], pi[5]), sp_pack<DT>(pi[6], pi[7]));
        }
    }
    // E weights for the lane's outputs: modes n = 16 w + 4 kg + j, columns
    // a = 16 ct + r16, weight Abar_n^{chunk - BW (a + 1)}.  Column tiles run
    // from the last down, the weight growing by Abar_n^{16 BW} per tile (fp32;
    // the starting weight and the step in float64 first).
    float2 E0[4], Zstep[4];
    float2 Bb[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int n = 16 * w + 4 * kg + j;
        double2 z = make_double2(0.0, 0.0);
        Bb[j] = make_float2(0.f, 0.f);
        if (n < m) {
            const long i = (long)h * m + n;
            z = make_double2(Abar[2 * i], Abar[2 * i + 1]);
            Bb[j] = make_float2(Bbar[2 * i], Bbar[2 * i + 1]);
        }
        const double2 zstep = sp_zpow(z, 16 * BW);
        const double2 p = sp_zpow(z, chunk - BW * (16 * (NCT - 1) + r16 + 1));
        E0[j] = make_float2((float)p.x, (float)p.y);
        Zstep[j] = make_float2((float)zstep.x, (float)zstep.y);
    }

    // this wave's slices q = w + 4 s of a staged row (s < nsl; waves past the
    // last slice copy slice w again into the never-read slot): the lane's
    // source element within the chunk row
    const int slices = row_b / 1024;             // chunk % 512 == 0
    const int nsl = (slices + 3) / 4;            // copies per wave per row (1..8)
    auto src_elem = [&](int q) {
        const int b = 1024 * q + 16 * lane;
        const int a = b / RB, slot = (b % RB) / 16;
        const int c = slot ^ ((a / RPB) % SPR);
        return BW * a + 8 * c;
    };
    // copies of chunk row rr into buffer (rr - r0) % CS_NS
    auto issue = [&](int rr) {
        const int bb = rr / nchunk, cc = rr % nchunk;
        // the row's address and the buffer, in scalar registers (wave-uniform)
        const uint64_t sp = (uint64_t)(uintptr_t)(u + ((long)bb * H + h) * L + (long)cc * chunk);
        const uint64_t spu = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(sp >> 32)) << 32) |
                             (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)sp);
        const uint16_t *src = (const uint16_t *)(uintptr_t)spu;
        const uint32_t st = lds0 + (uint32_t)(((rr - r0) % CS_NS) * row_b);
        for (int sl = 0; sl < nsl; ++sl) {
            const int q = w + 4 * sl;
            const bool real = q < slices;
            const uint32_t vo = 2u * (uint32_t)src_elem(real ? q : w);
            const uint32_t la = __builtin_amdgcn_readfirstlane(real ? st + (uint32_t)q * 1024 : dummy);
            asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, %2"
                         :
                         : "v"(vo), "s"(la), "s"(src)
                         : "memory", "m0");
        }
    };
    auto store_row = [&](int rr) {   // wave 0: the 64 sums of row rr from res[(rr - r0) & 1]
        const int bb = rr / nchunk, cc = rr % nchunk;
        const long crow = ((long)bb * H + h) * nchunk + cc;
        if (lane < m) states[crow * m + lane] = res[((rr - r0) & 1) * 64 + lane];
    };

    issue(r0);
    for (int rr = r0; rr < r1; ++rr) {
        // this row's copies landed for this wave, then for every wave; the
        // reads of the buffer refilled below (the previous row's) are done.
        // lgkmcnt(0) as well: the previous row's sums, written to res by
        // every wave, must have reached LDS before wave 0 reads them below
        // (a barrier alone does not wait for LDS writes in flight)
        __builtin_amdgcn_s_waitcnt(0x070);   // vmcnt(0) lgkmcnt(0)
        asm volatile("s_barrier" ::: "memory");
        if (w == 0 && rr > r0) store_row(rr - 1);
        // the next row's copies (none past the last row: the tail below
        // reuses the ring, so no copy may land there after the loop)
        if (rr + 1 < r1) issue(rr + 1);
        const char *us = cs_lds + ((rr - r0) % CS_NS) * row_b;
        sp_f4 sre = {0.f, 0.f, 0.f, 0.f}, sim = {0.f, 0.f, 0.f, 0.f};
        float2 E[4] = {E0[0], E0[1], E0[2], E0[3]};
#pragma unroll
        for (int ct = NA_MAX / 16 - 1; ct >= 0; --ct) {
            if (FULL || ct < NCT) {
                sp_f4 accr = {0.f, 0.f, 0.f, 0.f}, acci = {0.f, 0.f, 0.f, 0.f};
                const int a = 16 * ct + r16;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    // B operand: column a, reduction b = 32 ks + 8 kg .. + 7 (16-byte chunk 4 ks + kg)
                    const int c = 4 * ks + kg;
                    const uint4 bv = *(const uint4 *)(us + a * RB + 16 * (c ^ ((a / RPB) % SPR)));
                    accr = sp_mfma<DT>(Are[ks], bv, accr);
                    acci = sp_mfma<DT>(Aim[ks], bv, acci);
                }
                // lane: rows (modes) 4 kg + j, column a = 16 ct + r16
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    sre[j] = fmaf(E[j].x, accr[j], fmaf(-E[j].y, acci[j], sre[j]));
                    sim[j] = fmaf(E[j].x, acci[j], fmaf(E[j].y, accr[j], sim[j]));
                    E[j] = cmul(E[j], Zstep[j]);
                }
            }
        }
        // reduce over the 16 columns held by lanes r16 = 0..15
#pragma unroll
        for (int o = 1; o < 16; o <<= 1)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                sre[j] += __shfl_xor(sre[j], o);
                sim[j] += __shfl_xor(sim[j], o);
            }
        if (r16 == 0) {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                res[((rr - r0) & 1) * 64 + 16 * w + 4 * kg + j] = cmul(Bb[j], make_float2(sre[j], sim[j]));
        }
    }
    __syncthreads();   // the last row's sums are in LDS; every copy has landed
    if (w == 0) store_row(r1 - 1);
    if (tail.fuse) {
        // every chunk sum of the channel is written and visible to the
        // workgroup (a workgroup-scope fence: the readers are this
        // workgroup's waves, and a device-scope one would write back the
        // L2); the row ring is free for the table
        __threadfence_block();
        __syncthreads();
        cs_state_tail(tail, Abar, states, B, H, m, chunk, nchunk, h, (uint4 *)cs_lds);
    }
}

bool chunk_states_mfma_ok(int chunk, int dtype) {
    return (dtype == F16 || dtype == BF16) && chunk % 1024 == 0 && chunk <= SPM_CHUNK;
}

hipError_t launch_chunk_states_mfma(const void *u, const float *Abar, const float *Bbar, int B, int H,
                                    int L, int m, int chunk, int dtype, float2 *states, hipStream_t s,
                                    const StateTail *tail, bool *fused) {
    const int rows_per_ch = B * (L / chunk);
    const uint16_t *u16 = (const uint16_t *)u;
    const bool wide = chunk % 2048 == 0;   // 128-wide blocks need 16 columns per tile: chunk / 128 % 16 == 0
    const bool big = chunk > 8192;         // multiple of 2048 here, so wide
    const size_t lds = chunk_states_lds(chunk);
    // Workgroups per channel: a workgroup walks its rows one after another,
    // the grid runs in ceil(workgroups / resident) rounds.  Take the count in
    // 1..8 (at least 4 rows each where the channel has them) that minimises
    // rounds x (rows per workgroup + 1), the 1 standing for a workgroup's
    // set-up (its power tables in float64).
    auto pick_wg = [&](const void *fn) {
        int per_cu = 0, dev = 0, cus = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, lds) != hipSuccess || per_cu < 1) per_cu = 1;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
            cus = 1;
        const long resident = (long)per_cu * cus;
        int best = 1;
        long best_cost = -1;
        for (int w = 1; w <= 8; ++w) {
            if (w > 1 && rows_per_ch < 4 * w) break;
            const long rounds = ((long)H * w + resident - 1) / resident;
            const long cost = rounds * ((rows_per_ch + w - 1) / w + 1);
            if (best_cost < 0 || cost < best_cost) {
                best_cost = cost;
                best = w;
            }
        }
        return best;
    };
#define H3_CS_LAUNCH(DTV, BWV, CMV)                                                                              \
    do {                                                                                                         \
        auto fn = chunk == CMV ? chunk_states_mfma<DTV, BWV, CMV, true> : chunk_states_mfma<DTV, BWV, CMV, false>; \
        (void)hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);      \
        const int wg = pick_wg((const void *)fn);                                                                \
        StateTail tl{};                                                                                          \
        if (tail && wg == 1 && (size_t)CS_NS * chunk * 2 >= (size_t)CORR_TAB_U4 * 16) {                         \
            tl = *tail;                                                                                          \
            tl.fuse = 1;                                                                                         \
            if (fused) *fused = true;                                                                            \
        }                                                                                                        \
        hipLaunchKernelGGL(fn, dim3(H * wg), dim3(256), lds, s, u16, Abar, Bbar, B, H, L, m, chunk, wg, states,  \
                           tl);                                                                                  \
    } while (0)
    if (dtype == BF16) {
        if (big) H3_CS_LAUNCH(BF16, 128, 16384);
        else if (wide) H3_CS_LAUNCH(BF16, 128, 8192);
        else H3_CS_LAUNCH(BF16, 64, 8192);
    } else {
        if (big) H3_CS_LAUNCH(F16, 128, 16384);
        else if (wide) H3_CS_LAUNCH(F16, 128, 8192);
        else H3_CS_LAUNCH(F16, 64, 8192);
    }
#undef H3_CS_LAUNCH
    return hipGetLastError();
}

// -------------------------------------------- initial-state term, MFMA form ---
// corr[c N' + t] = 2 Re sum_n W_n Abar_n^t,  W_n = C_n x^(c)_n Abar_n  (so the
// term is 2 Re sum_n C_n Abar_n^{t+1} x^(c)_n, the M_xy x^(c) of Algorithm 2).
// With t = 64 a + b:  corr = 2 sum_k Pm[a][k] Qm[k][b],
//   Pm[a][k] = Re (W_k E[a][k]) (k < 64), -Im (W_{k-64} E[a][k-64]) (k >= 64),
//   Qm[k][b] = Re Abar_k^b (k < 64), Im Abar_{k-64}^b (k >= 64),
//   E[a][n] = Abar_n^{64 a}.
// Per channel the tables E and Q (powers in float64, stored fp16) sit in LDS;
// per chunk row W is scaled by a power of two to max |W| in [1/2, 1) before
// rounding to fp16, and the scale is undone in fp32.  Output in the I/O dtype.
// Workgroup (4 waves): one channel, a set of its chunk rows; wave w owns
// tiles a = 16 (TPW w) .. 16 (TPW (w + 1)) - 1 of every chunk (TPW = NAM / 64
// tiles per wave), all 64 columns b.  NAM = 128 serves chunks up to 8192, 256
// chunks up to 16384 (the E table then takes 69.6 KB of LDS instead of 34.8).
typedef _Float16 cr_h2 __attribute__((ext_vector_type(2)));
constexpr int CR_NA = 256;   // largest a-range (chunk / 64) of the matrix-core form

template <int DT, int NAM>
__global__ __launch_bounds__(256) void state_correction_mfma(const float *Abar, const float2 *corr_W,
                                                             int B, int H, int m, int chunk, int nchunk,
                                                             int wg_per_ch, uint16_t *corr) {
    constexpr int TPW = NAM / 64;
    __shared__ __attribute__((aligned(16))) uint32_t Et[NAM][64 + 4];       // E[a][n], fp16 complex
    __shared__ __attribute__((aligned(16))) uint16_t Qt[64][128 + 8];       // Qm[k][b] as [b][k]
    __shared__ float2 Ws[64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int r16 = lane & 15, kg = lane >> 4;
    const int h = blockIdx.x / wg_per_ch, part = blockIdx.x % wg_per_ch;
    const int NA = chunk / 64;
    const int rows_per_ch = B * nchunk;
    const int per = (rows_per_ch + wg_per_ch - 1) / wg_per_ch;
    const int r0 = part * per, r1 = min(r0 + per, rows_per_ch);
    {
        const int n = tid & 63, q = tid >> 6;
        double2 z = make_double2(0.0, 0.0);
        if (n < m) z = make_double2(Abar[2 * ((long)h * m + n)], Abar[2 * ((long)h * m + n) + 1]);
        // Q: b = 16 q .. 16 q + 15
        double2 p = sp_zpow(z, 16 * q);
        for (int j = 0; j < 16; ++j) {
            Qt[16 * q + j][n] = __builtin_bit_cast(uint16_t, (_Float16)p.x);
            Qt[16 * q + j][64 + n] = __builtin_bit_cast(uint16_t, (_Float16)p.y);
            p = sp_zmul(p, z);
        }
        // E: a = q, q + 4, ... (stride 4)
        const double2 z64 = sp_zpow(z, 64), z256 = sp_zpow(z64, 4);
        double2 e = sp_zpow(z64, q);
        for (int a = q; a < NA; a += 4) {
            cr_h2 v = {(_Float16)e.x, (_Float16)e.y};
            Et[a][n] = __builtin_bit_cast(uint32_t, v);
            e = sp_zmul(e, z256);
        }
    }
    __syncthreads();
    auto crow_of = [&](int rr) {
        const int bb = rr / nchunk, cc = rr % nchunk;
        return ((long)bb * H + h) * nchunk + cc;
    };
    // W of the next chunk row is loaded one row ahead
    float2 wnext = (r0 < r1 && lane < m) ? corr_W[crow_of(r0) * m + lane] : make_float2(0.f, 0.f);
    for (int rr = r0; rr < r1; ++rr) {
        const long crow = crow_of(rr);
        // W for this chunk row, scaled
        float2 wv = wnext;
        if (rr + 1 < r1 && lane < m) wnext = corr_W[crow_of(rr + 1) * m + lane];
        float mx = fmaxf(fabsf(wv.x), fabsf(wv.y));
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
        int ew = 0;
        if (mx > 0.f && mx < 3.0e38f) frexpf(mx, &ew);
        wv = make_float2(ldexpf(wv.x, -ew), ldexpf(wv.y, -ew));
        if (w == 0) Ws[lane] = wv;
        __syncthreads();
        // wave w: a-tiles TPW w .. TPW w + TPW - 1
#pragma unroll
        for (int at2 = 0; at2 < TPW; ++at2) {
            const int at = TPW * w + at2;
            if (16 * at >= NA) break;
            const int a = 16 * at + r16;
            // A fragments: k = 32 ks + 8 kg + i; n = k mod 64
            uint4 Af[4];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                uint32_t re[4], im[4];
#pragma unroll
                for (int i2 = 0; i2 < 4; ++i2) {
                    float pr[2], pim[2];
#pragma unroll
                    for (int ii = 0; ii < 2; ++ii) {
                        const int n = 32 * ks + 8 * kg + 2 * i2 + ii;
                        const cr_h2 e = __builtin_bit_cast(cr_h2, Et[a][n]);
                        const float2 wn = Ws[n];
                        const float er = (float)e.x, ei = (float)e.y;
                        pr[ii] = wn.x * er - wn.y * ei;
                        pim[ii] = -(wn.x * ei + wn.y * er);
                    }
                    re[i2] = sp_pack<F16>(pr[0], pr[1]);
                    im[i2] = sp_pack<F16>(pim[0], pim[1]);
                }
                Af[ks] = make_uint4(re[0], re[1], re[2], re[3]);
                Af[2 + ks] = make_uint4(im[0], im[1], im[2], im[3]);
            }
            // transposed product D[b][a] = sum_k Qm[k][b] Pm[a][k]: the Q tile
            // is the A operand and the P fragment the B operand (same
            // registers and addresses), so a lane ends up with four
            // consecutive t and writes them as one 8-byte store
            const float sc = ldexpf(2.0f, ew);
#pragma unroll
            for (int bt = 0; bt < 4; ++bt) {
                sp_f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const uint4 qv = *(const uint4 *)&Qt[16 * bt + r16][32 * ks + 8 * kg];
                    acc = sp_mfma<F16>(qv, Af[ks], acc);
                }
                // lane: rows b = 16 bt + 4 kg + j, column a = 16 at + r16
                const int t = 64 * (16 * at + r16) + 16 * bt + 4 * kg;
                uint2 o;
                if (DT == BF16) {
                    o.x = (uint32_t)f32_to_bf16(acc[0] * sc) | ((uint32_t)f32_to_bf16(acc[1] * sc) << 16);
                    o.y = (uint32_t)f32_to_bf16(acc[2] * sc) | ((uint32_t)f32_to_bf16(acc[3] * sc) << 16);
                } else {
                    o.x = sp_pack<F16>(acc[0] * sc, acc[1] * sc);
                    o.y = sp_pack<F16>(acc[2] * sc, acc[3] * sc);
                }
                *(uint2 *)(corr + crow * chunk + t) = o;
            }
        }
        __syncthreads();   // Ws is rewritten by the next chunk row
    }
}

bool state_correction_mfma_ok(int chunk, int dtype) {
    return (dtype == F16 || dtype == BF16) && chunk % 1024 == 0 && chunk / 64 <= CR_NA;
}

hipError_t launch_state_correction_mfma(const float *Abar, const float2 *corr_W, int B, int H, int m,
                                        int chunk, int nchunk, int dtype, void *corr, hipStream_t s) {
    const int rows_per_ch = B * nchunk;
    int wg = 1;
    while (H * wg < 1024 && rows_per_ch / (2 * wg) >= 4) wg *= 2;
    dim3 grid(H * wg), block(256);
    const bool big = chunk / 64 > 128;
    if (dtype == BF16) {
        if (big)
            hipLaunchKernelGGL((state_correction_mfma<BF16, 256>), grid, block, 0, s, Abar, corr_W, B, H, m, chunk, nchunk, wg, (uint16_t *)corr);
        else
            hipLaunchKernelGGL((state_correction_mfma<BF16, 128>), grid, block, 0, s, Abar, corr_W, B, H, m, chunk, nchunk, wg, (uint16_t *)corr);
    } else {
        if (big)
            hipLaunchKernelGGL((state_correction_mfma<F16, 256>), grid, block, 0, s, Abar, corr_W, B, H, m, chunk, nchunk, wg, (uint16_t *)corr);
        else
            hipLaunchKernelGGL((state_correction_mfma<F16, 128>), grid, block, 0, s, Abar, corr_W, B, H, m, chunk, nchunk, wg, (uint16_t *)corr);
    }
    return hipGetLastError();
}

// ---------------------------- per-channel tables of the fused state term ---
// For the L = 8192 and 16384 convs with the initial-state term fused in (their read-out
// computes 2 Re sum_n Abar_n^b V_n(a), t = 64 a + b, V_n(a) = W_n Abar_n^{64 a},
// on the matrix cores), per channel, in fp16 (re, im) pairs:
//   [0, 1024)     Abar_n^b as the A operand: uint4 (ib * 4 + kb) * 64 + 16 g + c
//                 holds b = 16 ib + c and modes n = 16 kb + 4 g + q in dword q
//   [1024, 1536)  Abar_n^{64 a}, a = 64 h2 + c: uint4 (h2 * 4 + kb) * 64 + 16 g + c,
//                 modes n = 16 kb + 4 g + q in dword q
//   [1536, 1552)  Abar_n^1024: uint4 kb * 4 + g, modes n = 16 kb + 4 g + q
//   [1552, 1568)  Abar_n^8192, the same layout (chunk 16384: a in [128, 256)
//                 takes Abar_n^{64 (a - 128)} times Abar_n^8192)
// Modes n >= m hold powers of 0 (their weights W_n are zero).  Powers in float64.
__device__ __forceinline__ uint32_t ct_h2(double2 p) {
    typedef _Float16 h2 __attribute__((ext_vector_type(2)));
    h2 v = {(_Float16)p.x, (_Float16)p.y};
    return __builtin_bit_cast(uint32_t, v);
}
// Channel h's table, assembled in ts (CORR_TAB_U4 uint4 of LDS) by a
// 256-thread workgroup, then written to dst in 16-byte pieces.
__device__ void corr_tables_body(const float *Abar, int h, int m, uint4 *ts, uint4 *dst) {
    const int tid = threadIdx.x, n = tid & 63, q4 = tid >> 6;
    uint32_t *t = (uint32_t *)ts;
    for (int i = tid; i < CORR_TAB_U4; i += 256) ts[i] = make_uint4(0, 0, 0, 0);   // unused tail
    __syncthreads();
    double2 z = make_double2(0.0, 0.0);
    if (n < m) z = make_double2(Abar[2 * ((long)h * m + n)], Abar[2 * ((long)h * m + n) + 1]);
    const int kb = n >> 4, g = (n >> 2) & 3, q = n & 3;
    // b = 16 q4 + i: ib = q4, c = i
    double2 p = sp_zpow(z, 16 * q4);
    for (int i = 0; i < 16; ++i) {
        t[((q4 * 4 + kb) * 64 + 16 * g + i) * 4 + q] = ct_h2(p);
        p = sp_zmul(p, z);
    }
    // a = 64 h2 + c with h2 = q4 >> 1, c = 8 (q4 & 1) + i
    const int h2 = q4 >> 1;
    const double2 z64 = sp_zpow(z, 64);
    double2 e = sp_zpow(z64, 64 * h2 + 8 * (q4 & 1));
    for (int i = 0; i < 8; ++i) {
        const int c = 8 * (q4 & 1) + i;
        t[(1024 + (h2 * 4 + kb) * 64 + 16 * g + c) * 4 + q] = ct_h2(e);
        e = sp_zmul(e, z64);
    }
    if (q4 == 0) t[(1536 + kb * 4 + g) * 4 + q] = ct_h2(sp_zpow(z, 1024));
    if (q4 == 1) t[(1552 + kb * 4 + g) * 4 + q] = ct_h2(sp_zpow(z, 8192));   // chunk 16384: a >= 128
    __syncthreads();
    for (int i = tid; i < CORR_TAB_U4; i += 256) dst[i] = ts[i];
}
__global__ __launch_bounds__(256) void corr_tables_kernel(const float *Abar, int H, int m, uint4 *tab) {
    __shared__ uint4 ts[CORR_TAB_U4];
    corr_tables_body(Abar, blockIdx.x, m, ts, tab + (long)blockIdx.x * CORR_TAB_U4);
}

hipError_t launch_corr_tables(const float *Abar, int H, int m, uint4 *tab, hipStream_t s) {
    if (m > 64) return hipErrorInvalidValue;
    hipLaunchKernelGGL(corr_tables_kernel, dim3(H), dim3(256), 0, s, Abar, H, m, tab);
    return hipGetLastError();
}

// ------------------------------------------------------------------ scan ---
// One thread per (row, mode): x <- Abar^{N'} x + s_c across the chunks.
// Writes corr_W[row, c, n] = C_n x^(c)_n Abar_n (so that the initial-state
// term of chunk c is 2 Re sum_n corr_W Abar_n^t) and x_final = x^(nchunk).
__global__ void state_scan_kernel(const float *Abar, const float *C, const float *x0,
                                  const float2 *states, int B, int H, int m, int chunk, int nchunk,
                                  float2 *corr_W, float *x_final) {
    const long gid = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (long)B * H * m) return;
    const int n = (int)(gid % m);
    const long row = gid / m;
    const int h = (int)(row % H);
    const long i = (long)h * m + n;
    const double ar = Abar[2 * i], ai = Abar[2 * i + 1];
    const float2 ab = make_float2((float)ar, (float)ai);
    const float2 cc = make_float2(C[2 * i], C[2 * i + 1]);
    const float2 cab = cmul(cc, ab);
    const float2 AN = cexp_scaled((double)chunk, 0.5 * log(ar * ar + ai * ai), atan2(ai, ar));
    float2 x = x0 ? make_float2(x0[2 * gid], x0[2 * gid + 1]) : make_float2(0.f, 0.f);
    for (int c = 0; c < nchunk; ++c) {
        const long ci = (row * nchunk + c) * m + n;
        corr_W[ci] = cmul(cab, x);
        x = cadd(cmul(AN, x), states[ci]);
    }
    if (x_final) {
        x_final[2 * gid] = x.x;
        x_final[2 * gid + 1] = x.y;
    }
}

// The same scan for the fused state term: one wavefront per (batch, channel)
// row, lane n = mode (modes n >= m idle).  For every chunk the weights
// W_n = C_n Abar_n x^(c)_n are written normalised, W / 2^e with max |W| in
// [1/2, 1), as fp16 (re, im) pairs, 64 per chunk row (zero beyond m), with
// the exponent e per chunk row.
// One wavefront: row = b H + h, lane n = mode.
__device__ void scan_w16_row(const float *Abar, const float *C, const float *x0, const float2 *states, long row,
                             int H, int m, int chunk, int nchunk, uint32_t *w16, int *wexp, float *x_final, int n) {
    const int h = (int)(row % H);
    const bool on = n < m;
    const long i = (long)h * m + n;
    float2 cab = make_float2(0.f, 0.f), AN = make_float2(0.f, 0.f), x = make_float2(0.f, 0.f);
    if (on) {
        const double ar = Abar[2 * i], ai = Abar[2 * i + 1];
        cab = cmul(make_float2(C[2 * i], C[2 * i + 1]), make_float2((float)ar, (float)ai));
        AN = cexp_scaled((double)chunk, 0.5 * log(ar * ar + ai * ai), atan2(ai, ar));
        if (x0) x = make_float2(x0[2 * (row * m + n)], x0[2 * (row * m + n) + 1]);
    }
    for (int c = 0; c < nchunk; ++c) {
        const float2 W = cmul(cab, x);
        float mx = fmaxf(fabsf(W.x), fabsf(W.y));
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
        int e = 0;
        if (mx > 0.f && mx < 3.0e38f) frexpf(mx, &e);
        typedef _Float16 h2 __attribute__((ext_vector_type(2)));
        const h2 v = {(_Float16)ldexpf(W.x, -e), (_Float16)ldexpf(W.y, -e)};
        const long rc = row * nchunk + c;
        w16[rc * 64 + n] = __builtin_bit_cast(uint32_t, v);
        if (n == 0) wexp[rc] = e;
        if (on) x = cadd(cmul(AN, x), states[rc * m + n]);
    }
    if (x_final && on) {
        x_final[2 * (row * m + n)] = x.x;
        x_final[2 * (row * m + n) + 1] = x.y;
    }
}
__global__ __launch_bounds__(256) void state_scan_w16_kernel(const float *Abar, const float *C, const float *x0,
                                                             const float2 *states, int B, int H, int m, int chunk,
                                                             int nchunk, uint32_t *w16, int *wexp, float *x_final) {
    const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= (long)B * H) return;   // whole wavefronts leave together
    scan_w16_row(Abar, C, x0, states, row, H, m, chunk, nchunk, w16, wexp, x_final, threadIdx.x & 63);
}

// The tail of the chunk-state kernel when one workgroup holds all chunk rows
// of channel h: its table of the fused state term (assembled in the kernel's
// LDS row ring, free by then) and the scan of its B rows, one wavefront per
// row.  The chunk sums were written by this workgroup and are read back.
__device__ void cs_state_tail(const StateTail &t, const float *Abar, const float2 *states, int B, int H, int m,
                              int chunk, int nchunk, int h, uint4 *lds) {
    corr_tables_body(Abar, h, m, lds, t.ctab + (long)h * CORR_TAB_U4);
    const int w = threadIdx.x >> 6;
    for (int b = w; b < B; b += 4)
        scan_w16_row(Abar, t.C, t.x0, states, (long)b * H + h, H, m, chunk, nchunk, t.w16, t.wexp, t.x_final,
                     threadIdx.x & 63);
}

hipError_t launch_state_scan_w16(const float *Abar, const float *C, const float *x0, const float2 *states,
                                 int B, int H, int m, int chunk, int nchunk, uint32_t *w16, int *wexp,
                                 float *x_final, hipStream_t s) {
    if (m > 64) return hipErrorInvalidValue;
    const long rows = (long)B * H;
    hipLaunchKernelGGL(state_scan_w16_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, Abar, C, x0,
                       states, B, H, m, chunk, nchunk, w16, wexp, x_final);
    return hipGetLastError();
}

hipError_t launch_chunk_states(const void *u, const float *Abar, const float *Bbar, int B, int H,
                               int L, int m, int chunk, int dtype, float2 *states, hipStream_t s,
                               const StateTail *tail, bool *fused) {
    if (fused) *fused = false;
    if (chunk_states_mfma_ok(chunk, dtype))
        return launch_chunk_states_mfma(u, Abar, Bbar, B, H, L, m, chunk, dtype, states, s, tail, fused);
    const int nchunk = L / chunk;
    const long ncr = (long)B * H * nchunk;
    const size_t lds = (size_t)chunk * sizeof(float) +
                       (size_t)(CS_T + CS_THREADS / H3_MAX_MODES_DEV) * H3_MAX_MODES_DEV * sizeof(float2);
    dim3 grid((unsigned)ncr), block(CS_THREADS);
    if (lds > 65536) {
        (void)hipFuncSetAttribute((const void *)chunk_states_kernel<F32>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        (void)hipFuncSetAttribute((const void *)chunk_states_kernel<F16>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        (void)hipFuncSetAttribute((const void *)chunk_states_kernel<BF16>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    }
    switch (dtype) {
        case F32:
            hipLaunchKernelGGL(chunk_states_kernel<F32>, grid, block, lds, s, u, Abar, Bbar, H, L, m, chunk, states);
            break;
        case F16:
            hipLaunchKernelGGL(chunk_states_kernel<F16>, grid, block, lds, s, u, Abar, Bbar, H, L, m, chunk, states);
            break;
        case BF16:
            hipLaunchKernelGGL(chunk_states_kernel<BF16>, grid, block, lds, s, u, Abar, Bbar, H, L, m, chunk, states);
            break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_state_scan(const float *Abar, const float *C, const float *x0,
                             const float2 *states, int B, int H, int m, int chunk, int nchunk,
                             float2 *corr_W, float *x_final, hipStream_t s) {
    const long n = (long)B * H * m;
    hipLaunchKernelGGL(state_scan_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, Abar, C,
                       x0, states, B, H, m, chunk, nchunk, corr_W, x_final);
    return hipGetLastError();
}

}  // namespace h3
