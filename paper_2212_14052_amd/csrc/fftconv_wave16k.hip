// Fused FFT convolution for L = 8192 (transform length N = 2L = 16384 =
// 4 x 4096) with four wavefronts per row pair (Sec. 4.1: kernel fusion +
// block FFT, at the fused-block length), gfx950, 16-bit I/O.
//
// With p = 4096 p3 + m (m < 4096; the zero-padded input vanishes for
// p3 >= 2), decimating the frequency by four (f = 4 f' + k3) gives
//   X[4 f' + k3] = DFT_4096[ w_16384^{k3 m} (x(m) + (-i)^{k3} x(4096 + m)) ](f').
// Wave k3 of the workgroup runs block k3 through the register-resident
// 4096-point pipeline of the one-wave kernel (three radix-16 layers on the
// matrix cores; see wave_common.h).  The block twiddle
//   w_16384^{k3 m} = w_64^{k3 p2} w_1024^{k3 p1} w_16384^{k3 p0},
//   m = 256 p2 + 16 p1 + p0,
// costs no instruction per point: the p2 factor scales the contraction side
// of the first layer's DFT matrix, the p1 factor rides on that layer's lane
// twiddles and the p0 factor scales the contraction side of the third
// layer's matrix.  The first layer contracts x(m) and x(4096 + m) together
// as two K steps of the MFMA (the second with (-i)^{k3} times the matrix),
// so the radix-4 butterfly needs no vector instruction either.
//
// Inverse: y(4096 t3 + m) = sum_k3 i^{t3 k3} w_16384^{-k3 m} IDFT_4096[Y_k3](m)
// for t3 = 0, 1 (outputs t < L only).  Each wave runs its block backwards up
// to the last radix-16 layer (the p0 and p1 factors again folded into a layer
// matrix and the lane twiddles).  The last layer's inputs are then exchanged
// through LDS so that wave w holds tiles p0 = 4w .. 4w + 3 of all four
// blocks, and the last layer, the w_64^{-k3 p2} factors and the radix-4
// butterfly over k3 run as one 64-point contraction (four K steps of the MFMA
// per output tile, two outputs t3 = 0, 1).
//
// The pair's input is staged once in LDS as interleaved complex (u_a, u_b)
// values, in the order the first layer reads them; every wave reads all of it
// and loads one quarter of it from HBM (prefetched into registers during the
// previous pair).  The kernel spectrum block of each wave stays in registers.
// D is folded into the kernel (k[0] += D).  16-bit inputs feed the first
// layer as they are (fp16 or bf16 MFMA); everything after it is fp16 with
// fp32 accumulation, with the power-of-two range control of the one-wave
// kernel.
#include "common.h"
#include "internal.h"
#include "wave_common.h"

namespace h3 {
namespace w16 {

using namespace wvc;

template <bool P2, bool SIG_A, class Pre, class Epi>
__device__ __forceinline__ void layer_sel(uint32_t *d, const Dft &F, Pre &&pre, Epi &&epi) {
    if constexpr (P2) layer2<SIG_A>(d, F, pre, epi);
    else layer<SIG_A>(d, F, pre, epi);
}

constexpr int N = 16384;
constexpr int L = 8192;
constexpr int NW = 4;           // waves per workgroup (one per frequency block)
constexpr int NT = 64 * NW;
constexpr int kU = 2048;        // uint4: input staging / last-layer exchange (32 KB)


// LDS tables: the one-wave kernel's L2 twiddles and per-lane DFT rows, then
// the last layer's matrix for each source block k3' as (real, imaginary)
// rows: entries conj(w_64^{(4 k2 + k3') p2}) / 4 for output row p2 = c and
// contraction point k2 = 4 g + i (lane l = 16 g + c).
constexpr int kTabG1 = 8 * 64;
constexpr int kTab16 = kTab + kTabG1;   // uint4
struct Half16 {
    uint32_t v[4 * kTab16];
};
constexpr Half16 make_half16() {
    const HalfTable base = make_half_table();
    Half16 t{};
    for (int i = 0; i < 4 * kTab; ++i) t.v[i] = base.v[i];
    for (int k3 = 0; k3 < 4; ++k3)
        for (int l = 0; l < 64; ++l)
            for (int i = 0; i < 4; ++i) {
                const long g = l >> 4, c = l & 15;
                const Cd v = cwd(-(4 * (4 * g + i) + k3) * c, 64);
                const double re = 0.25 * v.re, im = 0.25 * v.im;
                t.v[4 * (kTab + (2 * k3) * 64 + l) + i] = h2_bits(re, -im);
                t.v[4 * (kTab + (2 * k3 + 1) * 64 + l) + i] = h2_bits(im, re);
            }
    return t;
}
__device__ const Half16 kHalf16 = make_half16();

// Per-wave (k3) and per-lane factors, fp16 (re, im), 16 dwords per lane:
//   [0..3]  w_64^{k3 (4g+i)} / 2      first layer, contraction point i
//   [4..7]  w_1024^{k3 (4g+j)}         first layer's lane twiddles, row j
//   [8..11] w_16384^{k3 (4g+i)}        third layer, contraction point i
//   [12]    w_16384^{-k3 c}            inverse third layer, output row c
//   [13]    w_1024^{-k3 c}             inverse second layer's lane twiddles
//   [14,15] w_64^{-c}, w_64^{-2c}      last layer's rows, when not tabulated
struct Fac16 {
    uint32_t v[4 * 64 * 16];
};
constexpr Fac16 make_fac16() {
    Fac16 t{};
    for (int k3 = 0; k3 < 4; ++k3)
        for (int l = 0; l < 64; ++l) {
            const long g = l >> 4, c = l & 15;
            uint32_t *p = t.v + (k3 * 64 + l) * 16;
            for (int i = 0; i < 4; ++i) {
                const Cd a = cwd(k3 * (4 * g + i), 64);
                p[i] = h2_bits(0.5 * a.re, 0.5 * a.im);
                const Cd b = cwd(k3 * (4 * g + i), 1024);
                p[4 + i] = h2_bits(b.re, b.im);
                const Cd e = cwd(k3 * (4 * g + i), N);
                p[8 + i] = h2_bits(e.re, e.im);
            }
            const Cd r3 = cwd(-k3 * c, N), rx = cwd(-k3 * c, 1024);
            p[12] = h2_bits(r3.re, r3.im);
            p[13] = h2_bits(rx.re, rx.im);
            const Cd g1 = cwd(-c, 64), g2 = cwd(-2 * c, 64);
            p[14] = h2_bits(g1.re, g1.im);
            p[15] = h2_bits(g2.re, g2.im);
        }
    return t;
}
__device__ const Fac16 kFac16 = make_fac16();

// First layer: signal as the A operand, the two K steps x(m) (matrix Fa) and
// x(4096 + m) (matrix Fb) accumulated; operands straight from the staging
// buffer S (tile tau of half x at S[(16 x + tau) * 64 + lane]), two tiles
// ahead.  epi(tau, re, im) as in layer().
template <class OP, class Epi>
__device__ __forceinline__ void layer1(const uint4 *S, int lane, const OP &Far, const OP &Fai, const OP &Fbr,
                                       const OP &Fbi, Epi &&epi) {
    const f4_t z = {0.f, 0.f, 0.f, 0.f};
    auto mm = [&](uint4 x0, uint4 x1, f4_t &re, f4_t &im) {
        const OP a0 = __builtin_bit_cast(OP, x0), a1 = __builtin_bit_cast(OP, x1);
        re = mfma_acc(a1, Fbr, mfma_acc(a0, Far, z));
        im = mfma_acc(a1, Fbi, mfma_acc(a0, Fai, z));
    };
    f4_t re, im;
    mm(S[lane], S[16 * 64 + lane], re, im);
    uint4 n0 = S[64 + lane], n1 = S[17 * 64 + lane];
#pragma unroll
    for (int tau = 0; tau < 16; ++tau) {
        f4_t re1, im1;
        uint4 m0 = make_uint4(0, 0, 0, 0), m1 = m0;
        if (tau + 1 < 16) mm(n0, n1, re1, im1);
        if (tau + 2 < 16) {
            m0 = S[(tau + 2) * 64 + lane];
            m1 = S[(16 + tau + 2) * 64 + lane];
        }
        epi(tau, re, im);
        __builtin_amdgcn_sched_barrier(0);
        re = re1;
        im = im1;
        n0 = m0;
        n1 = m1;
    }
}

// One source block's contribution to the two output tiles of a half:
// D0 += G b, D1 += i^{k3'} G b, with the rotation done by choosing the
// matrix row kind and the sign of the data.
template <int K3P>
__device__ __forceinline__ void last_acc(uint4 gr4, uint4 gi4, uint4 b4, f4_t (&D)[4]) {
    const h8_t Ar = __builtin_bit_cast(h8_t, gr4), Ai = __builtin_bit_cast(h8_t, gi4);
    const h8_t b = __builtin_bit_cast(h8_t, b4);
    D[0] = mfma_acc(Ar, b, D[0]);
    D[1] = mfma_acc(Ai, b, D[1]);
    if constexpr (K3P == 0) {
        D[2] = mfma_acc(Ar, b, D[2]);
        D[3] = mfma_acc(Ai, b, D[3]);
    } else {
        const h8_t nb = __builtin_bit_cast(
            h8_t, make_uint4(b4.x ^ 0x80008000u, b4.y ^ 0x80008000u, b4.z ^ 0x80008000u, b4.w ^ 0x80008000u));
        if constexpr (K3P == 1) {   // i P: (-Im P, Re P)
            D[2] = mfma_acc(Ai, nb, D[2]);
            D[3] = mfma_acc(Ar, b, D[3]);
        } else if constexpr (K3P == 2) {   // -P
            D[2] = mfma_acc(Ar, nb, D[2]);
            D[3] = mfma_acc(Ai, nb, D[3]);
        } else {   // -i P: (Im P, -Re P)
            D[2] = mfma_acc(Ai, b, D[2]);
            D[3] = mfma_acc(Ar, nb, D[3]);
        }
    }
}

// Last layer for the wave's own tiles T = 4 w + tt: exchange, 64-point
// contraction with the radix-4 butterfly, output epilogue and stores.
//   D0 = sum_k3' G_k3' x_k3'           -> y(m)
//   D1 = sum_k3' i^{k3'} G_k3' x_k3'   -> y(4096 + m)
// (real parts row a, imaginary parts row b).  The exchange runs in two
// halves (tiles tt = 0, 1, then 2, 3 of every quarter) through a 32 KB
// buffer: slot ((source * 4 + destination) * 2 + tt % 2); every quarter,
// the wave's own included, passes through LDS, so no register index depends
// on the wave.  Source blocks are visited in order with their operands
// loaded one block ahead.  G_k3' comes from the LDS table G1, or (CORR 3,
// whose LDS holds the state-term tables instead) from the conjugate DFT rows
// times the lane's w_64^{-k3' c} (gf[k3' - 1]).
template <int DT, int CORR>
__device__ __forceinline__ void last_layer(uint32_t (&d)[64], uint4 *U, const uint4 *G1, const uint4 *Lc,
                                           const uint32_t (&gf)[3], int w, int lane, float sca, float scb, uint16_t *ya,
                                           uint16_t *yb, bool has_b, const void *cra, const void *crb, int ewa,
                                           int ewb) {
    const int g = lane >> 4, c = lane & 15;
    uint32_t pa0[8], pb0[8], pa1[8], pb1[8];   // packed outputs: [2 jj + half]
    const f4_t z = {0.f, 0.f, 0.f, 0.f};
    // this wave's share of the read-out below: row w >> 1, 16-byte pieces
    // i8 = (w & 1) 512 + 64 r + lane
    uint16_t *yrow = w < 2 ? ya : yb;
    const void *crow = w < 2 ? cra : crb;
    const bool active = w < 2 || has_b;
    uint4 c16[8];   // 16-bit correction term, loaded while the last layer runs
    uint4 wq[4];    // fused state term: the row's weights W for the lane's 16 modes
    auto kinds = [&](int k3p, uint4 &gr, uint4 &gi) {
        if constexpr (CORR != 3) {
            gr = G1[(2 * k3p) * 64 + lane];
            gi = G1[(2 * k3p + 1) * 64 + lane];
        } else if (k3p == 0) {
            gr = Lc[2 * 64 + lane];
            gi = Lc[3 * 64 + lane];
        } else {
            uint32_t R[4], I[4];
            const uint32_t ff[4] = {gf[k3p - 1], gf[k3p - 1], gf[k3p - 1], gf[k3p - 1]};
            kinds_scaled(Lc[3 * 64 + lane], ff, R, I);
            gr = make_uint4(R[0], R[1], R[2], R[3]);
            gi = make_uint4(I[0], I[1], I[2], I[3]);
        }
    };
#pragma unroll
    for (int half = 0; half < 2; ++half) {
        if (half == 1) __syncthreads();   // the first half's reads are done
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
            for (int t2 = 0; t2 < 2; ++t2) {
                const int T = 4 * q + 2 * half + t2;
                U[((w * 4 + q) * 2 + t2) * 64 + lane] = make_uint4(d[4 * T], d[4 * T + 1], d[4 * T + 2], d[4 * T + 3]);
            }
        if (CORR == 2 && half == 1) {
#pragma unroll
            for (int r = 0; r < 8; ++r)
                c16[r] = active ? ((const uint4 *)crow)[(w & 1) * 512 + r * 64 + lane] : make_uint4(0, 0, 0, 0);
        }
        __syncthreads();
        f4_t D[2][4] = {{z, z, z, z}, {z, z, z, z}};
        uint4 gr, gi;
        kinds(0, gr, gi);
        uint4 b0 = U[((0 * 4 + w) * 2 + 0) * 64 + lane], b1 = U[((0 * 4 + w) * 2 + 1) * 64 + lane];
#pragma unroll
        for (int k3p = 0; k3p < 4; ++k3p) {
            uint4 ngr = gr, ngi = gi, nb0 = b0, nb1 = b1;
            if (k3p + 1 < 4) {
                kinds(k3p + 1, ngr, ngi);
                nb0 = U[(((k3p + 1) * 4 + w) * 2 + 0) * 64 + lane];
                nb1 = U[(((k3p + 1) * 4 + w) * 2 + 1) * 64 + lane];
            }
            if (k3p == 0) {
                last_acc<0>(gr, gi, b0, D[0]);
                last_acc<0>(gr, gi, b1, D[1]);
            } else if (k3p == 1) {
                last_acc<1>(gr, gi, b0, D[0]);
                last_acc<1>(gr, gi, b1, D[1]);
            } else if (k3p == 2) {
                last_acc<2>(gr, gi, b0, D[0]);
                last_acc<2>(gr, gi, b1, D[1]);
            } else {
                last_acc<3>(gr, gi, b0, D[0]);
                last_acc<3>(gr, gi, b1, D[1]);
            }
            __builtin_amdgcn_sched_barrier(0);
            gr = ngr;
            gi = ngi;
            b0 = nb0;
            b1 = nb1;
        }
        if (CORR == 3 && half == 1) {
            // the row's weights for modes 16 kb + 4 g + (0..3): one uint4 per kb
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) wq[kb] = active ? ((const uint4 *)crow)[4 * kb + g] : make_uint4(0, 0, 0, 0);
        }
        // tiles 2 half (D[0]) and 2 half + 1 (D[1]) are consecutive points
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int s = 2 * jj + half;
            pa0[s] = pack_out<DT>(D[0][0][jj] * sca, D[1][0][jj] * sca);
            pb0[s] = pack_out<DT>(D[0][1][jj] * scb, D[1][1][jj] * scb);
            pa1[s] = pack_out<DT>(D[0][2][jj] * sca, D[1][2][jj] * sca);
            pb1[s] = pack_out<DT>(D[0][3][jj] * scb, D[1][3][jj] * scb);
        }
    }
    // outputs m = 256 (4 g + jj) + 16 c + 4 w + (0..3) of both rows go
    // through LDS (rows a, b as 8192 halves each), then out as 16-byte
    // chunks, each wave a contiguous quarter of the pair
    __syncthreads();   // every exchange read is done
    uint2 *Uo = (uint2 *)U;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
        const int m4 = (256 * (4 * g + jj) + 16 * c + 4 * w) >> 2;
        Uo[m4] = make_uint2(pa0[2 * jj], pa0[2 * jj + 1]);
        Uo[1024 + m4] = make_uint2(pa1[2 * jj], pa1[2 * jj + 1]);
        Uo[2048 + m4] = make_uint2(pb0[2 * jj], pb0[2 * jj + 1]);
        Uo[3072 + m4] = make_uint2(pb1[2 * jj], pb1[2 * jj + 1]);
    }
    __syncthreads();
    if constexpr (CORR == 3) {
        if (active) fused_state_term<DT, 2048>(U, G1, wq, w < 2 ? ewa : ewb, w >> 1, w & 1, lane, yrow);
        return;
    }
    if (active) {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int i8 = (w & 1) * 512 + r * 64 + lane;   // uint4 index within the row
            uint4 v = U[(w >> 1) * 1024 + i8];
            if constexpr (CORR != 0) {
                // state-passing initial-state term, added to the 16-bit outputs
                float cv[8];
                if constexpr (CORR == 1) {
                    const float4 c0 = ((const float4 *)crow)[2 * i8], c1 = ((const float4 *)crow)[2 * i8 + 1];
                    cv[0] = c0.x; cv[1] = c0.y; cv[2] = c0.z; cv[3] = c0.w;
                    cv[4] = c1.x; cv[5] = c1.y; cv[6] = c1.z; cv[7] = c1.w;
                } else {
                    const uint4 cr = c16[r];
                    const uint32_t cw[4] = {cr.x, cr.y, cr.z, cr.w};
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        cv[2 * e] = lo_f<DT>(cw[e]);
                        cv[2 * e + 1] = hi_f<DT>(cw[e]);
                    }
                }
                uint32_t vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    vw[e] = pack_out<DT>(lo_f<DT>(vw[e]) + cv[2 * e], hi_f<DT>(vw[e]) + cv[2 * e + 1]);
                v = make_uint4(vw[0], vw[1], vw[2], vw[3]);
            }
            *(uint4 *)(yrow + 8 * i8) = v;
        }
    }
}

}  // namespace w16

// ============================================================================
// CORR: 0 none, 1 float32 correction term, 2 correction term in the I/O dtype,
// 3 the term computed here from the chunk's weights W
template <int DT, int CORR>
__global__ __launch_bounds__(w16::NT) __attribute__((amdgpu_waves_per_eu(2))) void fftconv_wave16k_kernel(
    ConvArgs a, const float *k, int wg_per_ch, int pairs_per_ch) {
    using namespace w16;
    // Ytab + Lc, then the last layer's matrices, or (CORR 3) the channel's
    // state-term tables
    constexpr int kTabAll = CORR == 3 ? kTab + CORR_TAB_U4 : kTab16;
    __shared__ uint4 Tab[kTabAll];
    __shared__ uint4 U[kU];         // pair staging, then the last-layer exchange
    __shared__ float red[3 * NW];   // row a max | kernel spectrum max | row b max
    const uint4 *Ytab = Tab, *Lc = Tab + kTabY, *G1 = Tab + kTab;
    uint32_t *Ud = (uint32_t *)U;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // frequency block k3
    const int g = lane >> 4, c = lane & 15;
    const int h = blockIdx.x / wg_per_ch, part = blockIdx.x % wg_per_ch;
    const int per = (pairs_per_ch + wg_per_ch - 1) / wg_per_ch;
    const int q0 = part * per, q1 = min(q0 + per, pairs_per_ch);
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
    // This wave's quarter of a pair: half x = w >> 1, lane rows g = 2 (w & 1)
    // + gi; lane l holds c = l & 15, j = l >> 4, points m = 4096 x + 256 (4 g
    // + j) + 16 c + 8 hh .. + 7 of both rows (ra/rb[2 gi + hh]).
    const int xq = w >> 1, jq = lane >> 4;
    uint4 ra[4], rb[4];
    auto issue_loads = [&](int qq) {
        long oa, ob;
        rows(qq, oa, ob);
        const uint16_t *ua = u + oa, *ub = u + (ob >= 0 ? ob : oa);   // wave-uniform bases
#pragma unroll
        for (int gi = 0; gi < 2; ++gi) {
            const int off = 4096 * xq + 256 * (4 * (2 * (w & 1) + gi) + jq) + 16 * c;
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                ra[2 * gi + hh] = *(const uint4 *)(ua + off + 8 * hh);
                rb[2 * gi + hh] = *(const uint4 *)(ub + off + 8 * hh);
            }
        }
        if (ob < 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) rb[i] = make_uint4(0, 0, 0, 0);
        }
    };
    // staging position of point (x, T, lane row g, lane c, register j):
    // dword ((16 x + T) * 64 + 16 g + c) * 4 + j  (conflict-free writes)
    auto stage_at = [&](int gi, int T) { return ((16 * xq + T) * 64 + 16 * (2 * (w & 1) + gi) + c) * 4 + jq; };

    // ---- start-up loads: tables into LDS, factors, kernel row, first pair ----
#pragma unroll
    for (int r = 0; r < (kTabAll + NT - 1) / NT; ++r) {
        const int base = r * NT + 64 * w;   // kTab and CORR_TAB_U4 are multiples of 64
        if (base < kTabAll) {
            const uint4 *src = (CORR != 3 || base < kTab) ? (const uint4 *)kHalf16.v + base
                                                         : a.corr_tab + (long)h * CORR_TAB_U4 + (base - kTab);
            __builtin_amdgcn_global_load_lds((gvoid_t *)(src + lane), (lvoid_t *)(Tab + base), 16, 0, 0);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    uint32_t f1[4], xf[4], f3[4], g3, xh, gf[3];
    {
        const uint4 *fp = (const uint4 *)kFac16.v + (w * 64 + lane) * 4;
        const uint4 v0 = fp[0], v1 = fp[1], v2 = fp[2], v3 = fp[3];
        f1[0] = v0.x; f1[1] = v0.y; f1[2] = v0.z; f1[3] = v0.w;
        xf[0] = v1.x; xf[1] = v1.y; xf[2] = v1.z; xf[3] = v1.w;
        f3[0] = v2.x; f3[1] = v2.y; f3[2] = v2.z; f3[3] = v2.w;
        g3 = v3.x;
        xh = v3.y;
        gf[0] = v3.z;
        gf[1] = v3.w;
        gf[2] = cmul(v3.z, v3.w);   // w_64^{-3c}
    }
    float4 kq[8];   // [4 gi + s]: points m = ... + 16 c + 4 s .. + 3
    // CORR 3 with gen_C: the kernel row is formed here (below); lane n = mode
    // n loads C_n and Bbar_n instead
    const bool gen = CORR == 3 && a.gen_C != nullptr;   // uniform
    float2 gC = make_float2(0.f, 0.f), gB = make_float2(0.f, 0.f);
    if (gen) {
        if (lane < a.m_gen) {
            gC = ((const float2 *)a.gen_C)[(long)h * a.m_gen + lane];
            gB = ((const float2 *)a.gen_Bbar)[(long)h * a.m_gen + lane];
        }
    } else {
#pragma unroll
        for (int gi = 0; gi < 2; ++gi) {
            const int off = 4096 * xq + 256 * (4 * (2 * (w & 1) + gi) + jq) + 16 * c;
#pragma unroll
            for (int s = 0; s < 4; ++s) kq[4 * gi + s] = *(const float4 *)(k + (long)h * L + off + 4 * s);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (q0 < q1) issue_loads(q0);
    if (CORR == 3 && gen) {
        // k_t = 2 Re sum_n W_n Abar_n^t with W_n = C_n Bbar_n: the fused state
        // term's sum (Algorithm 2's M_xy form) with the kernel's weights; waves
        // 0 and 1 form t in [4096 w, 4096 w + 4096) in fp32 into U, then every
        // wave reads its points as from k.  W is normalised to max |W| in
        // [1/2, 1) (fp16), in the tables' unused tail.
        if (q0 < q1)
            __builtin_amdgcn_s_waitcnt(kWaitVm8);   // tables landed; the pair loads may be in flight
        else
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
        const float2 Wn = make_float2(gC.x * gB.x - gC.y * gB.y, gC.x * gB.y + gC.y * gB.x);
        const int ew = __builtin_amdgcn_readfirstlane(exp_of(wave_max(fmaxf(fabsf(Wn.x), fabsf(Wn.y)))));
        uint32_t *Wl = (uint32_t *)(Tab + kTab + 1568);   // 32 unused uint4 of the table
        __syncthreads();   // every wave's table copies landed
        if (w == 0) Wl[lane] = pk(ldexpf(Wn.x, -ew), ldexpf(Wn.y, -ew));
        __syncthreads();
        if (w < 2) {
            uint4 wq[4];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) wq[kb] = ((const uint4 *)Wl)[4 * kb + g];
            const float sc = ldexpf(2.0f, ew);
            float *Uf = (float *)U;
            state_term_core<false>(G1, wq, w, lane, [&](int t, f4_t D) {
                *(float4 *)(Uf + t) = make_float4(D[0] * sc, D[1] * sc, D[2] * sc, D[3] * sc);
            });
        }
        __syncthreads();
#pragma unroll
        for (int gi = 0; gi < 2; ++gi) {
            const int off = 4096 * xq + 256 * (4 * (2 * (w & 1) + gi) + jq) + 16 * c;
#pragma unroll
            for (int s = 0; s < 4; ++s) kq[4 * gi + s] = *(const float4 *)((const float *)U + off + 4 * s);
        }
    }

    // ---- kernel spectrum block w of channel h (F(k + D delta) 2^-ek / 128) ----
    uint32_t K[64];
    int kexp;
    uint32_t d[64];
    {
        if (tid == 0 && a.D) kq[0].x += a.D[h];   // point m = 0: wave 0, lane 0
        float mx = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            mx = fmaxf(mx, fmaxf(fmaxf(fabsf(kq[i].x), fabsf(kq[i].y)), fmaxf(fabsf(kq[i].z), fabsf(kq[i].w))));
        mx = wave_max(mx);
        if (lane == 0) red[w] = mx;
        // tables, factors and kernel row landed; only the first pair's 8
        // loads (issued last, if any) may still be in flight
        if (q0 < q1)
            __builtin_amdgcn_s_waitcnt(kWaitVm8);
        else
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
        __syncthreads();
        const int ek = __builtin_amdgcn_readfirstlane(exp_of(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))));
#pragma unroll
        for (int gi = 0; gi < 2; ++gi)
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const float4 v = kq[4 * gi + s];
                Ud[stage_at(gi, 4 * s + 0)] = pk(ldexpf(v.x, -ek), 0.f);
                Ud[stage_at(gi, 4 * s + 1)] = pk(ldexpf(v.y, -ek), 0.f);
                Ud[stage_at(gi, 4 * s + 2)] = pk(ldexpf(v.z, -ek), 0.f);
                Ud[stage_at(gi, 4 * s + 3)] = pk(ldexpf(v.w, -ek), 0.f);
            }
        __syncthreads();
        {
            uint32_t R[4], I[4], Rb[4], Ib[4];
            kinds_scaled(Lc[1 * 64 + lane], f1, R, I);
            kinds_rot(w, R, I, Rb, Ib);
            const Dft Fa = dft_of(R, I), Fb = dft_of(Rb, Ib);
            uint32_t xw[4], xs[4];
            twiddles_fwd(Lc[4 * 64 + lane], xf, xw, xs);
            layer1(U, lane, Fa.re, Fa.im, Fb.re, Fb.im, [&](int tau, f4_t re, f4_t im) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = cmul2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
            });
        }
        forward_mid(d, Lc, Ytab, lane);
        {
            uint32_t R[4], I[4];
            kinds_scaled(Lc[1 * 64 + lane], f3, R, I);
            layer<false>(d, dft_of(R, I), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) K[4 * tau + jj] = pk(re[jj], im[jj]);
            });
        }
        if (a.conj_k) {   // conjugated spectrum (correlation, the input gradient)
#pragma unroll
            for (int i = 0; i < 64; ++i) K[i] ^= 0x80000000u;
        }
        h2_t hmx = {0, 0}, hmn = {0, 0};
#pragma unroll
        for (int i = 0; i < 64; i += 2) {
            hmx = __builtin_elementwise_maximum(hmx, __builtin_elementwise_maximum(as_h2(K[i]), as_h2(K[i + 1])));
            hmn = __builtin_elementwise_minimum(hmn, __builtin_elementwise_minimum(as_h2(K[i]), as_h2(K[i + 1])));
        }
        float km = fmaxf(fmaxf((float)hmx.x, (float)hmx.y), fmaxf(-(float)hmn.x, -(float)hmn.y));
        km = wave_max(km);
        if (lane == 0) red[NW + w] = km;
        __syncthreads();   // red; every wave is done reading the staged kernel row
        const int e2 = __builtin_amdgcn_readfirstlane(
            exp_of(fmaxf(fmaxf(red[NW], red[NW + 1]), fmaxf(red[NW + 2], red[NW + 3]))));
        kexp = 6 + ek + e2;
        const _Float16 s2 = (_Float16)ldexpf(1.0f, -e2);
        const h2_t s22 = {s2, s2};
#pragma unroll
        for (int i = 0; i < 4; ++i) f3[i] = as_u32(as_h2(f3[i]) * s22);   // pairs' third layer carries 2^-e2
    }

    // ---- row pairs: all four waves on each pair ----
    for (int qq = q0; qq < q1; ++qq) {
        // the per-wave factors are loop-invariant; opaque here so that their
        // swizzled and negated forms are not hoisted out of the loop as well
#pragma unroll
        for (int i = 0; i < 4; ++i) asm volatile("" : "+v"(f1[i]), "+v"(xf[i]), "+v"(f3[i]));
        asm volatile("" : "+v"(g3), "+v"(xh));
        {
            const float mxa = wave_max(raw_max<DT>(ra)), mxb = wave_max(raw_max<DT>(rb));
            if (lane == 0) {
                red[w] = mxa;
                red[2 * NW + w] = mxb;
            }
        }
        __syncthreads();   // red; the previous pair's exchange reads are done
        const float gma = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
        const float gmb = fmaxf(fmaxf(red[2 * NW], red[2 * NW + 1]), fmaxf(red[2 * NW + 2], red[2 * NW + 3]));
        // one power-of-two scale per row (see the one-wave kernel): fp16
        // inputs stay as they are while both rows sit in [2^-4, 16) within a
        // factor of four of each other
        int ea = exp_of(gma), eb = exp_of(gmb);
        if (!(gma > 0.f)) ea = eb;
        if (!(gmb > 0.f)) eb = ea;
        int eua = 0, eub = 0;
        if (DT == BF16 || !(ea >= -3 && ea <= 4 && eb >= -3 && eb <= 4 && abs(ea - eb) <= 1)) {
            eua = ea;
            eub = eb;
        }
        eua = __builtin_amdgcn_readfirstlane(eua);
        eub = __builtin_amdgcn_readfirstlane(eub);
        // interleave (u_a, u_b) and stage; fp16 inputs out of range are
        // scaled here, bf16 inputs through the first layer's matrix
#pragma unroll
        for (int gi = 0; gi < 2; ++gi)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const uint4 va = ra[2 * gi + hh], vb = rb[2 * gi + hh];
                const uint32_t A4[4] = {va.x, va.y, va.z, va.w}, B4[4] = {vb.x, vb.y, vb.z, vb.w};
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    uint32_t lo = __builtin_amdgcn_perm(B4[s], A4[s], 0x05040100u);
                    uint32_t hi = __builtin_amdgcn_perm(B4[s], A4[s], 0x07060302u);
                    if (DT == F16 && (eua | eub) != 0) {
                        lo = pk(ldexpf((float)as_h2(lo).x, -eua), ldexpf((float)as_h2(lo).y, -eub));
                        hi = pk(ldexpf((float)as_h2(hi).x, -eua), ldexpf((float)as_h2(hi).y, -eub));
                    }
                    Ud[stage_at(gi, 8 * hh + 2 * s)] = lo;
                    Ud[stage_at(gi, 8 * hh + 2 * s + 1)] = hi;
                }
            }
        const bool more = qq + 1 < q1;
        if (more) issue_loads(qq + 1);
        __syncthreads();   // staged pair visible
        {
            uint32_t R[4], I[4], Rb[4], Ib[4];
            kinds_scaled(Lc[1 * 64 + lane], f1, R, I);
            kinds_rot(w, R, I, Rb, Ib);
            uint32_t xw[4], xs[4];
            twiddles_fwd(Lc[4 * 64 + lane], xf, xw, xs);
            auto epi = [&](int tau, f4_t re, f4_t im) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = cmul2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
            };
            if (DT == F16) {
                const Dft Fa = dft_of(R, I), Fb = dft_of(Rb, Ib);
                layer1(U, lane, Fa.re, Fa.im, Fb.re, Fb.im, epi);
            } else {
                const float sa = ldexpf(1.0f, -eua), sb = ldexpf(1.0f, -eub);
                bf8_t Far, Fai, Fbr, Fbi;
                kinds_bf16(R, I, sa, sb, Far, Fai);
                kinds_bf16(Rb, Ib, sa, sb, Fbr, Fbi);
                layer1(U, lane, Far, Fai, Fbr, Fbi, epi);
            }
        }
        __syncthreads();   // every wave is done reading the staged pair
        forward_mid<CORR == 0>(d, Lc, Ytab, lane);
        {
            // third layer (contraction side times w_16384^{k3 p0} 2^-e2) and
            // the pointwise product with the kernel spectrum block
            uint32_t R[4], I[4];
            kinds_scaled(Lc[1 * 64 + lane], f3, R, I);
            layer_sel<CORR == 0, false>(d, dft_of(R, I), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    // opaque per use: otherwise the (-im, re) companion of every
                    // spectrum value is hoisted out of the pair loop (64 more VGPRs)
                    uint32_t kk = K[4 * tau + jj];
                    asm volatile("" : "+v"(kk));
                    d[4 * tau + jj] = cmul(pk(re[jj], im[jj]), kk);
                }
            });
        }
        {
            // inverse third layer: output rows times w_16384^{-k3 c}
            uint32_t R[4], I[4];
            const uint32_t gg[4] = {g3, g3, g3, g3};
            kinds_scaled(Lc[3 * 64 + lane], gg, R, I);
            layer_sel<CORR == 0, false>(d, dft_of(R, I), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = pk(re[jj], im[jj]);
            });
        }
        swap_GT(d);
        {
            uint32_t e[64];
#pragma unroll
            for (int T = 0; T < 16; ++T) {
                const uint4 yv = Ytab[T * 64 + lane];
                e[4 * T + 0] = cmulc(d[pidx(T, 0)], yv.x);
                e[4 * T + 1] = cmulc(d[pidx(T, 1)], yv.y);
                e[4 * T + 2] = cmulc(d[pidx(T, 2)], yv.z);
                e[4 * T + 3] = cmulc(d[pidx(T, 3)], yv.w);
            }
#pragma unroll
            for (int i = 0; i < 64; ++i) d[i] = e[i];
        }
        {
            uint32_t xw[4], xs[4];
            twiddles_inv(Lc[4 * 64 + lane], xh, xw, xs);
            layer_sel<CORR == 0, true>(d, lds_dft(Lc, lane, true), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = cmul2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
            });
        }
        // the inverse second layer's outputs are complete here (otherwise its
        // epilogues drift into the exchange and keep MFMA results live)
#pragma unroll
        for (int i = 0; i < 64; ++i) asm volatile("" ::"v"(d[i]));
        long oa, ob;
        rows(qq, oa, ob);
        const float sca = ldexpf(1.0f, kexp + eua), scb = ldexpf(1.0f, kexp + eub);
        uint16_t *ya = y + oa, *yb = y + (ob >= 0 ? ob : oa);
        const long obc = ob >= 0 ? ob : oa;
        const void *cra = nullptr, *crb = nullptr;
        if (CORR == 1) {
            cra = (const float *)a.corr + oa;
            crb = (const float *)a.corr + obc;
        } else if (CORR == 2) {
            cra = (const uint16_t *)a.corr + oa;
            crb = (const uint16_t *)a.corr + obc;
        }
        int ewa = 0, ewb = 0;
        if (CORR == 3) {   // normalised weights W of chunk rows oa / L, obc / L
            cra = (const uint32_t *)a.corr + (oa / L) * 64;
            crb = (const uint32_t *)a.corr + (obc / L) * 64;
            ewa = a.corr_e[oa / L];
            ewb = a.corr_e[obc / L];
        }
        last_layer<DT, CORR>(d, U, G1, Lc, gf, w, lane, sca, scb, ya, yb, ob >= 0, cra, crb, ewa, ewb);
    }
}

bool fftconv_wave16k_supported(int L, int dtype) { return L == w16::L && (dtype == F16 || dtype == BF16); }

hipError_t launch_fftconv_wave16k(const ConvArgs &a, const float *k, hipStream_t s) {
    if (!fftconv_wave16k_supported(a.L, a.dtype)) return hipErrorInvalidValue;
    int pairs_per_ch;
    if (a.pair_mode == 0)
        pairs_per_ch = (a.B + 1) / 2;
    else
        pairs_per_ch = a.B * ((a.nchunk + 1) / 2);
    // two workgroups fit a CU: split a channel while fewer than ~2 per CU
    // and each still gets two pairs
    int wg_per_ch = 1;
    while ((long)a.H * wg_per_ch < 512 && pairs_per_ch >= 4 * wg_per_ch) wg_per_ch *= 2;
    dim3 grid(a.H * wg_per_ch), block(w16::NT);
    const int corr = a.corr == nullptr ? 0 : a.corr_tab != nullptr ? 3 : (a.corr16 ? 2 : 1);
    if (corr == 3 && (a.pair_mode != 1 || a.corr_e == nullptr)) return hipErrorInvalidValue;
#define H3_W16_LAUNCH(DTV, CV) \
    hipLaunchKernelGGL((fftconv_wave16k_kernel<DTV, CV>), grid, block, 0, s, a, k, wg_per_ch, pairs_per_ch)
    if (a.dtype == F16) {
        if (corr == 0) H3_W16_LAUNCH(F16, 0);
        else if (corr == 1) H3_W16_LAUNCH(F16, 1);
        else if (corr == 2) H3_W16_LAUNCH(F16, 2);
        else H3_W16_LAUNCH(F16, 3);
    } else {
        if (corr == 0) H3_W16_LAUNCH(BF16, 0);
        else if (corr == 1) H3_W16_LAUNCH(BF16, 1);
        else if (corr == 2) H3_W16_LAUNCH(BF16, 2);
        else H3_W16_LAUNCH(BF16, 3);
    }
#undef H3_W16_LAUNCH
    return hipGetLastError();
}

}  // namespace h3
