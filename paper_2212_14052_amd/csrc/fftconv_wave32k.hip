// Fused FFT convolution for L = 16384 (transform length N = 2L = 32768 =
// 8 x 4096) with eight wavefronts per row pair (Sec. 4.1: kernel fusion +
// block FFT past the 8192 length of the paper's fused block; Sec. 4.2 uses
// it as the state-passing chunk), gfx950, 16-bit I/O.
//
// With p = 4096 p3 + m (m < 4096; the zero-padded input vanishes for
// p3 >= 4), decimating the frequency by eight (f = 8 f' + k3) gives
//   X[8 f' + k3] = DFT_4096[ w_32768^{k3 m} sum_{p3 < 4} w_8^{k3 p3} x(4096 p3 + m) ](f').
// Wave k3 of the workgroup runs block k3 through the register-resident
// 4096-point pipeline of the one-wave kernel (three radix-16 layers on the
// matrix cores; see wave_common.h), as the L = 8192 kernel does with four
// blocks.  The block twiddle, with m = 256 p2 + 16 p1 + p0,
//   w_32768^{k3 m} = w_128^{k3 p2} w_2048^{k3 p1} w_32768^{k3 p0},
// costs no instruction per point: the p2 factor scales the contraction side
// of the first layer's DFT matrix, the p1 factor rides on that layer's lane
// twiddles and the p0 factor scales the contraction side of the third
// layer's matrix.  The first layer contracts the four quarters x(4096 p3 +
// m) together as four K steps of the MFMA, the matrix of step p3 being the
// first one times w_8^{k3 p3}: a rotation by a power of -i, for odd
// exponents of the matrix times w_8 (built once per pair).
//
// Inverse: y(4096 t3 + m) = sum_k3 w_8^{-t3 k3} w_32768^{-k3 m} IDFT_4096[Y_k3](m)
// for t3 = 0 .. 3 (outputs t < L only).  Each wave runs its block backwards
// up to the last radix-16 layer (the p0 and p1 factors again folded into a
// layer matrix and the lane twiddles).  The last layer's inputs are then
// exchanged through LDS so that wave w holds tiles p0 = 2 w and 2 w + 1 of
// all eight blocks, and the last layer, the w_128^{-k3 p2} factors and the
// radix-8 combination over k3 run as one 128-point contraction: eight K steps
// of the MFMA per output tile and quarter t3, the factor w_8^{-t3 k3} taken
// as a choice between the block's rows and the rows times w_8^{-1} and a
// rotation by a power of i (signs and a row swap).
//
// The pair's input is staged once in LDS (64 KB) as interleaved complex
// (u_a, u_b) values, in the order the first layer reads them; every wave
// reads all of it and loads one eighth of it from HBM (prefetched into
// registers during the previous pair).  The per-wave factors are read from
// their constant table where they are used (they would not fit in registers
// beside the spectrum block, the signal and the prefetched rows).  The kernel spectrum block of each
// wave stays in registers.  D is folded into the kernel (k[0] += D).  16-bit
// inputs feed the first layer as they are (fp16 or bf16 MFMA); everything
// after it is fp16 with fp32 accumulation, with the power-of-two range
// control of the one-wave kernel.
#include "common.h"
#include "internal.h"
#include "wave_common.h"

namespace h3 {
namespace w32 {

using namespace wvc;

constexpr int N = 32768;
constexpr int L = 16384;
constexpr int NW = 8;           // waves per workgroup (one per frequency block)
constexpr int NT = 64 * NW;
constexpr int kU = 4096;        // uint4: pair staging, last-layer exchange, output staging (64 KB)

// LDS tables: the one-wave kernel's L2 twiddles and per-lane DFT rows, then
// for each source block k3' the last layer's rows: kinds 0, 1 = (real,
// imaginary) rows of entries conj(w_128^{(8 k2 + k3') p2}) / 8, kinds 2, 3 =
// the same times exp(i pi / 4) = w_8^{-1}; output row p2 = c, contraction
// point k2 = 4 g + i (lane l = 16 g + c).
constexpr int kTabG = 4 * 8 * 64;
constexpr int kTab32 = kTab + kTabG;   // uint4
struct Half32 {
    uint32_t v[4 * kTab32];
};
constexpr Half32 make_half32() {
    const HalfTable base = make_half_table();
    Half32 t{};
    for (int i = 0; i < 4 * kTab; ++i) t.v[i] = base.v[i];
    const double r2 = 0.70710678118654752440;
    for (int k3 = 0; k3 < 8; ++k3)
        for (int l = 0; l < 64; ++l)
            for (int i = 0; i < 4; ++i) {
                const long g = l >> 4, c = l & 15;
                const Cd v = cwd(-(8 * (4 * g + i) + k3) * c, 128);
                const double re = 0.125 * v.re, im = 0.125 * v.im;
                const double re45 = (re - im) * r2, im45 = (re + im) * r2;
                t.v[4 * (kTab + (4 * k3 + 0) * 64 + l) + i] = h2_bits(re, -im);
                t.v[4 * (kTab + (4 * k3 + 1) * 64 + l) + i] = h2_bits(im, re);
                t.v[4 * (kTab + (4 * k3 + 2) * 64 + l) + i] = h2_bits(re45, -im45);
                t.v[4 * (kTab + (4 * k3 + 3) * 64 + l) + i] = h2_bits(im45, re45);
            }
    return t;
}
__device__ const Half32 kHalf32 = make_half32();

// Per-wave (k3) and per-lane factors, fp16 (re, im), 16 dwords per lane:
//   [0..3]  w_128^{k3 (4g+i)} / 4      first layer, contraction point i (the
//                                      1/4 keeps the four-quarter sum in range)
//   [4..7]  w_2048^{k3 (4g+j)}         first layer's lane twiddles, row j
//   [8..11] w_32768^{k3 (4g+i)}        third layer, contraction point i
//   [12]    w_32768^{-k3 c}            inverse third layer, output row c
//   [13]    w_2048^{-k3 c}             inverse second layer's lane twiddles
//   [14]    w_8                        the first layer's odd quarter factors
struct Fac32 {
    uint32_t v[8 * 64 * 16];
};
constexpr Fac32 make_fac32() {
    Fac32 t{};
    for (int k3 = 0; k3 < 8; ++k3)
        for (int l = 0; l < 64; ++l) {
            const long g = l >> 4, c = l & 15;
            uint32_t *p = t.v + (k3 * 64 + l) * 16;
            for (int i = 0; i < 4; ++i) {
                const Cd a = cwd(k3 * (4 * g + i), 128);
                p[i] = h2_bits(0.25 * a.re, 0.25 * a.im);
                const Cd b = cwd(k3 * (4 * g + i), 2048);
                p[4 + i] = h2_bits(b.re, b.im);
                const Cd e = cwd(k3 * (4 * g + i), N);
                p[8 + i] = h2_bits(e.re, e.im);
            }
            const Cd r3 = cwd(-k3 * c, N), rx = cwd(-k3 * c, 2048), q = cwd(1, 8);
            p[12] = h2_bits(r3.re, r3.im);
            p[13] = h2_bits(rx.re, rx.im);
            p[14] = h2_bits(q.re, q.im);
        }
    return t;
}
__device__ const Fac32 kFac32 = make_fac32();

// The four first-layer matrices of wave k3 as (real, imaginary) row kinds:
// step p3 is the base (R, I) times w_8^{k3 p3} = (-i)^{e / 2} for even
// e = k3 p3 mod 8, and (R45, I45) (the base times w_8) times (-i)^{(e-1)/2}
// for odd e.
__device__ __forceinline__ void quarter_rows(int k3, const uint32_t (&R)[4], const uint32_t (&I)[4],
                                             const uint32_t (&R45)[4], const uint32_t (&I45)[4],
                                             uint32_t (&Rq)[4][4], uint32_t (&Iq)[4][4]) {
#pragma unroll
    for (int p3 = 0; p3 < 4; ++p3) {
        const int e = (k3 * p3) & 7;
        const bool odd = (e & 1) != 0;   // wave-uniform; element-wise selects keep the rows in registers
        uint32_t Rs[4], Is[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            Rs[i] = odd ? R45[i] : R[i];
            Is[i] = odd ? I45[i] : I[i];
        }
        kinds_rot(e >> 1, Rs, Is, Rq[p3], Iq[p3]);
    }
}

// First layer: signal as the A operand, the four K steps x(4096 p3 + m)
// (matrix F_p3) accumulated; operands straight from the staging buffer S
// (tile tau of quarter x at S[(16 x + tau) * 64 + lane]), one tile ahead.
// epi(tau, re, im) as in layer().
template <class OP, class Epi>
__device__ __forceinline__ void layer1q(const uint4 *S, int lane, const OP (&Fr)[4], const OP (&Fi)[4], Epi &&epi) {
    const f4_t z = {0.f, 0.f, 0.f, 0.f};
    auto mm = [&](const uint4 (&x)[4], f4_t &re, f4_t &im) {
        re = z;
        im = z;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const OP a = __builtin_bit_cast(OP, x[q]);
            re = mfma_acc(a, Fr[q], re);
            im = mfma_acc(a, Fi[q], im);
        }
    };
    uint4 x[4], n[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) x[q] = S[(16 * q) * 64 + lane];
    f4_t re, im;
    mm(x, re, im);
#pragma unroll
    for (int q = 0; q < 4; ++q) n[q] = S[(16 * q + 1) * 64 + lane];
#pragma unroll
    for (int tau = 0; tau < 16; ++tau) {
        f4_t re1, im1;
        if (tau + 1 < 16) mm(n, re1, im1);
        if (tau + 2 < 16) {
#pragma unroll
            for (int q = 0; q < 4; ++q) n[q] = S[(16 * q + tau + 2) * 64 + lane];
        }
        epi(tau, re, im);
        __builtin_amdgcn_sched_barrier(0);
        re = re1;
        im = im1;
    }
}

// One source block's contribution to an output tile, for the quarters t3:
// re/im += rot^n(A) b with rot = multiplication by i, done by the choice of
// row kind and the sign of the data.
__device__ __forceinline__ void acc_rot(int n, h8_t Ar, h8_t Ai, h8_t b, h8_t nb, f4_t &re, f4_t &im) {
    if (n == 0) {
        re = mfma_acc(Ar, b, re);
        im = mfma_acc(Ai, b, im);
    } else if (n == 1) {   // i P: (-Im P, Re P)
        re = mfma_acc(Ai, nb, re);
        im = mfma_acc(Ar, b, im);
    } else if (n == 2) {   // -P
        re = mfma_acc(Ar, nb, re);
        im = mfma_acc(Ai, nb, im);
    } else {               // -i P: (Im P, -Re P)
        re = mfma_acc(Ai, b, re);
        im = mfma_acc(Ar, nb, im);
    }
}

// Last layer for the wave's tiles p0 = 2 w + tt (tt = 0, 1): exchange,
// 128-point contraction with the radix-8 combination, output through LDS.
//   y(4096 t3 + m) = sum_k3' w_8^{-t3 k3'} G_k3' x_k3'   (real parts row a,
// imaginary parts row b).  Round tt: every wave writes its tiles 2 q + tt
// (q = 0 .. 7) to slot (source * 8 + q) of the 64 KB buffer, then reads slot
// (k3' * 8 + w) of every source k3'.  The values of round 0 wait in fp32 and
// are packed with those of round 1 (adjacent points), staged in LDS as rows
// a and b, and stored by every wave as one contiguous eighth.
// CORR: 0 none, 1 float32 term, 2 term in the I/O dtype, added at the store;
// 3 the term computed here from the chunk rows' normalised weights (cra, crb:
// 64 fp16 complex each; exponents ewa, ewb) and the channel's tables CT.
template <int DT, int CORR>
__device__ __forceinline__ void last_layer32(uint32_t (&d)[64], uint4 *U, const uint4 *G, const uint4 *CT, int w,
                                             int lane, float sca, float scb, uint16_t *ya, uint16_t *yb, bool has_b,
                                             const void *cra, const void *crb, int ewa, int ewb) {
    const int g = lane >> 4, c = lane & 15;
    float v0[4][2][4];        // round 0: [t3][row a, b][jj], scaled
    uint32_t po[4][2][4];     // packed rounds 0 and 1
    const f4_t z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
        __syncthreads();   // U free: the staged pair (round 0) or round 0's reads (round 1) are done
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int T = 2 * q + tt;
            U[(w * 8 + q) * 64 + lane] = make_uint4(d[4 * T], d[4 * T + 1], d[4 * T + 2], d[4 * T + 3]);
        }
        __syncthreads();
        f4_t D[4][2] = {{z, z}, {z, z}, {z, z}, {z, z}};
        uint4 b4 = U[(0 * 8 + w) * 64 + lane];
#pragma unroll
        for (int k3p = 0; k3p < 8; ++k3p) {
            const uint4 gr = G[(4 * k3p + 0) * 64 + lane], gi = G[(4 * k3p + 1) * 64 + lane];
            const uint4 hr = G[(4 * k3p + 2) * 64 + lane], hi = G[(4 * k3p + 3) * 64 + lane];
            uint4 nb4 = b4;
            if (k3p + 1 < 8) nb4 = U[((k3p + 1) * 8 + w) * 64 + lane];
            const h8_t b = __builtin_bit_cast(h8_t, b4);
            const h8_t nb = __builtin_bit_cast(
                h8_t, make_uint4(b4.x ^ 0x80008000u, b4.y ^ 0x80008000u, b4.z ^ 0x80008000u, b4.w ^ 0x80008000u));
            const h8_t Gr = __builtin_bit_cast(h8_t, gr), Gi = __builtin_bit_cast(h8_t, gi);
            const h8_t Hr = __builtin_bit_cast(h8_t, hr), Hi = __builtin_bit_cast(h8_t, hi);
#pragma unroll
            for (int t3 = 0; t3 < 4; ++t3) {
                const int e = (t3 * k3p) & 7;   // factor exp(i pi e / 4)
                if (e & 1)
                    acc_rot(e >> 1, Hr, Hi, b, nb, D[t3][0], D[t3][1]);
                else
                    acc_rot(e >> 1, Gr, Gi, b, nb, D[t3][0], D[t3][1]);
            }
            __builtin_amdgcn_sched_barrier(0);
            b4 = nb4;
        }
#pragma unroll
        for (int t3 = 0; t3 < 4; ++t3)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const float va = D[t3][0][jj] * sca, vb = D[t3][1][jj] * scb;
                if (tt == 0) {
                    v0[t3][0][jj] = va;
                    v0[t3][1][jj] = vb;
                } else {
                    po[t3][0][jj] = pack_out<DT>(v0[t3][0][jj], va);
                    po[t3][1][jj] = pack_out<DT>(v0[t3][1][jj], vb);
                }
            }
    }
    // outputs t = 4096 t3 + 256 (4 g + jj) + 16 c + 2 w (+ 1) of both rows go
    // through LDS (rows a, b as 16384 halves each), then out as 16-byte
    // chunks, each wave a contiguous eighth of the pair
    uint4 cq[8];   // correction term (CORR 2), loaded while the outputs are staged
    uint4 wq[4];   // fused state term (CORR 3): the row's weights W for the lane's 16 modes
    const bool active = w < 4 || has_b;
    __syncthreads();   // every exchange read is done
    uint32_t *Ud = (uint32_t *)U;
#pragma unroll
    for (int t3 = 0; t3 < 4; ++t3)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int dw = 2048 * t3 + 128 * (4 * g + jj) + 8 * c + w;
            Ud[dw] = po[t3][0][jj];
            Ud[8192 + dw] = po[t3][1][jj];
        }
    uint16_t *yrow = w < 4 ? ya : yb;
    const void *crow = w < 4 ? cra : crb;
    if (CORR == 2) {
#pragma unroll
        for (int r = 0; r < 8; ++r)
            cq[r] = active ? ((const uint4 *)crow)[(w & 3) * 512 + r * 64 + lane] : make_uint4(0, 0, 0, 0);
    }
    if (CORR == 3) {   // modes 16 kb + 4 g + (0..3): one uint4 per kb
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
            wq[kb] = active ? ((const uint4 *)crow)[4 * kb + (lane >> 4)] : make_uint4(0, 0, 0, 0);
    }
    __syncthreads();
    if constexpr (CORR == 3) {
        if (active) fused_state_term<DT, 4096>(U, CT, wq, w < 4 ? ewa : ewb, w >> 2, w & 3, lane, yrow);
        return;
    }
    if (active) {
#pragma unroll
        for (int r = 0; r < 8; ++r) {
            const int i8 = (w & 3) * 512 + r * 64 + lane;   // uint4 index within the row
            uint4 v = U[(w >> 2) * 2048 + i8];
            if constexpr (CORR != 0) {
                float cv[8];
                if constexpr (CORR == 1) {
                    const float4 c0 = ((const float4 *)crow)[2 * i8], c1 = ((const float4 *)crow)[2 * i8 + 1];
                    cv[0] = c0.x; cv[1] = c0.y; cv[2] = c0.z; cv[3] = c0.w;
                    cv[4] = c1.x; cv[5] = c1.y; cv[6] = c1.z; cv[7] = c1.w;
                } else {
                    const uint32_t cw[4] = {cq[r].x, cq[r].y, cq[r].z, cq[r].w};
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

}  // namespace w32

// ============================================================================
template <int DT, int CORR>
__global__ __launch_bounds__(w32::NT) __attribute__((amdgpu_waves_per_eu(2))) void fftconv_wave32k_kernel(
    ConvArgs a, const float *k, int wg_per_ch, int pairs_per_ch) {
    using namespace w32;
    // Ytab + Lc, then the last layer's rows, then (CORR 3) the channel's
    // state-term tables
    constexpr int kTabAll = CORR == 3 ? kTab32 + CORR_TAB_U4 : kTab32;
    __shared__ uint4 Tab[kTabAll];
    __shared__ uint4 U[kU];         // pair staging, then the exchange and the output staging
    __shared__ float red[3 * NW];   // row a max | kernel spectrum max | row b max
    const uint4 *Ytab = Tab, *Lc = Tab + kTabY, *G = Tab + kTab, *CT = Tab + kTab32;
    uint32_t *Ud = (uint32_t *)U;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // frequency block k3
    const int c = lane & 15;
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
    // This wave's eighth of a pair: quarter x = w >> 1, lane rows g = 2 (w & 1)
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
        const int base = r * NT + 64 * w;   // kTab32 and CORR_TAB_U4 are multiples of 64
        if (base < kTabAll) {
            const uint4 *src = (CORR != 3 || base < kTab32) ? (const uint4 *)kHalf32.v + base
                                                            : a.corr_tab + (long)h * CORR_TAB_U4 + (base - kTab32);
            __builtin_amdgcn_global_load_lds((gvoid_t *)(src + lane), (lvoid_t *)(Tab + base), 16, 0, 0);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    // factor group i (0: f1, 1: xf, 2: f3, 3: g3 | xh | w8) of this wave and
    // lane; the index is opaque at every call so that the loads stay where
    // they are used instead of being hoisted out of the pair loop
    auto fac = [&](int i) {
        int idx = (w * 64 + lane) * 4 + i;
        asm volatile("" : "+v"(idx));
        return ((const uint4 *)kFac32.v)[idx];
    };
    auto u4 = [](uint4 v, uint32_t (&o)[4]) {
        o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
    };
    int e2 = 0;   // the spectrum's exponent: pairs' third layer carries 2^-e2
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
        // k_t = 2 Re sum_n W_n Abar_n^t with W_n = C_n Bbar_n, as in the
        // L = 8192 conv: waves 0 .. 3 form the quarters t in [4096 w, 4096 w
        // + 4096) in fp32 into U, then every wave reads its points as from k
        if (q0 < q1)
            __builtin_amdgcn_s_waitcnt(kWaitVm8);   // tables landed; the pair loads may be in flight
        else
            __builtin_amdgcn_s_waitcnt(kWaitVm0);
        const float2 Wn = make_float2(gC.x * gB.x - gC.y * gB.y, gC.x * gB.y + gC.y * gB.x);
        const int ew = __builtin_amdgcn_readfirstlane(exp_of(wave_max(fmaxf(fabsf(Wn.x), fabsf(Wn.y)))));
        uint32_t *Wl = (uint32_t *)(Tab + kTab32 + 1568);   // 32 unused uint4 of the table
        __syncthreads();   // every wave's table copies landed
        if (w == 0) Wl[lane] = pk(ldexpf(Wn.x, -ew), ldexpf(Wn.y, -ew));
        __syncthreads();
        if (w < 4) {
            uint4 wq[4];
            const int g = lane >> 4;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) wq[kb] = ((const uint4 *)Wl)[4 * kb + g];
            const float sc = ldexpf(2.0f, ew);
            float *Uf = (float *)U;
            state_term_core<true>(CT, wq, w, lane, [&](int t, f4_t D) {
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

    // first-layer rows of this wave: the base (contraction side times
    // w_128^{k3 p2} / 4) and the same times w_8
    auto first_rows = [&](uint32_t (&Rq)[4][4], uint32_t (&Iq)[4][4]) {
        uint32_t R[4], I[4], R45[4], I45[4], f1[4];
        u4(fac(0), f1);
        const uint32_t w8 = fac(3).z;
        kinds_scaled(Lc[1 * 64 + lane], f1, R, I);
        const uint32_t f45[4] = {cmul(f1[0], w8), cmul(f1[1], w8), cmul(f1[2], w8), cmul(f1[3], w8)};
        kinds_scaled(Lc[1 * 64 + lane], f45, R45, I45);
        quarter_rows(w, R, I, R45, I45, Rq, Iq);
    };

    // ---- kernel spectrum block w of channel h (F(k + D delta) 2^-ek / 256) ----
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
        float gm = red[0];
#pragma unroll
        for (int i = 1; i < NW; ++i) gm = fmaxf(gm, red[i]);
        const int ek = __builtin_amdgcn_readfirstlane(exp_of(gm));
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
            uint32_t Rq[4][4], Iq[4][4];
            first_rows(Rq, Iq);
            h8_t Fr[4], Fi[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const Dft F = dft_of(Rq[q], Iq[q]);
                Fr[q] = F.re;
                Fi[q] = F.im;
            }
            uint32_t xw[4], xs[4], xf[4];
            u4(fac(1), xf);
            twiddles_fwd(Lc[4 * 64 + lane], xf, xw, xs);
            layer1q(U, lane, Fr, Fi, [&](int tau, f4_t re, f4_t im) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = cmul2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
            });
        }
        forward_mid(d, Lc, Ytab, lane);
        {
            uint32_t R[4], I[4], f3[4];
            u4(fac(2), f3);
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
        float gk = red[NW];
#pragma unroll
        for (int i = 1; i < NW; ++i) gk = fmaxf(gk, red[NW + i]);
        e2 = __builtin_amdgcn_readfirstlane(exp_of(gk));
        // forward 1/256 per transform (first layer 1/16, then 1/4, 1/4);
        // inverse 1/128 (1/4, 1/4, last layer 1/8); N y = the unnormalised
        // inverse: y = out 256 256 128 / 32768 2^(eu + ek + e2)
        kexp = 8 + ek + e2;
    }
    const _Float16 s2 = (_Float16)ldexpf(1.0f, -e2);

    // ---- row pairs: all eight waves on each pair ----
    for (int qq = q0; qq < q1; ++qq) {
        {
            const float mxa = wave_max(raw_max<DT>(ra)), mxb = wave_max(raw_max<DT>(rb));
            if (lane == 0) {
                red[w] = mxa;
                red[2 * NW + w] = mxb;
            }
        }
        __syncthreads();   // red; the previous pair's output reads are done
        float gma = red[0], gmb = red[2 * NW];
#pragma unroll
        for (int i = 1; i < NW; ++i) {
            gma = fmaxf(gma, red[i]);
            gmb = fmaxf(gmb, red[2 * NW + i]);
        }
        // one power-of-two scale per row: fp16 inputs stay as they are while
        // both rows sit in [2^-4, 16) within a factor of four of each other
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
        // scaled here, bf16 inputs through the first layer's matrices
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
            uint32_t Rq[4][4], Iq[4][4];
            first_rows(Rq, Iq);
            uint32_t xw[4], xs[4], xf[4];
            u4(fac(1), xf);
            twiddles_fwd(Lc[4 * 64 + lane], xf, xw, xs);
            auto epi = [&](int tau, f4_t re, f4_t im) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = cmul2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
            };
            if (DT == F16) {
                h8_t Fr[4], Fi[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const Dft F = dft_of(Rq[q], Iq[q]);
                    Fr[q] = F.re;
                    Fi[q] = F.im;
                }
                layer1q(U, lane, Fr, Fi, epi);
            } else {
                const float sa = ldexpf(1.0f, -eua), sb = ldexpf(1.0f, -eub);
                bf8_t Fr[4], Fi[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) kinds_bf16(Rq[q], Iq[q], sa, sb, Fr[q], Fi[q]);
                layer1q(U, lane, Fr, Fi, epi);
            }
        }
        forward_mid(d, Lc, Ytab, lane);
        {
            // third layer (contraction side times w_32768^{k3 p0} 2^-e2) and
            // the pointwise product with the kernel spectrum block
            uint32_t R[4], I[4], f3[4];
            u4(fac(2), f3);
            const h2_t s22 = {s2, s2};
#pragma unroll
            for (int i = 0; i < 4; ++i) f3[i] = as_u32(as_h2(f3[i]) * s22);
            kinds_scaled(Lc[1 * 64 + lane], f3, R, I);
            layer<false>(d, dft_of(R, I), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
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
            // inverse third layer: output rows times w_32768^{-k3 c}
            uint32_t R[4], I[4];
            const uint32_t g3 = fac(3).x;
            const uint32_t gg[4] = {g3, g3, g3, g3};
            kinds_scaled(Lc[3 * 64 + lane], gg, R, I);
            layer<false>(d, dft_of(R, I), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
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
            const uint32_t xh = fac(3).y;
            twiddles_inv(Lc[4 * 64 + lane], xh, xw, xs);
            layer<true>(d, lds_dft(Lc, lane, true), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
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
        last_layer32<DT, CORR>(d, U, G, CT, w, lane, sca, scb, ya, yb, ob >= 0, cra, crb, ewa, ewb);
    }
}

bool fftconv_wave32k_supported(int L, int dtype) { return L == w32::L && (dtype == F16 || dtype == BF16); }

hipError_t launch_fftconv_wave32k(const ConvArgs &a, const float *k, hipStream_t s) {
    if (!fftconv_wave32k_supported(a.L, a.dtype)) return hipErrorInvalidValue;
    int pairs_per_ch;
    if (a.pair_mode == 0)
        pairs_per_ch = (a.B + 1) / 2;
    else
        pairs_per_ch = a.B * ((a.nchunk + 1) / 2);
    // one workgroup per CU (LDS): split a channel while fewer than ~one per
    // CU and each still gets two pairs
    int wg_per_ch = 1;
    while ((long)a.H * wg_per_ch < 256 && pairs_per_ch >= 4 * wg_per_ch) wg_per_ch *= 2;
    dim3 grid(a.H * wg_per_ch), block(w32::NT);
    const int corr = a.corr == nullptr ? 0 : a.corr_tab != nullptr ? 3 : (a.corr16 ? 2 : 1);
    if (corr == 3 && (a.pair_mode != 1 || a.corr_e == nullptr)) return hipErrorInvalidValue;
#define H3_W32_LAUNCH(DTV, CV) \
    hipLaunchKernelGGL((fftconv_wave32k_kernel<DTV, CV>), grid, block, 0, s, a, k, wg_per_ch, pairs_per_ch)
    if (a.dtype == F16) {
        if (corr == 0) H3_W32_LAUNCH(F16, 0);
        else if (corr == 1) H3_W32_LAUNCH(F16, 1);
        else if (corr == 2) H3_W32_LAUNCH(F16, 2);
        else H3_W32_LAUNCH(F16, 3);
    } else {
        if (corr == 0) H3_W32_LAUNCH(BF16, 0);
        else if (corr == 1) H3_W32_LAUNCH(BF16, 1);
        else if (corr == 2) H3_W32_LAUNCH(BF16, 2);
        else H3_W32_LAUNCH(BF16, 3);
    }
#undef H3_W32_LAUNCH
    return hipGetLastError();
}

}  // namespace h3
