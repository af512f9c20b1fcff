// Fused FFT convolution with one wavefront per transform (Sec. 4.1: kernel
// fusion + block FFT), gfx950, 16-bit I/O, L = 2048, transform length
// N = 2L = 4096 = 16^3.
//
// A wavefront holds a whole length-4096 complex signal in registers: lane
// l = 16 g + c (g = l / 16, c = l % 16) keeps 64 packed-fp16 complex values
// d[4 T + j], T, j = 0..15, 0..3.  Each of the three radix-16 layers of the
// block FFT is 16 pairs of v_mfma_f32_16x16x32_f16 (real and imaginary rows of
// the 16x16 DFT matrix), one pair per "tile" of 16 length-16 vectors.  The
// three base-16 digits of an index live in three slots:
//   C  = c           (the lane within a row of 16 lanes)
//   G  = 4 g + j     (the row of 16 lanes and the register within a tile)
//   T  = T           (the tile)
// An MFMA always contracts the digit in slot G.  With the signal as the A
// operand the output frequency lands in slot C and the digit that was in C
// moves to G (the matrix core transposes for free); with the signal as the B
// operand the frequency stays in G.  The one exchange of slot G with slot T
// that the three layers need is done in registers with v_permlane32_swap and
// v_permlane16_swap (gfx950), so no transform touches LDS.
//
// Forward DFT, input index p = 256 p2 + 16 p1 + p0, output X[k2 + 16 k1 +
// 256 k0] (decimation in frequency):
//   load           p2 : G, p1 : C, p0 : T
//   L1 (signal A)  DFT over p2 -> k2 : C, p1 : G      then * w_256^{k2 p1}
//   L2 (signal B)  DFT over p1 -> k1 : G              then * w_4096^{p0 (k2 + 16 k1)}
//   swap G <-> T   p0 : G, k1 : T
//   L3 (signal B)  DFT over p0 -> k0 : G
// The second transform is the inverse DFT run backwards with conjugated
// matrices and twiddles (L3^H, swap, conj twiddle, L2^H as A, conj twiddle,
// L1^H as B) and ends in the load layout, so outputs are written where the
// inputs were read.
//
// The skip term D u is folded into the kernel (k[0] += D): the length-2L
// circular convolution of the zero-padded row with k + D delta equals the
// causal convolution plus D u on t < L.
//
// Dynamic range: every DFT matrix carries a factor 1/4; the signal is scaled
// by a power of two when its max |u| leaves [2^-4, 16) and the kernel spectrum
// is normalised to max |K| in [1/2, 1), so no fp16 intermediate overflows; the
// scale factors are powers of two and are undone in fp32 at the output.
//
// One workgroup of 4 waves handles the row pairs of one channel (or a share
// of them): wave 0 first transforms the channel's kernel into LDS (the
// spectrum never reaches HBM); every wave then streams its own pairs.
#include "common.h"
#include "internal.h"
#include "wave_common.h"

namespace h3 {
namespace wv {

using namespace wvc;

constexpr int N = 4096;
constexpr int L = 2048;
constexpr int NW = 4;           // waves per workgroup
constexpr int NT = 64 * NW;

__device__ const HalfTable kHalf = make_half_table();

// The two-channel instance stages a compact copy of the table: the conjugate
// DFT rows are the direct rows with one half's sign flipped ((re, -im) ->
// (re, im) and (im, re) -> (-im, re)), so they are formed in registers, and
// the 2 KB saved let three workgroups (three waves per SIMD) share a CU.
// Layout: Ytab, then DFT rows (real, imaginary), L1 twiddles X and (-im, re).
constexpr int kTabC = kTabY + 4 * 64;
struct HalfTableC {
    uint32_t v[4 * kTabC];
};
constexpr HalfTableC make_half_table_c() {
    const HalfTable h = make_half_table();
    HalfTableC c{};
    for (int i = 0; i < 4 * (kTabY + 2 * 64); ++i) c.v[i] = h.v[i];
    for (int i = 0; i < 4 * 2 * 64; ++i) c.v[4 * (kTabY + 2 * 64) + i] = h.v[4 * (kTabY + 4 * 64) + i];
    return c;
}
__device__ const HalfTableC kHalfC = make_half_table_c();
// per-lane constant kinds in the full (CT false) and compact (CT true) layouts
template <bool CT> struct LcKind {
    static constexpr int X = CT ? 2 : 4, XS = CT ? 3 : 5;
};
template <bool CT>
__device__ __forceinline__ Dft lc_dft(const uint4 *Lc, int lane, bool conj) {
    if constexpr (!CT) {
        return lds_dft(Lc, lane, conj);
    } else {
        asm volatile("" ::: "memory");   // re-read per layer, do not keep live
        uint4 re = Lc[lane], im = Lc[64 + lane];
        if (conj) {
            re = make_uint4(re.x ^ 0x80000000u, re.y ^ 0x80000000u, re.z ^ 0x80000000u, re.w ^ 0x80000000u);
            im = make_uint4(im.x ^ 0x8000u, im.y ^ 0x8000u, im.z ^ 0x8000u, im.w ^ 0x8000u);
        }
        Dft F;
        F.re = __builtin_bit_cast(h8_t, re);
        F.im = __builtin_bit_cast(h8_t, im);
        return F;
    }
}

// Forward transform of a register-resident signal up to L3: L1 (signal A) +
// w_256 twiddle, L2 (signal B) + w_4096 twiddle written in P layout, swap.
template <bool CT>
__device__ __forceinline__ void forward_front(uint32_t (&d)[64], const uint4 *Lc, const uint4 *Ytab,
                                              int lane) {
    {
        const Dft F = lc_dft<CT>(Lc, lane, false);
        const uint4 X = Lc[LcKind<CT>::X * 64 + lane], Xs = Lc[LcKind<CT>::XS * 64 + lane];
        const uint32_t xw[4] = {X.x, X.y, X.z, X.w}, xs[4] = {Xs.x, Xs.y, Xs.z, Xs.w};
        layer2<true>(d, F, NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = cmul2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
        });
    }
    uint32_t e[64];
    {
        const Dft F = lc_dft<CT>(Lc, lane, false);
        layer2<false>(d, F, [&](int tau) { return Ytab[tau * 64 + lane]; },
                     [&](int tau, f4_t re, f4_t im, uint4 y) {
                         e[pidx(tau, 0)] = cmul(pk(re[0], im[0]), y.x);
                         e[pidx(tau, 1)] = cmul(pk(re[1], im[1]), y.y);
                         e[pidx(tau, 2)] = cmul(pk(re[2], im[2]), y.z);
                         e[pidx(tau, 3)] = cmul(pk(re[3], im[3]), y.w);
                     });
    }
#pragma unroll
    for (int i = 0; i < 64; ++i) d[i] = e[i];
    swap_GT(d);
}
// L1^H with the output epilogue.  Only outputs p2 < 8 (t < L) are kept, so
// one MFMA per tile suffices: its matrix Fc stacks the real rows 0..7 (rows
// 0..7 of the product: row a) over the imaginary rows 0..7 (rows 8..15: row
// b).  Lane (g, c) then holds, for tile tau, the outputs p2 = 4 (g & 1) + i,
// p1 = c, p0 = tau of row a (g < 2) or row b (g >= 2), times rem (REM), plus
// the correction term of that row (CORR), times the gate (GATE: the same
// points of the row at grow), packed two tiles at a time into d[8 s + i]
// (points p0 = 2 s, 2 s + 1).
template <int DT, int CORR, bool REM, bool GATE>
__device__ __forceinline__ void out_layer(uint32_t (&d)[64], const h8_t &Fc, float rem, const void *corr,
                                          long orow, int lane, const uint16_t *grow) {
    const int g = lane >> 4, c = lane & 15;
    const int pbase = 256 * (4 * (g & 1)) + 16 * c;
    // gate: gq[2 i + h] holds the gate at points p0 = 8 h .. 8 h + 7 of output
    // i; the second half (h = 1) is loaded while tiles 3 .. 7 run, so that
    // only 16 registers of it are live at a time
    uint4 gq[8];
    auto gate_loads = [&](int hh) {
#pragma unroll
        for (int i = 0; i < 4; ++i) gq[2 * i + hh] = *(const uint4 *)(grow + pbase + 256 * i + 8 * hh);
    };
    if constexpr (GATE) gate_loads(0);
    float pr[4];   // previous (even) tile's outputs
    auto mm = [&](int tau) {
        h8_t x = h8_of(d[4 * tau], d[4 * tau + 1], d[4 * tau + 2], d[4 * tau + 3]);
        asm volatile("" : "+v"(x));
        return mfma(Fc, x);
    };
    f4_t v = mm(0), vn = mm(1);
#pragma unroll
    for (int tau = 0; tau < 16; ++tau) {
        f4_t v1 = vn;
        if (tau + 2 < 16) vn = mm(tau + 2);
        if (GATE && tau == 3) gate_loads(1);
        float yv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) yv[i] = REM ? v[i] * rem : v[i];
        if (CORR != 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int p = pbase + 256 * i + tau;
                if (CORR == 2)
                    yv[i] += lo_f<DT>(((const uint16_t *)corr)[orow + p]);
                else
                    yv[i] += ((const float *)corr)[orow + p];
            }
        }
        if constexpr (GATE) {
            // gate values of this lane's points: gq[2 i + tau / 8], half tau % 8
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint4 q4 = gq[2 * i + (tau >> 3)];
                const uint32_t qw = (tau & 7) < 2 ? q4.x : (tau & 7) < 4 ? q4.y : (tau & 7) < 6 ? q4.z : q4.w;
                yv[i] *= (tau & 1) ? hi_f<DT>(qw) : lo_f<DT>(qw);
            }
        }
        if ((tau & 1) == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) pr[i] = yv[i];
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) d[4 * (tau - 1) + i] = pack_out<DT>(pr[i], yv[i]);
        }
        __builtin_amdgcn_sched_barrier(0);
        v = v1;
    }
}

}  // namespace wv

// ============================================================================
// CORR: 0 none, 1 float32 correction term, 2 correction term in the I/O dtype.
// CPW: channels per workgroup.  1: the four waves share one channel's row
// pairs.  2 (at most two row pairs per channel, e.g. batch 4): channels
// 2 hb and 2 hb + 1, both spectra computed by all four waves, then waves 0, 1
// take the first channel's pairs and waves 2, 3 the second's, so no wave
// idles while its workgroup holds the CU's LDS.
// GATE: the output is multiplied by a.gate (same layout as y) before rounding.
template <int DT, int CORR, int CPW, bool CT = false, bool GATE = false>
__global__ __launch_bounds__(wv::NT) __attribute__((amdgpu_waves_per_eu(CPW == 1 || CT ? 3 : 2))) void
fftconv_wave4096_kernel(ConvArgs a, const float *k, int wg_per_ch, int pairs_per_ch) {
    using namespace wv;
    // CT: the compact constant table (three workgroups per CU; two channels per
    // workgroup only)
    static_assert(!CT || CPW == 2, "compact table with two channels per workgroup");
    constexpr int kT = CT ? kTabC : kTab;
    __shared__ uint4 Tab[kT];         // Ytab (L2 twiddles per tile and lane) + Lc (per-lane constants)
    __shared__ uint4 Ks[CPW][16 * 64];   // kernel spectra per L3 quad and lane (also the spectrum's scratch)
    uint4 *Ytab = Tab, *Lc = Tab + kTabY;
    __shared__ float red[2 * NW];
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
    const int g = lane >> 4, c = lane & 15;
    const int hb = blockIdx.x / wg_per_ch, part = blockIdx.x % wg_per_ch;
    const int chw = CPW == 1 ? 0 : (w >> 1);   // this wave's channel within the workgroup
    const int h = hb * CPW + chw;              // this wave's channel
    const int wl = CPW == 1 ? w : (w & 1);     // this wave's index among its channel's waves
    constexpr int WPC = NW / CPW;              // waves per channel
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
    // raw loads of a pair: lanes g < 2 hold points p2 = 4 g + j (j = 0..3),
    // p1 = c, p0 = 0..15 of both rows (8 consecutive 16-bit values per uint4)
    uint4 ra[8], rb[8];
    auto issue_loads = [&](int qq) {
        long oa, ob;
        rows(qq, oa, ob);
        const long obl = ob >= 0 ? ob : oa;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            ra[i] = make_uint4(0, 0, 0, 0);
            rb[i] = make_uint4(0, 0, 0, 0);
        }
        if (g < 2) {
            const uint16_t *ua = u + oa, *ub = u + obl;   // wave-uniform bases
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int off = 256 * (4 * g + j) + 16 * c;
                ra[2 * j] = *(const uint4 *)(ua + off);
                ra[2 * j + 1] = *(const uint4 *)(ua + off + 8);
                rb[2 * j] = *(const uint4 *)(ub + off);
                rb[2 * j + 1] = *(const uint4 *)(ub + off + 8);
            }
        }
        if (ob < 0) {
#pragma unroll
            for (int i = 0; i < 8; ++i) rb[i] = make_uint4(0, 0, 0, 0);
        }
    };
    // Loads in the order they are needed: (1) the constant tables, straight
    // into LDS (1 KB per wave and instruction, no registers)
#pragma unroll
    for (int r = 0; r < (kT + NT - 1) / NT; ++r) {
        const int base = r * NT + 64 * w;   // this wave's 64 uint4
        if (base < kT)
            __builtin_amdgcn_global_load_lds((gvoid_t *)((const uint4 *)(CT ? kHalfC.v : kHalf.v) + base + lane),
                                             (lvoid_t *)(Tab + base), 16, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    // (2) this wave's L1 tiles of the kernel row: lane (g < 2, c) takes
    // k[256 (4 g + j) + 16 c + 4 w + t], t = 0..3, for j = 0..3 (tile
    // T = 4 w + t, point p2 = 4 g + j)
    float4 kq[CPW][4];
#pragma unroll
    for (int ch = 0; ch < CPW; ++ch) {
        const int hs = hb * CPW + ch;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            kq[ch][j] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (g < 2 && (CPW == 1 || hs < a.H))   // one channel per workgroup: always present
                kq[ch][j] = *(const float4 *)(k + (long)hs * L + 256 * (4 * g + j) + 16 * c + 4 * w);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    // (3) this wave's first pair, in flight during the kernel transform
    int qq = q0 + wl;
    bool have = (CPW == 1 || h < a.H) && qq < q1;
    if (have) issue_loads(qq);

    // ---- kernel spectrum of channel h, all waves: wave w runs tiles
    //      4 w .. 4 w + 3 of L1 and L2 and quads 4 w .. 4 w + 3 of L3; the
    //      swap between L2 and L3 goes through Ks.  Ks ends up holding
    //      F(k + D delta) 2^-ek / 64; the pairs' L3 matrix carries 2^-e2.
    int kexpc[CPW], e2c[CPW];
#pragma unroll
    for (int ch = 0; ch < CPW; ++ch) {
        const int hs = hb * CPW + ch;
        if (CPW > 1 && hs >= a.H) {   // workgroup-uniform: an odd channel count's missing second channel
            kexpc[ch] = 0;
            e2c[ch] = 0;
            continue;
        }
        if (tid == 0 && a.D) kq[ch][0].x += a.D[hs];   // k[0] += D: lane 0, point 0 of tile 0
        float mx = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            mx = fmaxf(mx, fmaxf(fmaxf(fabsf(kq[ch][j].x), fabsf(kq[ch][j].y)), fmaxf(fabsf(kq[ch][j].z), fabsf(kq[ch][j].w))));
        mx = wave_max(mx);
        if (lane == 0) red[w] = mx;
        // tables and kernel row landed; at most the 16 pair loads (issued
        // last) still in flight
        if (have)
            __builtin_amdgcn_s_waitcnt(kWaitVm16);
        else
            __builtin_amdgcn_s_waitcnt(kWaitVm0);   // no pair loads: everything must land
        __syncthreads();   // red, Ytab, Lc
        const int ek = __builtin_amdgcn_readfirstlane(exp_of(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))));
        uint32_t dq[16];   // quad t = tile 4 w + t, element j
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            dq[0 + j] = pk(ldexpf(kq[ch][j].x, -ek), 0.f);
            dq[4 + j] = pk(ldexpf(kq[ch][j].y, -ek), 0.f);
            dq[8 + j] = pk(ldexpf(kq[ch][j].z, -ek), 0.f);
            dq[12 + j] = pk(ldexpf(kq[ch][j].w, -ek), 0.f);
        }
        const Dft F = lc_dft<CT>(Lc, lane, false);
        {
            const uint4 X = Lc[LcKind<CT>::X * 64 + lane], Xs = Lc[LcKind<CT>::XS * 64 + lane];
            const uint32_t xw[4] = {X.x, X.y, X.z, X.w}, xs[4] = {Xs.x, Xs.y, Xs.z, Xs.w};
            layer<true, 4>(dq, F, NoPre{}, [&](int t, f4_t re, f4_t im, uint4) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) dq[4 * t + jj] = cmul2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
            });
        }
        layer<false, 4>(dq, F, [&](int t) { return Ytab[(4 * w + t) * 64 + lane]; },
                        [&](int t, f4_t re, f4_t im, uint4 yv) {
            dq[4 * t + 0] = cmul(pk(re[0], im[0]), yv.x);
            dq[4 * t + 1] = cmul(pk(re[1], im[1]), yv.y);
            dq[4 * t + 2] = cmul(pk(re[2], im[2]), yv.z);
            dq[4 * t + 3] = cmul(pk(re[3], im[3]), yv.w);
        });
        // after the swap, tile T = 4 w + t output jj sits in lane 16 w + c,
        // L3 quad 4 g + jj, element t: one 16-byte write per jj
#pragma unroll
        for (int jj = 0; jj < 4; ++jj)
            Ks[ch][(4 * g + jj) * 64 + 16 * w + c] = make_uint4(dq[jj], dq[4 + jj], dq[8 + jj], dq[12 + jj]);
        __syncthreads();
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const uint4 v = Ks[ch][(4 * w + t) * 64 + lane];
            dq[4 * t + 0] = v.x; dq[4 * t + 1] = v.y; dq[4 * t + 2] = v.z; dq[4 * t + 3] = v.w;
        }
        layer<false, 4>(dq, F, NoPre{}, [&](int t, f4_t re, f4_t im, uint4) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) dq[4 * t + jj] = pk(re[jj], im[jj]);
        });
        h2_t hmx = {0, 0}, hmn = {0, 0};
#pragma unroll
        for (int i = 0; i < 16; i += 2) {
            hmx = __builtin_elementwise_maximum(hmx, __builtin_elementwise_maximum(as_h2(dq[i]), as_h2(dq[i + 1])));
            hmn = __builtin_elementwise_minimum(hmn, __builtin_elementwise_minimum(as_h2(dq[i]), as_h2(dq[i + 1])));
        }
        float km = fmaxf(fmaxf((float)hmx.x, (float)hmx.y), fmaxf(-(float)hmn.x, -(float)hmn.y));
        km = wave_max(km);
        if (lane == 0) red[NW + w] = km;
        // conjugated spectrum (correlation, the input gradient): flip the
        // sign of every imaginary half
        const uint32_t cj = a.conj_k ? 0x80000000u : 0u;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            Ks[ch][(4 * w + t) * 64 + lane] =
                make_uint4(dq[4 * t] ^ cj, dq[4 * t + 1] ^ cj, dq[4 * t + 2] ^ cj, dq[4 * t + 3] ^ cj);
        __syncthreads();   // Ks complete
        const int e2v = __builtin_amdgcn_readfirstlane(
            exp_of(fmaxf(fmaxf(red[NW], red[NW + 1]), fmaxf(red[NW + 2], red[NW + 3]))));   // in [-6, 6]
        e2c[ch] = e2v;
        kexpc[ch] = 6 + ek + e2v;
    }
    const int kexp = (CPW == 1 || chw == 0) ? kexpc[0] : kexpc[CPW - 1];
    const int e2 = (CPW == 1 || chw == 0) ? e2c[0] : e2c[CPW - 1];

    // ---- row pairs of this wave ----
    uint32_t d[64];
    // One flag guards both the prefetch and the back edge, so the staged
    // registers are dead between their unpacking and the next prefetch.
    while (have) {
        // max |u| per row, then packing into (a + i b) complex fp16: p2 =
        // 4 g + j : G, p1 = c : C, p0 = T : tile
        float mxa, mxb;
        if (DT == F16) {
            h2_t amx = {0, 0}, amn = {0, 0}, bmx = {0, 0}, bmn = {0, 0};
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint32_t va[4] = {ra[i].x, ra[i].y, ra[i].z, ra[i].w}, vb[4] = {rb[i].x, rb[i].y, rb[i].z, rb[i].w};
#pragma unroll
                for (int e = 0; e < 4; e += 2) {
                    amx = __builtin_elementwise_maximum(amx, __builtin_elementwise_maximum(as_h2(va[e]), as_h2(va[e + 1])));
                    amn = __builtin_elementwise_minimum(amn, __builtin_elementwise_minimum(as_h2(va[e]), as_h2(va[e + 1])));
                    bmx = __builtin_elementwise_maximum(bmx, __builtin_elementwise_maximum(as_h2(vb[e]), as_h2(vb[e + 1])));
                    bmn = __builtin_elementwise_minimum(bmn, __builtin_elementwise_minimum(as_h2(vb[e]), as_h2(vb[e + 1])));
                }
            }
            mxa = fmaxf(fmaxf((float)amx.x, (float)amx.y), fmaxf(-(float)amn.x, -(float)amn.y));
            mxb = fmaxf(fmaxf((float)bmx.x, (float)bmx.y), fmaxf(-(float)bmn.x, -(float)bmn.y));
        } else {
            uint32_t ma = 0, mb = 0;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint32_t va[4] = {ra[i].x, ra[i].y, ra[i].z, ra[i].w}, vb[4] = {rb[i].x, rb[i].y, rb[i].z, rb[i].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t x = va[e] & 0x7fff7fffu, z = vb[e] & 0x7fff7fffu;
                    ma = max(ma, max(x & 0xffffu, x >> 16));
                    mb = max(mb, max(z & 0xffffu, z >> 16));
                }
            }
            mxa = __uint_as_float(ma << 16);
            mxb = __uint_as_float(mb << 16);
        }
        mxa = wave_max(mxa);
        mxb = wave_max(mxb);
        // Each row of the pair has its own power-of-two scale, so the rounding
        // of the shared fp16 transform stays at each row's own scale.  fp16
        // inputs are left as they are while both rows sit in [2^-4, 16) within
        // a factor of four of each other (the common case); bf16 inputs are
        // converted (and scaled) anyway.
        int ea = exp_of(mxa), eb = exp_of(mxb);
        if (!(mxa > 0.f)) ea = eb;   // an all-zero (or absent) row takes its partner's scale
        if (!(mxb > 0.f)) eb = ea;
        int eua = 0, eub = 0;
        if (DT == BF16 || !(ea >= -3 && ea <= 4 && eb >= -3 && eb <= 4 && abs(ea - eb) <= 1)) {
            eua = ea;
            eub = eb;
        }
        eua = __builtin_amdgcn_readfirstlane(eua);   // equal in all lanes
        eub = __builtin_amdgcn_readfirstlane(eub);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int hf = 0; hf < 2; ++hf) {
                const uint4 va = ra[2 * j + hf], vb = rb[2 * j + hf];
                const uint32_t A4[4] = {va.x, va.y, va.z, va.w}, B4[4] = {vb.x, vb.y, vb.z, vb.w};
#pragma unroll
                for (int s = 0; s < 4; ++s) {
                    const int T = 8 * hf + 2 * s;
                    if (DT == F16) {
                        d[4 * T + j] = __builtin_amdgcn_perm(B4[s], A4[s], 0x05040100u);
                        d[4 * (T + 1) + j] = __builtin_amdgcn_perm(B4[s], A4[s], 0x07060302u);
                    } else {
                        d[4 * T + j] = pk(ldexpf(lo_f<DT>(A4[s]), -eua), ldexpf(lo_f<DT>(B4[s]), -eub));
                        d[4 * (T + 1) + j] = pk(ldexpf(hi_f<DT>(A4[s]), -eua), ldexpf(hi_f<DT>(B4[s]), -eub));
                    }
                }
            }
        }
        if (DT == F16 && (eua | eub) != 0) {
            // in float32: 2^-e may leave fp16's range
#pragma unroll
            for (int i = 0; i < 64; ++i) d[i] = pk(ldexpf((float)as_h2(d[i]).x, -eua), ldexpf((float)as_h2(d[i]).y, -eub));
        }

        forward_front<CT>(d, Lc, Ytab, lane);
        // L3 (matrix scaled by 2^-e2, the spectrum's normalisation) +
        // pointwise product with the kernel spectrum (quads in P layout)
        Dft F3 = lc_dft<CT>(Lc, lane, false);
        F3.re = h8_scale(F3.re, (_Float16)ldexpf(1.0f, -e2));
        F3.im = h8_scale(F3.im, (_Float16)ldexpf(1.0f, -e2));
        layer2<false>(d, F3, [&](int tau) { return Ks[chw][tau * 64 + lane]; },
                     [&](int tau, f4_t re, f4_t im, uint4 kk) {
            d[4 * tau + 0] = cmul(pk(re[0], im[0]), kk.x);
            d[4 * tau + 1] = cmul(pk(re[1], im[1]), kk.y);
            d[4 * tau + 2] = cmul(pk(re[2], im[2]), kk.z);
            d[4 * tau + 3] = cmul(pk(re[3], im[3]), kk.w);
        });
        // inverse: L3^H, swap, conj twiddle (back to quad-per-tile layout),
        // L2^H (signal A) + conj twiddle, L1^H
        layer2<false>(d, lc_dft<CT>(Lc, lane, true), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = pk(re[jj], im[jj]);
        });
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
            const uint4 X = Lc[LcKind<CT>::X * 64 + lane], Xs = Lc[LcKind<CT>::XS * 64 + lane];
            const uint32_t xw[4] = {X.x, X.y, X.z, X.w}, xs[4] = {Xs.x, Xs.y, Xs.z, Xs.w};
            layer2<true>(d, lc_dft<CT>(Lc, lane, true), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = cmulc2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
            });
        }
        // L1^H: outputs p2 = 4 g + i (kept for g < 2), p1 = c, p0 = tile.
        // The output scales 2^(kexp + eua), 2^(kexp + eub) ride on the DFT matrix as far as fp16
        // allows; any remainder is applied in fp32.
        long oa, ob;
        rows(qq, oa, ob);
        // The real rows of L1^H make row a (lanes g < 2 of the product), the
        // imaginary rows row b (lanes g >= 2): each carries its own row's scale.
        const int sea = kexp + eua, seb = kexp + eub;
        const int sfa = min(max(sea, -10), 14), srema = sea - sfa;
        const int sfb = min(max(seb, -10), 14), sremb = seb - sfb;
        const bool lane_b = g >= 2;
        h8_t Fc;
        {
            asm volatile("" ::: "memory");
            const bool hi = c >= 8;   // imaginary rows: lane c - 8's imaginary DFT row
            uint4 r;
            if constexpr (!CT) {
                r = hi ? Lc[3 * 64 + lane - 8] : Lc[2 * 64 + lane];
            } else {
                r = hi ? Lc[64 + lane - 8] : Lc[lane];
                const uint32_t f = hi ? 0x8000u : 0x80000000u;
                r = make_uint4(r.x ^ f, r.y ^ f, r.z ^ f, r.w ^ f);
            }
            Fc = h8_scale(__builtin_bit_cast(h8_t, r), (_Float16)ldexpf(1.0f, hi ? sfb : sfa));
        }
        // branch-free epilogue (a branch inside it lets the compiler hoist
        // all of the layer's MFMAs above it); the rare remainder scale picks
        // a second instance of the layer instead
        const long obc = ob >= 0 ? ob : oa;   // row b's correction read from row a if absent
        const long orow = lane_b ? obc : oa;
        // gate of the lane's 64 outputs (row a or b; a missing row b reads row a's)
        const uint16_t *grow = GATE ? (const uint16_t *)a.gate + orow : nullptr;
        if ((srema | sremb) == 0)
            out_layer<DT, CORR, false, GATE>(d, Fc, 1.0f, a.corr, orow, lane, grow);
        else
            out_layer<DT, CORR, true, GATE>(d, Fc, ldexpf(1.0f, lane_b ? sremb : srema), a.corr, orow, lane, grow);
        if (!lane_b || ob >= 0) {
            uint16_t *yrow = y + orow;
            const int gl = g & 1;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int off = 256 * (4 * gl + i) + 16 * c;
                *(uint4 *)(yrow + off) = make_uint4(d[i], d[8 + i], d[16 + i], d[24 + i]);
                *(uint4 *)(yrow + off + 8) = make_uint4(d[32 + i], d[40 + i], d[48 + i], d[56 + i]);
            }
        }
        // next pair's loads, consumed at the top of the next iteration
        qq += WPC;
        have = qq < q1;
        if (have) issue_loads(qq);
    }
}

// ============================================================================
// Kernel gradient of the convolution at L = 2048, 16-bit I/O (the appendix on
// the backward pass): dk[h] = Re IFFT( sum_b conj(F u_b) . F dy_b )[:L], with
// rows paired as above (the real part of the pair product is the sum of the two
// rows' correlations; the cross terms land in the imaginary part), and
// dD[h] = sum_{b,t} u dy = dk[h][0].
//
// One workgroup per channel.  Each wave takes row pairs q = w, w + 4, ...:
// the forward transform of the u pair (as in the convolution, through L3) is
// kept in packed fp16; the forward transform of the dy pair ends in an L3
// epilogue that forms conj(Zu) . Zdy in float32 from the matrix-core outputs,
// undoes both inputs' power-of-two scales and adds it into a float32 spectrum
// in LDS (the four waves in turn).  Wave 0 then normalises the summed
// spectrum to a power of two, runs the inverse of the
// convolution (L3^H, swap, conj twiddle, L2^H, L1^H) and writes dk in float32.
// Scales: the forward leaves F(z) 2^-e / 64 (three matrices carrying 1/4), so
// the accumulated spectrum is S = sum conj(F z_u) F z_dy / 4096; with S scaled
// by 2^-es the inverse returns 64 IFFT(S 2^-es), hence dk = Re(out) 2^(es + 6).
namespace wv {

// Raw 16-bit loads of a row pair (layout of the convolution's loads); rows
// past the batch read as zero.
__device__ __forceinline__ void load_pair_raw(const uint16_t *x, long oa, long ob, int g, int c, uint4 (&ra)[8],
                                              uint4 (&rb)[8]) {
    const long obl = ob >= 0 ? ob : oa;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        ra[i] = make_uint4(0, 0, 0, 0);
        rb[i] = make_uint4(0, 0, 0, 0);
    }
    if (g < 2) {
        const uint16_t *xa = x + oa, *xb = x + obl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int off = 256 * (4 * g + j) + 16 * c;
            ra[2 * j] = *(const uint4 *)(xa + off);
            ra[2 * j + 1] = *(const uint4 *)(xa + off + 8);
            rb[2 * j] = *(const uint4 *)(xb + off);
            rb[2 * j + 1] = *(const uint4 *)(xb + off + 8);
        }
    }
    if (ob < 0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) rb[i] = make_uint4(0, 0, 0, 0);
    }
}

// Pack a raw pair into the complex signal d = (a + i b) 2^-e (load layout of
// the transform), e the power of two that brings max |x| below 1 (0 when the
// fp16 values need no scaling).  Returns e (wave-uniform).
template <int DT>
__device__ __forceinline__ int pack_pair(const uint4 (&ra)[8], const uint4 (&rb)[8], uint32_t (&d)[64]) {
    uint32_t mb = 0;
    float mx;
    if (DT == F16) {
        h2_t hmx = {0, 0}, hmn = {0, 0};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t v[8] = {ra[i].x, ra[i].y, ra[i].z, ra[i].w, rb[i].x, rb[i].y, rb[i].z, rb[i].w};
#pragma unroll
            for (int e = 0; e < 8; e += 2) {
                hmx = __builtin_elementwise_maximum(hmx, __builtin_elementwise_maximum(as_h2(v[e]), as_h2(v[e + 1])));
                hmn = __builtin_elementwise_minimum(hmn, __builtin_elementwise_minimum(as_h2(v[e]), as_h2(v[e + 1])));
            }
        }
        mx = fmaxf(fmaxf((float)hmx.x, (float)hmx.y), fmaxf(-(float)hmn.x, -(float)hmn.y));
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t v[8] = {ra[i].x, ra[i].y, ra[i].z, ra[i].w, rb[i].x, rb[i].y, rb[i].z, rb[i].w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t m = v[e] & 0x7fff7fffu;
                mb = max(mb, max(m & 0xffffu, m >> 16));
            }
        }
        mx = __uint_as_float(mb << 16);
    }
    mx = wave_max(mx);
    int eu = 0;
    if (DT == BF16 || !(mx >= 0.0625f && mx < 16.0f)) eu = exp_of(mx);
    eu = __builtin_amdgcn_readfirstlane(eu);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            const uint4 va = ra[2 * j + hf], vb = rb[2 * j + hf];
            const uint32_t A4[4] = {va.x, va.y, va.z, va.w}, B4[4] = {vb.x, vb.y, vb.z, vb.w};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const int T = 8 * hf + 2 * s;
                if (DT == F16) {
                    d[4 * T + j] = __builtin_amdgcn_perm(B4[s], A4[s], 0x05040100u);
                    d[4 * (T + 1) + j] = __builtin_amdgcn_perm(B4[s], A4[s], 0x07060302u);
                } else {
                    d[4 * T + j] = pk(ldexpf(lo_f<DT>(A4[s]), -eu), ldexpf(lo_f<DT>(B4[s]), -eu));
                    d[4 * (T + 1) + j] = pk(ldexpf(hi_f<DT>(A4[s]), -eu), ldexpf(hi_f<DT>(B4[s]), -eu));
                }
            }
        }
    }
    if (DT == F16 && eu != 0) {
        // in float32: 2^-eu may leave fp16's range
#pragma unroll
        for (int i = 0; i < 64; ++i) d[i] = pk(ldexpf((float)as_h2(d[i]).x, -eu), ldexpf((float)as_h2(d[i]).y, -eu));
    }
    // packing complete here: the raw registers are dead before the transform
#pragma unroll
    for (int i = 0; i < 64; ++i) asm volatile("" : "+v"(d[i]));
    return eu;
}

}  // namespace wv

template <int DT>
__global__ __launch_bounds__(wv::NT) __attribute__((amdgpu_waves_per_eu(3))) void wgrad_wave4096_kernel(
    const uint16_t *u, const uint16_t *dy, int B, int H, int ngroup, float *dk, float *dD) {
    using namespace wv;
    __shared__ uint4 Tab[kTabC];   // the compact table: three workgroups per CU
    // summed spectrum, planar (re, im), index (tau * 4 + jj) * 64 + lane (lanes
    // on consecutive banks); then the dk staging buffer
    __shared__ float S[2 * kN];
    uint4 *Ytab = Tab, *Lc = Tab + kTabY;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, c = lane & 15;
    const int h = blockIdx.x / ngroup, grp = blockIdx.x % ngroup;
    const int npairs = (B + 1) / 2;
    const int qq = NW * grp + w;   // this wave's row pair (at most one)
    const bool have = qq < npairs;
#pragma unroll
    for (int r = 0; r < (kTabC + NT - 1) / NT; ++r) {
        const int base = r * NT + 64 * w;
        if (base < kTabC)
            __builtin_amdgcn_global_load_lds((gvoid_t *)((const uint4 *)kHalfC.v + base + lane),
                                             (lvoid_t *)(Tab + base), 16, 0, 0);
    }
    uint4 ra[8], rb[8];
    uint32_t d[64], zu[64];
    uint32_t *zs = (uint32_t *)S + w * (2 * kN / NW);   // this wave's quarter of S
    const long oa = ((long)(2 * qq) * H + h) * L;
    const long ob = (2 * qq + 1 < B) ? oa + (long)H * L : -1;
    if (have) load_pair_raw(u, oa, ob, g, c, ra, rb);
    __builtin_amdgcn_s_waitcnt(kWaitVm0);
    __syncthreads();   // tables
    int ep = 0;
    if (have) {
        const int eu = pack_pair<DT>(ra, rb, d);
        forward_front<true>(d, Lc, Ytab, lane);
        layer<false>(d, lc_dft<true>(Lc, lane, false), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) zu[4 * tau + jj] = pk(re[jj], im[jj]);
        });
        // the upper half of u's spectrum waits in this wave's quarter of S
        // (free until the products are summed), the lower half in registers
#pragma unroll
        for (int i = 32; i < 64; ++i) zs[(i - 32) * 64 + lane] = zu[i];
        // dy's loads after the u transform (the empty asm pins the kept zu
        // values before them): raw, transform and spectrum registers are
        // never live at once (three waves per SIMD)
#pragma unroll
        for (int i = 0; i < 32; ++i) asm volatile("" : "+v"(zu[i])::"memory");
        load_pair_raw(dy, oa, ob, g, c, ra, rb);
        const int eg = pack_pair<DT>(ra, rb, d);
        forward_front<true>(d, Lc, Ytab, lane);
        // conj(Zu) . Zdy in float32 from the matrix-core outputs, packed back
        // into zu at 2^-7 (both transforms are below 1448 in modulus, so the
        // product stays below 2^14)
        layer<false>(d, lc_dft<true>(Lc, lane, false), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int i = 4 * tau + jj;
                const h2_t a = as_h2(i < 32 ? zu[i] : zs[(i - 32) * 64 + lane]);
                const float ar = (float)a.x, ai = (float)a.y;
                zu[4 * tau + jj] = pk((ar * re[jj] + ai * im[jj]) * 0.0078125f, (ar * im[jj] - ai * re[jj]) * 0.0078125f);
            }
        });
        ep = eu + eg + 7;
    }
    __syncthreads();   // every wave has read its quarter of S back
    // the waves add their products into S in turn (wave 0 stores), scaled
    // back by 2^ep: S = sum conj(F z_u) F z_dy / 4096
    const float sc = ldexpf(1.0f, ep);
#pragma unroll 1
    for (int turn = 0; turn < NW; ++turn) {
        if (w == turn && (have || turn == 0)) {
#pragma unroll
            for (int i = 0; i < 64; ++i) {
                const int si = i * 64 + lane;   // i = 4 tau + jj
                const h2_t p = as_h2(zu[i]);
                const float pr = have ? (float)p.x * sc : 0.f, pi = have ? (float)p.y * sc : 0.f;
                if (turn == 0) {
                    S[si] = pr;
                    S[kN + si] = pi;
                } else {
                    S[si] += pr;
                    S[kN + si] += pi;
                }
            }
        }
        __syncthreads();
    }
    if (w != 0) return;   // no barrier below: wave 0 alone runs the inverse

    float mx = 0.f;
#pragma unroll
    for (int i = 0; i < 64; ++i) mx = fmaxf(mx, fmaxf(fabsf(S[i * 64 + lane]), fabsf(S[kN + i * 64 + lane])));
    mx = wave_max(mx);
    const int es = __builtin_amdgcn_readfirstlane(exp_of(mx));
#pragma unroll
    for (int tau = 0; tau < 16; ++tau)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int si = (4 * tau + jj) * 64 + lane;
            d[4 * tau + jj] = pk(ldexpf(S[si], -es), ldexpf(S[kN + si], -es));
        }
    // the inverse of the convolution
    layer<false>(d, lc_dft<true>(Lc, lane, true), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = pk(re[jj], im[jj]);
    });
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
        const uint4 X = Lc[LcKind<true>::X * 64 + lane], Xs = Lc[LcKind<true>::XS * 64 + lane];
        const uint32_t xw[4] = {X.x, X.y, X.z, X.w}, xs[4] = {Xs.x, Xs.y, Xs.z, Xs.w};
        layer<true>(d, lc_dft<true>(Lc, lane, true), NoPre{}, [&](int tau, f4_t re, f4_t im, uint4) {
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) d[4 * tau + jj] = cmulc2(pk(re[jj], im[jj]), xw[jj], xs[jj]);
        });
    }
    // L1^H: lane (g < 2, c), tile tau, element i holds t = 256 (4 g + i) + 16 c + tau;
    // the real part is dk.  Staged through LDS (S is free) for coalesced stores.
    float *stage = S;
    const float osc = ldexpf(1.0f, es + 6);
    layer<false>(d, lc_dft<true>(Lc, lane, true), NoPre{}, [&](int tau, f4_t re, f4_t, uint4) {
        if (g < 2) {
#pragma unroll
            for (int i = 0; i < 4; ++i) stage[256 * (4 * g + i) + 16 * c + tau] = re[i] * osc;
        }
    });
    // other lanes' staging writes visible before the reads (one wave: no barrier)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    // group grp's share: rows grp H + h of dk and dD (ngroup = 1: the outputs)
    float *dkh = dk + ((long)grp * H + h) * L;
#pragma unroll
    for (int r = 0; r < L / 256; ++r) {
        const int t = 256 * r + 4 * lane;
        if (dk) *(float4 *)(dkh + t) = *(const float4 *)(stage + t);
    }
    if (lane == 0 && dD) dD[(long)grp * H + h] = stage[0];
}

bool fftconv_wave_supported(int L, int dtype) { return L == wv::L && (dtype == F16 || dtype == BF16); }

// partial sums of the workgroup groups of a channel
__global__ __launch_bounds__(256) void wgrad_reduce_kernel(const float *pk_, const float *pd, int ngroup, int H,
                                                           float *dk, float *dD) {
    const long n = (long)H * wv::L / 4;
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (dk && i < n) {
        float4 acc = ((const float4 *)pk_)[i];
        for (int gi = 1; gi < ngroup; ++gi) {
            const float4 v = ((const float4 *)pk_)[(long)gi * n + i];
            acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
        }
        ((float4 *)dk)[i] = acc;
    }
    if (dD && i < H) {
        float a = 0.f;
        for (int gi = 0; gi < ngroup; ++gi) a += pd[(long)gi * H + i];
        dD[i] = a;
    }
}

int wgrad_wave_groups(int B) { return ((B + 1) / 2 + wv::NW - 1) / wv::NW; }

size_t wgrad_wave_workspace(int B, int H) {
    const int ng = wgrad_wave_groups(B);
    if (ng <= 1) return 0;
    return (size_t)ng * H * wv::L * sizeof(float) + (size_t)ng * H * sizeof(float);
}

hipError_t launch_wgrad_wave(const void *u, const void *dy, int B, int H, int dtype, float *dk, float *dD,
                             void *ws, hipStream_t s) {
    if (dtype != F16 && dtype != BF16) return hipErrorInvalidValue;
    const int ng = wgrad_wave_groups(B);
    float *pk_ = dk, *pd = dD;
    if (ng > 1) {   // partial sums per group in the workspace, then one reduction
        if (!ws) return hipErrorInvalidValue;
        pk_ = dk ? (float *)ws : nullptr;
        pd = dD ? (float *)ws + (size_t)ng * H * wv::L : nullptr;
    }
    const dim3 grid(H * ng), block(wv::NT);
    if (dtype == F16)
        hipLaunchKernelGGL(wgrad_wave4096_kernel<F16>, grid, block, 0, s, (const uint16_t *)u, (const uint16_t *)dy,
                           B, H, ng, pk_, pd);
    else
        hipLaunchKernelGGL(wgrad_wave4096_kernel<BF16>, grid, block, 0, s, (const uint16_t *)u, (const uint16_t *)dy,
                           B, H, ng, pk_, pd);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || ng == 1) return e;
    const long n = (long)H * wv::L / 4;
    hipLaunchKernelGGL(wgrad_reduce_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, pk_, pd, ng, H, dk,
                       dD);
    return hipGetLastError();
}

hipError_t launch_fftconv_wave(const ConvArgs &a, const float *k, hipStream_t s) {
    if (!fftconv_wave_supported(a.L, a.dtype)) return hipErrorInvalidValue;
    int pairs_per_ch;
    if (a.pair_mode == 0)
        pairs_per_ch = (a.B + 1) / 2;
    else
        pairs_per_ch = a.B * ((a.nchunk + 1) / 2);
    // split a channel over several workgroups only while the chip would hold
    // fewer than ~2 waves per SIMD and each wave still gets a pair
    int wg_per_ch = 1;
    while ((long)a.H * wg_per_ch * wv::NW < 2048 && pairs_per_ch >= 2 * wv::NW * wg_per_ch) wg_per_ch *= 2;
    dim3 grid(a.H * wg_per_ch), block(wv::NT);
    const int corr = a.corr == nullptr ? 0 : (a.corr16 ? 2 : 1);
    if (corr == 0 && a.pair_mode == 0 && pairs_per_ch <= 2 && wg_per_ch == 1 && a.H >= 2) {
        // two channels per workgroup: every wave has a row pair.  From two
        // workgroups per CU on (512 and more) the instance with the compact
        // table runs three per CU (B = 4: 51 -> 48 us at H = 2560, 337 -> 300
        // us at H = 20480); below that its extra instructions only cost (19
        // -> 20 us at H = 768)
        const dim3 grid2((a.H + 1) / 2);
        const bool ct = grid2.x >= 512;
#define H3_WAVE2_LAUNCH(DTV, CTV, GV) \
    hipLaunchKernelGGL((fftconv_wave4096_kernel<DTV, 0, 2, CTV, GV>), grid2, block, 0, s, a, k, 1, pairs_per_ch)
#define H3_WAVE2_CT(DTV, GV) \
    do {                                   \
        if (ct) H3_WAVE2_LAUNCH(DTV, true, GV); \
        else H3_WAVE2_LAUNCH(DTV, false, GV);   \
    } while (0)
        if (a.dtype == F16) {
            if (a.gate) H3_WAVE2_CT(F16, true);
            else H3_WAVE2_CT(F16, false);
        } else {
            if (a.gate) H3_WAVE2_CT(BF16, true);
            else H3_WAVE2_CT(BF16, false);
        }
#undef H3_WAVE2_CT
#undef H3_WAVE2_LAUNCH
        return hipGetLastError();
    }
#define H3_WAVE_LAUNCH(DTV, CV) \
    hipLaunchKernelGGL((fftconv_wave4096_kernel<DTV, CV, 1>), grid, block, 0, s, a, k, wg_per_ch, pairs_per_ch)
    if (a.gate) {
        if (corr != 0 || a.pair_mode != 0) return hipErrorInvalidValue;
        if (a.dtype == F16)
            hipLaunchKernelGGL((fftconv_wave4096_kernel<F16, 0, 1, false, true>), grid, block, 0, s, a, k, wg_per_ch,
                               pairs_per_ch);
        else
            hipLaunchKernelGGL((fftconv_wave4096_kernel<BF16, 0, 1, false, true>), grid, block, 0, s, a, k, wg_per_ch,
                               pairs_per_ch);
        return hipGetLastError();
    }
    if (a.dtype == F16) {
        if (corr == 0) H3_WAVE_LAUNCH(F16, 0);
        else if (corr == 1) H3_WAVE_LAUNCH(F16, 1);
        else H3_WAVE_LAUNCH(F16, 2);
    } else {
        if (corr == 0) H3_WAVE_LAUNCH(BF16, 0);
        else if (corr == 1) H3_WAVE_LAUNCH(BF16, 1);
        else H3_WAVE_LAUNCH(BF16, 2);
    }
#undef H3_WAVE_LAUNCH
    return hipGetLastError();
}

}  // namespace h3
