// Pieces shared by the matrix-core forward kernels: kernel arguments, the LDS
// tile set, staging of one chunk (global -> registers -> LDS), the chunk-local
// prefix sums and the temporal write matrix.  NTH is the workgroup size.
#pragma once

#include "cyfa_mfma_common.h"
#include "cyfa_mixer.h"

namespace cyfa {

struct MfmaArgs {
    FwdParams p;
    int P;               // segments per (b, h)
    int cps;             // chunks per segment
    int nchunks;         // chunks per sequence
    int chunk;           // chunk length (32 or 64)
    const __bf16 *Mz;    // [H][128][128]  row = slot i', column = internal basis j; times scale log2(e)
    __bf16 *seg_state;   // [B*H*P][2*128*128] accumulator-dump layout, bf16: segment
                         // contributions, then the states entering each segment
    float *fin_state;    // [B*H][2*128*128] same layout, fp32: state after the last segment
    double *seg_span;    // [B*H*P] clock span of each segment (reduced mod m)
    double *seg_gsum;    // [B*H*P] sum of log alpha over each segment
    double *seg_origin;  // [B*H*P] absolute clock at each segment start (reduced)
    double *final_lam;   // [B*H] local clock after the last segment (reduced)
    int has_init;        // segment-entry states are read from seg_state
    int zero_init;       // no initial state: the first segment starts from zero (its entry
                         // state is neither written by the scan nor read)
    int want_final;      // last segment dumps its final state into fin_state
    int hv;              // 128-channel column blocks per head (1: d = 128, 2: d = 256).  The
                         // pre-pass, the segment scan and the final-state conversion treat
                         // each block as a head of its own (a "virtual head", index
                         // hv h + block): the states of a 256-channel head are two 128 x 128
                         // pairs, and the per-token scalars are shared by its blocks.
    MixIn mix;           // fused layer forward only: the mixer's weights and gate inputs (p.q,
                         // p.k, p.v are then the raw projections and p.o the layer output)
};


namespace mfma {

typedef _Float16 half2v __attribute__((ext_vector_type(2)));
typedef _Float16 half8v __attribute__((ext_vector_type(8)));

struct Tiles {
    __bf16 *Qs, *Ks, *Vs, *As, *Ads, *Ss, *Xs, *Ws, *Os, *Stage, *Mt;
    float2 *red;
    half2v *CS;
    float *Gs;      // chunk-local prefix sums of log alpha
    float *gam;     // row scale of the inter-chunk terms: exp(G_r + L)
    float *betas;
    float *decw;    // multiplier of A_dec rows
    float *urev;    // clock at each row reduced mod m, divided by m (revolutions, in [0, 1))
    float *ctl;     // [0]: factor applied to the carried states this chunk, [1]: log scale L after it,
                    // [2]: 1 when the chunk's decay factors into a row scale (A_dec tile), else 0
    float4 *bw;     // per row, for the temporal-write builder: amplitude beta sqrt(2/m) times the
                    // row's decay factor (when its tile holds A_dec), urev, cos and sin of 2 pi urev
};

// n entries per array (the chunk length or 64); block size scalar_bytes(n)
__device__ __forceinline__ void scalars_at(Tiles &t, char *base, int n = 64) {
    t.Gs = reinterpret_cast<float *>(base);
    t.gam = t.Gs + n;
    t.betas = t.gam + n;
    t.decw = t.betas + n;
    t.urev = t.decw + n;
    t.ctl = reinterpret_cast<float *>(t.urev + n);
    t.bw = reinterpret_cast<float4 *>(t.ctl + 4);      // 16-byte aligned for n a multiple of 4
}
__host__ __device__ constexpr int scalar_bytes(int n) { return n * (4 + 4 + 4 + 4 + 4 + 16) + 16; }

// Segment-boundary states travel in bf16 (the precision in which the chunk
// products consume them); the carried states themselves accumulate in fp32.
// Lane-major dump layout, one (virtual) head's pair per kStateFloats block: two
// 16-byte loads per accumulator.
__device__ __forceinline__ void load_state(const __bf16 *st, int w, int lane, f32x16 (&kacc)[4],
                                           f32x16 (&vacc)[4]) {
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        const bf16x8 k0 = *reinterpret_cast<const bf16x8 *>(st + dump_off(w, x, lane, 0));
        const bf16x8 k1 = *reinterpret_cast<const bf16x8 *>(st + dump_off(w, x, lane, 8));
        const bf16x8 v0 = *reinterpret_cast<const bf16x8 *>(st + 128 * 128 + dump_off(w, x, lane, 0));
        const bf16x8 v1 = *reinterpret_cast<const bf16x8 *>(st + 128 * 128 + dump_off(w, x, lane, 8));
#pragma unroll
        for (int v = 0; v < 8; ++v) {
            kacc[x][v] = (float)k0[v];
            kacc[x][v + 8] = (float)k1[v];
            vacc[x][v] = (float)v0[v];
            vacc[x][v + 8] = (float)v1[v];
        }
    }
}

// fp32 dump (the final state), four 16-byte stores per accumulator
__device__ __forceinline__ void dump_state(float *st, int w, int lane, const f32x16 (&kacc)[4],
                                           const f32x16 (&vacc)[4]) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            *reinterpret_cast<float4 *>(st + dump_off(w, x, lane, 4 * q)) =
                make_float4(kacc[x][4 * q], kacc[x][4 * q + 1], kacc[x][4 * q + 2], kacc[x][4 * q + 3]);
            *reinterpret_cast<float4 *>(st + 128 * 128 + dump_off(w, x, lane, 4 * q)) =
                make_float4(vacc[x][4 * q], vacc[x][4 * q + 1], vacc[x][4 * q + 2], vacc[x][4 * q + 3]);
        }
}

// Global -> register prefetch of one chunk: CC NTH/16 x 16-byte pieces per thread
// per tensor (rows (NTH/16) it + tid / 16, columns 8 (tid % 16)), plus one
// token's scalars on the first CC lanes.
template <int CC, int NTH = NT>
struct Prefetch {
    static constexpr int kIt = CC * 16 / NTH;
    uint4 q[kIt], k[kIt], v[kIt];
    float g, dl, be;
};

// Tb: tokens of this sequence (rows at or past it read as zero, scalars as 0).
// kMix: the per-token scalars are the gate activations of the mixer's projections
// (mx), computed as the standalone prologue computes them.
template <int CC, bool kWithQ, int NTH = NT, bool kMix = false>
__device__ __forceinline__ void load_chunk(const FwdParams &p, int b, int h, int t0, int Tb, int tid,
                                           Prefetch<CC, NTH> &pf, const MixIn *mx = nullptr) {
    constexpr int kRows = NTH / 16;                  // rows per pass
    // Uniform chunk base (scalar registers) plus a fixed 32-bit per-lane byte offset:
    // no per-lane 64-bit address arithmetic.  Rows past the sequence read as zero.
    const size_t row_el = (size_t)p.H * D;           // elements between consecutive tokens
    const size_t base = (seq_row0(p, b) + t0) * row_el + (size_t)h * D;
    const char *q = reinterpret_cast<const char *>(static_cast<const __bf16 *>(p.q) + base);
    const char *k = reinterpret_cast<const char *>(static_cast<const __bf16 *>(p.k) + base);
    const char *v = reinterpret_cast<const char *>(static_cast<const __bf16 *>(p.v) + base);
    const int r0 = tid >> 4;
    const unsigned loff = (unsigned)(r0 * (int)row_el + (tid & 15) * 8) * 2u;
    const unsigned pass = (unsigned)(kRows * row_el * 2);
    const uint4 zero = make_uint4(0, 0, 0, 0);
    // (uniform part added first, so that the loads take a scalar base and a 32-bit
    // vector offset)
    auto ld = [&](const char *base_it) { return *reinterpret_cast<const uint4 *>(base_it + loff); };
    if (t0 + CC <= Tb) {                             // whole chunk in range (uniform)
#pragma unroll
        for (int it = 0; it < Prefetch<CC, NTH>::kIt; ++it) {
            if (kWithQ) pf.q[it] = ld(q + it * pass);
            pf.k[it] = ld(k + it * pass);
            pf.v[it] = ld(v + it * pass);
        }
    } else {
#pragma unroll
        for (int it = 0; it < Prefetch<CC, NTH>::kIt; ++it) {
            const bool in = t0 + r0 + kRows * it < Tb;
            if (kWithQ) pf.q[it] = in ? ld(q + it * pass) : zero;
            pf.k[it] = in ? ld(k + it * pass) : zero;
            pf.v[it] = in ? ld(v + it * pass) : zero;
        }
    }
    if (tid < 64) {
        const int t = t0 + tid;
        const size_t sbase = (seq_row0(p, b) + t0) * p.H + h;
        // opaque per chunk: otherwise base + lane offset is kept per lane (64-bit)
        // across the whole chunk loop
        const unsigned soff = (unsigned)opq(tid * p.H);
        if (tid < CC && t < Tb) {
            if constexpr (kMix) {
                pf.dl = mix_sigm((mx->z_delta + sbase)[soff] + (mx->b_delta ? mx->b_delta[h] : 0.f));
                pf.g = mx->z_alpha ? -mx->A[h] * mix_softplus((mx->z_alpha + sbase)[soff] +
                                                              (mx->b_alpha ? mx->b_alpha[h] : 0.f))
                                   : 0.f;
                pf.be = mx->z_beta ? mix_sigm((mx->z_beta + sbase)[soff]) : 1.f;
            } else {
                pf.dl = (p.delta + sbase)[soff];
                pf.g = p.log_alpha ? (p.log_alpha + sbase)[soff] : 0.f;
                pf.be = p.beta ? (p.beta + sbase)[soff] : 1.f;
            }
        } else {
            pf.dl = 0.f;   // rows past the chunk or the sequence: no shift, no decay, no write
            pf.g = 0.f;
            pf.be = 0.f;
        }
    }
}

// Registers -> LDS, row-major tiles (Q padded to stride QS; K and V padded too,
// or swizzled when kSwzKV).  Each group of 16 lanes stores one whole row.
template <int CC, bool kWithQ, int NTH = NT, bool kSwzKV = false>
__device__ __forceinline__ void store_chunk(const Tiles &s, int tid, const Prefetch<CC, NTH> &pf) {
    constexpr int kRows = NTH / 16;
    static_assert(kRows % 4 == 0, "row passes keep the swizzle phase");
    const int off = (tid >> 4) * QS + (tid & 15) * 8;
    const int kvs = kSwzKV ? SWS : QS;
    const int kvo = kSwzKV ? swz_elem(tid >> 4, (tid & 15) * 8) : off;
#pragma unroll
    for (int it = 0; it < Prefetch<CC, NTH>::kIt; ++it) {
        if (kWithQ) *reinterpret_cast<uint4 *>(s.Qs + off + kRows * it * QS) = pf.q[it];
        *reinterpret_cast<uint4 *>(s.Ks + kvo + kRows * it * kvs) = pf.k[it];
        *reinterpret_cast<uint4 *>(s.Vs + kvo + kRows * it * kvs) = pf.v[it];
    }
}

// Wave 0: chunk-local inclusive prefix sums of log alpha (float) and of the
// clock increments (double, continuing the carried clock), reduced mod m.
// Lanes past the chunk hold zeros, so entry 63 equals the chunk total.
//
// Carried states are kept as Kbar = exp(L) Kt (same L for Vbar).  Normally a
// chunk only adds to Kt: Kt += K^T (A exp(-G_r - L)) and L += G_C, which is
// Kbar <- gamma^C Kbar + K^T (A gamma^C / gamma^r) (App. B, Eq. app-scalar-chunk)
// without touching the state registers.  When exp(+-(G_r + L)) could leave
// [e^-60, e^60] the chunk instead rescales Kt by exp(L + G_C), uses
// A gamma^C / gamma^r and restarts L at 0.
// NSC: entries of the scalar arrays (lanes >= NSC hold no token and write nothing)
// kEps: for the kernels whose A tile holds A_dec: gam holds the row scale eps_r
// of a "factored" chunk (below) and ctl[2] says whether the chunk is one.
template <int CC, int NTH = NT, int NSC = 64, bool kEps = false>
__device__ __forceinline__ void chunk_scans(const Tiles &s, int lane, int m, const Prefetch<CC, NTH> &pf,
                                            double &carry, double &gsum, float &L) {
    const double inv_m = 1.0 / (double)m;
    const float G = wave_incl_scan(pf.g);
    const double lam = carry + wave_incl_scan((double)pf.dl);
    const float GC = lane63(G);
    const float gabs = wave_max_nonneg(fabsf(G));
    const bool lazy = fabsf(L) + gabs <= 60.f;
    // Factored chunk: Gamma_rs = eps_r decw_s with both factors within e^+-60, so
    // with A_dec in place of A every intra-chunk term is eps_r (S A_dec).  Lazy:
    // eps_r = exp(G_r + L) = gam_r.  Eager with a chunk range |G_C| <= 60: the
    // states are rescaled by exp(L + G_C) before the inter-chunk products and
    // eps_r = exp(G_r - G_C); that factor must stay a normal fp32 number (the
    // first tokens' inter-chunk terms depend on the rescaled states), hence
    // |L| + |G_C| <= 80.  Otherwise the kernel applies Gamma per score entry and
    // gam_r before the intra products, and rescales the states after them.
    const bool factored = lazy || (gabs <= 60.f && fabsf(L) + gabs <= 80.f);
    if (lane < NSC) {
        const int ol = opq(lane);                   // one address register for the five writes
        s.Gs[ol] = G;
        s.gam[ol] = (kEps && !lazy && factored) ? __expf(G - GC) : __expf(G + L);
        const float dw = lazy ? __expf(-G - L) : __expf(GC - G);
        s.decw[ol] = dw;
        s.betas[ol] = pf.be;
        const double q = lam * inv_m;               // clock in revolutions of the m-slot ring
        const float u = (float)(q - floor(q));
        s.urev[ol] = u;
        // builder record: its tile holds A_dec (pre-pass; fused kernel when factored)
        // or A (fused kernel otherwise)
        float s1, c1;
        sincos_rev(u, &s1, &c1);
        const float amp = pf.be * sqrtf(2.f / (float)m) * ((!kEps || factored) ? dw : 1.f);
        s.bw[ol] = make_float4(amp, u, c1, s1);
    }
    const float state_factor = lazy ? 1.f : __expf(L + GC);
    L = lazy ? L + GC : 0.f;
    if (lane == 0) {
        s.ctl[0] = state_factor;
        s.ctl[1] = L;
        s.ctl[2] = factored ? 1.f : 0.f;
    }
    const double last = lane63(lam);
    carry = reduce_clock(last, (double)m, inv_m);
    gsum += (double)GC;
}

// Temporal write matrix for the chunk (Eq. app-temporal-writes):
// A_r = beta_r U(-lambda_r) b, i.e. beta_r [sqrt(2/m) cos th_j, -sqrt(2/m) sin th_j]
// on pair j and beta_r / sqrt(m) on DC, th_j = 2 pi j lambda_r / m.  The copy
// A_dec has row r scaled by gamma^C / gamma^r (right rescaling, Eq. app-chunk-rescale).
// kA: write A and the (cos, sin) table; kAd: write A_dec.
// Thread (r = tid / TPR, q = tid % TPR) fills internal columns NCOL q .. NCOL q + NCOL-1
// of row r; the last quarter also holds DC (column 126) and padding (127).  The
// phases advance by angle addition from an accurately reduced start.
template <int CC, bool kA, bool kAd, int NTH = NT>
__device__ __forceinline__ void build_writes(const Tiles &s, int tid, int m) {
    constexpr int TPR = NTH / CC;         // threads per row
    constexpr int NCOL = 128 / TPR;       // columns per thread
    constexpr int NP = NCOL / 2;          // pairs per thread
    static_assert(NP % 4 == 0, "whole 8-column groups per thread");
    const int r = tid / TPR, q = tid % TPR;
    const int J = (m - 1) >> 1;
    const float dc = 1.0f / sqrtf((float)m);
    const float bac = s.betas[r] * sqrtf(2.0f / (float)m);
    const float wdec = s.decw[r];
    const double u = s.urev[r];                      // revolutions per unit frequency (float:
                                                     // the phases it starts are far finer
                                                     // than A's bf16 rounding)
    float s1, c1, sn, cs;
    sincos_rev((float)u, &s1, &c1);
    {
        double rev = (double)(NP * q + 1) * u;
        rev -= floor(rev);
        sincos_rev((float)rev, &sn, &cs);
    }
    // Emitted 4 pairs (8 columns) at a time: few values live at once.
#pragma unroll
    for (int k8 = 0; k8 < NP / 4; ++k8) {
        bf16x8 a8, ad8;
        half8v cs8;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int j = NP * q + 1 + 4 * k8 + jj;
            const bool live = j <= J && j <= 63;
            const float cv = live ? cs : 0.f;
            const float sv = live ? sn : 0.f;
            float a0 = bac * cv, a1 = -bac * sv;
            if (q == TPR - 1 && k8 == NP / 4 - 1 && jj == 3) {
                a0 = s.betas[r] * dc;            // internal column 126: DC
                a1 = 0.f;                        // 127: padding
            }
            a8[2 * jj] = (__bf16)a0;
            a8[2 * jj + 1] = (__bf16)a1;
            ad8[2 * jj] = (__bf16)(a0 * wdec);
            ad8[2 * jj + 1] = (__bf16)(a1 * wdec);
            // table entry 63 (internal columns 126, 127: DC and padding) is (1, 0),
            // so the token-wise rotations pass those columns through unchanged
            cs8[2 * jj] = (_Float16)(j == 64 ? 1.f : cv);
            cs8[2 * jj + 1] = (_Float16)sv;
            const float nc = cs * c1 - sn * s1;
            const float ns = sn * c1 + cs * s1;
            cs = nc;
            sn = ns;
        }
        if (kA) {
            *reinterpret_cast<bf16x8 *>(s.As + r * QS + NCOL * q + 8 * k8) = a8;
            *reinterpret_cast<half8v *>(s.CS + r * 64 + NP * q + 4 * k8) = cs8;
        }
        if (kAd) *reinterpret_cast<bf16x8 *>(s.Ads + r * QS + NCOL * q + 8 * k8) = ad8;
    }
}

// The temporal write matrix stored into a swizzled tile (A or A_dec, as the
// chunk scans decided: row r is amp_r [cos th_j, -sin th_j] on pair j and
// amp_r / sqrt(2) on DC, amp_r = beta_r sqrt(2/m) times the row's decay factor
// when the tile holds A_dec), 16 threads per row so that each group of 16 lanes
// stores one whole row, and (kTab) a (cos, sin) table of row stride CSW half2
// words.  Thread (r, q) fills internal columns 8q .. 8q+7 (pairs 4q+1 .. 4q+4)
// of rows r = tid / 16 + (NTH / 16) it; q = 15 also holds DC (column 126) and the
// padding (127).  One 16-byte read gives a row's amplitude, clock phase u and
// unit step (cos, sin)(2 pi u); the start phase (4q+1) u mod 1 is taken in fp32:
// u < 1 and 4q+1 <= 61 keep its error below 4e-6 revolutions, far under the bf16
// and f16 rounding of the tile and the table.
template <int CC, bool kTab, int NTH, int CSW>
__device__ __forceinline__ void build_writes_swz(const Tiles &s, __bf16 *tile, int tid, int m) {
    constexpr int RPP = NTH / 16;                    // rows per pass
    static_assert(CC % RPP == 0 && RPP % 4 == 0, "whole passes with a fixed swizzle phase");
    const int q = tid & 15, r0 = tid >> 4;
    const int J = (m - 1) >> 1;
    const int pc = swz_elem(r0, 8 * q) - r0 * SWS;   // stored column of this thread's chunk
    // rows one after another: interleaving them raises the register peak of the
    // fused kernel, which holds the carried states and the prefetched chunk here
#pragma unroll 1
    for (int it = 0; it < CC / RPP; ++it) {
        const int r = r0 + RPP * it;
        const float4 rec = s.bw[r];
        const float amp = rec.x, u = rec.y, c1 = rec.z, s1 = rec.w;
        float sn, cs;
        sincos_rev(__builtin_amdgcn_fractf((float)(4 * q + 1) * u), &sn, &cs);
        bf16x8 a8;
        half8v cs8;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int j = 4 * q + 1 + jj;
            const bool live = j <= J && j <= 63;
            const float cv = live ? cs : 0.f;
            const float sv = live ? sn : 0.f;
            float a0 = amp * cv, a1 = -amp * sv;
            if (jj == 3 && q == 15) {
                a0 = amp * 0.70710678118654752f;     // internal column 126: DC
                a1 = 0.f;                            // 127: padding
            }
            a8[2 * jj] = (__bf16)a0;
            a8[2 * jj + 1] = (__bf16)a1;
            // table entry 63 (DC and padding) is (1, 0): the token-wise rotations
            // pass those columns through unchanged
            cs8[2 * jj] = (_Float16)(j == 64 ? 1.f : cv);
            cs8[2 * jj + 1] = (_Float16)sv;
            if (jj < 3) {
                const float nc = cs * c1 - sn * s1;
                const float ns = sn * c1 + cs * s1;
                cs = nc;
                sn = ns;
            }
        }
        *reinterpret_cast<bf16x8 *>(tile + r * SWS + pc) = a8;
        if (kTab) *reinterpret_cast<half8v *>(s.CS + r * CSW + 4 * q) = cs8;
    }
}

}  // namespace mfma
}  // namespace cyfa
