// Matrix-core (bf16 MFMA) forward for slot counts 127 < m <= 255 (m* = 256 storage
// rows, the largest slot count of the paper's ablation), d_k = d_v = 128, 32-token
// chunks, bf16 inputs with fp32 accumulation.
//
// The computation of the 128-row fused kernel (App. B: clock and log-decay prefix
// sums, temporal writes A (Eq. app-temporal-writes), key pass (Eq.
// app-cyfa-key-chunk), token-wise softmax readout (Eq. cyfa-two-pass, middle line),
// value pass (Eq. app-cyfa-value-chunk)) over the doubled slot space.  Per chunk
// (token rows t, s; gamma_t = exp(G_t), rho_s = exp(G_C - G_s), Gamma_ts = exp(G_t -
// G_s) for s <= t; Kbar, Vbar the states entering the chunk):
//   p = gamma (.) Q Kbar^T + (Q K^T (.) Gamma) A            [32 x 256]
//   X = U(lambda) p (scale folded into M);  W = softmax over the slots of M X
//   u = U(-lambda) M^T W                                      [32 x 256]
//   o = gamma (.) u Vbar + (u A^T (.) Gamma) V                [32 x 128]
//   Kbar <- exp(G_C) Kbar + (rho (.) A)^T K,  Vbar likewise with V.
//
// One eight-wave workgroup (two waves per SIMD, one workgroup per compute unit)
// walks a chunk group of a sequence with both 256 x 128 fp32 states in MFMA
// accumulators (groups > 1 fill the chip when B H is small):
//   Kbar: wave w holds slots i = 32 w + lane % 32 and all 128 channels (four
//     accumulators, the transposed product D[c][i]), so the key pass and its slot
//     logits are formed per wave without reductions;
//   Vbar: wave w holds channel block 32 (w % 4) + lane % 32 of slots 128 (w / 4) ..
//     + 127 (four accumulators D[i][c], one per 32-slot block), so each wave forms
//     the value output of its channel block over half the slots; the upper half's
//     waves hand their partial outputs to the lower half's through LDS.
// The bf16 readout matrix Mz = zs M (zs = scale log2 e) and its transpose are read
// from global memory (L2) as MFMA operands: at 128 KiB each they do not fit in LDS
// beside the chunk tiles.  Tiles are padded rows: [32][128] at 288 bytes, [32][256]
// at 544 bytes (each row 8 banks after the previous one).
//
// Chunk groups: wide_contrib_kernel (b, h, group) forms each group's own contribution
// to the absolute-clock states at its end (zero entering state, App. B's recurrence
// unrolled), its total log decay and the clock entering it (a double-precision sum of
// every earlier increment); the forward's workgroup for group g then starts from
// (K0, V0) decayed through groups 0 .. g-1 plus each earlier contribution decayed
// through the groups after it.  Absolute-clock states need no rotation between
// groups.  The contributions stay fp32 in the workspace, in the accumulators' own
// lane-major layout.
//
// Internal basis order: pair j = 1 .. 127 at (2j-2, 2j-1), DC at 254, padding 255;
// the ABI's state arrays [B][H][256][128] use the paper order (0 = DC, 2j-1, 2j).
#include "cyfa_internal.h"
#include "cyfa_mfma_common.h"
#include "cyfa_rows.h"
#include "cyfa_prep.h"

#include <hip/hip_ext.h>

namespace cyfa {

using namespace mfma;

namespace {

constexpr int kC = 32;              // tokens per chunk
constexpr int kNT = 512;            // eight waves
constexpr int kR = kWideRows;       // 256 storage rows
constexpr int kDCw = kR - 2;        // internal index of DC
constexpr int PS = 144, PSB = 288;  // [32][128] tiles
constexpr int PW = 272, PWB = 544;  // [32][256] tiles
constexpr int SSB = 40;             // [32][32] score tiles

__device__ __forceinline__ int paper_row_w(int i) { return i < kDCw ? i + 1 : (i == kDCw ? 0 : kR - 1); }
__device__ __forceinline__ bool row_active_w(int i, int m) { return i < m - 1 || i == kDCw; }
__device__ __forceinline__ float uniform(float x) {
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}
__device__ __forceinline__ float opqf(float x) {
    asm volatile("" : "+v"(x));
    return x;
}
__device__ __forceinline__ const char *cbyte(const __bf16 *T) { return reinterpret_cast<const char *>(T); }
__device__ __forceinline__ char *cbyte(__bf16 *T) { return reinterpret_cast<char *>(T); }

// Lane offsets (bytes) into the padded tiles.
struct Sw {
    int row, st, tr;        // [32][128]: row operand, 8-byte pieces, transposed operand
    int roww, stw, trw;     // [32][256]: the same
    int cp;                 // 16-byte pieces of whole [32][128] rows: row tid/16, columns 8 (tid%16)
};
__device__ __forceinline__ Sw make_sw(int tid) {
    const int lane = tid & 63, l32 = lane & 31, hl = lane >> 5;
    Sw z;
    z.row = l32 * PSB + 16 * hl;
    z.st = l32 * PSB + 8 * hl;
    z.tr = 2 * tr_off(PS, lane);
    z.roww = l32 * PWB + 16 * hl;
    z.stw = l32 * PWB + 8 * hl;
    z.trw = 2 * tr_off(PW, lane);
    z.cp = (tid >> 4) * PSB + (tid & 15) * 16;
    return z;
}
// Row operand of a [32][256] tile: element [lane%32][16 ks + 8 (lane/32) + p].
__device__ __forceinline__ bf16x8 srow_w(const __bf16 *T, int ks, const Sw &z) {
    return *reinterpret_cast<const bf16x8 *>(cbyte(T) + z.roww + 32 * ks);
}
// Row operand in the permuted k order of a fed-back accumulator (columns 16 ks +
// 4 (lane/32) .. +3 and 16 ks + 8 + 4 (lane/32) .. +3 of row lane%32).
__device__ __forceinline__ bf16x8 perm8(const char *p) {
    const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(p);
    const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(p + 16);
    bf16x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
}
__device__ __forceinline__ bf16x8 sperm(const __bf16 *T, int ks, const Sw &z) { return perm8(cbyte(T) + z.st + 32 * ks); }
__device__ __forceinline__ bf16x8 sperm_w(const __bf16 *T, int ks, const Sw &z) {
    return perm8(cbyte(T) + z.stw + 32 * ks);
}
// Transposed operands: element [k0 + 8 (lane/32) + p][n0 + lane % 32].
__device__ __forceinline__ bf16x8 stro(const __bf16 *T, int k0, int n0, const Sw &z) {
    return lds8_tr(reinterpret_cast<const __bf16 *>(cbyte(T) + z.tr) + k0 * PS + n0, PS);
}
__device__ __forceinline__ bf16x8 stro_w(const __bf16 *T, int k0, int n0, const Sw &z) {
    return lds8_tr(reinterpret_cast<const __bf16 *>(cbyte(T) + z.trw) + k0 * PW + n0, PW);
}
// A 32 x 32 output block D[mr][n] (lane: n = lane % 32; register v: mr = 8 (v / 4) +
// 4 (lane / 32) + v % 4) stored as bf16 at row n, columns col0 + mr.
__device__ __forceinline__ void store_block(__bf16 *T, int col0, const f32x16 &acc, const Sw &z) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (__bf16)acc[4 * g4 + e];
        *reinterpret_cast<bf16x4 *>(cbyte(T) + z.st + 2 * (col0 + 8 * g4)) = o;
    }
}
__device__ __forceinline__ void store_block_w(__bf16 *T, int col0, const f32x16 &acc, const Sw &z) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (__bf16)acc[4 * g4 + e];
        *reinterpret_cast<bf16x4 *>(cbyte(T) + z.stw + 2 * (col0 + 8 * g4)) = o;
    }
}
// Row operand of a score tile: element [row][k0 + 8 (lane/32) + p].
__device__ __forceinline__ bf16x8 rd_row(const __bf16 *S, int row, int k0, int hl) {
    return lds8(S + row * SSB + k0 + 8 * hl);
}
// The operand's k indices k0 + 8 (lane/32) + p scaled by f[p].
__device__ __forceinline__ bf16x8 scale_k(bf16x8 v, const float *f) {
    const float4 a = *reinterpret_cast<const float4 *>(f);
    const float4 b = *reinterpret_cast<const float4 *>(f + 4);
    const float d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    bf16x8 r;
#pragma unroll
    for (int q = 0; q < 8; ++q) r[q] = (__bf16)((float)v[q] * d[q]);
    return r;
}
// Row operand of a [256][256] bf16 matrix in global memory (L2): element [r0 +
// lane%32][16 ks + 8 (lane/32) + p].
__device__ __forceinline__ bf16x8 grow(const __bf16 *Mg, int ks) {
    return *reinterpret_cast<const bf16x8 *>(Mg + 16 * ks);
}
template <int N>
__device__ __forceinline__ void scale_acc(f32x16 (&acc)[N], float f) {
#pragma unroll
    for (int x = 0; x < N; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[x][v] *= f;
}

// ---- chunk staging (one 16-byte piece of each [32][128] tile per thread) ------
// (The lane's offsets are recomputed at every call, opaque to the compiler: kept live
// across the chunk loop as 64-bit addresses they would be spilled, and every reload
// would wait for all of the wave's outstanding loads.)
__device__ __forceinline__ void load_row1(const __bf16 *base, size_t row_stride, int n, int tid, uint4 &o) {
    tid = opq(tid);
    const int r = tid >> 4, c8 = (tid & 15) * 8;
    const uint4 v = *reinterpret_cast<const uint4 *>(base + (size_t)min(r, max(n - 1, 0)) * row_stride + c8);
    o = r < n ? v : make_uint4(0, 0, 0, 0);
}
__device__ __forceinline__ void store_row1(__bf16 *T, const uint4 &o, const Sw &z) {
    *reinterpret_cast<uint4 *>(cbyte(T) + z.cp) = o;
}
__device__ __forceinline__ void copy_row1_out(const __bf16 *T, __bf16 *dst, size_t row_stride, int nrows, int tid,
                                              const Sw &z) {
    const int r = tid >> 4, c8 = (tid & 15) * 8;
    if (r < nrows)
        *reinterpret_cast<uint4 *>(dst + (size_t)r * row_stride + c8) =
            *reinterpret_cast<const uint4 *>(cbyte(T) + z.cp);
}

// Per-token scalars of a chunk (lanes 0..31 of wave 0; zero past the sequence: no
// shift, no decay, no write).
struct Tok {
    float g, dl, be;
};
__device__ __forceinline__ void load_tok(const FwdParams &p, size_t row0, int h, int t0, int Tb, int tid, Tok &k) {
    k.g = 0.f;
    k.dl = 0.f;
    k.be = 0.f;
    const int t = t0 + tid;
    if (tid < kC && t < Tb) {
        const size_t si = (row0 + t) * p.H + h;
        k.g = p.log_alpha ? p.log_alpha[si] : 0.f;
        k.dl = p.delta[si];
        k.be = p.beta ? p.beta[si] : 1.f;
    }
}

// Chunk scalars in LDS.
struct Sc {
    float G[kC];      // chunk-local inclusive sums of log alpha
    float gam[kC];    // exp(G_t) (times the carried states' scale)
    float rho[kC];    // exp(G_C - G_s) (likewise)
    float urev[kC];   // clock after token t over m, mod 1 (revolutions)
    float4 bw[kC];    // write-builder record: amplitude, urev, cos and sin of 2 pi urev
    float ea[kC];     // exp(G_t) and exp(-G_t): Gamma_ts = ea_t eb_s when every |G_t| <= 60
    float eb[kC];
    float ctl[4];     // [0] factor on the carried states before the chunk, [1] before their
                      // update, [2] 1 while lazily scaled, [3] 1 when Gamma factors into ea, eb
};

// Wave 0: prefix sums of the chunk and the builder records; carry is the clock
// entering the chunk (reduced), advanced past it.  The carried states are held as
// exp(Ls) times the registers: a chunk's decay moves Ls (gam_t = exp(G_t + Ls) scales
// the inter-chunk terms, rho_s = exp(-Ls - G_s) the update operand, then Ls += G_C)
// instead of rescaling every accumulator; when an exponent could leave [-60, 60] the
// chunk is eager (registers times exp(Ls) first, Ls restarts at 0, plain gam and rho,
// registers times exp(G_C) before the update).
__device__ __forceinline__ void chunk_scalars(Sc &s, int lane, int m, const Tok &k, double &carry, float Ls) {
    lane = opq(lane);                               // per-lane LDS offsets recomputed, not spilled
    const double inv_m = 1.0 / (double)m;
    const float G = wave_incl_scan(k.g);
    const double lam = carry + wave_incl_scan((double)k.dl);
    const float GC = lane63(G);
    const float gabs = wave_max_nonneg(fabsf(G));
    const bool lazy = fabsf(Ls) + gabs <= 60.f;
    if (lane < kC) {
        s.G[lane] = G;
        s.ea[lane] = __expf(G);
        s.eb[lane] = __expf(-G);
        s.gam[lane] = lazy ? __expf(G + Ls) : __expf(G);
        s.rho[lane] = lazy ? __expf(-Ls - G) : __expf(GC - G);
        const double q = lam * inv_m;
        const float u = (float)(q - floor(q));
        s.urev[lane] = u;
        float s1, c1;
        sincos_rev(u, &s1, &c1);
        s.bw[lane] = make_float4(k.be * sqrtf(2.f / (float)m), u, c1, s1);
    }
    if (lane == 0) {
        s.ctl[0] = lazy ? 1.f : __expf(Ls);
        s.ctl[1] = lazy ? 1.f : __expf(GC);
        s.ctl[2] = lazy ? 1.f : 0.f;
        s.ctl[3] = gabs <= 60.f ? 1.f : 0.f;
    }
    carry = reduce_clock(lane63(lam), (double)m, inv_m);
}
__device__ __forceinline__ float next_scale(const Sc &s, float Ls) {
    return s.ctl[2] != 0.f ? Ls + s.G[kC - 1] : 0.f;
}

// Temporal write rows (Eq. app-temporal-writes) into a [32][256] tile: amp_t [cos
// th_j, -sin th_j] on pair j (internal columns 2j-2, 2j-1), amp_t / sqrt 2 = beta_t /
// sqrt m on DC (254), 0 on 255.  Thread (row tid/32 + 16 it, q = tid % 32) fills
// columns 8q .. 8q+7 (pairs 4q+1 .. 4q+4); the phases advance by angle addition
// from a start reduced in revolutions.
__device__ __forceinline__ void build_A(const Sc &s, __bf16 *T, int tid, int m) {
    const int q = tid & 31, r0 = tid >> 5;
    const int J = (m - 1) >> 1;
#pragma unroll 1
    for (int it = 0; it < 2; ++it) {
        const int r = r0 + 16 * it;
        const float4 rec = s.bw[r];
        const float amp = rec.x, u = rec.y, c1 = rec.z, s1 = rec.w;
        float sn, cs;
        sincos_rev(__builtin_amdgcn_fractf((float)(4 * q + 1) * u), &sn, &cs);
        bf16x8 a8;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const int j = 4 * q + 1 + jj;
            const bool live = j <= J;
            float a0 = live ? amp * cs : 0.f, a1 = live ? -amp * sn : 0.f;
            if (jj == 3 && q == 31) {
                a0 = amp * 0.70710678118654752f;
                a1 = 0.f;
            }
            a8[2 * jj] = (__bf16)a0;
            a8[2 * jj + 1] = (__bf16)a1;
            if (jj < 3) {
                const float nc = cs * c1 - sn * s1;
                const float ns = sn * c1 + cs * s1;
                cs = nc;
                sn = ns;
            }
        }
        *reinterpret_cast<bf16x8 *>(cbyte(T) + r * PWB + 16 * q) = a8;
    }
}

// (cos, sin) of 2 pi j urev for the eight pairs of a lane's 16 slots in wave w's
// 32-slot block: pair e (registers 2e, 2e+1) has frequency j = 16w + 4(e/2) + 2hl +
// e%2 + 1.  Inactive pairs, DC and padding get (1, 0).
__device__ __forceinline__ void lane_phases(float u, int w, int hl, int m, float (&c)[8], float (&s)[8]) {
    const int J = (m - 1) >> 1;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int j = 16 * w + 4 * (e >> 1) + 2 * hl + (e & 1) + 1;
        c[e] = 1.f;
        s[e] = 0.f;
        if (j <= J) sincos_rev(__builtin_amdgcn_fractf((float)j * u), &s[e], &c[e]);
    }
}
// acc <- mul U(SIGN lambda) acc on a lane's pairs; DC and padding are multiplied by mul.
template <int SIGN>
__device__ __forceinline__ void rotate(f32x16 &a, const float (&c)[8], const float (&s)[8], float mul) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const float x0 = a[2 * e], x1 = a[2 * e + 1];
        const float sn = SIGN > 0 ? s[e] : -s[e];
        a[2 * e] = mul * (c[e] * x0 - sn * x1);
        a[2 * e + 1] = mul * (sn * x0 + c[e] * x1);
    }
}

// One 16 x 16 block of a causal 32 x 32 score tile into S (bf16, [32][SSB]):
// S[nr][mr] = Gamma_{nr, mr} sum_k Am[mr][k] Bn[nr][k] for mr in m0 .., nr in n0 ..
// (mr <= nr), over KS k-steps of 32 columns of tiles with row stride STR
// (v_mfma_f32_16x16x32: lane nr = n0 + lane % 16, registers mr = m0 + 4 (lane / 16) + q).
template <int KS, int STR>
__device__ __forceinline__ void score_block(const __bf16 *Am, int m0, const __bf16 *Bn, int n0, __bf16 *S,
                                            const Sc &sc, int lane) {
    const int l16 = lane & 15, g = lane >> 4;
    const int nr = n0 + l16, mb = m0 + 4 * g;
    bf16x4 o = bf16x4{};
    if (m0 <= n0) {
        f32x4 acc = zero_acc4();
        const __bf16 *ap = Am + (m0 + l16) * STR + 8 * g;
        const __bf16 *bp = Bn + nr * STR + 8 * g;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) acc = mma16(lds8(ap + 32 * ks), lds8(bp + 32 * ks), acc);
        const bool fac = uniform(sc.ctl[3]) != 0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int mr = mb + q;
            const float gm = fac ? sc.ea[nr] * sc.eb[mr] : __expf(sc.G[nr] - sc.G[mr]);
            o[q] = (__bf16)(mr <= nr ? acc[q] * gm : 0.f);
        }
    }
    *reinterpret_cast<bf16x4 *>(S + nr * SSB + mb) = o;
}

// ---- state in / out (ABI layout [B][H][256][128], paper row order) ------------
// Key state (kacc[x]: slot i = 32 w + lane % 32, channel c = 32 x + 8 (v/4) + 4 (lane/32) + v%4).
__device__ __forceinline__ void add_key_state(f32x16 (&acc)[4], const float *S, float f, int w, int lane, int m) {
    const int i = 32 * w + (lane & 31);
    if (!row_active_w(i, m)) return;
    const float *row = S + (size_t)paper_row_w(i) * 128 + 4 * (lane >> 5);
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
            const float4 q = *reinterpret_cast<const float4 *>(row + 32 * x + 8 * v4);
            acc[x][4 * v4] = fmaf(f, q.x, acc[x][4 * v4]);
            acc[x][4 * v4 + 1] = fmaf(f, q.y, acc[x][4 * v4 + 1]);
            acc[x][4 * v4 + 2] = fmaf(f, q.z, acc[x][4 * v4 + 2]);
            acc[x][4 * v4 + 3] = fmaf(f, q.w, acc[x][4 * v4 + 3]);
        }
}
__device__ __forceinline__ void store_key_state(float *S, const f32x16 (&acc)[4], float f, int w, int lane, int m) {
    const int i = 32 * w + (lane & 31);
    const bool live = row_active_w(i, m);
    float *row = S + (size_t)paper_row_w(i) * 128 + 4 * (lane >> 5);
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4)
            *reinterpret_cast<float4 *>(row + 32 * x + 8 * v4) =
                live ? make_float4(f * acc[x][4 * v4], f * acc[x][4 * v4 + 1], f * acc[x][4 * v4 + 2],
                                   f * acc[x][4 * v4 + 3])
                     : make_float4(0.f, 0.f, 0.f, 0.f);
}
// Value state (vacc[j]: slot i = 128 hh + 32 j + 8 (v/4) + 4 (lane/32) + v%4, channel
// c = 32 cb + lane % 32).
__device__ __forceinline__ int value_slot(int hh, int j, int v, int hl) {
    return 128 * hh + 32 * j + 8 * (v >> 2) + 4 * hl + (v & 3);
}
__device__ __forceinline__ void add_value_state(f32x16 (&acc)[4], const float *S, float f, int hh, int cb, int lane,
                                                int m) {
    const int c = 32 * cb + (lane & 31), hl = lane >> 5;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int i = value_slot(hh, j, v, hl);
            if (row_active_w(i, m)) acc[j][v] = fmaf(f, S[(size_t)paper_row_w(i) * 128 + c], acc[j][v]);
        }
}
__device__ __forceinline__ void store_value_state(float *S, const f32x16 (&acc)[4], float f, int hh, int cb, int lane,
                                                  int m) {
    const int c = 32 * cb + (lane & 31), hl = lane >> 5;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int i = value_slot(hh, j, v, hl);
            S[(size_t)paper_row_w(i) * 128 + c] = row_active_w(i, m) ? f * acc[j][v] : 0.f;
        }
}

// ---- chunk-group contributions (bf16, lane-major: wave w, accumulator x, lane, register;
// the precision in which the chunk products consume the state)
constexpr int kStateW = kR * 128;                   // elements of one 256 x 128 state
__device__ __forceinline__ int dump_w(int w, int x, int lane) { return ((w * 4 + x) * 64 + lane) * 16; }
__device__ __forceinline__ void store_dump(__bf16 *E, const f32x16 (&acc)[4], int w, int lane) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            bf16x8 o;
#pragma unroll
            for (int v = 0; v < 8; ++v) o[v] = (__bf16)acc[x][8 * hf + v];
            *reinterpret_cast<bf16x8 *>(E + dump_w(w, x, lane) + 8 * hf) = o;
        }
}
// a lane's part of one state of one contribution: [x][half] pieces of 8 registers
__device__ __forceinline__ void load_dump(bf16x8 (&e)[8], const __bf16 *E, int w, int lane) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) e[2 * x + hf] = *reinterpret_cast<const bf16x8 *>(E + dump_w(w, x, lane) + 8 * hf);
}
__device__ __forceinline__ void add_dump(f32x16 (&acc)[4], const bf16x8 (&e)[8], float f) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[x][v] = fmaf(f, (float)e[2 * x + (v >> 3)][v & 7], acc[x][v]);
}

struct WideArgs {
    FwdParams p;
    const __bf16 *Mz, *MzT;  // [H][256][256] readout matrix times scale log2 e, and its transpose
    int groups, cpg;         // chunk groups per sequence, chunks per group
    __bf16 *Ef;              // [BH][groups][2][kStateW] each group's own contribution (K, V), bf16
    float *Gg;               // [BH][groups] total log decay of each group
    double *gclk;            // [BH][groups] clock entering each group (reduced mod m)
    float *S0;               // [BH][2][kStateW] copy of (K0, V0) (groups > 1: the states may be
                             // overwritten in place by the last group)
};

// Sum over tokens [t_lo, t_hi) of x[t * stride] in double over the workgroup (eight
// loads in flight per thread); every thread gets the sum.  red: 8 doubles of LDS.
__device__ __forceinline__ double block_token_sum(const float *x, int stride, int t_lo, int t_hi, double *red,
                                                  int tid) {
    double ds = 0.0;
    for (int t0 = t_lo; t0 < t_hi; t0 += 8 * kNT) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int t = t0 + u * kNT + tid;
            v[u] = t < t_hi ? x[(size_t)t * stride] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) ds += (double)v[u];
    }
    for (int o = 32; o > 0; o >>= 1) ds += __shfl_xor(ds, o);
    if ((tid & 63) == 0) red[tid >> 6] = ds;
    __syncthreads();
    double tot = 0.0;
#pragma unroll
    for (int i = 0; i < kNT / 64; ++i) tot += red[i];
    __syncthreads();
    return tot;
}

// ---- LDS map (bytes) ------------------------------------------------------------
struct Lay {
    static constexpr int T1 = kC * PSB;            // [32][128] tile
    static constexpr int T2 = kC * PWB;            // [32][256] tile
    static constexpr int TS = kC * SSB * 2;        // score tile
    static constexpr int Q = 0;                    // Q, then the output tile
    static constexpr int K = Q + T1;
    static constexpr int V = K + T1;
    static constexpr int A = V + T1;               // temporal writes
    static constexpr int X = A + T2;               // X, then u
    static constexpr int W = X + T2;               // W, then the upper half's partial outputs
    static constexpr int S1 = W + T2;              // Gamma (.) Q K^T
    static constexpr int S2 = S1 + TS;             // Gamma (.) u A^T
    static constexpr int RED = S2 + TS;            // softmax partials [8 waves][32 tokens] float2
    static constexpr int SC = RED + 8 * kC * 8;
    static constexpr int BYTES = SC + (int)sizeof(Sc);
    static_assert(4 * 64 * 16 * 4 <= T2, "partial outputs fit the W tile");
    static_assert(BYTES <= 160 * 1024, "one workgroup per compute unit");
};

__global__ __launch_bounds__(kNT, 1) void wide_forward_kernel(WideArgs a) {
    using L = Lay;
    __shared__ __attribute__((aligned(256))) char smem[L::BYTES];
    const FwdParams &p = a.p;
    const __bf16 *Mz = a.Mz, *MzT = a.MzT;
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31, hl = lane >> 5;
    const int hh = w >> 2, cb = w & 3;             // value-state slot half and channel block
    const int m = p.m;
    const int Tb = seq_tokens(p, b);
    const size_t row0 = seq_row0(p, b);
    // this group's chunks, up to the sequence's last one
    const int c_begin = g * a.cpg, c_end = min(c_begin + a.cpg, (Tb + kC - 1) / kC);
    Sc &sc = *lds_at<Sc>(smem, L::SC);
    __bf16 *Qt = lds_at<__bf16>(smem, L::Q), *Kt = lds_at<__bf16>(smem, L::K), *Vt = lds_at<__bf16>(smem, L::V);
    __bf16 *At = lds_at<__bf16>(smem, L::A), *Xt = lds_at<__bf16>(smem, L::X), *Wt = lds_at<__bf16>(smem, L::W);
    __bf16 *S1 = lds_at<__bf16>(smem, L::S1), *S2 = lds_at<__bf16>(smem, L::S2);
    float2 *red = lds_at<float2>(smem, L::RED);
    float *part = lds_at<float>(smem, L::W);
    const Sw z = make_sw(tid);
    const float zs = p.scale * 1.4426950408889634f;     // Mz = zs M: logits in log2 units
    const float inv_zs = 1.f / zs;
    // this lane's rows of the readout matrix and of its transpose (slot / basis 32 w + l32)
    const __bf16 *Mrow = Mz + ((size_t)h * kR + 32 * w + l32) * kR + 8 * hl;
    const __bf16 *MTrow = MzT + ((size_t)h * kR + 32 * w + l32) * kR + 8 * hl;

    f32x16 kacc[4], vacc[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        kacc[x] = zero_acc();
        vacc[x] = zero_acc();
    }
    const size_t sb = (size_t)bh * kStateW;
    double carry;
    if (a.groups == 1) {
        if (p.K0) add_key_state(kacc, p.K0 + sb, 1.f, w, lane, m);
        if (p.V0) add_value_state(vacc, p.V0 + sb, 1.f, hh, cb, lane, m);
        carry = reduce_clock(p.clock0 ? p.clock0[bh] : 0.0, (double)m, 1.0 / (double)m);
    } else {
        // state entering the group: each earlier group's contribution decayed through
        // the groups after it, plus (K0, V0) decayed through all earlier groups
        // (key states first, then value states, two contributions per memory round trip)
        const float *Gg = a.Gg + (size_t)bh * a.groups;
        const __bf16 *Eb = a.Ef + (size_t)bh * a.groups * 2 * kStateW;
        auto sum_groups = [&](f32x16 (&acc)[4], int sv) {
            float tl = 0.f;                       // log decay of groups q+1 .. g-1
            for (int q = g - 1; q >= 0; q -= 2) {
                bf16x8 e0[8], e1[8];
                load_dump(e0, Eb + ((size_t)q * 2 + sv) * kStateW, w, lane);
                if (q >= 1) load_dump(e1, Eb + ((size_t)(q - 1) * 2 + sv) * kStateW, w, lane);
                add_dump(acc, e0, __expf(tl));
                tl += Gg[q];
                if (q >= 1) {
                    add_dump(acc, e1, __expf(tl));
                    tl += Gg[q - 1];
                }
            }
        };
        sum_groups(kacc, 0);
        sum_groups(vacc, 1);
        float tail = 0.f;                         // log decay of groups 0 .. g-1
        for (int q = 0; q < g; ++q) tail += Gg[q];
        const float *S0 = a.S0 + (size_t)bh * 2 * kStateW;
        if (p.K0) add_key_state(kacc, S0, __expf(tail), w, lane, m);
        if (p.V0) add_value_state(vacc, S0 + kStateW, __expf(tail), hh, cb, lane, m);
        carry = a.gclk[(size_t)bh * a.groups + g];
    }

    const size_t rs = (size_t)p.H * 128;
    const __bf16 *qin = static_cast<const __bf16 *>(p.q), *kin = static_cast<const __bf16 *>(p.k);
    const __bf16 *vin = static_cast<const __bf16 *>(p.v);
    __bf16 *o = static_cast<__bf16 *>(p.o);
    uint4 rq, rk, rv;
    Tok tk;
    auto prefetch = [&](int c) {
        const int t0 = c * kC, n = min(kC, Tb - t0);
        const size_t base = ((row0 + t0) * p.H + h) * 128;
        load_row1(qin + base, rs, n, tid, rq);
        load_row1(kin + base, rs, n, tid, rk);
        load_row1(vin + base, rs, n, tid, rv);
        load_tok(p, row0, h, t0, Tb, tid, tk);
    };
    if (c_begin < c_end) prefetch(c_begin);
    float Ls = 0.f;                                   // carried states: exp(Ls) x registers
    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * kC, n = min(kC, Tb - t0);
        // -- stage the chunk and its scalars
        store_row1(Qt, rq, z);
        store_row1(Kt, rk, z);
        store_row1(Vt, rv, z);
        if (w == 0) chunk_scalars(sc, lane, m, tk, carry, Ls);
        if (c + 1 < c_end) prefetch(c + 1);
        lds_barrier();
        {
            const float pre = uniform(sc.ctl[0]);
            if (pre != 1.f) {
                scale_acc(kacc, pre);
                scale_acc(vacc, pre);
            }
        }
        build_A(sc, At, tid, m);
        if (w < 4) score_block<4, PS>(Kt, 16 * (w & 1), Qt, 16 * (w >> 1), S1, sc, lane);   // S1[t][s]
        // -- key pass: p = gamma (.) Q Kbar^T + S1 A (D[slot][t]); then the key state update
        const float gr = sc.gam[l32];
        f32x16 pacc = zero_acc();
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) pacc = mma(acc_to_operand(kacc[ks >> 1], ks & 1), sperm(Qt, ks, z), pacc);
#pragma unroll
        for (int v = 0; v < 16; ++v) pacc[v] *= gr;
        lds_barrier();
        const float post = uniform(sc.ctl[1]);
        if (post != 1.f) scale_acc(kacc, post);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const bf16x8 at = stro_w(At, 16 * ks, 32 * w, z);
            pacc = mma(at, rd_row(S1, l32, 16 * ks, hl), pacc);
            const bf16x8 ad = scale_k(at, sc.rho + 16 * ks + 8 * hl);
#pragma unroll
            for (int x = 0; x < 4; ++x) kacc[x] = mma(stro(Kt, 16 * ks, 32 * x, z), ad, kacc[x]);
        }
        // -- X = U(lambda) p (the scale is folded into Mz); the padding column carries 1
        {
            float pc[8], ps[8];
            lane_phases(opqf(sc.urev[l32]), w, hl, m, pc, ps);
            rotate<1>(pacc, pc, ps, 1.f);
            if (w == 7 && hl == 1) pacc[15] = 1.f;
            store_block_w(Xt, 32 * w, pacc, z);
        }
        lds_barrier();
        // -- slot logits of this wave's 32 slots (log2 units; inactive slots about -1e30)
        f32x16 wr = zero_acc();
#pragma unroll
        for (int ks = 0; ks < 16; ++ks) wr = mma(grow(Mrow, ks), srow_w(Xt, ks, z), wr);
        {
            if (p.logits && l32 < n) {
                float *lg = p.logits + ((row0 + t0 + l32) * p.H + h) * m;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int slot = 32 * w + 8 * (v >> 2) + 4 * hl + (v & 3);
                    if (slot < m) lg[slot] = wr[v] * 0.69314718055994531f;
                }
            }
            float mx = wr[0];
#pragma unroll
            for (int v = 1; v < 16; ++v) mx = fmaxf(mx, wr[v]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
#pragma unroll
            for (int v = 0; v < 16; ++v) wr[v] = __builtin_amdgcn_exp2f(wr[v] - mx);
            float sm = 0.f;
#pragma unroll
            for (int v = 0; v < 16; ++v) sm += wr[v];
            sm += __shfl_xor(sm, 32);
            if (hl == 0) red[w * kC + l32] = make_float2(mx, sm);
            lds_barrier();
            float M = red[l32].x;
#pragma unroll
            for (int x = 1; x < 8; ++x) M = fmaxf(M, red[x * kC + l32].x);
            float Lsum = 0.f;
#pragma unroll
            for (int x = 0; x < 8; ++x) {
                const float2 pr = red[x * kC + l32];
                Lsum += pr.y * __builtin_amdgcn_exp2f(pr.x - M);
            }
            const float f = __builtin_amdgcn_exp2f(mx - M) / Lsum;
#pragma unroll
            for (int v = 0; v < 16; ++v) wr[v] *= f;
        }
        store_block_w(Wt, 32 * w, wr, z);
        lds_barrier();
        // -- u = U(-lambda) M^T W of this wave's 32 basis coordinates, in X's place
        {
            f32x16 ya = zero_acc();
#pragma unroll
            for (int ks = 0; ks < 16; ++ks) ya = mma(grow(MTrow, ks), srow_w(Wt, ks, z), ya);
            float pc[8], ps[8];
            lane_phases(opqf(sc.urev[l32]), w, hl, m, pc, ps);
            rotate<-1>(ya, pc, ps, inv_zs);
            store_block_w(Xt, 32 * w, ya, z);
        }
        lds_barrier();
        // -- value pass: o = gamma (.) u Vbar + S2 V, this wave's channel block over its
        //    slot half (D[c][t]); then the value state update
        if (w < 4) score_block<8, PW>(At, 16 * (w & 1), Xt, 16 * (w >> 1), S2, sc, lane);   // S2[t][s]
        f32x16 oacc = zero_acc();
#pragma unroll
        for (int ks = 0; ks < 8; ++ks)
            oacc = mma(acc_to_operand(vacc[ks >> 1], ks & 1), sperm_w(Xt, 8 * hh + ks, z), oacc);
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[v] *= gr;
        if (post != 1.f) scale_acc(vacc, post);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const bf16x8 vb = stro(Vt, 16 * ks, 32 * cb, z);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                vacc[j] = mma(scale_k(stro_w(At, 16 * ks, 128 * hh + 32 * j, z), sc.rho + 16 * ks + 8 * hl), vb,
                              vacc[j]);
        }
        if (hh == 1) {
            float *dst = part + ((w - 4) * 64 + lane) * 16;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                *reinterpret_cast<float4 *>(dst + 4 * q) =
                    make_float4(oacc[4 * q], oacc[4 * q + 1], oacc[4 * q + 2], oacc[4 * q + 3]);
        }
        lds_barrier();
        if (hh == 0) {
            const float *src = part + (w * 64 + lane) * 16;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float4 e = *reinterpret_cast<const float4 *>(src + 4 * q);
                oacc[4 * q] += e.x;
                oacc[4 * q + 1] += e.y;
                oacc[4 * q + 2] += e.z;
                oacc[4 * q + 3] += e.w;
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) oacc = mma(stro(Vt, 16 * ks, 32 * cb, z), rd_row(S2, l32, 16 * ks, hl), oacc);
            store_block(Qt, 32 * cb, oacc, z);          // o[t][c], in Q's place
        }
        Ls = next_scale(sc, Ls);
        lds_barrier();
        copy_row1_out(Qt, o + ((row0 + t0) * p.H + h) * 128, rs, n, tid, z);
        lds_barrier();
    }
    // the last group ends with the final states (chunks past a sequence change nothing)
    if (g == a.groups - 1) {
        const float f = __expf(Ls);
        if (p.K_out) store_key_state(p.K_out + sb, kacc, f, w, lane, m);
        if (p.V_out) store_value_state(p.V_out + sb, vacc, f, hh, cb, lane, m);
        if (p.clock_out && tid == 0) p.clock_out[bh] = carry;
    }
}

// Each chunk group's own contribution (groups > 1; launched before the forward):
// sum_t exp(G_end - G_t) a_t [k_t | v_t]^T over the group's tokens, a plain weighted
// sum, so every token's decay to the group end is one factor in [0, 1] folded into its
// write row (no running rescale; G_end, the group's total log decay, is reduced
// first).  64-token steps: every wave runs the step's clock and decay scans itself
// (lane = token), builds 8 of the decayed write rows (taking its token's phase and
// amplitude from the scanning lane), and after one barrier updates its state blocks
// from the shared tiles.  The last group's contribution is never read, so its
// workgroup copies (K0, V0) for the forward's prologues instead and forms only its
// total log decay.
constexpr int kCS = 64;                             // tokens per step
__global__ __launch_bounds__(kNT, 1) void wide_contrib_kernel(WideArgs a) {
    constexpr int TK = kCS * PSB;                   // [64][128] tile
    constexpr int TA = kCS * PWB;                   // [64][256] tile
    __shared__ __attribute__((aligned(256))) char smem[2 * TK + TA];
    __shared__ double red[kNT / 64];
    const FwdParams &p = a.p;
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int hh = w >> 2, cb = w & 3;
    const int m = p.m;
    const int Tb = seq_tokens(p, b);
    const size_t row0 = seq_row0(p, b);
    const int t_begin = min(g * a.cpg * kC, Tb), t_end = min((g + 1) * a.cpg * kC, Tb);
    const size_t tok0 = row0 * p.H + h;
    const size_t pi = (size_t)bh * a.groups + g;
    const bool last = g == a.groups - 1;
    const size_t rs = (size_t)p.H * 128;
    const __bf16 *kin = static_cast<const __bf16 *>(p.k), *vin = static_cast<const __bf16 *>(p.v);
    // K, V pieces: rows tid/16 + 32 it, 16-byte column block tid%16; token `lane`'s scalars
    uint4 rk[2], rv[2];
    float dl, gg, be;
    auto prefetch = [&](int t0) {
        const int tq = opq(tid);
        const int r = tq >> 4, c8 = (tq & 15) * 8;
        const size_t base = ((row0 + t0) * p.H + h) * 128 + c8;
#pragma unroll
        for (int it = 0; it < 2; ++it) {
            const int rr = r + 32 * it;
            const bool in = t0 + rr < t_end;
            rk[it] = in ? *reinterpret_cast<const uint4 *>(kin + base + (size_t)rr * rs) : make_uint4(0, 0, 0, 0);
            rv[it] = in ? *reinterpret_cast<const uint4 *>(vin + base + (size_t)rr * rs) : make_uint4(0, 0, 0, 0);
        }
        const int t = t0 + lane;
        const size_t si = (row0 + t) * p.H + h;
        const bool tin = t < t_end;
        dl = tin ? p.delta[si] : 0.f;
        gg = (tin && p.log_alpha) ? p.log_alpha[si] : 0.f;
        be = tin ? (p.beta ? p.beta[si] : 1.f) : 0.f;
    };
    // the first step's rows are in flight while the two sums below are formed
    if (!last && t_begin < t_end) prefetch(t_begin);
    // clock entering the group: clock0 plus every increment before it (double)
    const double c_in = reduce_clock((p.clock0 ? p.clock0[bh] : 0.0) +
                                         block_token_sum(p.delta + tok0, p.H, 0, t_begin, red, tid),
                                     (double)m, 1.0 / (double)m);
    if (tid == 0) a.gclk[pi] = c_in;
    const double G_end = p.log_alpha ? block_token_sum(p.log_alpha + tok0, p.H, t_begin, t_end, red, tid) : 0.0;
    if (tid == 0) a.Gg[pi] = (float)G_end;
    if (last) {
        float *S0 = a.S0 + (size_t)bh * 2 * kStateW;
        const size_t sb = (size_t)bh * kStateW;
        for (int e = 4 * tid; e < kStateW; e += 4 * kNT) {
            if (p.K0) *reinterpret_cast<float4 *>(S0 + e) = *reinterpret_cast<const float4 *>(p.K0 + sb + e);
            if (p.V0) *reinterpret_cast<float4 *>(S0 + kStateW + e) = *reinterpret_cast<const float4 *>(p.V0 + sb + e);
        }
        return;
    }
    __bf16 *Kt = lds_at<__bf16>(smem, 0), *Vt = lds_at<__bf16>(smem, TK), *Adt = lds_at<__bf16>(smem, 2 * TK);
    const double dm = (double)m, inv_m = 1.0 / (double)m;
    const float amp0 = sqrtf(2.f / (float)m);
    const int J = (m - 1) >> 1;
    f32x16 kacc[4], vacc[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        kacc[x] = zero_acc();
        vacc[x] = zero_acc();
    }
    double carry = c_in, gsum = 0.0;
    for (int t0 = t_begin; t0 < t_end; t0 += kCS) {
        const int tq = opq(tid);
        const Sw z = make_sw(tq);
        {
            const int r = tq >> 4, c16 = (tq & 15) * 16;
#pragma unroll
            for (int it = 0; it < 2; ++it) {
                *reinterpret_cast<uint4 *>(cbyte(Kt) + (r + 32 * it) * PSB + c16) = rk[it];
                *reinterpret_cast<uint4 *>(cbyte(Vt) + (r + 32 * it) * PSB + c16) = rv[it];
            }
        }
        // the step's scans on every wave (lane = token): clock (double, absolute from the
        // group's entering clock) and the decay from the token to the group end
        float u, amp;
        {
            const double lam = carry + wave_incl_scan((double)dl);
            const float Gl = wave_incl_scan(gg);
            const float rem = (float)(G_end - gsum);
            const double q = lam * inv_m;
            u = (float)(q - floor(q));
            amp = be * amp0 * __expf(rem - Gl);
            carry = reduce_clock(lane63(lam), dm, inv_m);
            gsum += (double)lane63(Gl);
        }
        if (t0 + kCS < t_end) prefetch(t0 + kCS);
        {
            // decayed write rows: thread (row 8 w + lane / 8, eighth e = lane % 8) fills
            // columns 32 e .. 32 e + 31 (pairs 16 e + 1 .. 16 e + 16; DC and padding at
            // 254, 255), from four starts advanced by angle addition
            const int lq = opq(lane);
            const int r = 8 * w + (lq >> 3), e = lq & 7;
            const float ur = __shfl(u, r), ar = __shfl(amp, r);
            float s1, c1;
            sincos_rev(ur, &s1, &c1);
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
                float sn, cs;
                sincos_rev(__builtin_amdgcn_fractf((float)(16 * e + 4 * qq + 1) * ur), &sn, &cs);
                bf16x8 d8;
#pragma unroll
                for (int jj = 0; jj < 4; ++jj) {
                    const int j = 16 * e + 4 * qq + 1 + jj;
                    const bool live = j <= J;
                    float a0 = live ? ar * cs : 0.f, a1 = live ? -ar * sn : 0.f;
                    if (j == kR / 2) {                          // internal columns 254, 255
                        a0 = ar * 0.70710678118654752f;
                        a1 = 0.f;
                    }
                    d8[2 * jj] = (__bf16)a0;
                    d8[2 * jj + 1] = (__bf16)a1;
                    if (jj < 3) {
                        const float nc = cs * c1 - sn * s1;
                        const float ns = sn * c1 + cs * s1;
                        cs = nc;
                        sn = ns;
                    }
                }
                *reinterpret_cast<bf16x8 *>(cbyte(Adt) + r * PWB + 64 * e + 16 * qq) = d8;
            }
        }
        lds_barrier();
#pragma unroll
        for (int ks = 0; ks < kCS / 16; ++ks) {
            const bf16x8 ad = stro_w(Adt, 16 * ks, 32 * w, z);
#pragma unroll
            for (int x = 0; x < 4; ++x) kacc[x] = mma(stro(Kt, 16 * ks, 32 * x, z), ad, kacc[x]);
            const bf16x8 vb = stro(Vt, 16 * ks, 32 * cb, z);
#pragma unroll
            for (int j = 0; j < 4; ++j) vacc[j] = mma(stro_w(Adt, 16 * ks, 128 * hh + 32 * j, z), vb, vacc[j]);
        }
        lds_barrier();
    }
    __bf16 *E = a.Ef + pi * 2 * kStateW;
    store_dump(E, kacc, w, lane);
    store_dump(E + kStateW, vacc, w, lane);
}

}  // namespace

bool mfma_wide_supported(const FwdParams &p) {
    return p.dtype == 1 && p.dk == 128 && p.dv == 128 && p.m > kMaxActive && p.m <= kMaxActiveWide &&
           (p.chunk == 32 || p.chunk == 64);
}

int mfma_wide_auto_groups(const FwdParams &p) {
    // one eight-wave workgroup per compute unit: split sequences into chunk groups
    // until B H G covers the 256 compute units
    const int nc = (p.T + kC - 1) / kC;
    const int BH = p.B * p.H;
    int g = (256 + BH - 1) / BH;
    if (g > nc) g = nc;
    return g < 1 ? 1 : g;
}

namespace {
struct WideWs {
    size_t mz, mzt, ef, gg, gclk, s0, total;
};
WideWs wide_ws(const FwdParams &p, int groups) {
    auto up = [](size_t x) { return (x + 255) / 256 * 256; };
    const size_t BH = (size_t)p.B * p.H, G = groups;
    WideWs L{};
    size_t off = 0;
    L.mz = off;
    off += up((size_t)p.H * kR * kR * 2);
    L.mzt = off;
    off += up((size_t)p.H * kR * kR * 2);
    if (groups > 1) {
        L.ef = off;
        off += up(BH * G * 2 * kStateW * 2);
        L.gg = off;
        off += up(BH * G * 4);
        L.gclk = off;
        off += up(BH * G * 8);
        L.s0 = off;
        off += up(BH * 2 * kStateW * 4);
    }
    L.total = off;
    return L;
}
}  // namespace

size_t mfma_wide_workspace_bytes(const FwdParams &p, int groups) { return wide_ws(p, groups).total; }

hipError_t launch_fwd_mfma_wide(const FwdParams &p, int groups, void *ws, hipStream_t st, hipEvent_t ev_start,
                                hipEvent_t ev_stop) {
    char *base = static_cast<char *>(ws);
    const WideWs L = wide_ws(p, groups);
    WideArgs a{};
    a.p = p;
    a.Mz = reinterpret_cast<const __bf16 *>(base + L.mz);
    a.MzT = reinterpret_cast<const __bf16 *>(base + L.mzt);
    const int nc = (p.T + kC - 1) / kC;
    a.cpg = nc > 0 ? (nc + groups - 1) / groups : 1;
    a.groups = nc > 0 ? (nc + a.cpg - 1) / a.cpg : 1;      // no empty trailing group
    if (a.groups > 1) {
        a.Ef = reinterpret_cast<__bf16 *>(base + L.ef);
        a.Gg = reinterpret_cast<float *>(base + L.gg);
        a.gclk = reinterpret_cast<double *>(base + L.gclk);
        a.S0 = reinterpret_cast<float *>(base + L.s0);
    }
    hipError_t e = launch_readout_prep_wide_bf16(p.H, p.m, p.R, const_cast<__bf16 *>(a.Mz),
                                                 const_cast<__bf16 *>(a.MzT), p.scale * 1.4426950408889634f, st);
    if (e != hipSuccess) return e;
    const dim3 grid(p.B * p.H, a.groups);
    if (a.groups > 1) {
        hipLaunchKernelGGL(wide_contrib_kernel, grid, dim3(kNT), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipExtLaunchKernelGGL(wide_forward_kernel, grid, dim3(kNT), 0, st, ev_start, ev_stop, 0, a);
    return hipGetLastError();
}

}  // namespace cyfa
