// Matrix-core (bf16 MFMA) backward of the chunk-wise CyFA forward: bf16 inputs,
// d_k = d_v = 128, m <= 127, 32-token chunks.
//
// The gradients are those of the vector-ALU backward (reverse mode of the
// absolute-clock recurrence and readout, Sec. 3.2 Eqs. cyfa-absolute-recurrence
// and cyfa-absolute-readout, chunk by chunk as in App. B; the clock increments
// receive the reverse cumulative sum of the per-token clock gradients, Eq.
// app-clock-gradient-accumulation; the per-token formulas are written out at
// the top of cyfa_bwd_valu.hip).  Here every dense product runs on bf16
// matrix-core tiles with fp32 accumulation, and the states stay in MFMA
// accumulators while a workgroup walks its chunk group:
//   (1) fwd_contrib_kernel (b, h, group): the group's own contribution to the
//       states at its end (zero entering state; not for the last group, whose
//       contribution no walk reads), the clock entering the group and the group's
//       total log decay.
//   (2) readout_kernel (b, h, group): forms the state entering its group from
//       (K0, V0) and the earlier groups' contributions, then walks the group's
//       chunks forward with both states in accumulators, recomputes the key
//       pass p, X, the slot weights W and u, and forms du, the readout's adjoint
//       (dY, dW, dZ, dX, dp), dq, the group's part of dM, <q, dq> + <u, du> and
//       the clock gradients of X and u; u and dp go to the workspace in bf16 for
//       (3) and (4).  The last group ends with the final states and forms the
//       final-state loss <dK_T, Kbar_T> + <dV_T, Vbar_T>.
//   (3) adj_contrib_kernel (b, h, group > 0): the group's own contribution to
//       the adjoint states entering it from its tokens (zero adjoint at its end).
//   (4) grad_kernel (b, h, group): forms the adjoint at its group's end from
//       (dK_T, dV_T) and the later groups' contributions, then walks the group's
//       chunks in reverse with both adjoint states in accumulators: dk, dv, da and
//       from da the gradient of beta and the clock gradient of the write a_t, and
//       dL/dG.  The first group ends at the sequence start: dK0, dV0.
// The reverse cumulative sums (dlog_alpha, ddelta, dclock0) and dR = dM Phi^T
// are the vector-ALU backward's last two kernels (launch_bwd_tail).
//
// Within a chunk (token rows r, s; G_r the chunk-local inclusive sum of log
// alpha; gamma_r = exp(G_r); rho_s = exp(G_C - G_s); Gamma_rs = exp(G_r - G_s)
// for s <= r, else 0; Kbar, Vbar the states entering the chunk; DK', DV' the
// adjoint states at its end):
//   p  = gamma (.) Q Kbar^T + (Q K^T (.) Gamma) A      du = gamma (.) dO Vbar^T + (dO V^T (.) Gamma) A
//   dq = gamma (.) dP Kbar  + (dP A^T (.) Gamma) K
//   dk = rho (.) A DK' + (dP A^T (.) Gamma)^T Q         dv = rho (.) A DV' + (U A^T (.) Gamma)^T dO
//   da = rho (.) (K DK'^T + V DV'^T) + (Q K^T (.) Gamma)^T dP + (dO V^T (.) Gamma)^T U
//   Kbar <- exp(G_C) Kbar + (rho (.) A)^T K,   DK'_prev = exp(G_C) DK' + (gamma (.) dP)^T Q
// (Vbar, DV' likewise with V and (gamma (.) U)^T dO).
//
// Basis order inside: the matrix-core kernels' internal order (pair j at
// (2j-2, 2j-1), DC at 126, padding 127), so a rotation acts on two consecutive
// accumulator registers of one lane.  The ABI's state arrays (paper order) are
// converted where they are read or written; dM leaves in paper column order.
//
// State accumulators, four per wave (x = 0..3): wave w holds basis rows
// i = 32 w + lane % 32 and columns c = 32 x + 8 (v / 4) + 4 (lane / 32) + v % 4 of
// a 128 x 128 state in register v, i.e. the transposed product D[c][i]; the key
// and the value state (and their adjoints) alike.  Fed back as an A operand
// (acc_to_operand) it supplies rows i and the permuted k indices c (the other
// operand is then read with lds8_perm).  The workspace copies use the same
// lane-major dump layout (dump_off).
#include "cyfa_bwd.h"
#include "cyfa_mfma_common.h"
#include "cyfa_prep.h"

namespace cyfa {

using namespace mfma;

namespace {

constexpr int kC = kBwdMfmaChunk;   // tokens per chunk
constexpr int kNT = 256;            // threads per workgroup (four waves)
constexpr int kT32 = kC * 288;      // bytes of a padded [32][128] bf16 tile (row stride 144)
constexpr int kT128 = 128 * 288;    // bytes of a padded [128][128] bf16 tile
constexpr int SSB = 40;             // row stride (bf16) of a [32][32] score tile
constexpr int kTS = kC * SSB * 2;   // bytes of a score tile
constexpr int kSE = 128 * 128;      // floats of one 128 x 128 state
constexpr int kCombBlocks = kBwdFinParts;
constexpr float kTwoPi = 6.283185307179586f;

struct Args {
    BwdParams p;        // shapes, inputs and outputs; nc / Tpad count 32-token chunks;
                        // p.udu, p.dlam, p.dG, p.dMp, p.fin as for the shared last kernels
    const __bf16 *Mz;   // [H][128][128] readout matrix times zs = scale log2 e (internal columns)
    float *Ef;          // [BH][G][2][kSE] forward states: group contributions, then entering states
    float *Ea;          // [BH][G][2][kSE] adjoint states: group contributions, then the adjoints at
                        // each group's end
    float *Gg;          // [BH][G] total log decay of each group
    double *gclk;       // [BH][G] clock entering each group (reduced mod m)
    double *cclk;       // [BH][nc] clock entering each chunk (reduced mod m)
    __bf16 *U, *dP;     // [BH][Tpad][128] u_t and dp_t, internal basis order
};

// a value every lane holds alike, moved to a scalar register
__device__ __forceinline__ float uniform(float x) {
    return __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(x)));
}
// opaque copy: a value recomputed from it is not merged with an earlier computation
__device__ __forceinline__ float opqf(float x) {
    asm volatile("" : "+v"(x));
    return x;
}

__device__ __forceinline__ int tokens_of(const BwdParams &p, int b) {
    return p.lens ? min(max(p.lens[b], 0), p.T) : p.T;
}

// internal basis index -> paper row (a bijection of 0..127; rows i < m-1 and DC are active)
__device__ __forceinline__ int paper_row(int i) { return i < 126 ? i + 1 : (i == 126 ? 0 : 127); }
__device__ __forceinline__ bool row_active(int i, int m) { return i < m - 1 || i == 126; }

// element e of the dump layout -> (internal row i, column c)
__device__ __forceinline__ void dump_coords(int e, int &i, int &c) {
    const int w = e >> 12, x = (e >> 10) & 3, lane = (e >> 4) & 63, v = e & 15;
    i = 32 * w + (lane & 31);
    c = 32 * x + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}

__device__ __forceinline__ void load_acc(const float *E, int w, int lane, f32x16 (&acc)[4]) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 f = *reinterpret_cast<const float4 *>(E + dump_off(w, x, lane, 4 * q));
            acc[x][4 * q] = f.x;
            acc[x][4 * q + 1] = f.y;
            acc[x][4 * q + 2] = f.z;
            acc[x][4 * q + 3] = f.w;
        }
}
__device__ __forceinline__ void store_acc(float *E, int w, int lane, const f32x16 (&acc)[4]) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *reinterpret_cast<float4 *>(E + dump_off(w, x, lane, 4 * q)) =
                make_float4(acc[x][4 * q], acc[x][4 * q + 1], acc[x][4 * q + 2], acc[x][4 * q + 3]);
}
template <int N>
__device__ __forceinline__ void scale_acc(f32x16 (&acc)[N], float f) {
#pragma unroll
    for (int x = 0; x < N; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[x][v] *= f;
}
// two accumulators of wave block w: column blocks x0, x0 + 1
__device__ __forceinline__ void store_acc2(float *E, int w, int x0, int lane, const f32x16 (&acc)[2]) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *reinterpret_cast<float4 *>(E + dump_off(w, x0 + j, lane, 4 * q)) =
                make_float4(acc[j][4 * q], acc[j][4 * q + 1], acc[j][4 * q + 2], acc[j][4 * q + 3]);
}
// The helpers below take N accumulators of one wave, column blocks x0 .. x0+N-1 of
// the basis rows 32 w + lane % 32 (the four-wave kernels hold N = 4 from x0 = 0).
// acc += f * (a state in the ABI layout [128 paper rows][128], active rows only)
template <int N>
__device__ __forceinline__ void add_abi_state(f32x16 (&acc)[N], const float *S, float f, int w, int x0, int lane,
                                              int m) {
    const int i = 32 * w + (lane & 31);
    if (!row_active(i, m)) return;
    const float *row = S + (size_t)paper_row(i) * 128 + 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < N; ++j)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
            const float4 q = *reinterpret_cast<const float4 *>(row + 32 * (x0 + j) + 8 * v4);
            acc[j][4 * v4] = fmaf(f, q.x, acc[j][4 * v4]);
            acc[j][4 * v4 + 1] = fmaf(f, q.y, acc[j][4 * v4 + 1]);
            acc[j][4 * v4 + 2] = fmaf(f, q.z, acc[j][4 * v4 + 2]);
            acc[j][4 * v4 + 3] = fmaf(f, q.w, acc[j][4 * v4 + 3]);
        }
}
// acc += f * (a state in the dump layout)
template <int N>
__device__ __forceinline__ void add_dump_state(f32x16 (&acc)[N], const float *E, float f, int w, int x0, int lane) {
#pragma unroll
    for (int j = 0; j < N; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 e = *reinterpret_cast<const float4 *>(E + dump_off(w, x0 + j, lane, 4 * q));
            acc[j][4 * q] = fmaf(f, e.x, acc[j][4 * q]);
            acc[j][4 * q + 1] = fmaf(f, e.y, acc[j][4 * q + 1]);
            acc[j][4 * q + 2] = fmaf(f, e.z, acc[j][4 * q + 2]);
            acc[j][4 * q + 3] = fmaf(f, e.w, acc[j][4 * q + 3]);
        }
}
// sum over the lane's elements of S (ABI layout, active rows) times acc
template <int N>
__device__ __forceinline__ float dot_abi_state(const f32x16 (&acc)[N], const float *S, int w, int x0, int lane,
                                               int m) {
    const int i = 32 * w + (lane & 31);
    if (!S || !row_active(i, m)) return 0.f;
    const float *row = S + (size_t)paper_row(i) * 128 + 4 * (lane >> 5);
    float t = 0.f;
#pragma unroll
    for (int j = 0; j < N; ++j)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
            const float4 q = *reinterpret_cast<const float4 *>(row + 32 * (x0 + j) + 8 * v4);
            t = fmaf(q.x, acc[j][4 * v4], t);
            t = fmaf(q.y, acc[j][4 * v4 + 1], t);
            t = fmaf(q.z, acc[j][4 * v4 + 2], t);
            t = fmaf(q.w, acc[j][4 * v4 + 3], t);
        }
    return t;
}
// f * acc into a state in the ABI layout (rows that are not active written as 0)
template <int N>
__device__ __forceinline__ void store_abi_state(float *S, const f32x16 (&acc)[N], float f, int w, int x0, int lane,
                                                int m) {
    const int i = 32 * w + (lane & 31);
    const bool act = row_active(i, m);
    float *row = S + (size_t)paper_row(i) * 128 + 4 * (lane >> 5);
#pragma unroll
    for (int j = 0; j < N; ++j)
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4)
            *reinterpret_cast<float4 *>(row + 32 * (x0 + j) + 8 * v4) =
                act ? make_float4(f * acc[j][4 * v4], f * acc[j][4 * v4 + 1], f * acc[j][4 * v4 + 2],
                                  f * acc[j][4 * v4 + 3])
                    : make_float4(0.f, 0.f, 0.f, 0.f);
}

// ---- padded tiles ----------------------------------------------------------------
// [rows][128] bf16 tiles with a row stride of PS = 144 elements (288 bytes: each row
// starts 8 banks after the previous one).  Transposed operands (sixteen lanes read 32
// bytes from each of four consecutive rows) and row operands (eight lanes read 16 bytes
// from each of eight consecutive rows) are then free of bank conflicts; 8-byte
// accesses of sixteen consecutive rows at one column meet rows r and r + 8 in the same
// banks.  Every offset is a lane constant plus a compile-time term, which the LDS
// instructions take as their immediate offset.
constexpr int PS = 144;
constexpr int PSB = PS * 2;                 // row stride in bytes

struct Sw {
    int row;    // row operand: row lane%32, columns 8 (lane/32) ..          (+ 32 ks bytes)
    int st;     // 8-byte pieces: row lane%32, columns 4 (lane/32) ..        (+ 2 col bytes)
    int tr;     // transposed operand (tr_off)                               (+ rows, columns)
    int cp;     // 16-byte pieces of whole rows: row tid/16, columns 8 (tid%16) ..
};
__device__ __forceinline__ Sw make_sw(int tid) {
    const int lane = tid & 63, l32 = lane & 31, hl = lane >> 5;
    Sw z;
    z.row = l32 * PSB + 16 * hl;
    z.st = l32 * PSB + 8 * hl;
    z.tr = 2 * tr_off(PS, lane);
    z.cp = (tid >> 4) * PSB + (tid & 15) * 16;
    return z;
}
__device__ __forceinline__ const char *cbyte(const __bf16 *T) { return reinterpret_cast<const char *>(T); }
__device__ __forceinline__ char *cbyte(__bf16 *T) { return reinterpret_cast<char *>(T); }

// Row operand: element [r0 + lane%32][16 ks + 8 (lane/32) + p].
__device__ __forceinline__ bf16x8 srow(const __bf16 *T, int r0, int ks, const Sw &z) {
    return *reinterpret_cast<const bf16x8 *>(cbyte(T) + z.row + r0 * PSB + 32 * ks);
}
// Row operand in the permuted k order of a fed-back accumulator: columns
// 16 ks + 4 (lane/32) .. +3 and 16 ks + 8 + 4 (lane/32) .. +3 of row lane%32.
__device__ __forceinline__ bf16x8 sperm(const __bf16 *T, int ks, const Sw &z) {
    const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(cbyte(T) + z.st + 32 * ks);
    const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(cbyte(T) + z.st + 32 * ks + 16);
    bf16x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
}
// Transposed operand: element [k0 + 8 (lane/32) + p][n0 + lane % 32].
__device__ __forceinline__ bf16x8 stro(const __bf16 *T, int k0, int n0, const Sw &z) {
    return lds8_tr(reinterpret_cast<const __bf16 *>(cbyte(T) + z.tr) + k0 * PS + n0, PS);
}
// Accumulators as bf16 rows of a [128][PS] tile: row 32 w + lane%32, columns
// 32 (x0 + j) + 8 g4 + 4 (lane/32) .. +3 per store.
template <int N>
__device__ __forceinline__ void dump_tile(__bf16 *T, int w, int x0, const f32x16 (&acc)[N], const Sw &z) {
    char *b = cbyte(T) + z.st + 32 * w * PSB;
#pragma unroll
    for (int j = 0; j < N; ++j)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            bf16x4 o;
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = (__bf16)acc[j][4 * g4 + e];
            *reinterpret_cast<bf16x4 *>(b + 2 * (32 * (x0 + j) + 8 * g4)) = o;
        }
}
// A 32 x 32 output block D[m][n] in registers (lane: n = lane % 32; register v:
// m = 8 (v / 4) + 4 (lane / 32) + v % 4) stored as bf16 rows of a [32][PS] tile at
// row n, columns col0 + m.
__device__ __forceinline__ void store_block(__bf16 *T, int col0, const f32x16 &acc, const Sw &z) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (__bf16)acc[4 * g4 + e];
        *reinterpret_cast<bf16x4 *>(cbyte(T) + z.st + 2 * (col0 + 8 * g4)) = o;
    }
}
// The same block read back as floats.
__device__ __forceinline__ void load_block(const __bf16 *T, int col0, f32x16 &acc, const Sw &z) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
        const bf16x4 x4 = *reinterpret_cast<const bf16x4 *>(cbyte(T) + z.st + 2 * (col0 + 8 * g4));
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[4 * g4 + e] = (float)x4[e];
    }
}
// Row operand of a padded score tile (row stride SSB): element [row][k0 + 8 (lane/32) + p].
__device__ __forceinline__ bf16x8 rd_row(const __bf16 *T, int stride, int row, int k0, int hl) {
    return lds8(T + row * stride + k0 + 8 * hl);
}
// The operand's eight k indices k0 + 8 (lane/32) + p scaled by f[p] (f points at entry k0 + 8 (lane/32)).
__device__ __forceinline__ bf16x8 scale_k(bf16x8 v, const float *f) {
    const float4 a = *reinterpret_cast<const float4 *>(f);
    const float4 b = *reinterpret_cast<const float4 *>(f + 4);
    const float d[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    bf16x8 r;
#pragma unroll
    for (int q = 0; q < 8; ++q) r[q] = (__bf16)((float)v[q] * d[q]);
    return r;
}

// ---- chunk staging ---------------------------------------------------------
// 32 rows x 128 bf16 (two 16-byte pieces per thread: rows tid/16 and tid/16 + 16,
// columns 8 (tid % 16)); rows at or past n read as zero.
struct Rows2 {
    uint4 r[2];
};
// (Rows past n are read from a clamped row of the chunk, which exists: the chunk
// starts inside the tensor, and then set to zero.)
__device__ __forceinline__ void load_rows(const __bf16 *base, size_t row_stride, int n, int tid, Rows2 &o) {
    const int r0 = tid >> 4, c8 = (tid & 15) * 8;
    const int last = max(n - 1, 0);
#pragma unroll
    for (int it = 0; it < 2; ++it) {
        const int r = r0 + 16 * it;
        const uint4 v = *reinterpret_cast<const uint4 *>(base + (size_t)min(r, last) * row_stride + c8);
        o.r[it] = r < n ? v : make_uint4(0, 0, 0, 0);
    }
}
__device__ __forceinline__ void store_rows(__bf16 *T, const Rows2 &o, const Sw &z) {
#pragma unroll
    for (int it = 0; it < 2; ++it) *reinterpret_cast<uint4 *>(cbyte(T) + 16 * PSB * it + z.cp) = o.r[it];
}

// 512-thread variant: one 16-byte piece per thread (row tid/16, columns 8 (tid % 16)).
// kOpq: the lane's offsets are recomputed at every call, opaque to the compiler (in the
// reverse walk, kept live across the chunk loop as 64-bit addresses they are spilled,
// and every reload waits for all of the wave's outstanding loads).
template <bool kOpq = false>
__device__ __forceinline__ void load_row1(const __bf16 *base, size_t row_stride, int n, int tid, uint4 &o) {
    if (kOpq) tid = opq(tid);
    const int r = tid >> 4, c8 = (tid & 15) * 8;
    const uint4 v = *reinterpret_cast<const uint4 *>(base + (size_t)min(r, max(n - 1, 0)) * row_stride + c8);
    o = r < n ? v : make_uint4(0, 0, 0, 0);
}
__device__ __forceinline__ void store_row1(__bf16 *T, const uint4 &o, const Sw &z) {
    *reinterpret_cast<uint4 *>(cbyte(T) + z.cp) = o;
}

// Per-token scalars of a chunk (lanes 0..31 of wave 0; zero elsewhere and past the
// sequence: no shift, no decay, no write).
struct Tok {
    float g, dl, be;
};
__device__ __forceinline__ void load_tok(const BwdParams &p, int b, int h, int t0, int Tb, int tid, Tok &k) {
    k.g = 0.f;
    k.dl = 0.f;
    k.be = 0.f;
    const int t = t0 + tid;
    if (tid < kC && t < Tb) {
        const size_t si = ((size_t)b * p.T + t) * p.H + h;
        k.g = p.log_alpha ? p.log_alpha[si] : 0.f;
        k.dl = p.delta[si];
        k.be = p.beta ? p.beta[si] : 1.f;
    }
}

// Chunk scalars in LDS.
struct Sc {
    float G[kC];      // chunk-local inclusive sums of log alpha
    float gam[kC];    // exp(G_r) (times the carried states' scale where a kernel keeps one)
    float rho[kC];    // exp(G_C - G_r) (likewise)
    float urev[kC];   // clock after token r over m, mod 1 (revolutions)
    float4 bw[kC];    // write-builder record: amplitude, urev, cos and sin of 2 pi urev
    float ea[kC];     // exp(G_r) and exp(-G_r): Gamma_rs = ea_r eb_s when every |G_r| <= 60
    float eb[kC];
    float ctl[4];     // lazily scaled kernels: [0] factor applied to the carried states
                      // before the chunk, [1] factor applied before their update; [3]: 1 when
                      // Gamma factors into ea, eb
};
constexpr int kScBytes = sizeof(Sc);
static_assert(kScBytes % 16 == 0, "scalar block");

// Wave 0: prefix sums of the chunk and the builder records; carry is the clock
// entering the chunk (reduced), advanced past it.  dec_amp: the write rows carry
// their right decay rho_r (A_dec).
//
// Lazily scaled carried states (kLazy: the forward walk's states, kLazyAdj: the
// reverse walk's adjoint states) are held as exp(Ls) times the registers, so that a
// chunk's decay changes Ls instead of every accumulator.  Forward walk: gam_r =
// exp(G_r + Ls) scales the inter-chunk terms and rho_s = exp(-Ls - G_s) the update
// operand, then Ls += G_C.  Reverse walk: rho_s = exp(G_C - G_s + Ls) scales the
// inter-chunk terms and gam_r = exp(G_r - G_C - Ls) the update operand, then Ls +=
// G_C.  When an exponent could leave [-60, 60] the chunk is eager: the registers
// are first multiplied by exp(Ls) (ctl[0]), Ls restarts at 0, gam and rho take their
// plain values and the registers are multiplied by exp(G_C) (ctl[1]) before the
// update.  Every thread tracks Ls itself from the same LDS values.
enum { kPlain = 0, kLazy = 1, kLazyAdj = 2 };
// kOpq: the lane's LDS offsets are recomputed at every call rather than kept (and
// spilled) across the reverse walk's chunk loop.
template <int kMode, bool kOpq = false>
__device__ __forceinline__ void chunk_scalars(Sc &s, int lane, int m, const Tok &k, double &carry, bool dec_amp,
                                              float Ls = 0.f) {
    if (kOpq) lane = opq(lane);
    const double inv_m = 1.0 / (double)m;
    const float G = wave_incl_scan(k.g);
    const double lam = carry + wave_incl_scan((double)k.dl);
    const float GC = lane63(G);
    const float gabs = wave_max_nonneg(fabsf(G));
    bool lazy = false;
    if (kMode != kPlain) lazy = fabsf(Ls) + (kMode == kLazyAdj ? 2.f : 1.f) * gabs <= 60.f;
    if (lane < kC) {
        s.G[lane] = G;
        s.ea[lane] = __expf(G);
        s.eb[lane] = __expf(-G);
        float gam = __expf(G), rho = __expf(GC - G);
        if (lazy) {
            if (kMode == kLazy) {
                gam = __expf(G + Ls);
                rho = __expf(-Ls - G);
            } else {
                rho = __expf(GC - G + Ls);
                gam = __expf(G - GC - Ls);
            }
        }
        s.gam[lane] = gam;
        s.rho[lane] = rho;
        const double q = lam * inv_m;
        const float u = (float)(q - floor(q));
        s.urev[lane] = u;
        float s1, c1;
        sincos_rev(u, &s1, &c1);
        s.bw[lane] = make_float4(k.be * sqrtf(2.f / (float)m) * (dec_amp ? rho : 1.f), u, c1, s1);
    }
    if (lane == 0) {
        s.ctl[0] = lazy ? 1.f : __expf(Ls);
        s.ctl[1] = lazy ? 1.f : __expf(GC);
        s.ctl[2] = lazy ? 1.f : 0.f;
        s.ctl[3] = gabs <= 60.f ? 1.f : 0.f;
    }
    carry = reduce_clock(lane63(lam), (double)m, inv_m);
}
// Every thread: the carried log scale after the chunk (from the chunk's control words).
__device__ __forceinline__ float next_scale(const Sc &s, float Ls) {
    return s.ctl[2] != 0.f ? Ls + s.G[kC - 1] : 0.f;
}

// Temporal write rows (Eq. app-temporal-writes) into a padded [32][PS] tile:
// amp_r [cos th_j, -sin th_j] on pair j (internal columns 2j-2, 2j-1), amp_r /
// sqrt 2 = beta_r / sqrt m on DC (126), 0 on 127.  Thread (row tid/16 + 16 it,
// q = tid % 16) fills columns 8q .. 8q+7 (pairs 4q+1 .. 4q+4); the phases advance
// by angle addition from a start reduced in revolutions.
template <int NTH = kNT>
__device__ __forceinline__ void build_A(const Sc &s, __bf16 *T, int tid, int m, const Sw &z) {
    const int q = tid & 15, r0 = tid >> 4;
    const int J = (m - 1) >> 1;
#pragma unroll 1
    for (int it = 0; it < kC * 16 / NTH; ++it) {
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
            if (jj == 3 && q == 15) {
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
        *reinterpret_cast<bf16x8 *>(cbyte(T) + 16 * PSB * it + z.cp) = a8;
    }
}

// (cos, sin) of 2 pi j urev for the eight pairs of a lane's 16 rows in wave w's
// 32-row block: pair e (registers 2e, 2e+1) is internal rows 32w + 8(e/2) + 4hl +
// 2(e%2) (+1), frequency j = 16w + 4(e/2) + 2hl + e%2 + 1.  Inactive pairs, DC and
// padding get (1, 0).
__device__ __forceinline__ int pair_freq(int w, int hl, int e) { return 16 * w + 4 * (e >> 1) + 2 * hl + (e & 1) + 1; }
__device__ __forceinline__ void lane_phases(float u, int w, int hl, int m, float (&c)[8], float (&s)[8]) {
    const int J = (m - 1) >> 1;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int j = pair_freq(w, hl, e);
        c[e] = 1.f;
        s[e] = 0.f;
        if (j <= J) sincos_rev(__builtin_amdgcn_fractf((float)j * u), &s[e], &c[e]);
    }
}
// acc <- mul U(SIGN lambda) acc on a lane's pairs (U(tau): rotation by +2 pi j tau / m
// of the (cos, sin) pair); DC and padding are multiplied by mul.
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
// Clock-gradient part of Z = U(+-lambda) y over a lane's active pairs:
// sum_j j (dZ_sin Z_cos - dZ_cos Z_sin); the gradient is +-(2 pi / m) times its
// sum over all pairs.
__device__ __forceinline__ float rot_part(const f32x16 &dz, const f32x16 &z, int w, int hl, int m) {
    const int J = (m - 1) >> 1;
    float acc = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int j = pair_freq(w, hl, e);
        if (j <= J) acc = fmaf((float)j, dz[2 * e + 1] * z[2 * e] - dz[2 * e] * z[2 * e + 1], acc);
    }
    return acc;
}

// One 16 x 16 block of a masked 32 x 32 score tile into S (bf16, [32][SSB]):
// D[mr][nr] = sum_k Am[mr][k] Bn[nr][k] over 128 columns for mr in m0 .. m0+15 and nr in
// n0 .. n0+15 (v_mfma_f32_16x16x32: lane nr = n0 + lane % 16, registers mr = m0 +
// 4 (lane / 16) + q), times Gamma and stored at S[nr][mr .. mr+3].  kLaneLater: nr is
// the later token (Gamma_{nr,mr}, mr <= nr); otherwise mr is (Gamma_{mr,nr}, mr >= nr).
// A block on the zero side of the diagonal is written as zeros without products.
// Gamma is ea eb when the chunk factors (every |G_r| <= 60), else exp of the difference.
template <bool kLaneLater>
__device__ __forceinline__ void score_block(const __bf16 *Am, int m0, const __bf16 *Bn, int n0, __bf16 *S,
                                            const Sc &sc, int lane) {
    const int l16 = lane & 15, g = lane >> 4;
    const int nr = n0 + l16, mb = m0 + 4 * g;
    bf16x4 o = bf16x4{};
    if (kLaneLater ? m0 <= n0 : m0 >= n0) {
        f32x4 acc = zero_acc4();
        const __bf16 *ap = Am + (m0 + l16) * PS + 8 * g;
        const __bf16 *bp = Bn + nr * PS + 8 * g;
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) acc = mma16(lds8(ap + 32 * ks), lds8(bp + 32 * ks), acc);
        const bool fac = uniform(sc.ctl[3]) != 0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int mr = mb + q;
            float gm;
            if (fac) gm = kLaneLater ? sc.ea[nr] * sc.eb[mr] : sc.ea[mr] * sc.eb[nr];
            else gm = __expf(kLaneLater ? sc.G[nr] - sc.G[mr] : sc.G[mr] - sc.G[nr]);
            o[q] = (__bf16)((kLaneLater ? mr <= nr : mr >= nr) ? acc[q] * gm : 0.f);
        }
    }
    *reinterpret_cast<bf16x4 *>(S + nr * SSB + mb) = o;
}

// Rows 0 .. nrows-1 of a [32][PS] tile to global memory (row r at dst + r row_stride):
// each group of sixteen lanes writes one whole 256-byte row.
__device__ __forceinline__ void copy_rows_out(const __bf16 *T, __bf16 *dst, size_t row_stride, int nrows, int tid,
                                              const Sw &z) {
    const int r0 = tid >> 4, c8 = (tid & 15) * 8;
#pragma unroll
    for (int it = 0; it < 2; ++it) {
        const int r = r0 + 16 * it;
        if (r < nrows)
            *reinterpret_cast<uint4 *>(dst + (size_t)r * row_stride + c8) =
                *reinterpret_cast<const uint4 *>(cbyte(T) + 16 * PSB * it + z.cp);
    }
}

// Per-token output row: token l32 of the chunk, columns 32w + 4hl + 8 g4 .. +3.
__device__ __forceinline__ void store_out(__bf16 *dst, const f32x16 &acc, bool live) {
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = (__bf16)(live ? acc[4 * g4 + e] : 0.f);
        *reinterpret_cast<bf16x4 *>(dst + 8 * g4) = o;
    }
}
// <the lane's part of a bf16 tile block (as store_block), accumulator>
__device__ __forceinline__ float dot_block(const __bf16 *T, int col0, const f32x16 &acc, const Sw &z) {
    float s = 0.f;
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4) {
        const bf16x4 x = *reinterpret_cast<const bf16x4 *>(cbyte(T) + z.st + 2 * (col0 + 8 * g4));
#pragma unroll
        for (int e = 0; e < 4; ++e) s = fmaf((float)x[e], acc[4 * g4 + e], s);
    }
    return s;
}

constexpr int kNT8 = 512;                           // eight-wave kernels

// Sum of a per-token scalar x[t * stride] over tokens [t_lo, t_hi) in double, over the
// whole workgroup (kNT8 threads, eight loads in flight per thread); every thread gets
// the sum.  red: kNT8 / 64 doubles of LDS.
__device__ __forceinline__ double block_token_sum(const float *x, int stride, int t_lo, int t_hi, double *red,
                                                  int tid) {
    double ds = 0.0;
    for (int t0 = t_lo; t0 < t_hi; t0 += 8 * kNT8) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int t = t0 + u * kNT8 + tid;
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
    for (int i = 0; i < kNT8 / 64; ++i) tot += red[i];
    __syncthreads();
    return tot;
}
// ---------------------------------------------------------------------------
// (1) group contributions to the forward states and the group's clock entry.
// Eight waves: wave w8 holds basis rows 32 (w8 % 4) .. and column blocks 2 (w8 / 4),
// 2 (w8 / 4) + 1 of both states (two waves per SIMD: the chunk loop waits on LDS and
// global loads, which the second wave covers).  The last group's contribution is
// never read (no walk starts after it), so its workgroups form only its clock entry
// and total log decay.
struct CLay {
    static constexpr int K = 0, V = kT32, A = 2 * kT32, SC = 3 * kT32, RED = SC + kScBytes;
    static constexpr int BYTES = RED + kNT8 / 64 * 8;
};
__global__ __launch_bounds__(kNT8, 1) void fwd_contrib_kernel(Args a) {
    using L = CLay;
    __shared__ __attribute__((aligned(256))) char smem[L::BYTES];
    const BwdParams &p = a.p;
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63, w8 = tid >> 6, wi = w8 & 3, xh = w8 >> 2;
    const int m = p.m;
    const int Tb = tokens_of(p, b);
    const int c_begin = g * p.cpg, c_end = min(c_begin + p.cpg, p.nc);
    Sc &sc = *lds_at<Sc>(smem, L::SC);
    __bf16 *Kt = lds_at<__bf16>(smem, L::K), *Vt = lds_at<__bf16>(smem, L::V), *At = lds_at<__bf16>(smem, L::A);
    // clock entering the group: clock0 plus every increment before it (double)
    double *red = lds_at<double>(smem, L::RED);
    const size_t tok0 = (size_t)b * p.T * p.H + h;
    double carry = reduce_clock((p.clock0 ? p.clock0[bh] : 0.0) +
                                          block_token_sum(p.delta + tok0, p.H, 0, min(c_begin * kC, Tb), red, tid),
                                      (double)m, 1.0 / (double)m);
    if (tid == 0) a.gclk[(size_t)bh * p.groups + g] = carry;
    if (g == p.groups - 1) {
        // the last group's contribution is not read: only its total log decay
        const double gs = p.log_alpha ? block_token_sum(p.log_alpha + tok0, p.H, min(c_begin * kC, Tb),
                                                        min(c_end * kC, Tb), red, tid)
                                      : 0.0;
        if (tid == 0) a.Gg[(size_t)bh * p.groups + g] = (float)gs;
        return;
    }
    const Sw z = make_sw(tid);
    f32x16 kacc[2], vacc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        kacc[j] = zero_acc();
        vacc[j] = zero_acc();
    }
    const size_t rs = (size_t)p.H * 128;
    const __bf16 *kin = static_cast<const __bf16 *>(p.k), *vin = static_cast<const __bf16 *>(p.v);
    uint4 rk, rv;
    Tok tk;
    auto prefetch = [&](int c) {
        const int t0 = c * kC, n = min(kC, Tb - t0);
        const size_t base = (((size_t)b * p.T + t0) * p.H + h) * 128;
        load_row1(kin + base, rs, n, tid, rk);
        load_row1(vin + base, rs, n, tid, rv);
        load_tok(p, b, h, t0, Tb, tid, tk);
    };
    if (c_begin < c_end) prefetch(c_begin);
    double gsum = 0.0;
    float Ls = 0.f;                                   // states: exp(Ls) x registers
    for (int c = c_begin; c < c_end; ++c) {
        store_row1(Kt, rk, z);
        store_row1(Vt, rv, z);
        if (w8 == 0) chunk_scalars<kLazy>(sc, lane, m, tk, carry, true, Ls);
        if (c + 1 < c_end) prefetch(c + 1);
        lds_barrier();
        build_A<kNT8>(sc, At, tid, m, z);
        gsum += (double)sc.G[kC - 1];
        {
            const float f = uniform(sc.ctl[0]) * uniform(sc.ctl[1]);
            if (f != 1.f) {
                scale_acc(kacc, f);
                scale_acc(vacc, f);
            }
        }
        Ls = next_scale(sc, Ls);
        lds_barrier();
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const bf16x8 ad = stro(At, 16 * ks, 32 * wi, z);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                kacc[j] = mma(stro(Kt, 16 * ks, 32 * (2 * xh + j), z), ad, kacc[j]);
                vacc[j] = mma(stro(Vt, 16 * ks, 32 * (2 * xh + j), z), ad, vacc[j]);
            }
        }
        lds_barrier();
    }
    scale_acc(kacc, __expf(Ls));
    scale_acc(vacc, __expf(Ls));
    float *E = a.Ef + ((size_t)bh * p.groups + g) * 2 * kSE;
    store_acc2(E, wi, 2 * xh, lane, kacc);
    store_acc2(E + kSE, wi, 2 * xh, lane, vacc);
    if (tid == 0) a.Gg[(size_t)bh * p.groups + g] = (float)gsum;
}

// ---------------------------------------------------------------------------
// (2) readout recomputation and its adjoint, per (sequence, chunk group).
// LDS: padded [32][PS] tiles Q, K, V, dO, A, X, W (later dp), dY (later scale dZ);
// [128][PS] tiles of the entering key state (bf16) and the readout matrix; three
// score tiles; chunk scalars; per-token reduction slots.
struct RLay {
    static constexpr int Q = 0, K = kT32, V = 2 * kT32, O = 3 * kT32, A = 4 * kT32;
    static constexpr int X = 5 * kT32, W = 6 * kT32, Y = 7 * kT32;
    static constexpr int KB = 8 * kT32, MZ = KB + kT128;
    static constexpr int S1 = MZ + kT128, S2 = S1 + kTS, S3 = S2 + kTS;
    static constexpr int SC = S3 + kTS;
    static constexpr int R1 = SC + kScBytes, R2 = R1 + 4 * kC * 8, R3 = R2 + 4 * kC * 4;
    static constexpr int BYTES = R3 + 4 * kC * 8;
    static_assert(BYTES <= 160 * 1024, "one workgroup per compute unit");
};
__global__ __launch_bounds__(kNT, 1) void readout_kernel(Args a) {
    using L = RLay;
    __shared__ __attribute__((aligned(256))) char smem[L::BYTES];
    const BwdParams &p = a.p;
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31, hl = lane >> 5, h4 = 4 * hl;
    const int m = p.m;
    const int Tb = tokens_of(p, b);
    const int c_begin = g * p.cpg, c_end = min(c_begin + p.cpg, p.nc);
    Sc &sc = *lds_at<Sc>(smem, L::SC);
    __bf16 *Qt = lds_at<__bf16>(smem, L::Q), *Kt = lds_at<__bf16>(smem, L::K), *Vt = lds_at<__bf16>(smem, L::V);
    __bf16 *Ot = lds_at<__bf16>(smem, L::O), *At = lds_at<__bf16>(smem, L::A), *Xt = lds_at<__bf16>(smem, L::X);
    __bf16 *Wt = lds_at<__bf16>(smem, L::W), *Yt = lds_at<__bf16>(smem, L::Y);
    __bf16 *KB = lds_at<__bf16>(smem, L::KB), *MZ = lds_at<__bf16>(smem, L::MZ);
    __bf16 *S1 = lds_at<__bf16>(smem, L::S1), *S2 = lds_at<__bf16>(smem, L::S2), *S3 = lds_at<__bf16>(smem, L::S3);
    float2 *red1 = lds_at<float2>(smem, L::R1);
    float *red2 = lds_at<float>(smem, L::R2);
    float2 *red3 = lds_at<float2>(smem, L::R3);
    const Sw z = make_sw(tid);
    const float scale = p.scale;
    const float zs = scale * 1.4426950408889634f;   // the LDS readout matrix is zs M
    const float inv_zs = 1.f / zs;

    {
        const __bf16 *Mh = a.Mz + (size_t)h * 128 * 128;
#pragma unroll
        for (int it = 0; it < 8; ++it) {
            const int e = it * kNT + tid, row = e >> 4, c0 = (e & 15) * 8;
            *reinterpret_cast<uint4 *>(cbyte(MZ) + 16 * PSB * it + z.cp) =
                *reinterpret_cast<const uint4 *>(Mh + row * 128 + c0);
        }
    }
    f32x16 kacc[4], vacc[4], macc[4];
    {
        // state entering the group: (K0, V0) decayed through the earlier groups, plus each
        // earlier group's contribution decayed through the groups after it
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            kacc[x] = zero_acc();
            vacc[x] = zero_acc();
            macc[x] = zero_acc();
        }
        const float *Gg = a.Gg + (size_t)bh * p.groups;
        float tail = 0.f;                         // log decay of groups q+1 .. g-1
        for (int q = g - 1; q >= 0; --q) {
            const float f = __expf(tail);
            const float *E = a.Ef + ((size_t)bh * p.groups + q) * 2 * kSE;
            add_dump_state(kacc, E, f, w, 0, lane);
            add_dump_state(vacc, E + kSE, f, w, 0, lane);
            tail += Gg[q];
        }
        const size_t sb = (size_t)bh * kStoreRows * 128;
        if (p.K0) add_abi_state(kacc, p.K0 + sb, __expf(tail), w, 0, lane, m);
        if (p.V0) add_abi_state(vacc, p.V0 + sb, __expf(tail), w, 0, lane, m);
    }
    double carry = a.gclk[(size_t)bh * p.groups + g];
    const size_t rs = (size_t)p.H * 128;
    const __bf16 *qin = static_cast<const __bf16 *>(p.q), *kin = static_cast<const __bf16 *>(p.k);
    const __bf16 *vin = static_cast<const __bf16 *>(p.v), *oin = static_cast<const __bf16 *>(p.dout);
    __bf16 *gq = static_cast<__bf16 *>(p.gq);
    Rows2 pq, pk, pv, po;
    Tok tk;
    auto prefetch = [&](int c) {
        const int t0 = c * kC, n = min(kC, Tb - t0);
        const size_t base = (((size_t)b * p.T + t0) * p.H + h) * 128;
        load_rows(qin + base, rs, n, tid, pq);
        load_rows(kin + base, rs, n, tid, pk);
        load_rows(vin + base, rs, n, tid, pv);
        load_rows(oin + base, rs, n, tid, po);
        load_tok(p, b, h, t0, Tb, tid, tk);
    };
    if (c_begin < c_end) prefetch(c_begin);

    float Ls = 0.f;                                   // carried states: exp(Ls) x registers
    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * kC, n = min(kC, Tb - t0);
        // -- A: stage the chunk and its scalars; entering key state in bf16; writes
        store_rows(Qt, pq, z);
        store_rows(Kt, pk, z);
        store_rows(Vt, pv, z);
        store_rows(Ot, po, z);
        if (w == 0) {
            if (lane == 0) a.cclk[(size_t)bh * p.nc + c] = carry;
            chunk_scalars<kLazy>(sc, lane, m, tk, carry, false, Ls);
        }
        lds_barrier();
        {
            const float pre = uniform(sc.ctl[0]);
            if (pre != 1.f) {
                scale_acc(kacc, pre);
                scale_acc(vacc, pre);
            }
        }
        dump_tile(KB, w, 0, kacc, z);
        build_A(sc, At, tid, m, z);
        lds_barrier();
        // -- B: scores, inter-chunk terms of p and du, state update; prefetch the next chunk
        const float gr = sc.gam[l32];
        // S1[r][s] = Gamma (q_r . k_s), S2[r][s] = Gamma (do_r . v_s): wave w forms the 16 x 16
        // block (r block w / 2, s block w % 2) of each
        score_block<true>(Kt, 16 * (w & 1), Qt, 16 * (w >> 1), S1, sc, lane);
        score_block<true>(Vt, 16 * (w & 1), Ot, 16 * (w >> 1), S2, sc, lane);
        f32x16 pacc = zero_acc(), dacc = zero_acc();
        {
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                pacc = mma(srow(KB, 32 * w, ks, z), srow(Qt, 0, ks, z), pacc);
                dacc = mma(acc_to_operand(vacc[ks >> 1], ks & 1), sperm(Ot, ks, z), dacc);
            }
        }
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            pacc[v] *= gr;
            dacc[v] *= gr;
        }
        {
            const float post = uniform(sc.ctl[1]);
            if (post != 1.f) {
                scale_acc(kacc, post);
                scale_acc(vacc, post);
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 ad = scale_k(stro(At, 16 * ks, 32 * w, z), sc.rho + 16 * ks + 8 * hl);
#pragma unroll
                for (int x = 0; x < 4; ++x) {
                    kacc[x] = mma(stro(Kt, 16 * ks, 32 * x, z), ad, kacc[x]);
                    vacc[x] = mma(stro(Vt, 16 * ks, 32 * x, z), ad, vacc[x]);
                }
            }
        }
        Ls = next_scale(sc, Ls);
        lds_barrier();
        // -- C: intra-chunk terms; X = U(lambda) p (scale folded into M); slot logits
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const bf16x8 at = stro(At, 16 * ks, 32 * w, z);
            pacc = mma(at, rd_row(S1, SSB, l32, 16 * ks, hl), pacc);
            dacc = mma(at, rd_row(S2, SSB, l32, 16 * ks, hl), dacc);
        }
        float pc[8], ps[8];
        lane_phases(opqf(sc.urev[l32]), w, hl, m, pc, ps);
        rotate<1>(pacc, pc, ps, 1.f);                 // X' = U(lambda) p;  X = scale X'
        {
            f32x16 xs = pacc;
            if (w == 3 && hl == 1) xs[15] = 1.f;      // column 127 = 1: inactive slots get the mask logit
            store_block(Xt, 32 * w, xs, z);
        }
        lds_barrier();
        f32x16 wr = zero_acc();                       // slot logits (log2 units), then W
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) wr = mma(srow(MZ, 32 * w, ks, z), srow(Xt, 0, ks, z), wr);
        {
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
            if (hl == 0) red1[w * kC + l32] = make_float2(mx, sm);
            lds_barrier();
            float2 pr[4];
#pragma unroll
            for (int x = 0; x < 4; ++x) pr[x] = red1[x * kC + l32];
            const float M = fmaxf(fmaxf(pr[0].x, pr[1].x), fmaxf(pr[2].x, pr[3].x));
            float Lsum = 0.f;
#pragma unroll
            for (int x = 0; x < 4; ++x) Lsum += pr[x].y * __builtin_amdgcn_exp2f(pr[x].x - M);
            const float f = __builtin_amdgcn_exp2f(mx - M) / Lsum;
#pragma unroll
            for (int v = 0; v < 16; ++v) wr[v] *= f;
        }
        store_block(Wt, 32 * w, wr, z);
        {
            f32x16 dy = dacc;                          // dY = U(lambda) du
            rotate<1>(dy, pc, ps, 1.f);
            if (w == 3 && hl == 1) dy[15] = 0.f;
            store_block(Yt, 32 * w, dy, z);
        }
        lds_barrier();
        // -- D: u = U(-lambda) M^T W; dW = M dY; dM += W dY^T
        float tsum, tclk;
        float qc[8], qs[8];                            // the phases again (short live ranges)
        lane_phases(opqf(sc.urev[l32]), w, hl, m, qc, qs);
        {
            f32x16 ya = zero_acc();
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) ya = mma(stro(MZ, 16 * ks, 32 * w, z), srow(Wt, 0, ks, z), ya);
            rotate<-1>(ya, qc, qs, inv_zs);
            store_block(Ot, 32 * w, ya, z);            // u, staged in dO's place
            float ud = 0.f;
#pragma unroll
            for (int v = 0; v < 16; ++v) ud = fmaf(ya[v], dacc[v], ud);
            tsum = ud;
            tclk = -rot_part(dacc, ya, w, hl, m);
        }
        f32x16 dw = zero_acc();
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) dw = mma(srow(MZ, 32 * w, ks, z), srow(Yt, 0, ks, z), dw);
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const bf16x8 wa = stro(Wt, 16 * ks, 32 * w, z);
#pragma unroll
            for (int x = 0; x < 4; ++x) macc[x] = mma(wa, stro(Yt, 16 * ks, 32 * x, z), macc[x]);
        }
        {
            float sw = 0.f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                dw[v] *= inv_zs;
                sw = fmaf(wr[v], dw[v], sw);
            }
            sw += __shfl_xor(sw, 32);
            if (hl == 0) red2[w * kC + l32] = sw;
        }
        lds_barrier();
        copy_rows_out(Ot, a.U + ((size_t)bh * p.Tpad + t0) * 128, 128, kC, tid, z);
        {
            const float sW = (red2[l32] + red2[kC + l32]) + (red2[2 * kC + l32] + red2[3 * kC + l32]);
            // dZ = W (.) (dW - <W, dW>), stored times scale in the dY tile's place
#pragma unroll
            for (int v = 0; v < 16; ++v) dw[v] = wr[v] * (dw[v] - sW) * scale;
            store_block(Yt, 32 * w, dw, z);
        }
        lds_barrier();
        // -- E: dX = M^T dZ; dM += dZ X^T; dp = scale U(-lambda) dX; prefetch the next chunk
        if (c + 1 < c_end) prefetch(c + 1);
        {
            f32x16 xa = zero_acc();
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) xa = mma(stro(MZ, 16 * ks, 32 * w, z), srow(Yt, 0, ks, z), xa);
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 za = stro(Yt, 16 * ks, 32 * w, z);
#pragma unroll
                for (int x = 0; x < 4; ++x) macc[x] = mma(za, stro(Xt, 16 * ks, 32 * x, z), macc[x]);
            }
            const float fx = inv_zs / scale;
#pragma unroll
            for (int v = 0; v < 16; ++v) xa[v] *= fx;
            f32x16 xt;                                 // X' from its tile
            load_block(Xt, 32 * w, xt, z);
            tclk += scale * rot_part(xa, xt, w, hl, m);
            rotate<-1>(xa, qc, qs, scale);
            store_block(Wt, 32 * w, xa, z);
        }
        lds_barrier();
        copy_rows_out(Wt, a.dP + ((size_t)bh * p.Tpad + t0) * 128, 128, kC, tid, z);
        // -- F: dq = gamma (.) dP Kbar + (dP A^T (.) Gamma) K
        score_block<true>(At, 16 * (w & 1), Wt, 16 * (w >> 1), S3, sc, lane);   // S3[r][s] = Gamma (dp_r . a_s)
        f32x16 qa = zero_acc();
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) qa = mma(stro(KB, 16 * ks, 32 * w, z), srow(Wt, 0, ks, z), qa);
#pragma unroll
        for (int v = 0; v < 16; ++v) qa[v] *= gr;
        lds_barrier();
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) qa = mma(stro(Kt, 16 * ks, 32 * w, z), rd_row(S3, SSB, l32, 16 * ks, hl), qa);
        tsum += dot_block(Qt, 32 * w, qa, z);
        if (l32 >= n) qa = zero_acc();                 // rows past the sequence: dq = 0
        store_block(Xt, 32 * w, qa, z);                // dq, staged in X's place
        tsum += __shfl_xor(tsum, 32);
        tclk += __shfl_xor(tclk, 32);
        if (hl == 0) red3[w * kC + l32] = make_float2(tsum, tclk);
        lds_barrier();
        copy_rows_out(Xt, gq + (((size_t)b * p.T + t0) * p.H + h) * 128, (size_t)p.H * 128, min(kC, p.T - t0), tid, z);
        if (w == 0 && lane < kC) {
            float s1 = 0.f, s2 = 0.f;
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                const float2 v = red3[x * kC + lane];
                s1 += v.x;
                s2 += v.y;
            }
            const size_t ti = (size_t)bh * p.Tpad + t0 + lane;
            const bool lv = lane < n;
            p.udu[ti] = lv ? s1 : 0.f;
            p.dlam[ti] = lv ? s2 * (kTwoPi / (float)m) : 0.f;
        }
    }
    // the last group holds the final states: the loss <dK_T, Kbar_T> + <dV_T, Vbar_T>
    if (g == p.groups - 1) {
        const size_t sb = (size_t)bh * kStoreRows * 128;
        float t = __expf(Ls) * (dot_abi_state(kacc, p.dK_T ? p.dK_T + sb : nullptr, w, 0, lane, m) +
                                dot_abi_state(vacc, p.dV_T ? p.dV_T + sb : nullptr, w, 0, lane, m));
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) t += __shfl_xor(t, o);
        if (lane == 0) {
            p.fin[(size_t)bh * kCombBlocks + w] = t;
            p.fin[(size_t)bh * kCombBlocks + 4 + w] = 0.f;
        }
    }
    // the group's dM in paper column order
    float *dMo = p.dMp + ((size_t)bh * p.groups + g) * 128 * 128;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        const int col = paper_row(32 * x + l32);
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int j = 32 * w + 8 * (v >> 2) + h4 + (v & 3);
            dMo[j * 128 + col] = macc[x][v];
        }
    }
}

// ---------------------------------------------------------------------------
// (3) group contributions to the adjoint states (reverse over the group's chunks,
// zero adjoint at its end): DK <- exp(G_C) DK + (gamma (.) dP)^T Q, DV likewise
// with (gamma (.) U)^T dO.  Eight waves, split as in (1).
struct ALay {
    static constexpr int Q = 0, O = kT32, U = 2 * kT32, P = 3 * kT32, SC = 4 * kT32;
    static constexpr int BYTES = SC + kScBytes;
};
__global__ __launch_bounds__(kNT8, 1) void adj_contrib_kernel(Args a) {
    using L = ALay;
    __shared__ __attribute__((aligned(256))) char smem[L::BYTES];
    const BwdParams &p = a.p;
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H;
    if (g == 0) return;                               // the first group's contribution is not read
    const int tid = threadIdx.x, lane = tid & 63, w8 = tid >> 6, wi = w8 & 3, xh = w8 >> 2, hl = lane >> 5;
    const int Tb = tokens_of(p, b);
    const int c_begin = g * p.cpg, c_end = min(c_begin + p.cpg, p.nc);
    Sc &sc = *lds_at<Sc>(smem, L::SC);
    __bf16 *Qt = lds_at<__bf16>(smem, L::Q), *Ot = lds_at<__bf16>(smem, L::O);
    __bf16 *Ut = lds_at<__bf16>(smem, L::U), *Pt = lds_at<__bf16>(smem, L::P);
    const Sw z = make_sw(tid);
    f32x16 kacc[2], vacc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        kacc[j] = zero_acc();
        vacc[j] = zero_acc();
    }
    const size_t rs = (size_t)p.H * 128;
    const __bf16 *qin = static_cast<const __bf16 *>(p.q), *oin = static_cast<const __bf16 *>(p.dout);
    uint4 rq, ro, ru, rp;
    Tok tk;
    auto prefetch = [&](int c) {
        const int t0 = c * kC, n = min(kC, Tb - t0);
        const size_t base = (((size_t)b * p.T + t0) * p.H + h) * 128;
        const size_t wb = ((size_t)bh * p.Tpad + t0) * 128;
        load_row1(qin + base, rs, n, tid, rq);
        load_row1(oin + base, rs, n, tid, ro);
        load_row1(a.U + wb, 128, kC, tid, ru);
        load_row1(a.dP + wb, 128, kC, tid, rp);
        tk.g = 0.f;
        tk.dl = 0.f;
        tk.be = 0.f;
        if (tid < kC && t0 + tid < Tb && p.log_alpha) tk.g = p.log_alpha[((size_t)b * p.T + t0 + tid) * p.H + h];
    };
    if (c_begin < c_end) prefetch(c_end - 1);
    float Ls = 0.f;                                   // adjoint states: exp(Ls) x registers
    double clk = 0.0;                                 // (the clock is not used here)
    for (int c = c_end - 1; c >= c_begin; --c) {
        store_row1(Qt, rq, z);
        store_row1(Ot, ro, z);
        store_row1(Ut, ru, z);
        store_row1(Pt, rp, z);
        if (w8 == 0) chunk_scalars<kLazyAdj>(sc, lane, 3, tk, clk, false, Ls);
        if (c > c_begin) prefetch(c - 1);
        lds_barrier();
        {
            const float f = uniform(sc.ctl[0]) * uniform(sc.ctl[1]);
            if (f != 1.f) {
                scale_acc(kacc, f);
                scale_acc(vacc, f);
            }
        }
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const float *gk = sc.gam + 16 * ks + 8 * hl;
            const bf16x8 bp = scale_k(stro(Pt, 16 * ks, 32 * wi, z), gk);
            const bf16x8 bu = scale_k(stro(Ut, 16 * ks, 32 * wi, z), gk);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                kacc[j] = mma(stro(Qt, 16 * ks, 32 * (2 * xh + j), z), bp, kacc[j]);
                vacc[j] = mma(stro(Ot, 16 * ks, 32 * (2 * xh + j), z), bu, vacc[j]);
            }
        }
        Ls = next_scale(sc, Ls);
        lds_barrier();
    }
    scale_acc(kacc, __expf(Ls));
    scale_acc(vacc, __expf(Ls));
    float *E = a.Ea + ((size_t)bh * p.groups + g) * 2 * kSE;
    store_acc2(E, wi, 2 * xh, lane, kacc);
    store_acc2(E + kSE, wi, 2 * xh, lane, vacc);
}

// ---------------------------------------------------------------------------
// (4) token gradients, per (sequence, chunk group), chunks in reverse.
// Eight waves, two per SIMD: wave w8 holds column blocks 2 (w8 / 4), 2 (w8 / 4) + 1 of
// both adjoint states for the basis rows 32 (w8 % 4) ..; waves 0-3 form da for basis
// rows 32 (w8 % 4) .. and its per-token terms (dbeta, the write's clock term), waves
// 4-7 dk and dv for columns 32 (w8 % 4) .. and <k, dk> + <v, dv>.
// LDS: padded [32][PS] tiles Q, K, V, dO, U, dP, A; [128][PS] tiles of the adjoint
// states at the chunk's end (bf16; their first 32 rows then stage dk and dv); four
// score tiles stored [s][r]; scalars; per-token reduction slots.
struct GLay {
    static constexpr int Q = 0, K = kT32, V = 2 * kT32, O = 3 * kT32, U = 4 * kT32, P = 5 * kT32, A = 6 * kT32;
    static constexpr int DK = 7 * kT32, DV = DK + kT128;
    static constexpr int T1 = DV + kT128, T2 = T1 + kTS, T3 = T2 + kTS, T4 = T3 + kTS;
    static constexpr int SC = T4 + kTS, RED = SC + kScBytes;
    static constexpr int BYTES = RED + 8 * kC * 16;
    static_assert(BYTES <= 160 * 1024, "one workgroup per compute unit");
};
__global__ __launch_bounds__(kNT8, 1) void grad_kernel(Args a) {
    using L = GLay;
    __shared__ __attribute__((aligned(256))) char smem[L::BYTES];
    const BwdParams &p = a.p;
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63, w8 = tid >> 6, wi = w8 & 3, xh = w8 >> 2;
    const int l32 = lane & 31, hl = lane >> 5;
    const int m = p.m;
    const int Tb = tokens_of(p, b);
    const int c_begin = g * p.cpg, c_end = min(c_begin + p.cpg, p.nc);
    Sc &sc = *lds_at<Sc>(smem, L::SC);
    __bf16 *Qt = lds_at<__bf16>(smem, L::Q), *Kt = lds_at<__bf16>(smem, L::K), *Vt = lds_at<__bf16>(smem, L::V);
    __bf16 *Ot = lds_at<__bf16>(smem, L::O), *Ut = lds_at<__bf16>(smem, L::U), *Pt = lds_at<__bf16>(smem, L::P);
    __bf16 *At = lds_at<__bf16>(smem, L::A), *DKt = lds_at<__bf16>(smem, L::DK), *DVt = lds_at<__bf16>(smem, L::DV);
    __bf16 *T1 = lds_at<__bf16>(smem, L::T1), *T2 = lds_at<__bf16>(smem, L::T2);
    __bf16 *T3 = lds_at<__bf16>(smem, L::T3), *T4 = lds_at<__bf16>(smem, L::T4);
    float4 *red = lds_at<float4>(smem, L::RED);
    const Sw z = make_sw(tid);
    const int x0 = 2 * xh;                          // this wave's column blocks x0, x0 + 1
    f32x16 kacc[2], vacc[2];
    {
        // adjoint at the group's end: (dK_T, dV_T) decayed through the later groups, plus
        // each later group's own contribution decayed through the groups before it
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            kacc[j] = zero_acc();
            vacc[j] = zero_acc();
        }
        const float *Gg = a.Gg + (size_t)bh * p.groups;
        float head = 0.f;                         // log decay of groups g+1 .. q-1
        for (int q = g + 1; q < p.groups; ++q) {
            const float f = __expf(head);
            const float *E = a.Ea + ((size_t)bh * p.groups + q) * 2 * kSE;
            add_dump_state(kacc, E, f, wi, x0, lane);
            add_dump_state(vacc, E + kSE, f, wi, x0, lane);
            head += Gg[q];
        }
        const size_t sb = (size_t)bh * kStoreRows * 128;
        if (p.dK_T) add_abi_state(kacc, p.dK_T + sb, __expf(head), wi, x0, lane, m);
        if (p.dV_T) add_abi_state(vacc, p.dV_T + sb, __expf(head), wi, x0, lane, m);
    }
    const size_t rs = (size_t)p.H * 128;
    const __bf16 *qin = static_cast<const __bf16 *>(p.q), *kin = static_cast<const __bf16 *>(p.k);
    const __bf16 *vin = static_cast<const __bf16 *>(p.v), *oin = static_cast<const __bf16 *>(p.dout);
    __bf16 *gk = static_cast<__bf16 *>(p.gk), *gv = static_cast<__bf16 *>(p.gv);
    uint4 pq, pk, pv, po, pu, pp;
    Tok tk;
    double pclk = 0.0;
    float pudu = 0.f, pdl = 0.f;
    auto prefetch = [&](int c) {
        const int t0 = c * kC, n = min(kC, Tb - t0);
        const size_t base = (((size_t)b * p.T + t0) * p.H + h) * 128;
        const size_t wb = ((size_t)bh * p.Tpad + t0) * 128;
        load_row1<true>(qin + base, rs, n, tid, pq);
        load_row1<true>(kin + base, rs, n, tid, pk);
        load_row1<true>(vin + base, rs, n, tid, pv);
        load_row1<true>(oin + base, rs, n, tid, po);
        load_row1<true>(a.U + wb, 128, kC, tid, pu);
        load_row1<true>(a.dP + wb, 128, kC, tid, pp);
        load_tok(p, b, h, t0, Tb, tid, tk);
        // the readout walk's per-token terms and the chunk's entering clock
        pclk = a.cclk[(size_t)bh * p.nc + c];
        pudu = 0.f;
        pdl = 0.f;
        if (tid < kC) {
            pudu = p.udu[(size_t)bh * p.Tpad + t0 + tid];
            pdl = p.dlam[(size_t)bh * p.Tpad + t0 + tid];
        }
    };
    if (c_begin < c_end) prefetch(c_end - 1);
    const float sq2m = sqrtf(2.f / (float)m), dcw = 1.f / sqrtf((float)m);
    const int J = (m - 1) >> 1;

    float Ls = 0.f;                                   // adjoint states: exp(Ls) x registers
    for (int c = c_end - 1; c >= c_begin; --c) {
        const int t0 = c * kC, n = min(kC, Tb - t0);
        // -- A: stage, scalars (clock entering the chunk from the forward walk), adjoint
        //    states at the chunk's end in bf16, writes
        store_row1(Qt, pq, z);
        store_row1(Kt, pk, z);
        store_row1(Vt, pv, z);
        store_row1(Ot, po, z);
        store_row1(Ut, pu, z);
        store_row1(Pt, pp, z);
        const float cur_udu = pudu, cur_dl = pdl;    // this chunk's (the prefetch moves on)
        if (w8 == 0) {
            double carry = pclk;
            chunk_scalars<kLazyAdj, true>(sc, lane, m, tk, carry, false, Ls);
        }
        lds_barrier();
        {
            const float pre = uniform(sc.ctl[0]);
            if (pre != 1.f) {
                scale_acc(kacc, pre);
                scale_acc(vacc, pre);
            }
        }
        dump_tile(DKt, wi, x0, kacc, z);
        dump_tile(DVt, wi, x0, vacc, z);
        build_A<kNT8>(sc, At, tid, m, z);
        lds_barrier();
        // -- B: score tiles (stored [s][r]; the 16 x 16 block (s block wi / 2, r block wi % 2)
        //    of T1, T2 on waves 0-3 and of T3, T4 on waves 4-7); inter-chunk terms of da
        //    (waves 0-3) or of dk, dv (waves 4-7); adjoint update; prefetch
        const float rs_ = sc.rho[l32];
        f32x16 r0 = zero_acc(), r1 = zero_acc();     // da, or dk and dv
        {
            const int m0 = 16 * (wi & 1), n0 = 16 * (wi >> 1);
            if (xh == 0) {
                score_block<false>(Qt, m0, Kt, n0, T1, sc, lane);   // T1[s][r] = Gamma (q_r . k_s)
                score_block<false>(Ot, m0, Vt, n0, T2, sc, lane);   // T2[s][r] = Gamma (do_r . v_s)
            } else {
                score_block<false>(Pt, m0, At, n0, T3, sc, lane);   // T3[s][r] = Gamma (dp_r . a_s)
                score_block<false>(Ut, m0, At, n0, T4, sc, lane);   // T4[s][r] = Gamma (u_r . a_s)
            }
        }
        if (xh == 0) {
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                r0 = mma(srow(DKt, 32 * wi, ks, z), srow(Kt, 0, ks, z), r0);
                r0 = mma(srow(DVt, 32 * wi, ks, z), srow(Vt, 0, ks, z), r0);
            }
#pragma unroll
            for (int v = 0; v < 16; ++v) r0[v] *= rs_;
        } else {
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                const bf16x8 ar = srow(At, 0, ks, z);
                r0 = mma(stro(DKt, 16 * ks, 32 * wi, z), ar, r0);
                r1 = mma(stro(DVt, 16 * ks, 32 * wi, z), ar, r1);
            }
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                r0[v] *= rs_;
                r1[v] *= rs_;
            }
        }
        {
            const float post = uniform(sc.ctl[1]);
            if (post != 1.f) {
                scale_acc(kacc, post);
                scale_acc(vacc, post);
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const float *gk8 = sc.gam + 16 * ks + 8 * hl;
                const bf16x8 bp = scale_k(stro(Pt, 16 * ks, 32 * wi, z), gk8);
                const bf16x8 bu = scale_k(stro(Ut, 16 * ks, 32 * wi, z), gk8);
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    kacc[j] = mma(stro(Qt, 16 * ks, 32 * (x0 + j), z), bp, kacc[j]);
                    vacc[j] = mma(stro(Ot, 16 * ks, 32 * (x0 + j), z), bu, vacc[j]);
                }
            }
        }
        Ls = next_scale(sc, Ls);
        if (c > c_begin) prefetch(c - 1);
        lds_barrier();
        // -- C: intra-chunk terms and the per-token terms
        float t1 = 0.f, t2 = 0.f, t3 = 0.f;
        if (xh == 0) {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                r0 = mma(stro(Pt, 16 * ks, 32 * wi, z), rd_row(T1, SSB, l32, 16 * ks, hl), r0);
                r0 = mma(stro(Ut, 16 * ks, 32 * wi, z), rd_row(T2, SSB, l32, 16 * ks, hl), r0);
            }
            // dbeta = <da, U(-lambda) b>; clock term of a = beta U(-lambda) b
            float pc[8], ps[8];
            lane_phases(sc.urev[l32], wi, hl, m, pc, ps);
            const float amp = sc.bw[l32].x;            // beta sqrt(2/m)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int j = pair_freq(wi, hl, e);
                if (j <= J) {
                    t2 = fmaf(sq2m, pc[e] * r0[2 * e] - ps[e] * r0[2 * e + 1], t2);
                    // j (da_sin a_cos - da_cos a_sin) with a_cos = amp c, a_sin = -amp s
                    t3 = fmaf((float)j * amp, r0[2 * e + 1] * pc[e] + r0[2 * e] * ps[e], t3);
                }
            }
            if (wi == 3 && hl == 1) t2 = fmaf(dcw, r0[14], t2);   // DC (internal row 126)
        } else {
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                r0 = mma(stro(Qt, 16 * ks, 32 * wi, z), rd_row(T3, SSB, l32, 16 * ks, hl), r0);
                r1 = mma(stro(Ot, 16 * ks, 32 * wi, z), rd_row(T4, SSB, l32, 16 * ks, hl), r1);
            }
            t1 = dot_block(Kt, 32 * wi, r0, z) + dot_block(Vt, 32 * wi, r1, z);
            if (l32 >= n) {                            // rows past the sequence: dk = dv = 0
                r0 = zero_acc();
                r1 = zero_acc();
            }
            store_block(DKt, 32 * wi, r0, z);          // dk, dv staged in the first rows of the
            store_block(DVt, 32 * wi, r1, z);          // adjoint-state tiles (read only in B)
        }
        t1 += __shfl_xor(t1, 32);
        t2 += __shfl_xor(t2, 32);
        t3 += __shfl_xor(t3, 32);
        if (hl == 0) red[w8 * kC + l32] = make_float4(t1, t2, t3, 0.f);
        lds_barrier();
        {
            const size_t go = (((size_t)b * p.T + t0) * p.H + h) * 128;
            const int nr = min(kC, p.T - t0);
            if (tid < 256) copy_rows_out(DKt, gk + go, (size_t)p.H * 128, nr, tid, z);
            else copy_rows_out(DVt, gv + go, (size_t)p.H * 128, nr, tid - 256, make_sw(tid - 256));
        }
        if (w8 == 0 && lane < kC) {
            float s1 = 0.f, s2 = 0.f, s3 = 0.f;
#pragma unroll
            for (int x = 0; x < 8; ++x) {
                const float4 v = red[x * kC + lane];
                s1 += v.x;
                s2 += v.y;
                s3 += v.z;
            }
            const size_t ti = (size_t)bh * p.Tpad + t0 + lane;
            const bool lv = lane < n;
            p.dG[ti] = lv ? cur_udu - s1 : 0.f;
            p.dlam[ti] = lv ? cur_dl - s3 * (kTwoPi / (float)m) : 0.f;
            if (p.gbeta && t0 + lane < p.T) p.gbeta[((size_t)b * p.T + t0 + lane) * p.H + h] = lv ? s2 : 0.f;
        }
    }
    // the first group ends at the sequence start: its adjoints are dK0, dV0
    if (g == 0) {
        const size_t sb = (size_t)bh * kStoreRows * 128;
        const float f = __expf(Ls);
        if (p.gK0) store_abi_state(p.gK0 + sb, kacc, f, wi, x0, lane, m);
        if (p.gV0) store_abi_state(p.gV0 + sb, vacc, f, wi, x0, lane, m);
    }
}

}  // namespace

int bwd_mfma_auto_groups(int B, int T, int H) {
    const int nc = (T + kC - 1) / kC;
    const int BH = B * H;
    int g = (256 + BH - 1) / BH;
    if (g > nc) g = nc;
    return g < 1 ? 1 : g;
}

// Layout (each piece 256-byte aligned): Mz, Ef, Ea, Gg, gclk, cclk, U, dP, udu, dlam,
// dG, dMp, fin.
size_t bwd_mfma_workspace_bytes(int B, int T, int H, int groups) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const size_t BH = (size_t)B * H, nc = ((size_t)T + kC - 1) / kC, Tpad = nc * kC, G = groups;
    size_t n = al((size_t)H * 128 * 128 * 2);
    n += 2 * al(BH * G * 2 * kSE * 4);
    n += al(BH * G * 4) + al(BH * G * 8) + al(BH * nc * 8);
    n += 2 * al(BH * Tpad * 128 * 2);
    n += 3 * al(BH * Tpad * 4);
    n += al(BH * G * 128 * 128 * 4);
    n += al(BH * kCombBlocks * 4);
    return n;
}

hipError_t launch_bwd_mfma(BwdParams p, void *ws, hipStream_t s) {
    auto al = [](size_t x) { return (x + 255) / 256 * 256; };
    const size_t BH = (size_t)p.B * p.H, nc = p.nc, Tpad = p.Tpad, G = p.groups;
    char *w = static_cast<char *>(ws);
    auto take = [&](size_t bytes) { char *r = w; w += al(bytes); return r; };
    Args a{};
    __bf16 *Mz = reinterpret_cast<__bf16 *>(take((size_t)p.H * 128 * 128 * 2));
    a.Mz = Mz;
    a.Ef = reinterpret_cast<float *>(take(BH * G * 2 * kSE * 4));
    a.Ea = reinterpret_cast<float *>(take(BH * G * 2 * kSE * 4));
    a.Gg = reinterpret_cast<float *>(take(BH * G * 4));
    a.gclk = reinterpret_cast<double *>(take(BH * G * 8));
    a.cclk = reinterpret_cast<double *>(take(BH * nc * 8));
    a.U = reinterpret_cast<__bf16 *>(take(BH * Tpad * 128 * 2));
    a.dP = reinterpret_cast<__bf16 *>(take(BH * Tpad * 128 * 2));
    p.udu = reinterpret_cast<float *>(take(BH * Tpad * 4));
    p.dlam = reinterpret_cast<float *>(take(BH * Tpad * 4));
    p.dG = reinterpret_cast<float *>(take(BH * Tpad * 4));
    p.dMp = reinterpret_cast<float *>(take(BH * G * 128 * 128 * 4));
    p.fin = reinterpret_cast<float *>(take(BH * kCombBlocks * 4));
    a.p = p;
    hipError_t e = launch_readout_prep(p.H, p.m, p.R, nullptr, Mz, p.scale * 1.4426950408889634f, s);
    if (e != hipSuccess) return e;
    const dim3 block(kNT), grp(BH, G);
    hipLaunchKernelGGL(fwd_contrib_kernel, grp, dim3(kNT8), 0, s, a);
    hipLaunchKernelGGL(readout_kernel, grp, block, 0, s, a);
    hipLaunchKernelGGL(adj_contrib_kernel, grp, dim3(kNT8), 0, s, a);
    hipLaunchKernelGGL(grad_kernel, grp, dim3(kNT8), 0, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_bwd_tail(p, s);
}

}  // namespace cyfa
