// Fused chunk forward for 64-token chunks on eight waves (bf16 MFMA 16x16x32).
//
// Same computation as the four-wave kernel (App. B: key pass, token-wise
// softmax readout, value pass, state recurrence), laid out for two waves per
// SIMD on one sequence segment: wave w owns columns 16w .. 16w+15 of both
// carried states (Kbar^T: rows d, columns i; Vbar: rows i, columns c), 8 + 8
// accumulator tiles of 16 x 16, i.e. 32 + 32 registers per lane.  Every product
// of the chunk is split by those 16 output columns (or, for the two readout
// products, by 16 slots / 16 basis rows), so all eight waves share each step.
//
// v_mfma_f32_16x16x32_bf16 (l = lane, l16 = l % 16, g = l / 16):
//   A (16 x 32): A[l16][8g + p]   B (32 x 16): B[8g + p][l16]   D: D[4g + r][l16]
// A state accumulator pair (row tiles 2ks, 2ks+1) fed back as a B operand
// supplies k = 32ks + {4g..4g+3, 16+4g..16+4g+3}; the A operand of those
// products is read in the same permuted order.
#include "cyfa_mfma_chunk.h"

#include <hip/hip_ext.h>

namespace cyfa {

using namespace mfma;

namespace {

constexpr int W8 = 512;         // threads per workgroup
constexpr int CK = 64;          // chunk length

struct LayW8 {
    static constexpr int TILE = CK * QS * 2;
    static constexpr int SSC = CK + 8;                  // score tile row stride
    static constexpr int Q = 0;                         // Q -> X -> W
    static constexpr int K = Q + TILE;                  // K -> O''
    static constexpr int V = K + TILE;
    static constexpr int A = V + TILE;                  // A -> output staging
    static constexpr int AD = A + TILE;                 // A_dec
    static constexpr int S = AD + TILE;                 // scores [CK][SSC]
    static constexpr int CS = S + CK * SSC * 2;         // (cos, sin) [CK][64] half pairs
    static constexpr int MT = CS + CK * 64 * 4;         // readout matrix [128][QS]
    static constexpr int RED = MT + 128 * QS * 2;       // softmax (max, sum) [8 waves][CK]
    static constexpr int SC = RED + 8 * CK * 8;         // per-token scalars
    static constexpr int BYTES = SC + scalar_bytes(64);
    static_assert(BYTES <= 160 * 1024, "LDS budget");
};

// Lane offset (elements) for transposed 16x16x32 operands from a row-major tile:
// with base = tile + tr16_off, the operand element (n = l16, k = 8g + p) of the
// tile block at (k0, n0) is lds8_tr(base + k0 * stride + n0, stride), i.e.
// tile[k0 + 8g + p][n0 + l16].
__device__ __forceinline__ int tr16_off(int stride, int lane) {
    const int s = lane & 15, g = lane >> 4;
    return (8 * g + (s >> 2)) * stride + 4 * (s & 3);
}

// permuted-k A operand: columns {4g..4g+3} and {16+4g..16+4g+3} of a k-step,
// `p` already pointing at row base + 4g + 32 ks
__device__ __forceinline__ bf16x8 lds8_perm16(const __bf16 *p) {
    const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(p);
    const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(p + 16);
    bf16x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
}

// two state accumulator tiles as one bf16 B operand (k-step of 32)
__device__ __forceinline__ bf16x8 acc_pair(const f32x4 &x, const f32x4 &y) {
    bf16x8 r;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        r[q] = (__bf16)x[q];
        r[4 + q] = (__bf16)y[q];
    }
    return r;
}

// One 16 x 16 block (rb, sb) of the causal score tile: (A_rows B_rows^T) (.) Gamma,
// k = 128 along the rows of both operand tiles; blocks above the diagonal are zero.
// Sw: this lane's score-tile entry (row 4g, column l16) of block (0, 0).
__device__ __forceinline__ void score_block16(const Tiles &s, const __bf16 *An, const __bf16 *Bn,
                                              __bf16 *Sw, int rb, int sb, int lane) {
    const int l16 = lane & 15, g = lane >> 4;
    const int scol = 16 * sb + l16;
    const int row0 = 16 * rb + 4 * g;
    __bf16 *sw = Sw + 16 * rb * LayW8::SSC + 16 * sb;
    if (sb > rb) {
#pragma unroll
        for (int r = 0; r < 4; ++r) sw[r * LayW8::SSC] = (__bf16)0.f;
        return;
    }
    f32x4 acc = zero_acc4();
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
        acc = mma16(lds8(An + 16 * rb * QS + 32 * ks), lds8(Bn + 16 * sb * QS + 32 * ks), acc);
    const float Gs_col = s.Gs[scol];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const float val = scol <= row0 + r ? acc[r] * __expf(s.Gs[row0 + r] - Gs_col) : 0.f;
        sw[r * LayW8::SSC] = (__bf16)val;
    }
}

// The 12 blocks the intra-chunk products read (lower triangle, diagonal, and the
// two zero blocks (0,1), (2,3) that complete their 32-wide k-steps): wave w
// takes block w and, for w < 4, block 8 + w.
__device__ __forceinline__ void score_tiles16(const Tiles &s, const __bf16 *An, const __bf16 *Bn,
                                              __bf16 *Sw, int w, int lane) {
    constexpr int kRb[12] = {0, 0, 1, 1, 2, 2, 2, 2, 3, 3, 3, 3};
    constexpr int kSb[12] = {0, 1, 0, 1, 0, 1, 2, 3, 0, 1, 2, 3};
    score_block16(s, An, Bn, Sw, kRb[w], kSb[w], lane);
    if (w < 4) score_block16(s, An, Bn, Sw, kRb[8 + w], kSb[8 + w], lane);
}

__device__ __forceinline__ void load_state16(const __bf16 *st, int col, int g4, f32x4 (&kacc)[8],
                                             f32x4 (&vacc)[8]) {
#pragma unroll
    for (int x = 0; x < 8; ++x)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            kacc[x][r] = (float)st[dump_index_K(col, 16 * x + g4 + r)];
            vacc[x][r] = (float)st[dump_index_V(16 * x + g4 + r, col)];
        }
}

__device__ __forceinline__ void dump_state16(float *st, int col, int g4, const f32x4 (&kacc)[8],
                                             const f32x4 (&vacc)[8], float f) {
#pragma unroll
    for (int x = 0; x < 8; ++x)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            st[dump_index_K(col, 16 * x + g4 + r)] = f * kacc[x][r];
            st[dump_index_V(16 * x + g4 + r, col)] = f * vacc[x][r];
        }
}

__global__ __launch_bounds__(W8, 1) void chunk64_w8_kernel(MfmaArgs a) {
    using Ly = LayW8;
    constexpr int SSC = Ly::SSC;
    __shared__ __attribute__((aligned(16))) char smem[Ly::BYTES];
    Tiles s{};
    s.Qs = reinterpret_cast<__bf16 *>(smem + Ly::Q);
    s.Xs = s.Qs;
    s.Ws = s.Qs;
    s.Ks = reinterpret_cast<__bf16 *>(smem + Ly::K);
    s.Os = s.Ks;
    s.Vs = reinterpret_cast<__bf16 *>(smem + Ly::V);
    s.As = reinterpret_cast<__bf16 *>(smem + Ly::A);
    s.Stage = s.As;
    s.Ads = reinterpret_cast<__bf16 *>(smem + Ly::AD);
    s.Ss = reinterpret_cast<__bf16 *>(smem + Ly::S);
    s.CS = reinterpret_cast<half2v *>(smem + Ly::CS);
    s.Mt = reinterpret_cast<__bf16 *>(smem + Ly::MT);
    s.red = reinterpret_cast<float2 *>(smem + Ly::RED);
    scalars_at(s, smem + Ly::SC);

    const FwdParams &p = a.p;
    const int bh = blockIdx.x / a.P, seg = blockIdx.x % a.P;
    const int b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int l16 = lane & 15, g = lane >> 4, g4 = 4 * g;
    const int m = p.m;
    const int c_begin = seg * a.cps, c_end = min(c_begin + a.cps, a.nchunks);
    const int Tb = seq_tokens(p, b);
    const int col = 16 * w + l16;                     // this lane's state / output column
    // U(theta) on a (cos, sin) column pair held by lanes (2k, 2k+1)
    const float sgn = (l16 & 1) ? 1.f : -1.f;
    // the readout matrix is M times zs = scale log2(e) (logits in log2 units); the
    // readout weights are divided by zs to compensate
    const float zs = __int_as_float(__builtin_amdgcn_readfirstlane(
        __float_as_int(p.scale * 1.4426950408889634f)));

    // Per-lane operand bases, one opaque byte offset per access pattern; every
    // unrolled access below adds a compile-time constant below 64 KiB.
    constexpr int TE = Ly::TILE / 2;                  // tile size in elements
    const int trl = tr16_off(QS, lane);
    const __bf16 *Qp = lds_at<__bf16>(smem, opq(Ly::Q + 2 * (l16 * QS + g4)));      // permuted-k rows
    const __bf16 *Op = Qp + TE;                                                     // (K tile)
    const __bf16 *Qn = lds_at<__bf16>(smem, opq(Ly::Q + 2 * (l16 * QS + 8 * g)));   // natural-k rows
    const __bf16 *Kn = Qn + TE;
    const __bf16 *On = Kn;
    const __bf16 *An = Qn + 3 * TE;
    const __bf16 *Sn = lds_at<__bf16>(smem, opq(Ly::S + 2 * (l16 * SSC + 8 * g)));
    __bf16 *Sw = lds_at<__bf16>(smem, opq(Ly::S + 2 * (g4 * SSC + l16)));
    const __bf16 *Mn = lds_at<__bf16>(smem, opq(Ly::MT + 2 * (col * QS + 8 * g)));   // M rows 16w + l16
    const __bf16 *Mtr = lds_at<__bf16>(smem, opq(Ly::MT + 2 * (trl + 16 * w)));     // M columns 16w + l16
    const __bf16 *Atr = lds_at<__bf16>(smem, opq(Ly::A + 2 * (trl + 16 * w)));
    const __bf16 *Vtr = lds_at<__bf16>(smem, opq(Ly::V + 2 * (trl + 16 * w)));
    const __bf16 *ADw = lds_at<__bf16>(smem, opq(Ly::AD + 2 * (trl + 16 * w)));
    const __bf16 *ADtr = lds_at<__bf16>(smem, opq(Ly::AD + 2 * trl));
    const __bf16 *Ktr = lds_at<__bf16>(smem, opq(Ly::K + 2 * trl));
    // accumulator-row bases: row 4g (+ 16 rt + r), column col
    __bf16 *Xw = lds_at<__bf16>(smem, opq(Ly::Q + 2 * (g4 * QS + col)));
    __bf16 *Stw = Xw + 3 * TE;                                                      // A tile
    const half2v *CSx = lds_at<half2v>(smem, opq(Ly::CS + 4 * (g4 * 64 + (col >> 1))));
    const float *gam_r = lds_at<float>(smem, opq(Ly::SC + 4 * (64 + g4)));         // gam + 4g
    // token-row bases: row l16 (+ 16 rt), columns 16w + 4g ..
    __bf16 *Ww = lds_at<__bf16>(smem, opq(Ly::Q + 2 * (l16 * QS + 16 * w + g4)));
    __bf16 *O2w = Ww + TE;
    const half2v *CSy = lds_at<half2v>(smem, opq(Ly::CS + 4 * (l16 * 64 + 8 * w + 2 * g)));
    float2 *redw = lds_at<float2>(smem, opq(Ly::RED + 8 * (w * CK + l16)));
    const float2 *redr = lds_at<float2>(smem, opq(Ly::RED + 8 * l16));
    const __bf16 *Stg = lds_at<__bf16>(smem, opq(Ly::A + 2 * ((tid >> 4) * QS + (tid & 15) * 8)));

    {
        // readout matrix M_h (slot rows, internal basis columns), resident for the segment
        const __bf16 *Mh = a.Mz + (size_t)h * 128 * 128;
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int e = it * W8 + tid;
            const int row = e >> 4, c0 = (e & 15) * 8;
            *reinterpret_cast<uint4 *>(s.Mt + row * QS + c0) =
                *reinterpret_cast<const uint4 *>(Mh + row * 128 + c0);
        }
    }
    f32x4 kacc[8], vacc[8];
    const __bf16 *slot_state = a.seg_state + ((size_t)bh * a.P + seg) * kStateFloats;
    if (a.has_init && !(seg == 0 && a.zero_init)) {
        load_state16(slot_state, col, g4, kacc, vacc);
    } else {
#pragma unroll
        for (int x = 0; x < 8; ++x) {
            kacc[x] = f32x4{};
            vacc[x] = f32x4{};
        }
    }
    double carry = 0.0, gsum = 0.0;
    float logf = 0.f;                                 // carried states are exp(logf) x registers
    Prefetch<CK, W8> pf;
    load_chunk<CK, true, W8>(p, b, h, c_begin * CK, Tb, tid, pf);
    __bf16 *o = static_cast<__bf16 *>(p.o);

    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * CK;
        const int n = min(CK, Tb - t0);
        // -- A: stage the chunk, prefix sums, temporal writes; prefetch the next chunk
        store_chunk<CK, true, W8>(s, tid, pf);
        if (w == 0) chunk_scans<CK, W8>(s, lane, m, pf, carry, gsum, logf);
        __syncthreads();
        if (c + 1 < c_end) load_chunk<CK, true, W8>(p, b, h, t0 + CK, Tb, tid, pf);
        build_writes<CK, true, true, W8>(s, tid, m);
        __syncthreads();
        // -- B: key pass.  O' = gamma (.) Q Kbar^T + (Q K^T (.) Gamma) A
        score_tiles16(s, Qn, Kn, Sw, w, lane);
        f32x4 oacc[4];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) oacc[rt] = zero_acc4();
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const bf16x8 kb = acc_pair(kacc[2 * ks], kacc[2 * ks + 1]);
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
                oacc[rt] = mma16(lds8_perm16(Qp + 16 * rt * QS + 32 * ks), kb, oacc[rt]);
        }
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int r = 0; r < 4; ++r) oacc[rt][r] *= gam_r[16 * rt + r];
        __syncthreads();
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int ks = 0; ks <= (rt >> 1); ++ks)      // causal: row tile rt sees tokens < 32 (rt/2 + 1)
                oacc[rt] = mma16(lds8(Sn + 16 * rt * SSC + 32 * ks), lds8_tr(Atr + 32 * ks * QS, QS),
                                 oacc[rt]);
        {
            // key state: Kbar^T <- gamma^C Kbar^T + K^T A_dec (decay kept in L)
            const float sf = s.ctl[0];
            if (sf != 1.f) {
#pragma unroll
                for (int x = 0; x < 8; ++x)
#pragma unroll
                    for (int r = 0; r < 4; ++r) kacc[x][r] *= sf;
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 adw = lds8_tr(ADw + 32 * ks * QS, QS);
#pragma unroll
                for (int db = 0; db < 8; ++db)
                    kacc[db] = mma16(lds8_tr(Ktr + 32 * ks * QS + 16 * db, QS), adw, kacc[db]);
            }
        }
        // -- middle step 1: X_r = U(lambda_r) O'_r -> X tile (Q's)
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ro = 16 * rt + r;                  // row - 4g
                const float self = oacc[rt][r];
                const float part = swap_pair(self);
                const half2v cs = CSx[ro * 64];
                Xw[ro * QS] = (__bf16)fmaf(sgn * (float)cs[1], part, (float)cs[0] * self);
            }
        __syncthreads();
        // -- middle step 2: slot logits Z^T = M X^T; wave w owns slots 16w .. 16w+15
        f32x4 zacc[4];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) zacc[rt] = zero_acc4();
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const bf16x8 ma = lds8(Mn + 32 * ks);
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) zacc[rt] = mma16(ma, lds8(Qn + 16 * rt * QS + 32 * ks), zacc[rt]);
        }
        // -- middle step 3: softmax over the m active slots: 4 in-lane, across the
        //    four lane groups, then one (max, sum) exchange between the 8 waves
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            float mx = -INFINITY;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                if (16 * w + g4 + r >= m) zacc[rt][r] = -INFINITY;
                mx = fmaxf(mx, zacc[rt][r]);
            }
            mx = fmaxf(mx, swap16(mx));
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            // a wave whose slots are all inactive contributes (-inf, 0)
            const float mref = mx == -INFINITY ? 0.f : mx;
            float sm = 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) sm += __builtin_amdgcn_exp2f(zacc[rt][r] - mref);
            sm += swap16(sm);
            sm += __shfl_xor(sm, 32);
            const int tok = 16 * rt + l16;
            if (g == 0) redw[16 * rt] = make_float2(mx, sm);
            if (p.logits && tok < n) {
                // the accumulators hold log2(e) z; report z
                float *lg = p.logits + ((seq_row0(p, b) + t0 + tok) * p.H + h) * m;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int slot = 16 * w + g4 + r;
                    if (slot < m) lg[slot] = zacc[rt][r] * 0.69314718055994531f;
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            const int tok = 16 * rt + l16;
            float2 pr[8];
#pragma unroll
            for (int x = 0; x < 8; ++x) pr[x] = redr[x * CK + 16 * rt];
            float M = pr[0].x;
#pragma unroll
            for (int x = 1; x < 8; ++x) M = fmaxf(M, pr[x].x);
            float Lsum = 0.f;
#pragma unroll
            for (int x = 0; x < 8; ++x) Lsum += pr[x].y * __builtin_amdgcn_exp2f(pr[x].x - M);
            const float inv = __builtin_amdgcn_rcpf(Lsum * zs);
            bf16x4 wv;
#pragma unroll
            for (int r = 0; r < 4; ++r) wv[r] = (__bf16)(__builtin_amdgcn_exp2f(zacc[rt][r] - M) * inv);
            *reinterpret_cast<bf16x4 *>(Ww + 16 * rt * QS) = wv;
        }
        __syncthreads();
        // -- middle step 4: O''_r = U(-lambda_r) M^T W_r as Y^T = M^T W^T; wave w owns
        //    basis rows 16w .. 16w+15, each (cos, sin) pair in consecutive registers
        {
            f32x4 yacc[4];
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) yacc[rt] = zero_acc4();
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const bf16x8 mt = lds8_tr(Mtr + 32 * ks * QS, QS);
#pragma unroll
                for (int rt = 0; rt < 4; ++rt) yacc[rt] = mma16(mt, lds8(Qn + 16 * rt * QS + 32 * ks), yacc[rt]);
            }
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                const half2v *csr = CSy + 16 * rt * 64;
                bf16x4 ov;
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    const half2v cs = csr[k2];
                    const float cv = (float)cs[0], sv = (float)cs[1];
                    const float yc = yacc[rt][2 * k2], ys = yacc[rt][2 * k2 + 1];
                    ov[2 * k2] = (__bf16)fmaf(sv, ys, cv * yc);
                    ov[2 * k2 + 1] = (__bf16)fmaf(-sv, yc, cv * ys);
                }
                *reinterpret_cast<bf16x4 *>(O2w + 16 * rt * QS) = ov;
            }
        }
        __syncthreads();
        // -- D: value pass.  O = gamma (.) O'' Vbar + (O'' A^T (.) Gamma) V
        score_tiles16(s, On, An, Sw, w, lane);
        f32x4 pacc[4];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) pacc[rt] = zero_acc4();
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const bf16x8 vb = acc_pair(vacc[2 * ks], vacc[2 * ks + 1]);
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
                pacc[rt] = mma16(lds8_perm16(Op + 16 * rt * QS + 32 * ks), vb, pacc[rt]);
        }
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int r = 0; r < 4; ++r) pacc[rt][r] *= gam_r[16 * rt + r];
        __syncthreads();
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int ks = 0; ks <= (rt >> 1); ++ks)
                pacc[rt] = mma16(lds8(Sn + 16 * rt * SSC + 32 * ks), lds8_tr(Vtr + 32 * ks * QS, QS),
                                 pacc[rt]);
        // output tile -> staging (A's tile, read last by the value scores)
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int r = 0; r < 4; ++r) Stw[(16 * rt + r) * QS] = (__bf16)pacc[rt][r];
        {
            // value state: Vbar <- gamma^C Vbar + A_dec^T V (decay kept in L)
            const float sf = s.ctl[0];
            if (sf != 1.f) {
#pragma unroll
                for (int x = 0; x < 8; ++x)
#pragma unroll
                    for (int r = 0; r < 4; ++r) vacc[x][r] *= sf;
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                const bf16x8 vw = lds8_tr(Vtr + 32 * ks * QS, QS);
#pragma unroll
                for (int ib = 0; ib < 8; ++ib)
                    vacc[ib] = mma16(lds8_tr(ADtr + 32 * ks * QS + 16 * ib, QS), vw, vacc[ib]);
            }
        }
        __syncthreads();
        {
            const int r0 = tid >> 4, d0 = (tid & 15) * 8;
#pragma unroll
            for (int it = 0; it < 2; ++it) {
                const int r = r0 + 32 * it;
                if (r < n)
                    *reinterpret_cast<uint4 *>(o + ((seq_row0(p, b) + t0 + r) * p.H + h) * D + d0) =
                        *reinterpret_cast<const uint4 *>(Stg + 32 * it * QS);
            }
        }
    }
    if (a.want_final && seg == a.P - 1) {
        dump_state16(a.fin_state + (size_t)bh * kStateFloats, col, g4, kacc, vacc, __expf(s.ctl[1]));
        if (tid == 0) a.final_lam[bh] = carry;
    }
}

}  // namespace

hipError_t launch_chunk64_w8(const MfmaArgs &a, int groups, hipStream_t st, hipEvent_t ev_start,
                             hipEvent_t ev_stop) {
    hipExtLaunchKernelGGL(chunk64_w8_kernel, dim3(groups), dim3(W8), 0, st, ev_start, ev_stop, 0, a);
    return hipGetLastError();
}

}  // namespace cyfa
