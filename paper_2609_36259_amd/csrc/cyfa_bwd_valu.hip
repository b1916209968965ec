// Vector-ALU backward of the chunk-wise CyFA forward (fp32 arithmetic).
//
// Gradients of L = sum_t <do_t, o_t> + <dK_T, Kbar_T> + <dV_T, Vbar_T> in the
// absolute-clock form (Sec. 3.2, Eqs. cyfa-absolute-recurrence and
// cyfa-absolute-readout), evaluated chunk by chunk as the forward is (App. B).
// Forward per token: a_t = beta_t U(-lambda_t) b (Eq. app-temporal-writes),
// Kbar_t = alpha_t Kbar_{t-1} + a_t k_t^T (Vbar likewise), p_t = Kbar_t q_t,
// X_t = scale U(lambda_t) p_t, Z_t = M X_t, W_t = softmax over the m active
// slots, u_t = U(-lambda_t) M^T W_t, o_t = Vbar_t^T u_t, with M = R Phi.
// Reverse mode:
//   du_t = Vbar_t do_t,  dY_t = U(lambda_t) du_t,  dW_t = M dY_t,
//   dZ_t = W_t (.) (dW_t - <W_t, dW_t>),  dX_t = M^T dZ_t,  dp_t = scale U(-lambda_t) dX_t,
//   dM = sum_t W_t dY_t^T + dZ_t X_t^T  and  dR = dM Phi^T,
//   adjoint states DK_t = dp_t q_t^T + alpha_{t+1} DK_{t+1},  DV_t = u_t do_t^T + alpha_{t+1} DV_{t+1}
//   (starting from dK_T, dV_T), dq_t = Kbar_t^T dp_t, dk_t = DK_t^T a_t, dv_t = DV_t^T a_t,
//   da_t = DK_t k_t + DV_t v_t,  dbeta_t = <da_t, U(-lambda_t) b>.
// Decay: with G_t = sum_{j<=t} log alpha_j every pair (t, s) of a pass carries
// exp(G_t - G_s), so dL/dG_t = <q_t, dq_t> - <k_t, dk_t> + <u_t, du_t> - <a_t, DV_t v_t>
// (plus <dK_T, Kbar_T> + <dV_T, Vbar_T> at the last token) and dlog_alpha_t is the
// reverse cumulative sum of dL/dG.  Clock: U(+-lambda_t) acts on the (cos, sin)
// pair j as a rotation by +-2 pi j lambda_t / m, whose derivative is the
// rotation generator; dL/dlambda_t collects the three rotations of token t (a_t,
// X_t, u_t) and ddelta_t = sum_{tau >= t} dL/dlambda_tau
// (Eq. app-clock-gradient-accumulation); dclock0 is the full sum.
//
// Within a chunk (rows r, s; gamma_r = exp(G_r), Gamma_rs = exp(G_r - G_s) for
// r >= s, rho_s = exp(G_C - G_s), entering states Kbar_c, Vbar_c, adjoints
// DK', DV' at the chunk's end):
//   p  = gamma (.) Q Kbar_c^T + (Q K^T (.) Gamma) A
//   du = gamma (.) dO Vbar_c  + (dO V^T (.) Gamma) A
//   dq = gamma (.) dP Kbar_c  + (dP A^T (.) Gamma) K
//   dk = (dP A^T (.) Gamma)^T Q + (rho (.) A) DK'
//   dv = (U A^T (.) Gamma)^T dO + (rho (.) A) DV'
//   da = (Q K^T (.) Gamma)^T dP + rho (.) K DK'^T + (dO V^T (.) Gamma)^T U + rho (.) V DV'^T
// Kernels: (1a) states entering every chunk from the chunk group's own tokens,
// per chunk group, and (1b) the states entering every group, per sequence; (2)
// readout recomputation and its adjoint, per chunk group; (3a, 3b) the same
// split for the adjoint states at every chunk's end, in reverse; (4) token
// gradients, per chunk group; (5) reverse cumulative sums, per sequence; (6)
// dR, per head.  The states are in absolute-clock coordinates, so a group's
// entering state reaches its chunks through the decay alone.
#include <type_traits>

#include "cyfa_bwd.h"
#include "cyfa_mfma_common.h"   // wave-level prefix sums (DPP)

namespace cyfa {

namespace {

constexpr int kC = kBwdChunk;
constexpr int kNT = 512;            // threads per workgroup (two waves per SIMD)
constexpr int kRP = kNT / kStoreRows; // threads sharing one state row in the row layouts
constexpr int kRQ = kC * kStoreRows / kNT;   // token rows per thread in the readout products
constexpr int kReadoutThreads = kNT;           // the readout kernel (1024 measured slower: spills)
constexpr int kLD = kStoreRows + 4; // padded row of a [token][basis] tile (16-byte rows)
constexpr float kTwoPi = 6.283185307179586f;
constexpr int kCombBlocks = kBwdFinParts;   // workgroups per sequence of the group-combine kernels

__device__ __forceinline__ float wsum(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}
__device__ __forceinline__ float wmax(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}

__device__ __forceinline__ int bwd_tokens(const BwdParams &p, int b) {
    if (p.cu) return min(max(p.cu[b + 1] - p.cu[b], 0), p.T);
    return p.lens ? min(max(p.lens[b], 0), p.T) : p.T;
}
// first row of sequence b in the [rows, H, ...] tensors
__device__ __forceinline__ size_t brow0(const BwdParams &p, int b) {
    return p.cu ? (size_t)p.cu[b] : (size_t)b * p.T;
}

// Per-chunk scalar tables.
struct ChunkTab {
    double lam[kC];                 // clock after token r, reduced mod m
    float G[kC];                    // sum of log alpha over the chunk's tokens 0..r
    float beta[kC];
    float2 cs[kC][64];              // (cos, sin) of 2 pi j lam_r / m at [r][j-1]
};

// Loads the chunk's scalars (rows at or past the sequence's end: no shift, no
// decay, no write), forms the clock and log-decay prefix sums and the phase
// table.  Ends with a barrier.
template <int NT = kNT>
__device__ void chunk_tables(const BwdParams &p, int b, int h, int t0, int Tb, double lam_in,
                             ChunkTab &s, int tid) {
    if (tid < kC) {
        const int t = t0 + tid;
        const bool live = t < Tb;
        const size_t si = (brow0(p, b) + t) * p.H + h;
        s.lam[tid] = live ? (double)p.delta[si] : 0.0;
        s.G[tid] = (live && p.log_alpha) ? p.log_alpha[si] : 0.f;
        s.beta[tid] = live ? (p.beta ? p.beta[si] : 1.f) : 0.f;
    }
    __syncthreads();
    if (tid == 0) {
        double lam = lam_in;
        float G = 0.f;
        for (int r = 0; r < kC; ++r) {
            lam = reduce_clock(lam + s.lam[r], p.m);
            s.lam[r] = lam;
            G += s.G[r];
            s.G[r] = G;
        }
    }
    __syncthreads();
    const int J = (p.m - 1) / 2;
    for (int e = tid; e < kC * 64; e += NT) {
        const int r = e >> 6, jj = e & 63;
        float c = 1.f, sn = 0.f;
        if (jj < J) clock_phase(s.lam[r], jj + 1, p.m, &c, &sn);
        s.cs[r][jj] = make_float2(c, sn);
    }
    __syncthreads();
}

// Temporal write rows A_r = beta_r U(-lambda_r) b (Eq. app-temporal-writes).
__device__ __forceinline__ float write_entry(const ChunkTab &s, int m, int r, int i, float be) {
    if (i == 0) return be * (1.f / sqrtf((float)m));
    if (i >= m) return 0.f;
    const float ac = sqrtf(2.f / (float)m);
    const float2 cs = s.cs[r][(i - 1) >> 1];
    return (i & 1) ? be * ac * cs.x : -be * ac * cs.y;
}
template <int NT = kNT>
__device__ void build_writes(const ChunkTab &s, int m, float (*A)[kLD], int tid) {
    for (int e = tid; e < kC * kStoreRows; e += NT) {
        const int r = e >> 7, i = e & 127;
        A[r][i] = write_entry(s, m, r, i, s.beta[r]);
    }
}

// Y_r <- mul * U(sign lambda_r) Y_r for every row, in place: element 0 is scaled,
// pair (2j-1, 2j) rotated by sign * 2 pi j lambda_r / m; padding rows untouched.
template <int NT = kNT>
__device__ void rotate_rows(float (*Y)[kLD], const ChunkTab &s, int m, float sign, float mul, int tid) {
    const int J = (m - 1) / 2;
    for (int e = tid; e < kC * 64; e += NT) {
        const int r = e >> 6, j = e & 63;
        if (j == 0) {
            Y[r][0] *= mul;
        } else if (j <= J) {
            const float2 cs = s.cs[r][j - 1];
            const float c = cs.x, sn = sign * cs.y;
            const float a = Y[r][2 * j - 1], bb = Y[r][2 * j];
            Y[r][2 * j - 1] = mul * (c * a - sn * bb);
            Y[r][2 * j] = mul * (sn * a + c * bb);
        }
    }
}

// dL/dlambda of Z = U(sign lambda) y given dZ (one row, one wave): the pair j
// contributes sign (2 pi j / m) (dZ_{2j} Z_{2j-1} - dZ_{2j-1} Z_{2j}).
__device__ __forceinline__ float rot_grad(const float *dZ, const float *Z, int m, float sign, int lane) {
    const int J = (m - 1) / 2, j = lane + 1;
    float acc = 0.f;
    if (j <= J) acc = (float)j * (dZ[2 * j] * Z[2 * j - 1] - dZ[2 * j - 1] * Z[2 * j]);
    return sign * (kTwoPi / (float)m) * wsum(acc);
}

// Products with the readout matrix over the m active entries, register-blocked:
// thread (column col = tid % 128, rows RQ (tid / 128) .. + RQ - 1, RQ = 16 * 128 /
// threads) keeps RQ independent sums.  TRANS = false: out_r = M in_r (out[r][i] = sum_j M[i][j] in[r][j]);
// TRANS = true: out_r = M^T in_r.  Entries >= m of out are 0.
template <bool TRANS, int NT = kNT>
__device__ void readout_product(const float (*Ms)[kLD], const float (*in)[kLD], float (*out)[kLD], int m,
                                int tid) {
    constexpr int RQ = kC * kStoreRows / NT;
    const int col = tid & 127, r0 = (tid >> 7) * RQ;
    float acc[RQ];
#pragma unroll
    for (int q = 0; q < RQ; ++q) acc[q] = 0.f;
    if (col < m) {
        // four entries per step (16-byte rows; entries m .. 127 of in are 0, and M
        // is 0 outside its active block, so running to a multiple of four is exact)
#pragma unroll 2
        for (int j = 0; j < m; j += 4) {
            float4 mv;
            if (TRANS) {
                mv = make_float4(Ms[j][col], Ms[j + 1][col], Ms[j + 2][col], Ms[j + 3][col]);
            } else {
                mv = *reinterpret_cast<const float4 *>(&Ms[col][j]);
            }
#pragma unroll
            for (int q = 0; q < RQ; ++q) {
                const float4 x = *reinterpret_cast<const float4 *>(&in[r0 + q][j]);
                acc[q] = fmaf(mv.x, x.x, fmaf(mv.y, x.y, fmaf(mv.z, x.z, fmaf(mv.w, x.w, acc[q]))));
            }
        }
    }
#pragma unroll
    for (int q = 0; q < RQ; ++q) out[r0 + q][col] = acc[q];
}

// out[r][i] += sum_s S[r][s] A[s][i] for a causal (lower-triangular) score tile S.
template <int NT = kNT>
__device__ void add_scores_times(const float (*S)[kC + 1], const float (*A)[kLD], float (*out)[kLD], int tid) {
    constexpr int RQ = kC * kStoreRows / NT;
    const int col = tid & 127, r0 = (tid >> 7) * RQ;
    float acc[RQ];
#pragma unroll
    for (int q = 0; q < RQ; ++q) acc[q] = out[r0 + q][col];
    for (int s = 0; s < r0 + RQ; ++s) {
        const float a = A[s][col];
#pragma unroll
        for (int q = 0; q < RQ; ++q) acc[q] = fmaf(S[r0 + q][s], a, acc[q]);
    }
#pragma unroll
    for (int q = 0; q < RQ; ++q) out[r0 + q][col] = acc[q];
}

template <typename Tin>
__device__ __forceinline__ float ld_row(const void *base, size_t row0, int t, int h, int c, int H, int D, bool live) {
    return live ? load_as_float(static_cast<const Tin *>(base), ((row0 + t) * H + h) * D + c) : 0.f;
}

// ---------------------------------------------------------------------------
// (1a) states entering every chunk from the chunk group's own tokens (the
// group starts from zero), per (sequence, group).  Thread t keeps column t % D
// of a state and its rows (t / D) NR .. + NR - 1 (NR = 128 D / threads), for the key
// state (D = d_k) and the value state (D = d_v): a wave shares its rows, so the
// write rows are broadcast reads and the stored state rows are coalesced.  The
// group's own final state goes to EcK/EcV[g], its total log decay to Gg.
template <int DK, int DV, typename Tin>
__global__ __launch_bounds__(kNT) void bwd_states_local_kernel(BwdParams p) {
    constexpr int NRK = DK * kStoreRows / kNT, NRV = DV * kStoreRows / kNT;
    __shared__ float Ks[kC][DK];
    __shared__ float Vs[kC][DV];
    __shared__ __attribute__((aligned(16))) float Aw[kC][kStoreRows];   // rho_r A_r
    __shared__ ChunkTab tab;
    __shared__ double dred[kNT];
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H, tid = threadIdx.x;
    const int ck = tid % DK, rk = (tid / DK) * NRK;
    const int cv = tid % DV, rv = (tid / DV) * NRV;
    const int m = p.m;
    const int Tb = bwd_tokens(p, b);
    const int c_begin = g * p.cpg, c_end = min(c_begin + p.cpg, p.nc);
    // clock at the group's first token: lambda_0 plus the increments before it
    {
        const int t_start = min(c_begin * kC, Tb);
        double ds = 0.0;
        for (int t = tid; t < t_start; t += kNT) ds += (double)p.delta[(brow0(p, b) + t) * p.H + h];
        dred[tid] = ds;
        __syncthreads();
        for (int w = kNT / 2; w > 0; w >>= 1) {
            if (tid < w) dred[tid] += dred[tid + w];
            __syncthreads();
        }
    }
    double lam = reduce_clock((p.clock0 ? p.clock0[bh] : 0.0) + dred[0], m);
    if (p.gclk && tid == 0) p.gclk[(size_t)bh * p.groups + g] = lam;
    float kst[NRK], vst[NRV];
#pragma unroll
    for (int ii = 0; ii < NRK; ++ii) kst[ii] = 0.f;
#pragma unroll
    for (int ii = 0; ii < NRV; ++ii) vst[ii] = 0.f;
    float Gl = 0.f;
    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * kC;
        if (p.Kst) {        // the forward's group pre-pass keeps only the group totals
            float *Kd = p.Kst + ((size_t)bh * p.nc + c) * kStoreRows * DK + ck;
            float *Vd = p.Vst + ((size_t)bh * p.nc + c) * kStoreRows * DV + cv;
#pragma unroll
            for (int ii = 0; ii < NRK; ++ii) Kd[(size_t)(rk + ii) * DK] = kst[ii];
#pragma unroll
            for (int ii = 0; ii < NRV; ++ii) Vd[(size_t)(rv + ii) * DV] = vst[ii];
            if (tid == 0) {
                p.clk[(size_t)bh * p.nc + c] = lam;
                p.Gin[(size_t)bh * p.nc + c] = Gl;
            }
        }
        for (int e = tid; e < kC * DK; e += kNT) {
            const int r = e / DK, cc = e % DK;
            Ks[r][cc] = ld_row<Tin>(p.k, brow0(p, b), t0 + r, h, cc, p.H, DK, t0 + r < Tb);
        }
        for (int e = tid; e < kC * DV; e += kNT) {
            const int r = e / DV, cc = e % DV;
            Vs[r][cc] = ld_row<Tin>(p.v, brow0(p, b), t0 + r, h, cc, p.H, DV, t0 + r < Tb);
        }
        chunk_tables(p, b, h, t0, Tb, lam, tab, tid);
        const float GC = tab.G[kC - 1], gC = __expf(GC);
        for (int e = tid; e < kC * kStoreRows; e += kNT) {
            const int r = e >> 7, i = e & 127;
            Aw[r][i] = write_entry(tab, m, r, i, tab.beta[r]) * __expf(GC - tab.G[r]);
        }
        __syncthreads();
#pragma unroll
        for (int ii = 0; ii < NRK; ++ii) kst[ii] *= gC;
#pragma unroll
        for (int ii = 0; ii < NRV; ++ii) vst[ii] *= gC;
#pragma unroll 1
        for (int r = 0; r < kC; ++r) {
            const float kr = Ks[r][ck], vr = Vs[r][cv];
#pragma unroll
            for (int ii = 0; ii < NRK; ++ii) kst[ii] = fmaf(Aw[r][rk + ii], kr, kst[ii]);
#pragma unroll
            for (int ii = 0; ii < NRV; ++ii) vst[ii] = fmaf(Aw[r][rv + ii], vr, vst[ii]);
        }
        lam = tab.lam[kC - 1];
        Gl += GC;
        __syncthreads();
    }
    float *Ko = p.EcK + ((size_t)bh * p.groups + g) * kStoreRows * DK + ck;
    float *Vo = p.EcV + ((size_t)bh * p.groups + g) * kStoreRows * DV + cv;
#pragma unroll
    for (int ii = 0; ii < NRK; ++ii) Ko[(size_t)(rk + ii) * DK] = kst[ii];
#pragma unroll
    for (int ii = 0; ii < NRV; ++ii) Vo[(size_t)(rv + ii) * DV] = vst[ii];
    if (tid == 0) p.Gg[(size_t)bh * p.groups + g] = Gl;
}

// (1b) states entering each group, per sequence, in group order:
// E_0 = (K0, V0), E_{g+1} = exp(Gg_g) E_g + (group g's own final state); EcK/EcV[g]
// are overwritten with E_g.  The final state gives <dK_T, Kbar_T> + <dV_T, Vbar_T>,
// the final-state term of dL/dG at the last token.
template <int DK, int DV>
__global__ __launch_bounds__(kNT) void bwd_states_combine_kernel(BwdParams p) {
    __shared__ float red[kNT / 64];
    const int bh = blockIdx.x, tid = threadIdx.x, m = p.m, G = p.groups;
    const int e0 = blockIdx.y * kNT + tid, es = kCombBlocks * kNT;
    const float *Gg = p.Gg + (size_t)bh * G;
    float acc = 0.f;
    for (int e = e0; e < kStoreRows * DK; e += es) {
        const bool act = e / DK < m;
        float E = (p.K0 && act) ? p.K0[(size_t)bh * kStoreRows * DK + e] : 0.f;
        for (int g = 0; g < G; ++g) {
            float *slot = p.EcK + ((size_t)bh * G + g) * kStoreRows * DK + e;
            const float own = *slot;
            *slot = E;
            E = fmaf(__expf(Gg[g]), E, own);
        }
        if (p.dK_T && act) acc = fmaf(p.dK_T[(size_t)bh * kStoreRows * DK + e], E, acc);
    }
    for (int e = e0; e < kStoreRows * DV; e += es) {
        const bool act = e / DV < m;
        float E = (p.V0 && act) ? p.V0[(size_t)bh * kStoreRows * DV + e] : 0.f;
        for (int g = 0; g < G; ++g) {
            float *slot = p.EcV + ((size_t)bh * G + g) * kStoreRows * DV + e;
            const float own = *slot;
            *slot = E;
            E = fmaf(__expf(Gg[g]), E, own);
        }
        if (p.dV_T && act) acc = fmaf(p.dV_T[(size_t)bh * kStoreRows * DV + e], E, acc);
    }
    acc = wsum(acc);
    if ((tid & 63) == 0) red[tid >> 6] = acc;
    __syncthreads();
    if (tid == 0) {
        float t = 0.f;
        for (int w = 0; w < kNT / 64; ++w) t += red[w];
        p.fin[(size_t)bh * kCombBlocks + blockIdx.y] = t;
    }
}

// ---------------------------------------------------------------------------
// (2) readout recomputation and its adjoint, per (sequence, chunk group).
template <int DK, int DV, typename Tin>
__global__ __launch_bounds__(kReadoutThreads) void bwd_readout_kernel(BwdParams p) {
    constexpr int NT = kReadoutThreads, RP = NT / kStoreRows;
    constexpr int KH = DK / RP, VH = DV / RP, MH = kStoreRows / RP;
    constexpr int DM = DK > DV ? DK : DV;
    __shared__ __attribute__((aligned(16))) float Ms[kStoreRows][kLD];
    __shared__ float In0[kC][DM + 1];       // Q, then dO
    __shared__ float In1[kC][DM + 1];       // K, then V
    __shared__ __attribute__((aligned(16))) float As[kC][kLD], Xs[kC][kLD], Ws[kC][kLD], Us[kC][kLD],
        dUs[kC][kLD], dWs[kC][kLD];
    __shared__ float S1[kC][kC + 1], S2[kC][kC + 1];
    __shared__ ChunkTab tab;
    __shared__ float dlu[kC];
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H, tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int i = tid / RP, part = tid % RP, m = p.m;
    const int Tb = bwd_tokens(p, b);
    const int c_begin = g * p.cpg, c_end = min(c_begin + p.cpg, p.nc);
    const float *Mh = p.M + (size_t)h * kStoreRows * kStoreRows;
    for (int e = tid; e < kStoreRows * kStoreRows; e += NT) Ms[e >> 7][e & 127] = Mh[e];
    float dMacc[MH];                        // dM[i][MH part .. MH part + MH - 1]
#pragma unroll
    for (int jj = 0; jj < MH; ++jj) dMacc[jj] = 0.f;

    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * kC;
        const size_t row0 = (size_t)bh * p.Tpad + t0;
        for (int e = tid; e < kC * DK; e += NT) {
            const int r = e / DK, cc = e % DK;
            const bool live = t0 + r < Tb;
            In0[r][cc] = ld_row<Tin>(p.q, brow0(p, b), t0 + r, h, cc, p.H, DK, live);
            In1[r][cc] = ld_row<Tin>(p.k, brow0(p, b), t0 + r, h, cc, p.H, DK, live);
        }
        chunk_tables<NT>(p, b, h, t0, Tb, p.clk[(size_t)bh * p.nc + c], tab, tid);
        build_writes<NT>(tab, m, As, tid);
        if (tid < kC * kC) {   // S1 = (Q K^T) (.) Gamma
            const int r = tid >> 4, s = tid & 15;
            float acc = 0.f;
            if (s <= r) {
#pragma unroll 4
                for (int cc = 0; cc < DK; ++cc) acc = fmaf(In0[r][cc], In1[s][cc], acc);
                acc *= __expf(tab.G[r] - tab.G[s]);
            }
            S1[r][s] = acc;
        }
        {   // p_r = gamma_r Kbar_c q_r (entering key state)
            const float *Kc = p.Kst + (((size_t)bh * p.nc + c) * kStoreRows + i) * DK + part * KH;
            const float *Ke = p.EcK + (((size_t)bh * p.groups + g) * kStoreRows + i) * DK + part * KH;
            const float dec = __expf(p.Gin[(size_t)bh * p.nc + c]);
            float kr[KH];
#pragma unroll
            for (int cc = 0; cc < KH; ++cc) kr[cc] = fmaf(dec, Ke[cc], Kc[cc]);
#pragma unroll 1
            for (int r = 0; r < kC; ++r) {
                float ps = 0.f;
#pragma unroll
                for (int cc = 0; cc < KH; ++cc) ps = fmaf(In0[r][part * KH + cc], kr[cc], ps);
#pragma unroll
                for (int o = 1; o < RP; o <<= 1) ps += __shfl_xor(ps, o);
                if (part == 0) Xs[r][i] = __expf(tab.G[r]) * ps;
            }
        }
        __syncthreads();
        // p += S1 A
        add_scores_times<NT>(S1, As, Xs, tid);
        __syncthreads();
        for (int e = tid; e < kC * DV; e += NT) {
            const int r = e / DV, cc = e % DV;
            const bool live = t0 + r < Tb;
            In0[r][cc] = ld_row<Tin>(p.dout, brow0(p, b), t0 + r, h, cc, p.H, DV, live);
            In1[r][cc] = ld_row<Tin>(p.v, brow0(p, b), t0 + r, h, cc, p.H, DV, live);
        }
        // X = scale U(lambda) p
        rotate_rows<NT>(Xs, tab, m, 1.f, p.scale, tid);
        __syncthreads();
        // Z = M X (active slots), S2 = (dO V^T) (.) Gamma
        readout_product<false, NT>(Ms, Xs, Ws, m, tid);
        if (tid < kC * kC) {
            const int r = tid >> 4, s = tid & 15;
            float acc = 0.f;
            if (s <= r) {
#pragma unroll 4
                for (int cc = 0; cc < DV; ++cc) acc = fmaf(In0[r][cc], In1[s][cc], acc);
                acc *= __expf(tab.G[r] - tab.G[s]);
            }
            S2[r][s] = acc;
        }
        __syncthreads();
        // W = softmax over the m active slots
        for (int r = wave; r < kC; r += NT / 64) {
            const float z0 = lane < m ? Ws[r][lane] : -INFINITY;
            const float z1 = lane + 64 < m ? Ws[r][lane + 64] : -INFINITY;
            const float mx = wmax(fmaxf(z0, z1));
            const float e0 = lane < m ? __expf(z0 - mx) : 0.f;
            const float e1 = lane + 64 < m ? __expf(z1 - mx) : 0.f;
            const float inv = 1.f / wsum(e0 + e1);
            Ws[r][lane] = e0 * inv;
            Ws[r][lane + 64] = e1 * inv;
        }
        __syncthreads();
        // Y = M^T W
        readout_product<true, NT>(Ms, Ws, Us, m, tid);
        __syncthreads();
        // u = U(-lambda) Y;  du_r = gamma_r Vbar_c do_r (entering value state)
        rotate_rows<NT>(Us, tab, m, -1.f, 1.f, tid);
        {
            const float *Vc = p.Vst + (((size_t)bh * p.nc + c) * kStoreRows + i) * DV + part * VH;
            const float *Ve = p.EcV + (((size_t)bh * p.groups + g) * kStoreRows + i) * DV + part * VH;
            const float dec = __expf(p.Gin[(size_t)bh * p.nc + c]);
            float vr[VH];
#pragma unroll
            for (int cc = 0; cc < VH; ++cc) vr[cc] = fmaf(dec, Ve[cc], Vc[cc]);
#pragma unroll 1
            for (int r = 0; r < kC; ++r) {
                float ps = 0.f;
#pragma unroll
                for (int cc = 0; cc < VH; ++cc) ps = fmaf(In0[r][part * VH + cc], vr[cc], ps);
#pragma unroll
                for (int o = 1; o < RP; o <<= 1) ps += __shfl_xor(ps, o);
                if (part == 0) dUs[r][i] = __expf(tab.G[r]) * ps;
            }
        }
        __syncthreads();
        // store u; du += S2 A
        for (int e = tid; e < kC * kStoreRows; e += NT) {
            const int r = e >> 7, ii = e & 127;
            p.U[(row0 + r) * kStoreRows + ii] = Us[r][ii];
        }
        add_scores_times<NT>(S2, As, dUs, tid);
        __syncthreads();
        // <u, du> and the clock gradient of u = U(-lambda) Y
        for (int r = wave; r < kC; r += NT / 64) {
            const float ud = wsum(Us[r][lane] * dUs[r][lane] + Us[r][lane + 64] * dUs[r][lane + 64]);
            const float gl = rot_grad(dUs[r], Us[r], m, -1.f, lane);
            if (lane == 0) {
                p.udu[row0 + r] = ud;
                dlu[r] = gl;
            }
        }
        __syncthreads();
        // dY = U(lambda) du
        rotate_rows<NT>(dUs, tab, m, 1.f, 1.f, tid);
        __syncthreads();
        // dW = M dY;  dM += W dY^T
        readout_product<false, NT>(Ms, dUs, dWs, m, tid);
#pragma unroll 1
        for (int r = 0; r < kC; ++r) {
            const float w = Ws[r][i];
#pragma unroll
            for (int jj = 0; jj < MH; ++jj) dMacc[jj] = fmaf(w, dUs[r][part * MH + jj], dMacc[jj]);
        }
        __syncthreads();
        // dZ = W (.) (dW - <W, dW>)
        for (int r = wave; r < kC; r += NT / 64) {
            const float w0 = Ws[r][lane], w1 = Ws[r][lane + 64];
            const float d0 = dWs[r][lane], d1 = dWs[r][lane + 64];
            const float sd = wsum(w0 * d0 + w1 * d1);
            dWs[r][lane] = w0 * (d0 - sd);
            dWs[r][lane + 64] = w1 * (d1 - sd);
        }
        __syncthreads();
        // dM += dZ X^T;  dX = M^T dZ (into the dY tile)
#pragma unroll 1
        for (int r = 0; r < kC; ++r) {
            const float dz = dWs[r][i];
#pragma unroll
            for (int jj = 0; jj < MH; ++jj) dMacc[jj] = fmaf(dz, Xs[r][part * MH + jj], dMacc[jj]);
        }
        __syncthreads();
        readout_product<true, NT>(Ms, dWs, dUs, m, tid);
        __syncthreads();
        // clock gradient of X = scale U(lambda) p, plus that of u
        for (int r = wave; r < kC; r += NT / 64) {
            const float gl = rot_grad(dUs[r], Xs[r], m, 1.f, lane);
            if (lane == 0) p.dlam[row0 + r] = dlu[r] + gl;
        }
        __syncthreads();
        // dp = scale U(-lambda) dX
        rotate_rows<NT>(dUs, tab, m, -1.f, p.scale, tid);
        __syncthreads();
        for (int e = tid; e < kC * kStoreRows; e += NT) {
            const int r = e >> 7, ii = e & 127;
            p.dP[(row0 + r) * kStoreRows + ii] = dUs[r][ii];
        }
        __syncthreads();
    }
    float *dMo = p.dMp + (((size_t)bh * p.groups + g) * kStoreRows + i) * kStoreRows + part * MH;
#pragma unroll
    for (int jj = 0; jj < MH; ++jj) dMo[jj] = dMacc[jj];
}

// ---------------------------------------------------------------------------
// (3a) adjoint states at every chunk's end from the chunk group's own later
// tokens (zero at the group's end), reverse over the group's chunks, per
// (sequence, group).  Thread layout as in (1a).  The adjoint of the state
// entering the group goes to AcK/AcV[g].
template <int DK, int DV, typename Tin>
__global__ __launch_bounds__(kNT) void bwd_adjoint_local_kernel(BwdParams p) {
    constexpr int NRK = DK * kStoreRows / kNT, NRV = DV * kStoreRows / kNT;
    __shared__ float Qs[kC][DK];
    __shared__ float dOs[kC][DV];
    __shared__ __attribute__((aligned(16))) float Wp[kC][kStoreRows];   // gamma_r dp_r
    __shared__ __attribute__((aligned(16))) float Wu[kC][kStoreRows];   // gamma_r u_r
    __shared__ float Gs[kC];
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H, tid = threadIdx.x;
    const int ck = tid % DK, rk = (tid / DK) * NRK;
    const int cv = tid % DV, rv = (tid / DV) * NRV;
    const int Tb = bwd_tokens(p, b);
    const int c_begin = g * p.cpg, c_end = min(c_begin + p.cpg, p.nc);
    float ak[NRK], av[NRV];
#pragma unroll
    for (int ii = 0; ii < NRK; ++ii) ak[ii] = 0.f;
#pragma unroll
    for (int ii = 0; ii < NRV; ++ii) av[ii] = 0.f;
    float Go = 0.f;
    for (int c = c_end - 1; c >= c_begin; --c) {
        const int t0 = c * kC;
        const size_t row0 = (size_t)bh * p.Tpad + t0;
        float *Kd = p.DKe + ((size_t)bh * p.nc + c) * kStoreRows * DK + ck;
        float *Vd = p.DVe + ((size_t)bh * p.nc + c) * kStoreRows * DV + cv;
#pragma unroll
        for (int ii = 0; ii < NRK; ++ii) Kd[(size_t)(rk + ii) * DK] = ak[ii];
#pragma unroll
        for (int ii = 0; ii < NRV; ++ii) Vd[(size_t)(rv + ii) * DV] = av[ii];
        if (tid == 0) p.Gout[(size_t)bh * p.nc + c] = Go;
        for (int e = tid; e < kC * DK; e += kNT) {
            const int r = e / DK, cc = e % DK;
            Qs[r][cc] = ld_row<Tin>(p.q, brow0(p, b), t0 + r, h, cc, p.H, DK, t0 + r < Tb);
        }
        for (int e = tid; e < kC * DV; e += kNT) {
            const int r = e / DV, cc = e % DV;
            dOs[r][cc] = ld_row<Tin>(p.dout, brow0(p, b), t0 + r, h, cc, p.H, DV, t0 + r < Tb);
        }
        if (tid < kC) {
            const int t = t0 + tid;
            Gs[tid] = (t < Tb && p.log_alpha) ? p.log_alpha[(brow0(p, b) + t) * p.H + h] : 0.f;
        }
        __syncthreads();
        if (tid == 0)
            for (int r = 1; r < kC; ++r) Gs[r] += Gs[r - 1];
        __syncthreads();
        for (int e = tid; e < kC * kStoreRows; e += kNT) {
            const int r = e >> 7, ii = e & 127;
            const float gr = __expf(Gs[r]);
            Wp[r][ii] = gr * p.dP[(row0 + r) * kStoreRows + ii];
            Wu[r][ii] = gr * p.U[(row0 + r) * kStoreRows + ii];
        }
        __syncthreads();
        const float gC = __expf(Gs[kC - 1]);
#pragma unroll
        for (int ii = 0; ii < NRK; ++ii) ak[ii] *= gC;
#pragma unroll
        for (int ii = 0; ii < NRV; ++ii) av[ii] *= gC;
#pragma unroll 1
        for (int r = 0; r < kC; ++r) {
            const float qr = Qs[r][ck], dor = dOs[r][cv];
#pragma unroll
            for (int ii = 0; ii < NRK; ++ii) ak[ii] = fmaf(Wp[r][rk + ii], qr, ak[ii]);
#pragma unroll
            for (int ii = 0; ii < NRV; ++ii) av[ii] = fmaf(Wu[r][rv + ii], dor, av[ii]);
        }
        Go += Gs[kC - 1];
        __syncthreads();
    }
    float *Ko = p.AcK + ((size_t)bh * p.groups + g) * kStoreRows * DK + ck;
    float *Vo = p.AcV + ((size_t)bh * p.groups + g) * kStoreRows * DV + cv;
#pragma unroll
    for (int ii = 0; ii < NRK; ++ii) Ko[(size_t)(rk + ii) * DK] = ak[ii];
#pragma unroll
    for (int ii = 0; ii < NRV; ++ii) Vo[(size_t)(rv + ii) * DV] = av[ii];
}

// (3b) adjoints at each group's end, per sequence, in reverse group order:
// A_{G-1} = (dK_T, dV_T), A_{g-1} = exp(Gg_g) A_g + (group g's own adjoint of its
// entering state); AcK/AcV[g] are overwritten with A_g, and the adjoint of the
// initial state is dK0, dV0.
template <int DK, int DV>
__global__ __launch_bounds__(kNT) void bwd_adjoint_combine_kernel(BwdParams p) {
    const int bh = blockIdx.x, tid = threadIdx.x, m = p.m, G = p.groups;
    const int e0 = blockIdx.y * kNT + tid, es = kCombBlocks * kNT;
    const float *Gg = p.Gg + (size_t)bh * G;
    for (int e = e0; e < kStoreRows * DK; e += es) {
        const bool act = e / DK < m;
        float A = (p.dK_T && act) ? p.dK_T[(size_t)bh * kStoreRows * DK + e] : 0.f;
        for (int g = G - 1; g >= 0; --g) {
            float *slot = p.AcK + ((size_t)bh * G + g) * kStoreRows * DK + e;
            const float own = *slot;
            *slot = A;
            A = fmaf(__expf(Gg[g]), A, own);
        }
        if (p.gK0) p.gK0[(size_t)bh * kStoreRows * DK + e] = act ? A : 0.f;
    }
    for (int e = e0; e < kStoreRows * DV; e += es) {
        const bool act = e / DV < m;
        float A = (p.dV_T && act) ? p.dV_T[(size_t)bh * kStoreRows * DV + e] : 0.f;
        for (int g = G - 1; g >= 0; --g) {
            float *slot = p.AcV + ((size_t)bh * G + g) * kStoreRows * DV + e;
            const float own = *slot;
            *slot = A;
            A = fmaf(__expf(Gg[g]), A, own);
        }
        if (p.gV0) p.gV0[(size_t)bh * kStoreRows * DV + e] = act ? A : 0.f;
    }
}

// ---------------------------------------------------------------------------
// (4) token gradients, per (sequence, chunk group).
// Column products (a sum over the 128 state rows) give thread (column cc, row
// block ih) the partial sums for all kC tokens; row products (a sum over state
// columns) give the kRP threads (row i, part) one state row, each a kRP-th of its columns.
template <int DK, int DV, typename Tin>
__global__ __launch_bounds__(kNT) void bwd_grad_kernel(BwdParams p) {
    constexpr int KH = DK / kRP, VH = DV / kRP;
    constexpr int IHK = kNT / DK, IHV = kNT / DV;          // row blocks of the column products
    // token rows per pass of the column products: all of them up to d = 128; two passes
    // at d = 256, which halves their partial-sum buffer so that the tiles fit LDS
    constexpr int kCP = (DK > 128 || DV > 128) ? kC / 2 : kC;
    __shared__ float Qs[kC][DK + 1], Ks[kC][DK + 1];
    __shared__ float Vs[kC][DV + 1], dOs[kC][DV + 1];
    __shared__ float dPs[kC][kLD], Us[kC][kLD], As[kC][kLD], dAK[kC][kLD], dAV[kC][kLD];
    __shared__ __attribute__((aligned(16))) float dPT[kStoreRows][kC];   // dp and A transposed:
    __shared__ __attribute__((aligned(16))) float AT[kStoreRows][kC];    // all tokens of a row in 64 bytes
    __shared__ float Sqk[kC][kC + 1], Sdpa[kC][kC + 1], Suoa[kC][kC + 1], Sdov[kC][kC + 1];
    __shared__ float red[kNT * kCP];
    __shared__ float qkp[2][kC][kNT / 64];    // <q, dq> and <k, dk> per token, per 64 columns
    __shared__ ChunkTab tab;
    const int bh = blockIdx.x, g = blockIdx.y, b = bh / p.H, h = bh % p.H, tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int i = tid / kRP, part = tid % kRP, m = p.m;
    const int Tb = bwd_tokens(p, b);
    const int c_begin = g * p.cpg, c_end = min(c_begin + p.cpg, p.nc);
    Tin *gq = static_cast<Tin *>(p.gq);
    Tin *gk = static_cast<Tin *>(p.gk);
    Tin *gv = static_cast<Tin *>(p.gv);
    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * kC;
        const size_t row0 = (size_t)bh * p.Tpad + t0;
        const size_t st = ((size_t)bh * p.nc + c) * kStoreRows;    // state row 0 of this chunk
        const size_t sg = ((size_t)bh * p.groups + g) * kStoreRows; // group carry row 0
        const float dec_in = __expf(p.Gin[(size_t)bh * p.nc + c]);
        const float dec_out = __expf(p.Gout[(size_t)bh * p.nc + c]);
        for (int e = tid; e < kC * DK; e += kNT) {
            const int r = e / DK, cc = e % DK;
            const bool live = t0 + r < Tb;
            Qs[r][cc] = ld_row<Tin>(p.q, brow0(p, b), t0 + r, h, cc, p.H, DK, live);
            Ks[r][cc] = ld_row<Tin>(p.k, brow0(p, b), t0 + r, h, cc, p.H, DK, live);
        }
        for (int e = tid; e < kC * DV; e += kNT) {
            const int r = e / DV, cc = e % DV;
            const bool live = t0 + r < Tb;
            Vs[r][cc] = ld_row<Tin>(p.v, brow0(p, b), t0 + r, h, cc, p.H, DV, live);
            dOs[r][cc] = ld_row<Tin>(p.dout, brow0(p, b), t0 + r, h, cc, p.H, DV, live);
        }
        for (int e = tid; e < kC * kStoreRows; e += kNT) {
            const int r = e >> 7, ii = e & 127;
            const float dp = p.dP[(row0 + r) * kStoreRows + ii];
            dPs[r][ii] = dp;
            dPT[ii][r] = dp;
            Us[r][ii] = p.U[(row0 + r) * kStoreRows + ii];
        }
        chunk_tables(p, b, h, t0, Tb, p.clk[(size_t)bh * p.nc + c], tab, tid);
        for (int e = tid; e < kC * kStoreRows; e += kNT) {
            const int r = e >> 7, i = e & 127;
            const float a = write_entry(tab, m, r, i, tab.beta[r]);
            As[r][i] = a;
            AT[i][r] = a;
        }
        __syncthreads();
        const float GC = tab.G[kC - 1];
        {   // the four masked score tiles: threads 0..255 the (q, k) and (do, v) tiles,
            // threads 256..511 the (dp, a) and (u, a) tiles
            const int half = tid / (kC * kC), e = tid % (kC * kC);
            const int r = e >> 4, s = e & 15;
            float a0 = 0.f, a1 = 0.f;
            if (s <= r) {
                const float gam = __expf(tab.G[r] - tab.G[s]);
                if (half == 0) {
#pragma unroll 4
                    for (int cc = 0; cc < DK; ++cc) a0 = fmaf(Qs[r][cc], Ks[s][cc], a0);
#pragma unroll 4
                    for (int cc = 0; cc < DV; ++cc) a1 = fmaf(dOs[r][cc], Vs[s][cc], a1);
                } else {
#pragma unroll 4
                    for (int ii = 0; ii < kStoreRows; ++ii) {
                        a0 = fmaf(dPs[r][ii], As[s][ii], a0);
                        a1 = fmaf(Us[r][ii], As[s][ii], a1);
                    }
                }
                a0 *= gam;
                a1 *= gam;
            }
            if (half == 0) {
                Sqk[r][s] = a0;
                Sdov[r][s] = a1;
            } else {
                Sdpa[r][s] = a0;
                Suoa[r][s] = a1;
            }
        }
        // dq = gamma_r (dP Kbar_c)[r] + (Sdpa K)[r], dk = (Sdpa^T Q)[s] + rho_s (A DK')[s] and
        // dv = (Suoa^T dO)[s] + rho_s (A DV')[s], written out as formed, kCP token rows per
        // pass; the per-token <q, dq> and <k, dk> are reduced on the way (per wave: 64
        // columns of one row)
        for (int r0 = 0; r0 < kC; r0 += kCP) {
            {
                const int cc = tid % DK, ih = tid / DK;
                constexpr int RB = kStoreRows / IHK;
                float acc[kCP];
#pragma unroll
                for (int r = 0; r < kCP; ++r) acc[r] = 0.f;
#pragma unroll 2
                for (int ii = ih * RB; ii < (ih + 1) * RB; ++ii) {
                    const float kb = fmaf(dec_in, p.EcK[(sg + ii) * DK + cc], p.Kst[(st + ii) * DK + cc]);
#pragma unroll
                    for (int q4 = 0; q4 < kCP / 4; ++q4) {
                        const float4 x = *reinterpret_cast<const float4 *>(&dPT[ii][r0 + 4 * q4]);
                        acc[4 * q4] = fmaf(x.x, kb, acc[4 * q4]);
                        acc[4 * q4 + 1] = fmaf(x.y, kb, acc[4 * q4 + 1]);
                        acc[4 * q4 + 2] = fmaf(x.z, kb, acc[4 * q4 + 2]);
                        acc[4 * q4 + 3] = fmaf(x.w, kb, acc[4 * q4 + 3]);
                    }
                }
#pragma unroll
                for (int r = 0; r < kCP; ++r) red[(ih * kCP + r) * DK + cc] = acc[r];
            }
            __syncthreads();
            for (int e = tid; e < kCP * DK; e += kNT) {
                const int r = r0 + e / DK, cc = e % DK;
                float sum = 0.f;
                for (int ih = 0; ih < IHK; ++ih) sum += red[(ih * kCP + r - r0) * DK + cc];
                float acc = __expf(tab.G[r]) * sum;
                for (int s = 0; s <= r; ++s) acc = fmaf(Sdpa[r][s], Ks[s][cc], acc);
                const float part = wsum(Qs[r][cc] * acc);
                if (lane == 0) qkp[0][r][cc >> 6] = part;
                const int t = t0 + r;
                if (t < p.T) store_from_float(gq, ((brow0(p, b) + t) * p.H + h) * DK + cc, t < Tb ? acc : 0.f);
            }
            __syncthreads();
            {
                const int cc = tid % DK, ih = tid / DK;
                constexpr int RB = kStoreRows / IHK;
                float acc[kCP];
#pragma unroll
                for (int r = 0; r < kCP; ++r) acc[r] = 0.f;
#pragma unroll 2
                for (int ii = ih * RB; ii < (ih + 1) * RB; ++ii) {
                    const float kb = fmaf(dec_out, p.AcK[(sg + ii) * DK + cc], p.DKe[(st + ii) * DK + cc]);
#pragma unroll
                    for (int q4 = 0; q4 < kCP / 4; ++q4) {
                        const float4 x = *reinterpret_cast<const float4 *>(&AT[ii][r0 + 4 * q4]);
                        acc[4 * q4] = fmaf(x.x, kb, acc[4 * q4]);
                        acc[4 * q4 + 1] = fmaf(x.y, kb, acc[4 * q4 + 1]);
                        acc[4 * q4 + 2] = fmaf(x.z, kb, acc[4 * q4 + 2]);
                        acc[4 * q4 + 3] = fmaf(x.w, kb, acc[4 * q4 + 3]);
                    }
                }
#pragma unroll
                for (int s2 = 0; s2 < kCP; ++s2) red[(ih * kCP + s2) * DK + cc] = acc[s2];
            }
            __syncthreads();
            for (int e = tid; e < kCP * DK; e += kNT) {
                const int s2 = r0 + e / DK, cc = e % DK;
                float sum = 0.f;
                for (int ih = 0; ih < IHK; ++ih) sum += red[(ih * kCP + s2 - r0) * DK + cc];
                float acc = __expf(GC - tab.G[s2]) * sum;
                for (int r = s2; r < kC; ++r) acc = fmaf(Sdpa[r][s2], Qs[r][cc], acc);
                const float part = wsum(Ks[s2][cc] * acc);
                if (lane == 0) qkp[1][s2][cc >> 6] = part;
                const int t = t0 + s2;
                if (t < p.T) store_from_float(gk, ((brow0(p, b) + t) * p.H + h) * DK + cc, t < Tb ? acc : 0.f);
            }
            __syncthreads();
            {
                const int cc = tid % DV, ih = tid / DV;
                constexpr int RB = kStoreRows / IHV;
                float acc[kCP];
#pragma unroll
                for (int r = 0; r < kCP; ++r) acc[r] = 0.f;
#pragma unroll 2
                for (int ii = ih * RB; ii < (ih + 1) * RB; ++ii) {
                    const float vb = fmaf(dec_out, p.AcV[(sg + ii) * DV + cc], p.DVe[(st + ii) * DV + cc]);
#pragma unroll
                    for (int q4 = 0; q4 < kCP / 4; ++q4) {
                        const float4 x = *reinterpret_cast<const float4 *>(&AT[ii][r0 + 4 * q4]);
                        acc[4 * q4] = fmaf(x.x, vb, acc[4 * q4]);
                        acc[4 * q4 + 1] = fmaf(x.y, vb, acc[4 * q4 + 1]);
                        acc[4 * q4 + 2] = fmaf(x.z, vb, acc[4 * q4 + 2]);
                        acc[4 * q4 + 3] = fmaf(x.w, vb, acc[4 * q4 + 3]);
                    }
                }
#pragma unroll
                for (int s2 = 0; s2 < kCP; ++s2) red[(ih * kCP + s2) * DV + cc] = acc[s2];
            }
            __syncthreads();
            for (int e = tid; e < kCP * DV; e += kNT) {
                const int s2 = r0 + e / DV, cc = e % DV;
                const int t = t0 + s2;
                if (t >= p.T) continue;
                float sum = 0.f;
                for (int ih = 0; ih < IHV; ++ih) sum += red[(ih * kCP + s2 - r0) * DV + cc];
                float acc = __expf(GC - tab.G[s2]) * sum;
                for (int r = s2; r < kC; ++r) acc = fmaf(Suoa[r][s2], dOs[r][cc], acc);
                store_from_float(gv, ((brow0(p, b) + t) * p.H + h) * DV + cc, t < Tb ? acc : 0.f);
            }
            __syncthreads();
        }
        // da, carried-state parts: rho_s (K DK'^T)[s][i] and rho_s (V DV'^T)[s][i];
        // thread (row i, part) sums its share of the columns for every token s
        {
            float ak[kC], av[kC];
#pragma unroll
            for (int s2 = 0; s2 < kC; ++s2) {
                ak[s2] = 0.f;
                av[s2] = 0.f;
            }
            const float *dkr = p.DKe + (st + i) * DK + part * KH;
            const float *dkc = p.AcK + (sg + i) * DK + part * KH;
#pragma unroll 1
            for (int cc = 0; cc < KH; cc += 4) {
                const float4 d0 = *reinterpret_cast<const float4 *>(dkr + cc);
                const float4 d1 = *reinterpret_cast<const float4 *>(dkc + cc);
                const float4 d = make_float4(fmaf(dec_out, d1.x, d0.x), fmaf(dec_out, d1.y, d0.y),
                                             fmaf(dec_out, d1.z, d0.z), fmaf(dec_out, d1.w, d0.w));
#pragma unroll
                for (int s2 = 0; s2 < kC; ++s2) {
                    const float *kk = &Ks[s2][part * KH + cc];
                    ak[s2] = fmaf(kk[0], d.x, fmaf(kk[1], d.y, fmaf(kk[2], d.z, fmaf(kk[3], d.w, ak[s2]))));
                }
            }
            const float *dvr = p.DVe + (st + i) * DV + part * VH;
            const float *dvc = p.AcV + (sg + i) * DV + part * VH;
#pragma unroll 1
            for (int cc = 0; cc < VH; cc += 4) {
                const float4 d0 = *reinterpret_cast<const float4 *>(dvr + cc);
                const float4 d1 = *reinterpret_cast<const float4 *>(dvc + cc);
                const float4 d = make_float4(fmaf(dec_out, d1.x, d0.x), fmaf(dec_out, d1.y, d0.y),
                                             fmaf(dec_out, d1.z, d0.z), fmaf(dec_out, d1.w, d0.w));
#pragma unroll
                for (int s2 = 0; s2 < kC; ++s2) {
                    const float *vv = &Vs[s2][part * VH + cc];
                    av[s2] = fmaf(vv[0], d.x, fmaf(vv[1], d.y, fmaf(vv[2], d.z, fmaf(vv[3], d.w, av[s2]))));
                }
            }
#pragma unroll
            for (int s2 = 0; s2 < kC; ++s2) {
                float a = ak[s2] + __shfl_xor(ak[s2], 1);
                float bv = av[s2] + __shfl_xor(av[s2], 1);
                a += __shfl_xor(a, 2);
                bv += __shfl_xor(bv, 2);
                if (part == 0) {
                    const float rho = __expf(GC - tab.G[s2]);
                    dAK[s2][i] = rho * a;
                    dAV[s2][i] = rho * bv;
                }
            }
        }
        __syncthreads();
        // da, intra-chunk parts; dAK then holds the whole da
        for (int e = tid; e < kC * kStoreRows; e += kNT) {
            const int s = e >> 7, ii = e & 127;
            float av = dAV[s][ii], ak = dAK[s][ii];
            for (int r = s; r < kC; ++r) {
                av = fmaf(Sdov[r][s], Us[r][ii], av);
                ak = fmaf(Sqk[r][s], dPs[r][ii], ak);
            }
            dAV[s][ii] = av;
            dAK[s][ii] = ak + av;
        }
        __syncthreads();
        // per token: dbeta, clock gradient of a, dL/dG; dq and dk rows out
        for (int s = wave; s < kC; s += kNT / 64) {
            const int t = t0 + s;
            float qdq = 0.f, kdk = 0.f;                // whole-token sums (every lane alike)
            for (int j = 0; j < DK / 64; ++j) {
                qdq += qkp[0][s][j];
                kdk += qkp[1][s][j];
            }
            const float adav = As[s][lane] * dAV[s][lane] + As[s][lane + 64] * dAV[s][lane + 64];
            // <da, U(-lambda) b>: DC entry and the (cos, -sin) pairs
            float db = 0.f;
            {
                const int J = (m - 1) / 2, j = lane + 1;
                if (j <= J) {
                    const float2 cs = tab.cs[s][j - 1];
                    db = sqrtf(2.f / (float)m) * (cs.x * dAK[s][2 * j - 1] - cs.y * dAK[s][2 * j]);
                }
                if (lane == 0) db += dAK[s][0] / sqrtf((float)m);
            }
            const float gl = rot_grad(dAK[s], As[s], m, -1.f, lane);
            const float sums = (qdq - kdk) - wsum(adav);
            db = wsum(db);
            if (lane == 0 && t < p.T) {
                const size_t ti = row0 + s;
                const bool live = t < Tb;
                p.dG[ti] = live ? sums + p.udu[ti] : 0.f;
                p.dlam[ti] = live ? p.dlam[ti] + gl : 0.f;
                if (p.gbeta) p.gbeta[(brow0(p, b) + t) * p.H + h] = live ? db : 0.f;
            }
        }
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// (5) reverse cumulative sums per sequence: dlog_alpha_t = sum_{tau >= t} dG_tau
// (with the final-state term at the last token), ddelta_t = sum_{tau >= t}
// dlambda_tau, dclock0 = sum_t dlambda_t, all in double.  Workgroup (b h, piece)
// handles one of kScanPieces consecutive pieces of the sequence: it sums the tokens
// after its piece itself (loads batched eight per thread), and within the piece each
// thread sums its own run of tokens; the sum of the later runs is the piece total
// minus an inclusive prefix over the threads (wave prefix sums, then one offset per
// wave).  The thread that ends at token 0 holds the whole sum, dclock0.
constexpr int kScanPieces = 8;
__global__ __launch_bounds__(kNT) void bwd_scan_kernel(BwdParams p) {
    constexpr int kW = kNT / 64;
    __shared__ double sG[kW], sL[kW];
    const int bh = blockIdx.x, pc = blockIdx.y, b = bh / p.H, h = bh % p.H, tid = threadIdx.x, lane = tid & 63,
              wv = tid >> 6;
    const int Tb = bwd_tokens(p, b);
    const float *dG = p.dG + (size_t)bh * p.Tpad;
    const float *dl = p.dlam + (size_t)bh * p.Tpad;
    float fin = 0.f;
    for (int u = 0; u < kCombBlocks; ++u) fin += p.fin[(size_t)bh * kCombBlocks + u];
    const int pp = (Tb + kScanPieces - 1) / kScanPieces;
    const int P0 = min(pc * pp, Tb), P1 = min(P0 + pp, Tb);
    // tokens after the piece
    double lG = 0.0, lL = 0.0;
    for (int t0 = P1; t0 < Tb; t0 += 8 * kNT) {
        float vg[8], vl[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int t = t0 + u * kNT + tid;
            vg[u] = t < Tb ? dG[t] : 0.f;
            vl[u] = t < Tb ? dl[t] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            lG += vg[u];
            lL += vl[u];
        }
    }
    if (P1 < Tb && tid == 0) lG += fin;
    for (int o = 32; o > 0; o >>= 1) {
        lG += __shfl_xor(lG, o);
        lL += __shfl_xor(lL, o);
    }
    if (lane == 0) {
        sG[wv] = lG;
        sL[wv] = lL;
    }
    __syncthreads();
    double LG = 0.0, LL = 0.0;
#pragma unroll
    for (int u = 0; u < kW; ++u) {
        LG += sG[u];
        LL += sL[u];
    }
    __syncthreads();
    const int per = (P1 - P0 + kNT - 1) / kNT;
    const int t_lo = min(P0 + tid * per, P1), t_hi = min(t_lo + per, P1);
    double aG = 0.0, aL = 0.0;
    for (int t = t_lo; t < t_hi; ++t) {
        aG += dG[t] + (t == Tb - 1 ? fin : 0.f);
        aL += dl[t];
    }
    const double iG = mfma::wave_incl_scan(aG), iL = mfma::wave_incl_scan(aL);
    if (lane == 63) {
        sG[wv] = iG;
        sL[wv] = iL;
    }
    __syncthreads();
    double oG = 0.0, oL = 0.0, TG = 0.0, TL = 0.0;
#pragma unroll
    for (int u = 0; u < kW; ++u) {
        if (u < wv) {
            oG += sG[u];
            oL += sL[u];
        }
        TG += sG[u];
        TL += sL[u];
    }
    double rg = LG + (TG - (oG + iG)), rl = LL + (TL - (oL + iL));   // sums over the later tokens
    for (int t = t_hi - 1; t >= t_lo; --t) {
        rg += dG[t] + (t == Tb - 1 ? fin : 0.f);
        rl += dl[t];
        const size_t si = (brow0(p, b) + t) * p.H + h;
        if (p.glog_alpha) p.glog_alpha[si] = (float)rg;
        p.gdelta[si] = (float)rl;
    }
    if (pc == 0 && tid == 0 && p.gclock0) p.gclock0[bh] = rl;       // t_lo = 0: every token
    for (int t = Tb + pc * kNT + tid; t < p.T; t += kScanPieces * kNT) {
        const size_t si = (brow0(p, b) + t) * p.H + h;
        if (p.glog_alpha) p.glog_alpha[si] = 0.f;
        p.gdelta[si] = 0.f;
    }
}

// ---------------------------------------------------------------------------
// (6) dR_h = (sum over sequences b and chunk groups of dM) Phi^T on the active
// m x m block (M = R Phi, Phi the real Fourier basis of App. A.1).  Workgroup
// (h, row block) handles kDRRows rows of dR, which need the same rows of dM only.
constexpr int kDRRows = 8;
__global__ __launch_bounds__(kNT) void bwd_dR_kernel(BwdParams p) {
    __shared__ float dM[kDRRows][kLD];
    __shared__ float tab[2][kStoreRows];
    const int h = blockIdx.x, i0 = blockIdx.y * kDRRows, tid = threadIdx.x, m = p.m;
    const int nb = p.B * p.groups;
    for (int e = tid; e < kDRRows * kStoreRows; e += kNT) {
        const int ii = e >> 7, j = e & 127;
        float s = 0.f;
        for (int u0 = 0; u0 < nb; u0 += 8) {
            float v[8];                             // eight loads in flight, summed in order
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int u = u0 + k, b = u / p.groups, g = u % p.groups;
                v[k] = u < nb ? p.dMp[(((size_t)(b * p.H + h) * p.groups + g) * kStoreRows + i0 + ii) * kStoreRows + j]
                              : 0.f;
            }
#pragma unroll
            for (int k = 0; k < 8; ++k)
                if (u0 + k < nb) s += v[k];
        }
        dM[ii][j] = s;
    }
    if (tid < m) {
        double sn, cs;
        sincospi(2.0 * (double)tid / (double)m, &sn, &cs);
        tab[0][tid] = (float)cs;
        tab[1][tid] = (float)sn;
    }
    __syncthreads();
    const float dc = 1.f / sqrtf((float)m), ac = sqrtf(2.f / (float)m);
    for (int e = tid; e < kDRRows * m; e += kNT) {
        const int ii = e / m, s = e % m;
        if (i0 + ii >= m) continue;
        float acc = dM[ii][0] * dc;
        int n = 0;                                  // l s mod m, advanced by s per step
        for (int l = 1; 2 * l < m; ++l) {
            n += s;
            if (n >= m) n -= m;
            acc = fmaf(dM[ii][2 * l - 1], ac * tab[0][n], acc);
            acc = fmaf(dM[ii][2 * l], ac * tab[1][n], acc);
        }
        p.gR[((size_t)h * m + i0 + ii) * m + s] = acc;
    }
}

template <int DK, int DV, typename Tin>
hipError_t launch_typed(const BwdParams &p, hipStream_t s) {
    const int BH = p.B * p.H;
    const dim3 block(kNT), grp(BH, p.groups);
    hipLaunchKernelGGL((bwd_states_local_kernel<DK, DV, Tin>), grp, block, 0, s, p);
    hipLaunchKernelGGL((bwd_states_combine_kernel<DK, DV>), dim3(BH, kCombBlocks), block, 0, s, p);
    hipLaunchKernelGGL((bwd_readout_kernel<DK, DV, Tin>), grp, dim3(kReadoutThreads), 0, s, p);
    hipLaunchKernelGGL((bwd_adjoint_local_kernel<DK, DV, Tin>), grp, block, 0, s, p);
    hipLaunchKernelGGL((bwd_adjoint_combine_kernel<DK, DV>), dim3(BH, kCombBlocks), block, 0, s, p);
    hipLaunchKernelGGL((bwd_grad_kernel<DK, DV, Tin>), grp, block, 0, s, p);
    return launch_bwd_tail(p, s);
}

template <int DK, int DV>
hipError_t launch_dtype(const BwdParams &p, hipStream_t s) {
    return p.dtype == 0 ? launch_typed<DK, DV, float>(p, s) : launch_typed<DK, DV, __hip_bfloat16>(p, s);
}

size_t align_up(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

hipError_t launch_bwd_tail(const BwdParams &p, hipStream_t s) {
    hipLaunchKernelGGL(bwd_scan_kernel, dim3(p.B * p.H, kScanPieces), dim3(kNT), 0, s, p);
    if (p.gR) hipLaunchKernelGGL(bwd_dR_kernel, dim3(p.H, kStoreRows / kDRRows), dim3(kNT), 0, s, p);
    return hipGetLastError();
}

int bwd_auto_groups(int B, int T, int H) {
    const int nc = (T + kC - 1) / kC;
    const int BH = B * H;
    int g = (512 + BH - 1) / BH;
    if (g > nc) g = nc;
    return g < 1 ? 1 : g;
}

// Layout (each piece 256-byte aligned): M, Kst, Vst, clk, DKe, DVe, EcK, EcV,
// AcK, AcV, Gin, Gout, Gg, U, dP, udu, dlam, dG, dMp, fin.
size_t bwd_workspace_bytes(int B, int T, int H, int dk, int dv, int groups) {
    const size_t BH = (size_t)B * H, nc = ((size_t)T + kC - 1) / kC, Tpad = nc * kC;
    const size_t st = BH * nc * kStoreRows * (size_t)(dk + dv) * 4;
    const size_t gc = BH * (size_t)groups * kStoreRows * (size_t)(dk + dv) * 4;
    size_t n = align_up(readout_f32_bytes(H));
    n += align_up(st);                                   // Kst + Vst
    n += align_up(BH * nc * 8);                          // clk
    n += align_up(st);                                   // DKe + DVe
    n += 2 * align_up(gc);                               // EcK + EcV, AcK + AcV
    n += 2 * align_up(BH * nc * 4) + align_up(BH * (size_t)groups * 4);   // Gin, Gout, Gg
    n += 2 * align_up(BH * Tpad * kStoreRows * 4);       // U, dP
    n += 3 * align_up(BH * Tpad * 4);                    // udu, dlam, dG
    n += align_up(BH * (size_t)groups * kStoreRows * kStoreRows * 4);
    n += align_up(BH * kCombBlocks * 4);
    return n;
}

size_t group_states_bytes(int B, int H, int dk, int dv, int groups) {
    const size_t BH = (size_t)B * H;
    return align_up(BH * (size_t)groups * kStoreRows * (size_t)(dk + dv) * 4) +
           align_up(BH * (size_t)groups * 4) + align_up(BH * kCombBlocks * 4) +
           align_up(BH * (size_t)groups * 8);
}

hipError_t launch_group_states(const FwdParams &f, int groups, int cpg, void *ws, const float **EcK,
                               const float **EcV, const double **Eclk, hipStream_t s) {
    BwdParams p{};
    p.B = f.B; p.T = f.T; p.H = f.H; p.dk = f.dk; p.dv = f.dv; p.m = f.m;
    p.nc = (f.T + kC - 1) / kC;
    p.Tpad = p.nc * kC;
    p.groups = groups;
    p.cpg = cpg;
    p.scale = f.scale; p.dtype = f.dtype;
    p.q = f.q; p.k = f.k; p.v = f.v;
    p.delta = f.delta; p.log_alpha = f.log_alpha; p.beta = f.beta; p.lens = f.lens; p.cu = f.cu;
    p.K0 = f.K0; p.V0 = f.V0; p.clock0 = f.clock0;
    const size_t BH = (size_t)f.B * f.H;
    char *w = static_cast<char *>(ws);
    auto take = [&w](size_t bytes) { char *r = w; w += align_up(bytes); return r; };
    const size_t gcar = BH * (size_t)groups * kStoreRows;
    p.EcK = reinterpret_cast<float *>(take(gcar * (size_t)(f.dk + f.dv) * 4));
    p.EcV = p.EcK + gcar * f.dk;
    p.Gg = reinterpret_cast<float *>(take(BH * (size_t)groups * 4));
    p.fin = reinterpret_cast<float *>(take(BH * kCombBlocks * 4));
    p.gclk = reinterpret_cast<double *>(take(BH * (size_t)groups * 8));
    *EcK = p.EcK;
    *EcV = p.EcV;
    *Eclk = p.gclk;
    const dim3 block(kNT), grp(f.B * f.H, groups), comb(f.B * f.H, kCombBlocks);
    auto go = [&](auto dk_tag, auto dv_tag) {
        constexpr int DK = decltype(dk_tag)::value, DV = decltype(dv_tag)::value;
        if (f.dtype == 0) {
            hipLaunchKernelGGL((bwd_states_local_kernel<DK, DV, float>), grp, block, 0, s, p);
        } else {
            hipLaunchKernelGGL((bwd_states_local_kernel<DK, DV, __hip_bfloat16>), grp, block, 0, s, p);
        }
        hipLaunchKernelGGL((bwd_states_combine_kernel<DK, DV>), comb, block, 0, s, p);
    };
    using I64 = std::integral_constant<int, 64>;
    using I128 = std::integral_constant<int, 128>;
    if (f.dk == 64 && f.dv == 64) go(I64{}, I64{});
    else if (f.dk == 64) go(I64{}, I128{});
    else if (f.dv == 64) go(I128{}, I64{});
    else go(I128{}, I128{});
    return hipGetLastError();
}

hipError_t launch_bwd_valu(BwdParams p, void *ws, hipStream_t s) {
    const size_t BH = (size_t)p.B * p.H, nc = p.nc, Tpad = p.Tpad;
    char *w = static_cast<char *>(ws);
    auto take = [&w](size_t bytes) { char *r = w; w += align_up(bytes); return r; };
    float *M = reinterpret_cast<float *>(take(readout_f32_bytes(p.H)));
    char *st = take(BH * nc * kStoreRows * (size_t)(p.dk + p.dv) * 4);
    p.Kst = reinterpret_cast<float *>(st);
    p.Vst = p.Kst + BH * nc * kStoreRows * p.dk;
    p.clk = reinterpret_cast<double *>(take(BH * nc * 8));
    char *ad = take(BH * nc * kStoreRows * (size_t)(p.dk + p.dv) * 4);
    p.DKe = reinterpret_cast<float *>(ad);
    p.DVe = p.DKe + BH * nc * kStoreRows * p.dk;
    const size_t gcar = BH * (size_t)p.groups * kStoreRows;
    p.EcK = reinterpret_cast<float *>(take(gcar * (size_t)(p.dk + p.dv) * 4));
    p.EcV = p.EcK + gcar * p.dk;
    p.AcK = reinterpret_cast<float *>(take(gcar * (size_t)(p.dk + p.dv) * 4));
    p.AcV = p.AcK + gcar * p.dk;
    p.Gin = reinterpret_cast<float *>(take(BH * nc * 4));
    p.Gout = reinterpret_cast<float *>(take(BH * nc * 4));
    p.Gg = reinterpret_cast<float *>(take(BH * (size_t)p.groups * 4));
    p.U = reinterpret_cast<float *>(take(BH * Tpad * kStoreRows * 4));
    p.dP = reinterpret_cast<float *>(take(BH * Tpad * kStoreRows * 4));
    p.udu = reinterpret_cast<float *>(take(BH * Tpad * 4));
    p.dlam = reinterpret_cast<float *>(take(BH * Tpad * 4));
    p.dG = reinterpret_cast<float *>(take(BH * Tpad * 4));
    p.dMp = reinterpret_cast<float *>(take(BH * (size_t)p.groups * kStoreRows * kStoreRows * 4));
    p.fin = reinterpret_cast<float *>(take(BH * kCombBlocks * 4));
    p.M = M;
    hipError_t e = launch_readout_prep(p.H, p.m, p.R, M, nullptr, 1.f, s);
    if (e != hipSuccess) return e;
    if (p.dk == 64 && p.dv == 64) return launch_dtype<64, 64>(p, s);
    if (p.dk == 64 && p.dv == 128) return launch_dtype<64, 128>(p, s);
    if (p.dk == 128 && p.dv == 64) return launch_dtype<128, 64>(p, s);
    if (p.dk == 256 && p.dv == 256) return launch_dtype<256, 256>(p, s);
    return launch_dtype<128, 128>(p, s);
}

}  // namespace cyfa
