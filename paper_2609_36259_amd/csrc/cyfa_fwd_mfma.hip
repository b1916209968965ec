// Matrix-core (bf16 MFMA) chunk-wise CyFA forward for d_k = d_v = 128, C = 64.
//
// Work decomposition.  Each (b, h) sequence is cut into P segments of whole
// chunks.  Four kernels run in order on the caller's stream:
//   1. segment_state_kernel  (b, h, p < P-1): the segment's own contribution to
//      the carried states, DeltaS_p = sum_t (decay to segment end) a_t [k_t | v_t]^T,
//      with the clock origin at the segment start, plus the segment's clock span
//      and log-decay total.  App. B's state recurrence run from a zero state.
//   2. segment_scan_kernel  (b, h): the states entering every segment,
//      S'_{p+1} = U(span_p) (exp(gsum_p) S'_p + DeltaS_p), each expressed with its
//      own segment-start clock origin.  Moving the origin rotates an
//      absolute-clock state by U(-c) and leaves the output unchanged
//      (App. A.4, Prop. 6), which is what makes the segments independent.
//   3. chunk_forward_kernel  (b, h, p): the fused forward of App. B over the
//      segment's chunks: clock/log-decay prefix sums, temporal write matrix
//      A (Eq. app-temporal-writes), key pass (Eq. app-cyfa-key-chunk), token-wise
//      softmax readout (Eq. cyfa-two-pass, middle line), value pass
//      (Eq. app-cyfa-value-chunk).  Both 128 x 128 fp32 states stay in MFMA
//      accumulators for the whole segment.
//   4. state_out_kernel  (b, h): rotates the last segment's final state back to
//      the absolute clock and writes it in the ABI layout (only when asked).
#include "cyfa_mfma_common.h"

namespace cyfa {

using namespace mfma;

struct MfmaArgs {
    FwdParams p;
    int P;               // segments per (b, h)
    int cps;             // chunks per segment
    int nchunks;         // chunks per sequence
    const __bf16 *Mz;    // [H][128][128]  row = slot i', column = internal basis j
    const __bf16 *My;    // [H][128][128]  row = internal basis j, column = slot i'
    float *seg_state;    // [B*H*P][2*128*128] accumulator-dump layout
    double *seg_span;    // [B*H*P] clock span of each segment (reduced mod m)
    double *seg_gsum;    // [B*H*P] sum of log alpha over each segment
    double *seg_origin;  // [B*H*P] absolute clock at each segment start (reduced)
    double *final_lam;   // [B*H] local clock after the last segment (reduced)
    int has_init;        // segment-entry states are read from seg_state
    int want_final;      // last segment dumps its final state into seg_state
};

namespace {

// ---- LDS map of the fused kernel (bytes) ----------------------------------
constexpr int R_Q = 0;                          // Q  [64][QS] bf16 -> X -> W
constexpr int R_K = R_Q + C * QS * 2;           // K  [64][QS] bf16 }  logits Z
constexpr int R_KT = R_K + C * QS * 2;          // K^T [128][TS] bf16 } [64][ZS] f32
constexpr int R_VT = R_KT + D * TS * 2;         // V^T [128][TS] bf16
constexpr int R_A = R_VT + D * TS * 2;          // A  [64][QS] bf16
constexpr int R_AT = R_A + C * QS * 2;          // A^T [128][TS] bf16 -> O'' [64][QS]
constexpr int R_ATD = R_AT + D * TS * 2;        // right-decayed A^T [128][TS] bf16
constexpr int R_S = R_ATD + D * TS * 2;         // scores [64][SS] bf16
constexpr int R_CS = R_S + C * SS * 2;          // (cos, sin) [64][64] half pairs
constexpr int R_SC = R_CS + C * 64 * 4;         // per-token scalars
constexpr int SMEM_BYTES = R_SC + 64 * (4 + 4 + 4 + 8) + 64;
static_assert(C * ZS * 4 <= R_VT - R_K, "logit tile must fit in the K / K^T region");
static_assert(C * QS * 2 <= D * TS * 2, "O'' must fit in the A^T region");
static_assert(SMEM_BYTES <= 160 * 1024, "LDS budget");

typedef _Float16 half2v __attribute__((ext_vector_type(2)));

union Piece {
    uint4 u;
    __bf16 b[8];
};

struct Tiles {
    __bf16 *Qs, *Ks, *KTs, *VTs, *As, *ATs, *ATds, *Ss, *Xs, *Ws, *Os;
    float *Zf;
    half2v *CS;
    float *Gs, *gam, *betas;
    double *lams;
    double *carry;
};

__device__ __forceinline__ Tiles tiles(char *smem) {
    Tiles t;
    t.Qs = reinterpret_cast<__bf16 *>(smem + R_Q);
    t.Xs = t.Qs;
    t.Ws = t.Qs;
    t.Ks = reinterpret_cast<__bf16 *>(smem + R_K);
    t.Zf = reinterpret_cast<float *>(smem + R_K);
    t.KTs = reinterpret_cast<__bf16 *>(smem + R_KT);
    t.VTs = reinterpret_cast<__bf16 *>(smem + R_VT);
    t.As = reinterpret_cast<__bf16 *>(smem + R_A);
    t.ATs = reinterpret_cast<__bf16 *>(smem + R_AT);
    t.Os = t.ATs;
    t.ATds = reinterpret_cast<__bf16 *>(smem + R_ATD);
    t.Ss = reinterpret_cast<__bf16 *>(smem + R_S);
    t.CS = reinterpret_cast<half2v *>(smem + R_CS);
    t.Gs = reinterpret_cast<float *>(smem + R_SC);
    t.gam = t.Gs + 64;
    t.betas = t.gam + 64;
    t.lams = reinterpret_cast<double *>(t.betas + 64);
    t.carry = t.lams + 64;
    return t;
}

// Global -> register prefetch of one chunk: 4 x 16-byte pieces per thread per
// tensor (rows r = e / 16, columns 8 (e % 16)), plus one token's scalars on wave 0.
struct Prefetch {
    uint4 q[4], k[4], v[4];
    float g, dl, be;
};

template <bool kWithQ>
__device__ __forceinline__ void load_chunk(const FwdParams &p, int b, int h, int t0, int tid,
                                           Prefetch &pf) {
    const uint4 zero = make_uint4(0, 0, 0, 0);
    const __bf16 *q = static_cast<const __bf16 *>(p.q);
    const __bf16 *k = static_cast<const __bf16 *>(p.k);
    const __bf16 *v = static_cast<const __bf16 *>(p.v);
#pragma unroll
    for (int it = 0; it < 4; ++it) {
        const int e = it * NT + tid;
        const int r = e >> 4, d0 = (e & 15) * 8;
        const int t = t0 + r;
        if (t < p.T) {
            const size_t off = (((size_t)b * p.T + t) * p.H + h) * D + d0;
            if (kWithQ) pf.q[it] = *reinterpret_cast<const uint4 *>(q + off);
            pf.k[it] = *reinterpret_cast<const uint4 *>(k + off);
            pf.v[it] = *reinterpret_cast<const uint4 *>(v + off);
        } else {
            if (kWithQ) pf.q[it] = zero;
            pf.k[it] = zero;
            pf.v[it] = zero;
        }
    }
    if (tid < 64) {
        const int t = t0 + tid;
        if (t < p.T) {
            const size_t si = ((size_t)b * p.T + t) * p.H + h;
            pf.dl = p.delta[si];
            pf.g = p.log_alpha ? p.log_alpha[si] : 0.f;
            pf.be = p.beta ? p.beta[si] : 1.f;
        } else {
            pf.dl = 0.f;   // tokens past the end: no shift, no decay, no write
            pf.g = 0.f;
            pf.be = 0.f;
        }
    }
}

// Registers -> LDS: Q and K row-major, K and V transposed.
template <bool kWithQ>
__device__ __forceinline__ void store_chunk(const Tiles &s, int tid, const Prefetch &pf) {
    const int r0 = tid >> 4, d0 = (tid & 15) * 8;
    __bf16 *qrow = s.Qs + r0 * QS + d0;
    __bf16 *krow = s.Ks + r0 * QS + d0;
    __bf16 *ktcol = s.KTs + d0 * TS + r0;
    __bf16 *vtcol = s.VTs + d0 * TS + r0;
#pragma unroll
    for (int it = 0; it < 4; ++it) {            // piece it: row r0 + 16 it
        if (kWithQ) {
            *reinterpret_cast<uint4 *>(qrow + 16 * it * QS) = pf.q[it];
            *reinterpret_cast<uint4 *>(krow + 16 * it * QS) = pf.k[it];
        }
        Piece pk, pv;
        pk.u = pf.k[it];
        pv.u = pf.v[it];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            ktcol[j * TS + 16 * it] = pk.b[j];
            vtcol[j * TS + 16 * it] = pv.b[j];
        }
    }
}

// Wave 0: chunk-local inclusive prefix sums of log alpha (float) and of the
// clock increments (double, continuing the carried clock), reduced mod m.
__device__ __forceinline__ void chunk_scans(const Tiles &s, int lane, int m, const Prefetch &pf,
                                            double &carry, double &gsum) {
    const float G = wave_incl_scan(pf.g, lane);
    const double lam = carry + wave_incl_scan((double)pf.dl, lane);
    s.Gs[lane] = G;
    s.gam[lane] = __expf(G);
    s.betas[lane] = pf.be;
    s.lams[lane] = reduce_clock(lam, m);
    const double last = __shfl(lam, 63);
    carry = reduce_clock(last, m);
    gsum += (double)__shfl(G, 63);
}

// Temporal write matrix for the chunk (Eq. app-temporal-writes):
// A_r = beta_r U(-lambda_r) b, i.e. beta_r [sqrt(2/m) cos th_j, -sqrt(2/m) sin th_j]
// on pair j and beta_r / sqrt(m) on DC, th_j = 2 pi j lambda_r / m.
// Thread (r = tid / 4, quarter q = tid % 4) handles frequencies 16q+1 .. 16q+16;
// the phases advance by angle addition from an accurately reduced start.
template <bool kFull>
__device__ __forceinline__ void build_writes(const Tiles &s, int tid, int m) {
    const int r = tid >> 2, q = tid & 3;
    const int J = (m - 1) >> 1;
    const float dc = 1.0f / sqrtf((float)m);
    const float ac = sqrtf(2.0f / (float)m);
    const float be = s.betas[r];
    const float wdec = __expf(s.Gs[63] - s.Gs[r]);
    const double u = s.lams[r] / (double)m;          // revolutions per unit frequency
    float s1, c1, sn, cs;
    sincos_rev((float)u, &s1, &c1);
    {
        const int j0 = 16 * q + 1;
        double rev = (double)j0 * u;
        rev -= floor(rev);
        sincos_rev((float)rev, &sn, &cs);
    }
    __bf16 *As_t = s.As + r * QS + 32 * q;
    __bf16 *ATs_t = s.ATs + 32 * q * TS + r;
    __bf16 *ATds_t = s.ATds + 32 * q * TS + r;
    half2v *CS_t = s.CS + r * 64 + 16 * q;
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) {
        const int j = 16 * q + 1 + jj;
        if (j <= 63) {
            const float cv = j <= J ? cs : 0.f;
            const float sv = j <= J ? sn : 0.f;
            const float a_c = be * ac * cv, a_s = -be * ac * sv;
            // internal columns 32 q + 2 jj (cos) and 32 q + 2 jj + 1 (sin)
            if (kFull) {
                CS_t[jj] = half2v{(_Float16)cv, (_Float16)sv};
                bf16x2 pr;
                pr[0] = (__bf16)a_c;
                pr[1] = (__bf16)a_s;
                *reinterpret_cast<bf16x2 *>(As_t + 2 * jj) = pr;
                ATs_t[(2 * jj) * TS] = (__bf16)a_c;
                ATs_t[(2 * jj + 1) * TS] = (__bf16)a_s;
            }
            ATds_t[(2 * jj) * TS] = (__bf16)(a_c * wdec);
            ATds_t[(2 * jj + 1) * TS] = (__bf16)(a_s * wdec);
        }
        const float nc = cs * c1 - sn * s1;
        const float ns = sn * c1 + cs * s1;
        cs = nc;
        sn = ns;
    }
    if (q == 3) {
        const float a0 = be * dc;
        if (kFull) {
            bf16x2 pr;
            pr[0] = (__bf16)a0;
            pr[1] = (__bf16)0.f;
            *reinterpret_cast<bf16x2 *>(s.As + r * QS + kDC) = pr;
            s.ATs[kDC * TS + r] = (__bf16)a0;
            s.ATs[(kDC + 1) * TS + r] = (__bf16)0.f;
        }
        s.ATds[kDC * TS + r] = (__bf16)(a0 * wdec);
        s.ATds[(kDC + 1) * TS + r] = (__bf16)0.f;
    }
}

// Carried-state updates of one chunk (App. B):
//   Kbar^T <- gamma^C Kbar^T + K^T (right-decayed A),  Vbar <- gamma^C Vbar + (right-decayed A)^T V
__device__ __forceinline__ void update_states(const Tiles &s, int w, int l32, int hl,
                                              f32x16 (&kacc)[4], f32x16 (&vacc)[4]) {
    const float gC = s.gam[63];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            kacc[x][v] *= gC;
            vacc[x][v] *= gC;
        }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
        const bf16x8 at_w = lds8(s.ATds + (32 * w + l32) * TS + 16 * ks + 8 * hl);
        const bf16x8 vt_w = lds8(s.VTs + (32 * w + l32) * TS + 16 * ks + 8 * hl);
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            const bf16x8 kt = lds8(s.KTs + (32 * x + l32) * TS + 16 * ks + 8 * hl);
            kacc[x] = mma(kt, at_w, kacc[x]);
            const bf16x8 atd = lds8(s.ATds + (32 * x + l32) * TS + 16 * ks + 8 * hl);
            vacc[x] = mma(atd, vt_w, vacc[x]);
        }
    }
}

// row offset (within a 64-row tile, excluding the lane's 4h) of accumulator register v of block blk
__device__ __forceinline__ constexpr int acc_off(int blk, int v) {
    return 32 * blk + 8 * (v >> 2) + (v & 3);
}

// Causal score tile (S (.) Gamma) for block (rb, sb) -> Ss (bf16).
__device__ __forceinline__ void score_tile(const Tiles &s, const __bf16 *Arow, const __bf16 *Brow,
                                           int rb, int sb, int l32, int hl) {
    f32x16 acc = zero_acc();
    const __bf16 *ap = Arow + (32 * rb + l32) * QS + 8 * hl;
    const __bf16 *bp = Brow + (32 * sb + l32) * QS + 8 * hl;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) acc = mma(lds8(ap + 16 * ks), lds8(bp + 16 * ks), acc);
    const int scol = 32 * sb + l32;
    const float Gs_col = s.Gs[scol];
    const float *Gr = s.Gs + 32 * rb + 4 * hl;
    __bf16 *Sr = s.Ss + (32 * rb + 4 * hl) * SS + scol;
    const int rbase = 32 * rb + 4 * hl;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
        const int ro = acc_off(0, v);
        const float val = scol <= rbase + ro ? acc[v] * __expf(Gr[ro] - Gs_col) : 0.f;
        Sr[ro * SS] = (__bf16)val;
    }
}

__device__ __forceinline__ void load_state(const float *st, int w, int lane, f32x16 (&kacc)[4],
                                           f32x16 (&vacc)[4]) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            kacc[x][v] = st[((w * 4 + x) * 16 + v) * 64 + lane];
            vacc[x][v] = st[128 * 128 + ((w * 4 + x) * 16 + v) * 64 + lane];
        }
}

__device__ __forceinline__ void dump_state(float *st, int w, int lane, const f32x16 (&kacc)[4],
                                           const f32x16 (&vacc)[4]) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            st[((w * 4 + x) * 16 + v) * 64 + lane] = kacc[x][v];
            st[128 * 128 + ((w * 4 + x) * 16 + v) * 64 + lane] = vacc[x][v];
        }
}

// ---- 1. per-segment state contributions -------------------------------------
__global__ __launch_bounds__(NT, 1) void segment_state_kernel(MfmaArgs a) {
    __shared__ __attribute__((aligned(16))) char smem[SMEM_BYTES];
    const Tiles s = tiles(smem);
    const int Pm1 = a.P - 1;
    const int bh = blockIdx.x / Pm1, p = blockIdx.x % Pm1;
    const int b = bh / a.p.H, h = bh % a.p.H;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31, hl = lane >> 5;
    const int c_begin = p * a.cps, c_end = min(c_begin + a.cps, a.nchunks);
    f32x16 kacc[4], vacc[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        kacc[x] = f32x16{};
        vacc[x] = f32x16{};
    }
    double carry = 0.0, gsum = 0.0;
    Prefetch pf;
    load_chunk<false>(a.p, b, h, c_begin * C, tid, pf);
    for (int c = c_begin; c < c_end; ++c) {
        store_chunk<false>(s, tid, pf);
        if (w == 0) chunk_scans(s, lane, a.p.m, pf, carry, gsum);
        __syncthreads();
        if (c + 1 < c_end) load_chunk<false>(a.p, b, h, (c + 1) * C, tid, pf);
        build_writes<false>(s, tid, a.p.m);
        __syncthreads();
        update_states(s, w, l32, hl, kacc, vacc);
        __syncthreads();
    }
    const size_t slot = (size_t)bh * a.P + p;
    dump_state(a.seg_state + slot * kStateFloats, w, lane, kacc, vacc);
    if (tid == 0) {
        a.seg_span[slot] = carry;
        a.seg_gsum[slot] = gsum;
    }
}

// ---- 2. states entering each segment ----------------------------------------
// grid (B*H, 32): each thread owns one rotation pair (internal i = 2 ip, 2 ip + 1)
// of one column c of the key or the value state, and walks the segments.
__global__ __launch_bounds__(NT) void segment_scan_kernel(MfmaArgs a) {
    const int bh = blockIdx.x;
    const int gidx = blockIdx.y * NT + threadIdx.x;          // 0 .. 2*64*128-1
    const int kind = gidx >> 13;                             // 0: key, 1: value
    const int ip = (gidx >> 7) & 63, col = gidx & 127;
    const int i0 = 2 * ip, i1 = 2 * ip + 1;
    const int m = a.p.m;
    const int j = ip + 1;                                    // frequency of the pair
    const bool rotates = ip < 63 && j <= (m - 1) / 2;
    const int o0 = kind ? dump_index_V(i0, col) : dump_index_K(i0, col);
    const int o1 = kind ? dump_index_V(i1, col) : dump_index_K(i1, col);
    const float *init = kind ? a.p.V0 : a.p.K0;
    const double c0 = a.p.clock0 ? a.p.clock0[bh] : 0.0;
    double x0 = 0.0, x1 = 0.0;
    if (init) {
        const int p0 = internal_to_paper(i0, m), p1 = internal_to_paper(i1, m);
        const size_t base = (size_t)bh * 128 * 128;
        x0 = p0 >= 0 ? (double)init[base + (size_t)p0 * 128 + col] : 0.0;
        x1 = p1 >= 0 ? (double)init[base + (size_t)p1 * 128 + col] : 0.0;
    }
    auto rot = [&](double tau) {                             // (x0, x1) <- U(tau) (x0, x1)
        if (!rotates) return;
        double rev = (double)j * reduce_clock(tau, m) / (double)m;
        rev -= floor(rev);
        double sn, cs;
        sincospi(2.0 * rev, &sn, &cs);
        const double y0 = cs * x0 - sn * x1;
        const double y1 = sn * x0 + cs * x1;
        x0 = y0;
        x1 = y1;
    };
    rot(c0);                      // initial state in the frame whose origin is clock0
    double origin = reduce_clock(c0, m);
    for (int q = 0; q < a.P; ++q) {
        const size_t slot = (size_t)bh * a.P + q;
        float *st = a.seg_state + slot * kStateFloats;
        if (gidx == 0) a.seg_origin[slot] = origin;
        float d0 = 0.f, d1 = 0.f;
        if (q < a.P - 1) {
            d0 = st[o0];
            d1 = st[o1];
        }
        st[o0] = (float)x0;
        st[o1] = (float)x1;
        if (q < a.P - 1) {
            const double gdec = exp(a.seg_gsum[slot]);
            x0 = gdec * x0 + (double)d0;
            x1 = gdec * x1 + (double)d1;
            rot(a.seg_span[slot]);
            origin = reduce_clock(origin + a.seg_span[slot], m);
        }
    }
}

// ---- 3. fused chunk forward ----------------------------------------------------
__global__ __launch_bounds__(NT, 1) void chunk_forward_kernel(MfmaArgs a) {
    __shared__ __attribute__((aligned(16))) char smem[SMEM_BYTES];
    const Tiles s = tiles(smem);
    const FwdParams &p = a.p;
    const int bh = blockIdx.x / a.P, seg = blockIdx.x % a.P;
    const int b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31, hl = lane >> 5;
    const int m = p.m;
    const int c_begin = seg * a.cps, c_end = min(c_begin + a.cps, a.nchunks);
    const int icol = 32 * w + l32;                   // this lane's internal column
    const int h4 = 4 * hl;

    // Per-lane bases: every unrolled LDS access below is base + compile-time offset.
    const __bf16 *Mzr = a.Mz + ((size_t)h * 128 + icol) * 128 + 8 * hl;   // B operand rows (L2)
    const __bf16 *Myr = a.My + ((size_t)h * 128 + icol) * 128 + 8 * hl;
    const float *gam_l = s.gam + h4;                                      // accumulator rows
    const half2v *CS_l = s.CS + h4 * 64 + (icol >> 1);
    __bf16 *X_l = s.Xs + h4 * QS + icol;                                  // also W's tile
    __bf16 *O2_l = s.Os + h4 * QS + icol;                                 // O'' and output staging
    float *Z_l = s.Zf + h4 * ZS + icol;
    const __bf16 *Qperm = s.Qs + l32 * QS + h4;                           // permuted-k A operands
    const __bf16 *Operm = s.Os + l32 * QS + h4;
    const __bf16 *Xa = s.Xs + l32 * QS + 8 * hl;                          // natural-k A operands
    const __bf16 *Sa = s.Ss + l32 * SS + 8 * hl;
    const __bf16 *ATb = s.ATs + icol * TS + 8 * hl;                       // natural-k B operands
    const __bf16 *ATdb = s.ATds + icol * TS + 8 * hl;
    const __bf16 *VTb = s.VTs + icol * TS + 8 * hl;
    const __bf16 *KTa = s.KTs + l32 * TS + 8 * hl;
    const __bf16 *ATda = s.ATds + l32 * TS + 8 * hl;

    f32x16 kacc[4], vacc[4];
    float *slot_state = a.seg_state + ((size_t)bh * a.P + seg) * kStateFloats;
    if (a.has_init) {
        load_state(slot_state, w, lane, kacc, vacc);
    } else {
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            kacc[x] = f32x16{};
            vacc[x] = f32x16{};
        }
    }
    double carry = 0.0, gsum = 0.0;
    Prefetch pf;
    load_chunk<true>(p, b, h, c_begin * C, tid, pf);
    __bf16 *o = static_cast<__bf16 *>(p.o);

    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * C;
        const int n = min(C, p.T - t0);
        // -- A: stage the chunk, prefix sums, temporal writes
        store_chunk<true>(s, tid, pf);
        if (w == 0) chunk_scans(s, lane, m, pf, carry, gsum);
        __syncthreads();
        if (c + 1 < c_end) load_chunk<true>(p, b, h, (c + 1) * C, tid, pf);
        build_writes<true>(s, tid, m);
        __syncthreads();
        // -- B: key pass.  O' = gamma (.) Q Kbar^T + (Q K^T (.) Gamma) A
        if (w < 3) score_tile(s, s.Qs, s.Ks, w == 0 ? 0 : 1, w == 2 ? 1 : 0, l32, hl);
        f32x16 oacc[2] = {zero_acc(), zero_acc()};
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            const bf16x8 kb = acc_to_operand(kacc[ks >> 1], ks & 1);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
                oacc[rb] = mma(lds8_perm(Qperm + 32 * rb * QS, 16 * ks, 0), kb, oacc[rb]);
        }
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[rb][v] *= gam_l[acc_off(rb, v)];
        __syncthreads();
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                if (rb == 0 && ks >= 2) continue;    // rows 0..31 see only columns 0..31
                oacc[rb] = mma(lds8(Sa + 32 * rb * SS + 16 * ks), lds8(ATb + 16 * ks), oacc[rb]);
            }
        {
            // key state: Kbar^T <- gamma^C Kbar^T + K^T (right-decayed A)
            const float gC = s.gam[63];
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int v = 0; v < 16; ++v) kacc[x][v] *= gC;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const bf16x8 at_w = lds8(ATdb + 16 * ks);
#pragma unroll
                for (int x = 0; x < 4; ++x) kacc[x] = mma(lds8(KTa + 32 * x * TS + 16 * ks), at_w, kacc[x]);
            }
        }
        // -- middle step 1: X_r = scale U(lambda_r) O'_r -> X tile (reuses Q's)
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int ro = acc_off(rb, v);
                const float self = oacc[rb][v];
                const float part = swap_pair(self);
                float x = 0.f;
                if (icol < kDC) {
                    const half2v cs = CS_l[ro * 64];
                    const float cc = (float)cs[0], sn = (float)cs[1];
                    x = (icol & 1) ? (sn * part + cc * self) : (cc * self - sn * part);
                } else if (icol == kDC) {
                    x = self;
                }
                X_l[ro * QS] = (__bf16)(p.scale * x);
            }
        __syncthreads();
        // -- middle step 2: slot logits Z = X M^T -> Z tile (reuses K / K^T)
        {
            bf16x8 mz[8];
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) mz[ks] = *reinterpret_cast<const bf16x8 *>(Mzr + 16 * ks);
            f32x16 zacc[2] = {zero_acc(), zero_acc()};
#pragma unroll
            for (int ks = 0; ks < 8; ++ks)
#pragma unroll
                for (int rb = 0; rb < 2; ++rb)
                    zacc[rb] = mma(lds8(Xa + 32 * rb * QS + 16 * ks), mz[ks], zacc[rb]);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                for (int v = 0; v < 16; ++v) Z_l[acc_off(rb, v) * ZS] = zacc[rb][v];
        }
        __syncthreads();
        // -- middle step 3: softmax over the m active slots -> W tile (reuses X's)
        {
            const int r = tid >> 2, q = tid & 3;
            const float *zr = s.Zf + r * ZS + 32 * q;
            float zv[32];
#pragma unroll
            for (int k4 = 0; k4 < 8; ++k4) {
                const float4 z4 = *reinterpret_cast<const float4 *>(zr + 4 * k4);
                zv[4 * k4] = z4.x;
                zv[4 * k4 + 1] = z4.y;
                zv[4 * k4 + 2] = z4.z;
                zv[4 * k4 + 3] = z4.w;
            }
            if (p.logits && r < n) {
                float *lg = p.logits + (((size_t)b * p.T + t0 + r) * p.H + h) * m + 32 * q;
#pragma unroll
                for (int k = 0; k < 32; ++k)
                    if (32 * q + k < m) lg[k] = zv[k];
            }
            float mx = -INFINITY;
#pragma unroll
            for (int k = 0; k < 32; ++k) {
                if (32 * q + k >= m) zv[k] = -INFINITY;
                mx = fmaxf(mx, zv[k]);
            }
            mx = fmaxf(mx, swap_pair(mx));
            mx = fmaxf(mx, swap_halves4(mx));
            float sum = 0.f;
#pragma unroll
            for (int k = 0; k < 32; ++k) {
                zv[k] = __expf(zv[k] - mx);
                sum += zv[k];
            }
            sum += swap_pair(sum);
            sum += swap_halves4(sum);
            const float inv = 1.f / sum;
            __bf16 *wr = s.Ws + r * QS + 32 * q;
#pragma unroll
            for (int k8 = 0; k8 < 4; ++k8) {
                bf16x8 wv;
#pragma unroll
                for (int k = 0; k < 8; ++k) wv[k] = (__bf16)(zv[8 * k8 + k] * inv);
                *reinterpret_cast<bf16x8 *>(wr + 8 * k8) = wv;
            }
        }
        __syncthreads();
        // -- middle step 4: O''_r = U(-lambda_r) M^T W_r -> O'' tile (reuses A^T's)
        {
            bf16x8 my[8];
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) my[ks] = *reinterpret_cast<const bf16x8 *>(Myr + 16 * ks);
            f32x16 yacc[2] = {zero_acc(), zero_acc()};
#pragma unroll
            for (int ks = 0; ks < 8; ++ks)
#pragma unroll
                for (int rb = 0; rb < 2; ++rb)
                    yacc[rb] = mma(lds8(Xa + 32 * rb * QS + 16 * ks), my[ks], yacc[rb]);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int ro = acc_off(rb, v);
                    const float self = yacc[rb][v];
                    const float part = swap_pair(self);
                    float x = 0.f;
                    if (icol < kDC) {
                        const half2v cs = CS_l[ro * 64];
                        const float cc = (float)cs[0], sn = (float)cs[1];
                        x = (icol & 1) ? (cc * self - sn * part) : (cc * self + sn * part);
                    } else if (icol == kDC) {
                        x = self;
                    }
                    O2_l[ro * QS] = (__bf16)x;
                }
        }
        __syncthreads();
        // -- D: value pass.  O = gamma (.) O'' Vbar + (O'' A^T (.) Gamma) V
        if (w < 3) score_tile(s, s.Os, s.As, w == 0 ? 0 : 1, w == 2 ? 1 : 0, l32, hl);
        f32x16 pacc[2] = {zero_acc(), zero_acc()};
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
            const bf16x8 vb = acc_to_operand(vacc[ks >> 1], ks & 1);
#pragma unroll
            for (int rb = 0; rb < 2; ++rb)
                pacc[rb] = mma(lds8_perm(Operm + 32 * rb * QS, 16 * ks, 0), vb, pacc[rb]);
        }
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v) pacc[rb][v] *= gam_l[acc_off(rb, v)];
        __syncthreads();
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                if (rb == 0 && ks >= 2) continue;
                pacc[rb] = mma(lds8(Sa + 32 * rb * SS + 16 * ks), lds8(VTb + 16 * ks), pacc[rb]);
            }
        // output tile -> staging (O'' is dead) for 16-byte global stores
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
#pragma unroll
            for (int v = 0; v < 16; ++v) O2_l[acc_off(rb, v) * QS] = (__bf16)pacc[rb][v];
        {
            // value state: Vbar <- gamma^C Vbar + (right-decayed A)^T V
            const float gC = s.gam[63];
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int v = 0; v < 16; ++v) vacc[x][v] *= gC;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
                const bf16x8 vt_w = lds8(VTb + 16 * ks);
#pragma unroll
                for (int x = 0; x < 4; ++x) vacc[x] = mma(lds8(ATda + 32 * x * TS + 16 * ks), vt_w, vacc[x]);
            }
        }
        __syncthreads();
        {
            const int r0 = tid >> 4, d0 = (tid & 15) * 8;
#pragma unroll
            for (int it = 0; it < 4; ++it) {
                const int r = r0 + 16 * it;
                if (r < n)
                    *reinterpret_cast<uint4 *>(o + (((size_t)b * p.T + t0 + r) * p.H + h) * D + d0) =
                        *reinterpret_cast<const uint4 *>(s.Os + r * QS + d0);
            }
        }
    }
    if (a.want_final && seg == a.P - 1) {
        dump_state(slot_state, w, lane, kacc, vacc);
        if (tid == 0) a.final_lam[bh] = carry;
    }
}

// ---- 4. final state in the ABI layout ------------------------------------------
// grid (B*H, 32): thread = one rotation pair of one column of K or V.
__global__ __launch_bounds__(NT) void state_out_kernel(MfmaArgs a) {
    const int bh = blockIdx.x;
    const int gidx = blockIdx.y * NT + threadIdx.x;
    const int kind = gidx >> 13;
    const int ip = (gidx >> 7) & 63, col = gidx & 127;
    const int i0 = 2 * ip, i1 = 2 * ip + 1;
    const int m = a.p.m;
    const int j = ip + 1;
    const size_t slot = (size_t)bh * a.P + (a.P - 1);
    const float *st = a.seg_state + slot * kStateFloats;
    const double origin = a.seg_origin[slot];
    double x0 = st[kind ? dump_index_V(i0, col) : dump_index_K(i0, col)];
    double x1 = st[kind ? dump_index_V(i1, col) : dump_index_K(i1, col)];
    if (ip < 63 && j <= (m - 1) / 2) {
        // local frame (origin at the last segment's start) -> absolute clock: U(-origin)
        double rev = (double)j * origin / (double)m;
        rev -= floor(rev);
        double sn, cs;
        sincospi(2.0 * rev, &sn, &cs);
        const double y0 = cs * x0 + sn * x1;
        const double y1 = -sn * x0 + cs * x1;
        x0 = y0;
        x1 = y1;
    }
    float *out = kind ? a.p.V_out : a.p.K_out;
    if (out) {
        const size_t base = (size_t)bh * 128 * 128;
        const int p0 = internal_to_paper(i0, m), p1 = internal_to_paper(i1, m);
        if (p0 >= 0) out[base + (size_t)p0 * 128 + col] = (float)x0;
        if (p1 >= 0) out[base + (size_t)p1 * 128 + col] = (float)x1;
        // padding rows m..127 of the ABI layout are written as zero
        for (int row = m + ip; row < 128; row += 64) out[base + (size_t)row * 128 + col] = 0.f;
    }
    if (gidx == 0 && a.p.clock_out) {
        // with no tokens the final state is the initial one and the local clock is 0
        const double fl = a.nchunks > 0 ? a.final_lam[bh] : 0.0;
        a.p.clock_out[bh] = reduce_clock(origin + fl, m);
    }
}

// Readout matrices in the two bf16 layouts the fused kernel reads.
__global__ __launch_bounds__(NT) void readout_pack_kernel(int m, const float *__restrict__ M,
                                                          __bf16 *__restrict__ Mz, __bf16 *__restrict__ My) {
    const int h = blockIdx.x;
    const float *Mh = M + (size_t)h * 128 * 128;
    __bf16 *Mzh = Mz + (size_t)h * 128 * 128;
    __bf16 *Myh = My + (size_t)h * 128 * 128;
    for (int e = blockIdx.y * NT + threadIdx.x; e < 128 * 128; e += gridDim.y * NT) {
        const int row = e >> 7, col = e & 127;
        // Mz[i'][j_int] = M[i'][paper(j_int)]
        const int pj = internal_to_paper(col, m);
        Mzh[e] = (__bf16)(pj >= 0 ? Mh[(size_t)row * 128 + pj] : 0.f);
        // My[j_int][i'] = M[i'][paper(j_int)]
        const int pr = internal_to_paper(row, m);
        Myh[e] = (__bf16)(pr >= 0 ? Mh[(size_t)col * 128 + pr] : 0.f);
    }
}

}  // namespace

// ---- host side --------------------------------------------------------------
bool mfma_supported(const FwdParams &p) {
    return p.dtype == 1 && p.dk == 128 && p.dv == 128 && p.chunk == 64;
}

namespace {
struct WsLayout {
    size_t mz, my, state, span, gsum, origin, flam, total;
};
WsLayout ws_layout(const FwdParams &p, int P) {
    auto up = [](size_t x) { return (x + 255) / 256 * 256; };
    WsLayout L{};
    size_t off = up(readout_f32_bytes(p.H));
    L.mz = off;
    off += up((size_t)p.H * 128 * 128 * 2);
    L.my = off;
    off += up((size_t)p.H * 128 * 128 * 2);
    const size_t nseg = (size_t)p.B * p.H * P;
    L.state = off;
    off += up(nseg * kStateFloats * 4);
    L.span = off;
    off += up(nseg * 8);
    L.gsum = off;
    off += up(nseg * 8);
    L.origin = off;
    off += up(nseg * 8);
    L.flam = off;
    off += up((size_t)p.B * p.H * 8);
    L.total = off;
    return L;
}
}  // namespace

size_t mfma_workspace_bytes(const FwdParams &p, int segments) {
    // bytes beyond the float readout block the host API reserves first
    return ws_layout(p, segments).total - (readout_f32_bytes(p.H) + 255) / 256 * 256;
}

int mfma_auto_segments(const FwdParams &p) {
    // one workgroup per compute unit: split sequences until B*H*P covers 256 CUs
    const int seqs = p.B * p.H;
    int P = (256 + seqs - 1) / seqs;
    const int nchunks = (p.T + C - 1) / C;
    if (P > nchunks) P = nchunks;
    return P < 1 ? 1 : P;
}

hipError_t launch_fwd_mfma(const FwdParams &p, int P, void *ws, hipStream_t st,
                           hipEvent_t ev_start, hipEvent_t ev_stop) {
    char *base = static_cast<char *>(ws);
    const WsLayout L = ws_layout(p, P);
    MfmaArgs a{};
    a.p = p;
    a.nchunks = (p.T + C - 1) / C;
    a.P = P;
    a.cps = (a.nchunks + P - 1) / P;
    if (a.nchunks > 0) a.P = (a.nchunks + a.cps - 1) / a.cps;   // no empty trailing segment
    if (a.P < 1) a.P = 1;
    a.Mz = reinterpret_cast<const __bf16 *>(base + L.mz);
    a.My = reinterpret_cast<const __bf16 *>(base + L.my);
    a.seg_state = reinterpret_cast<float *>(base + L.state);
    a.seg_span = reinterpret_cast<double *>(base + L.span);
    a.seg_gsum = reinterpret_cast<double *>(base + L.gsum);
    a.seg_origin = reinterpret_cast<double *>(base + L.origin);
    a.final_lam = reinterpret_cast<double *>(base + L.flam);
    a.want_final = (p.K_out || p.V_out || p.clock_out) ? 1 : 0;
    const bool scan = a.P > 1 || p.K0 || p.V0 || p.clock0 || a.want_final;
    a.has_init = scan ? 1 : 0;
    const int BH = p.B * p.H;

    hipLaunchKernelGGL(readout_pack_kernel, dim3(p.H, 8), dim3(NT), 0, st, p.m,
                       reinterpret_cast<const float *>(base), const_cast<__bf16 *>(a.Mz),
                       const_cast<__bf16 *>(a.My));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (a.P > 1 && a.nchunks > 0) {
        hipLaunchKernelGGL(segment_state_kernel, dim3(BH * (a.P - 1)), dim3(NT), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (scan) {
        hipLaunchKernelGGL(segment_scan_kernel, dim3(BH, 2 * 64 * 128 / NT), dim3(NT), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (ev_start && (e = hipEventRecord(ev_start, st)) != hipSuccess) return e;
    if (a.nchunks > 0) {
        hipLaunchKernelGGL(chunk_forward_kernel, dim3(BH * a.P), dim3(NT), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (ev_stop && (e = hipEventRecord(ev_stop, st)) != hipSuccess) return e;
    if (a.want_final) {
        hipLaunchKernelGGL(state_out_kernel, dim3(BH, 2 * 64 * 128 / NT), dim3(NT), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace cyfa
