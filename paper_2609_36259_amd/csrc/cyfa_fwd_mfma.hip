// Matrix-core (bf16 MFMA) chunk-wise CyFA forward for d_k = d_v = 128, chunks of 32 or 64.
//
// Work decomposition.  Each (b, h) sequence is cut into P segments of whole
// chunks.  Four kernels run in order on the caller's stream:
//   1. segment_state_kernel  (b, h, p < P-1): the segment's own contribution to
//      the carried states, DeltaS_p = sum_t (decay to segment end) a_t [k_t | v_t]^T,
//      with the clock origin at the segment start, plus the segment's clock span
//      and log-decay total.  App. B's state recurrence run from a zero state.
//      Extra blocks of the same launch form the bf16 readout matrix
//      M_h = R_h Phi (times scale log2 e) for step 3.
//   2. scan_prep_kernel  (b, h): the states entering every segment,
//      S'_{p+1} = U(span_p) (exp(gsum_p) S'_p + DeltaS_p), each expressed with its
//      own segment-start clock origin.  Moving the origin rotates an
//      absolute-clock state by U(-c) and leaves the output unchanged
//      (App. A.4, Prop. 6), which is what makes the segments independent.
//      The recurrence runs in fp32; the contributions and entering states are
//      stored in bf16, the precision in which the chunk products consume them.
//      (Without a pre-pass, extra blocks of this launch form the readout matrix,
//      or, without a scan either, its own launch does.)
//   3. chunk_forward_kernel  (b, h, p): the fused forward of App. B over the
//      segment's chunks: clock/log-decay prefix sums, temporal write matrix
//      A (Eq. app-temporal-writes), key pass (Eq. app-cyfa-key-chunk), token-wise
//      softmax readout (Eq. cyfa-two-pass, middle line), value pass
//      (Eq. app-cyfa-value-chunk).  Both 128 x 128 fp32 states stay in MFMA
//      accumulators for the whole segment.
//   4. state_out_kernel  (b, h): rotates the last segment's final state back to
//      the absolute clock and writes it in the ABI layout (only when asked).
#include "cyfa_mfma_chunk.h"
#include "cyfa_prep.h"

#include <hip/hip_ext.h>

namespace cyfa {

using namespace mfma;

namespace {

// rows of the readout matrix per workgroup when extra blocks of the pre-pass or the
// scan form it
constexpr int kPrepRows = 32;

// ---- LDS maps (bytes) ---------------------------------------------------------
// Fused kernel (32-token chunks).  Tiles read through the transpose read (K, V,
// A and the readout matrix M) are swizzled rows of 128; Q (then X, W) and O''
// are padded to stride QS.  K's region switches to the padded layout when O''
// replaces K.  Two workgroups share a compute unit, so the map stays within half
// of its 160 KiB: one temporal-write tile (A_dec for a chunk whose decay factors
// into a row scale, else A, whose state updates then decay the other operand),
// and the softmax partials share the score tile.
template <int CC>
struct Lay {
    static constexpr int RB = CC / 32;                 // 32-row blocks per tile
    static constexpr int SSC = CC + 8;                 // row stride of the score tile
    static constexpr int CSW = 68;                     // row stride (half2 words) of the (cos, sin) table
    static constexpr int TILE = CC * QS * 2;           // padded tile
    static constexpr int STILE = CC * SWS * 2;         // swizzled tile
    static constexpr int Q = 0;                        // Q   -> X -> W       (padded)
    static constexpr int K = Q + TILE;                 // K (swizzled) -> O'' (padded)
    static constexpr int V = K + TILE;                 // V   (swizzled)
    static constexpr int A = V + STILE;                // A   (temporal writes, swizzled)
    static constexpr int S = A + STILE;                // scores [CC][SSC] bf16 / softmax partials
    static constexpr int RED = S;                      // (max, sum) per wave x row, middle step only
    static constexpr int CS = S + CC * SSC * 2;        // (cos, sin) [CC][CSW] half pairs
    static constexpr int MT = CS + CC * CSW * 4;       // readout matrix [128][SWS] bf16 (swizzled)
    static constexpr int SC = MT + 128 * SWS * 2;      // per-token scalars (CC entries each)
    static constexpr int BYTES = SC + scalar_bytes(CC);
    static_assert(4 * CC * 8 <= CC * SSC * 2, "softmax partials fit the score tile");
    static_assert(K % 256 == 0 && V % 256 == 0 && A % 256 == 0 && MT % 256 == 0,
                  "swizzled tiles start on a bank-window boundary");
    static_assert(CC != 32 || BYTES <= 80 * 1024, "two workgroups per compute unit");
};

template <int CC>
__device__ __forceinline__ Tiles fused_tiles(char *smem) {
    using L = Lay<CC>;
    Tiles t{};
    t.Qs = reinterpret_cast<__bf16 *>(smem + L::Q);
    t.Xs = t.Qs;
    t.Ws = t.Qs;
    t.Ks = reinterpret_cast<__bf16 *>(smem + L::K);
    t.Os = t.Ks;
    t.Vs = reinterpret_cast<__bf16 *>(smem + L::V);
    t.As = reinterpret_cast<__bf16 *>(smem + L::A);
    t.Ads = nullptr;
    t.Ss = reinterpret_cast<__bf16 *>(smem + L::S);
    t.CS = reinterpret_cast<half2v *>(smem + L::CS);
    t.Mt = reinterpret_cast<__bf16 *>(smem + L::MT);
    t.red = reinterpret_cast<float2 *>(smem + L::RED);
    t.Stage = reinterpret_cast<__bf16 *>(smem + L::CS);
    scalars_at(t, smem + L::SC, CC);
    return t;
}

// One 16 x 16 block (rb, sb) of the causal score tile -> Ss (bf16), k = 128 along
// the rows of both operand tiles: token rows t from a padded tile, rows s from
// the swizzled tile at byte offset Boff (column block ks of a row is its first
// block's offset ^ 64 ks).  The decay Gamma_ts is applied only when the chunk is
// not factored (fac = false); otherwise the A tile holds A_dec and Gamma becomes
// a per-token scale of the whole pass.  Computed transposed, D[s][t], so that
// each lane stores four consecutive entries S[t][s .. s+3] at once.
template <int CC>
__device__ __forceinline__ void score_block(const Tiles &s, const __bf16 *Arow, char *smem, int Boff,
                                            int rb, int sb, int lane, bool fac) {
    constexpr int SSC = Lay<CC>::SSC;
    const int l16 = lane & 15, g = lane >> 4;
    f32x4 acc = zero_acc4();
    const __bf16 *ap = Arow + (16 * rb + l16) * QS + 8 * g;
    // one opaque copy of the base per call (an asm statement also fences the
    // scheduler, so none sits between the reads and products below)
    const int bo = opq(Boff + 2 * swz_elem(16 * sb + l16, 8 * g));
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
        acc = mma16(lds8(lds_at<__bf16>(smem, bo ^ (64 * ks))), lds8(ap + 32 * ks), acc);
    const int t = 16 * rb + l16;
    const int s0 = 16 * sb + 4 * g;
    if (!fac) {                                        // uniform
        const float Gt = s.Gs[t];
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] *= __expf(Gt - s.Gs[s0 + r]);
    }
    bf16x4 sv;
#pragma unroll
    for (int r = 0; r < 4; ++r) sv[r] = (__bf16)(s0 + r <= t ? acc[r] : 0.f);
    *reinterpret_cast<bf16x4 *>(s.Ss + t * SSC + s0) = sv;
}

// The 16 x 16 blocks of the causal CC x CC score tile that the intra-chunk
// products read (the lower triangle plus the upper halves of the 32 x 32
// diagonal blocks, which come out as zeros), spread evenly over the 4 waves.
template <int CC>
__device__ __forceinline__ void score_tiles(const Tiles &s, const __bf16 *Arow, char *smem, int Boff,
                                            int w, int lane, bool fac) {
    static_assert(CC == 32, "four-wave fused kernel: 32-token chunks");
    score_block<CC>(s, Arow, smem, Boff, w >> 1, w & 1, lane, fac);
}

__device__ __forceinline__ void scale_states(f32x16 (&kacc)[4], f32x16 (&vacc)[4], float f) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            kacc[x][v] *= f;
            vacc[x][v] *= f;
        }
}

// ---- mixer pieces of the fused layer forward ----------------------------------
// The layer forward (cyfa_forward_mixer) runs the mixer prologue inside the fused
// kernel's chunk staging and the epilogue on its output tile, with the standalone
// kernels' arithmetic (cyfa_mixer.hip) in the same order, so that its output is
// the bits of prologue -> forward -> epilogue.  Thread (tid) of the staging owns
// channel block cb = tid % 16 (channels 8 cb .. 8 cb + 7) of rows tid / 16 and
// tid / 16 + 16 of each tile -- the positions store_chunk writes -- and the 16
// threads of a row are consecutive lanes of one wave.  In the mixer variant the
// (cos, sin) table's LDS holds the convolution taps and three raw rows before
// the chunk (the halo); the rotations compute their table entries on the fly.
constexpr int kMixHead = 128;                             // channels per head
constexpr int kMixTapBytes = 3 * kMixHead * 4 * 4;        // [q, k, v][s][channel]: weight of x_{t-s}
constexpr int kMixHaloBytes = 3 * 3 * kMixHead * 2;       // [q, k, v][row -3 .. -1][channel] bf16
constexpr int kMixNormBytes = 3 * kMixHead * 4;           // g_q, g_k, g_o

struct MixLds {
    int taps, halo, norm;                                 // byte offsets in the workgroup's LDS
};

__device__ __forceinline__ void bf16x8_to_float(uint4 u, float *x) {
    const unsigned w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ uint4 float_to_bf16x8(const float *y) { return mix_pack_bf16x8(y); }
// sum over the 16 lanes of one row (the standalone kernels' head reduction)
__device__ __forceinline__ float mix_row_sum(float s) {
#pragma unroll
    for (int o = 1; o < kMixHead / 8; o <<= 1) s += __shfl_xor(s, o);
    return s;
}

// Per-segment set-up: taps (zero past the width, reversed so that s indexes
// x_{t-s}), RMSNorm weights, and the halo of the segment's first chunk (raw rows
// t0-3 .. t0-1 of the sequence, zero before its start).
template <bool kConv>
__device__ __forceinline__ void mix_setup(const MfmaArgs &a, const MixLds &L, char *smem, int b, int h, int t0,
                                          int tid, int nth) {
    const FwdParams &p = a.p;
    const MixIn &mx = a.mix;
    const int K = mx.K;
    for (int e = tid; e < 3 * kMixHead; e += nth) {
        const int which = e / kMixHead, ch = e % kMixHead;
        const float *g = which == 0 ? mx.gq : (which == 1 ? mx.gk : mx.g_o);
        lds_at<float>(smem, L.norm)[e] = g ? g[ch] : 1.f;
    }
    if (!kConv) return;
    for (int e = tid; e < 3 * kMixHead * 4; e += nth) {
        const int tensor = e / (kMixHead * 4), s = (e / kMixHead) % 4, ch = e % kMixHead;
        const float *W = tensor == 0 ? mx.wq : (tensor == 1 ? mx.wk : mx.wv);
        const float w = (W && s < K) ? W[((size_t)h * kMixHead + ch) * K + (K - 1 - s)] : 0.f;
        lds_at<float>(smem, L.taps)[e] = w;
    }
    const int Tb = seq_tokens(p, b);
    for (int e = tid; e < 3 * 3 * 16; e += nth) {
        const int tensor = e / 48, hr = (e / 16) % 3, cb = e % 16;
        const int t = t0 - 3 + hr;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (t >= 0 && t < Tb) {
            const void *X = tensor == 0 ? p.q : (tensor == 1 ? p.k : p.v);
            v = *reinterpret_cast<const uint4 *>(static_cast<const __bf16 *>(X) +
                                                 ((seq_row0(p, b) + t) * p.H + h) * kMixHead + 8 * cb);
        }
        *reinterpret_cast<uint4 *>(smem + L.halo + ((tensor * 3 + hr) * kMixHead + 8 * cb) * 2) = v;
    }
}

// ShortConv (+ SiLU) (+ RMSNorm for q, k) of this thread's rows tid/16 + 16 it
// (it < CC/16) of one tensor, from the raw tile (rows >= 0) and the halo (rows <
// 0), as bf16.  Rows past the sequence (tokens t0 + row >= Tb) come out as 0.
// tensor 0: q (padded tile), 1: k, 2: v (swizzled).
template <int CC>
__device__ __forceinline__ void mix_conv_rows(const MfmaArgs &a, const MixLds &L, char *smem, int tile, int tensor,
                                              int tid, int t0, int Tb, uint4 *outv) {
    const MixIn &mx = a.mix;
    // opaque per call: the addresses below are formed here, not held across the chunk loop
    const int tq = opq(tid);
    const int cb = tq & 15, r0 = tq >> 4;
    const float *W = tensor == 0 ? mx.wq : (tensor == 1 ? mx.wk : mx.wv);
    const bool conv = W != nullptr;
    const float *g = tensor == 0 ? mx.gq : (tensor == 1 ? mx.gk : nullptr);
#pragma unroll
    for (int it = 0; it < CC / 16; ++it) {
        const int r = r0 + 16 * it;
        // x_{t-s} for s = 0 .. 3 in the standalone kernel's order of products
        float y[8];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if (s > 0 && !conv) break;                     // uniform: only x_t is used
            const int rr = r - s;
            uint4 u;
            if (rr >= 0) {
                const int off = tensor == 0 ? 2 * (rr * QS + 8 * cb) : 2 * swz_elem(rr, 8 * cb);
                u = *reinterpret_cast<const uint4 *>(smem + tile + off);
            } else {
                u = *reinterpret_cast<const uint4 *>(smem + L.halo + ((tensor * 3 + rr + 3) * kMixHead + 8 * cb) * 2);
            }
            float x[8];
            bf16x8_to_float(u, x);
            if (!conv) {
#pragma unroll
                for (int i = 0; i < 8; ++i) y[i] = x[i];
            } else {
                const float *tp = lds_at<float>(smem, L.taps + ((tensor * 4 + s) * kMixHead + 8 * cb) * 4);
                const float4 w0 = *reinterpret_cast<const float4 *>(tp);
                const float4 w1 = *reinterpret_cast<const float4 *>(tp + 4);
                const float wv[8] = {w0.x, w0.y, w0.z, w0.w, w1.x, w1.y, w1.z, w1.w};
#pragma unroll
                for (int i = 0; i < 8; ++i) y[i] = fmaf(wv[i], x[i], s == 0 ? 0.f : y[i]);
            }
        }
        if (mx.act)
#pragma unroll
            for (int i = 0; i < 8; ++i) y[i] = y[i] * mix_sigm(y[i]);
        if (g) {
            float ss = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) ss = fmaf(y[i], y[i], ss);
            const float rn = rsqrtf(mix_row_sum(ss) / (float)kMixHead + mx.eps);
            const float4 g0 = *reinterpret_cast<const float4 *>(smem + L.norm + (tensor * kMixHead + 8 * cb) * 4);
            const float4 g1 = *reinterpret_cast<const float4 *>(smem + L.norm + (tensor * kMixHead + 8 * cb + 4) * 4);
            const float gr[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
            for (int i = 0; i < 8; ++i) y[i] *= rn * gr[i];
        }
        if (t0 + r >= Tb)
#pragma unroll
            for (int i = 0; i < 8; ++i) y[i] = 0.f;
        outv[it] = float_to_bf16x8(y);
    }
}

// The (cos, sin) table entries of pairs 4q + jj0 and 4q + jj0 + 1 for a token (its
// builder record rec), computed exactly as build_writes_swz computes them: the
// start phase of pair 4q, then jj angle-addition steps for entry jj.
__device__ __forceinline__ half2v mix_cs_entry(float4 rec, int q, int jj, int J) {
    const float u = rec.y, c1 = rec.z, s1 = rec.w;
    float sn, cs;
    sincos_rev(__builtin_amdgcn_fractf((float)(4 * q + 1) * u), &sn, &cs);
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        if (k >= jj) break;
        const float nc = cs * c1 - sn * s1;
        const float ns = sn * c1 + cs * s1;
        cs = nc;
        sn = ns;
    }
    const int j = 4 * q + 1 + jj;
    const bool live = j <= J && j <= 63;
    const float cv = live ? cs : 0.f;
    const float sv = live ? sn : 0.f;
    half2v e;
    e[0] = (_Float16)(j == 64 ? 1.f : cv);
    e[1] = (_Float16)sv;
    return e;
}
__device__ __forceinline__ void mix_cs_pair(float4 rec, int q, int jj0, int J, half2v &e0, half2v &e1) {
    e0 = mix_cs_entry(rec, q, jj0, J);
    e1 = mix_cs_entry(rec, q, jj0 + 1, J);
}

// Epilogue of one chunk: out = RMSNorm(o) g_o sigmoid(gate) for this thread's
// rows of the staged output tile (padded, in the Q tile's place).
template <int CC>
__device__ __forceinline__ void mix_epilogue(const MfmaArgs &a, const MixLds &L, char *smem, int tile, int b, int h,
                                             int t0, int Tb, int tid, const uint4 *gpf) {
    const FwdParams &p = a.p;
    const MixIn &mx = a.mix;
    const int tq = opq(tid);
    const int cb = tq & 15, r0 = tq >> 4;
    const float4 g0 = *reinterpret_cast<const float4 *>(smem + L.norm + (2 * kMixHead + 8 * cb) * 4);
    const float4 g1 = *reinterpret_cast<const float4 *>(smem + L.norm + (2 * kMixHead + 8 * cb + 4) * 4);
    const float gr[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
    __bf16 *out = static_cast<__bf16 *>(p.o);
#pragma unroll
    for (int it = 0; it < 2; ++it) {
        const int r = r0 + 16 * it, t = t0 + r;
        const bool live = t < Tb;
        float yt[8], gt[8];
        if (live) {
            bf16x8_to_float(*reinterpret_cast<const uint4 *>(smem + tile + 2 * (r * QS + 8 * cb)), yt);
            if (mx.gate) bf16x8_to_float(gpf[it], gt);
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) yt[i] = 0.f;
        }
        float ss = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) ss = fmaf(yt[i], yt[i], ss);
        const float rn = rsqrtf(mix_row_sum(ss) / (float)kMixHead + mx.eps);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float v = yt[i] * rn * gr[i];
            if (mx.gate && live) v *= mix_sigm(gt[i]);
            yt[i] = live ? v : 0.f;
        }
        if (t < p.T)
            *reinterpret_cast<uint4 *>(out + ((seq_row0(p, b) + t) * p.H + h) * kMixHead + 8 * cb) =
                float_to_bf16x8(yt);
    }
}

// Gate rows of this thread for a chunk (zero past the sequence), loaded during the
// chunk so that its epilogue does not wait for them.
__device__ __forceinline__ void mix_load_gate(const MfmaArgs &a, int b, int h, int t0, int Tb, int tid, uint4 *gpf) {
    const FwdParams &p = a.p;
    const int tq = opq(tid);
    const int cb = tq & 15, r0 = tq >> 4;
    const int avail = Tb - t0;
    gpf[0] = make_uint4(0, 0, 0, 0);
    gpf[1] = gpf[0];
    if (!a.mix.gate || avail <= 0) return;                 // uniform
#pragma unroll
    for (int it = 0; it < 2; ++it) {
        const int r = min(r0 + 16 * it, avail - 1);        // rows past the sequence re-read its last
        gpf[it] = *reinterpret_cast<const uint4 *>(static_cast<const __bf16 *>(a.mix.gate) +
                                                   ((seq_row0(p, b) + t0 + r) * p.H + h) * kMixHead + 8 * cb);
    }
}

// ---- 1. per-segment state contributions -------------------------------------
// DeltaS_p = sum_t exp(G_end - G_t) a_t [k_t | v_t]^T over the segment's tokens,
// with a_t = beta_t U(-lambda_t) b the temporal write (Eq. app-temporal-writes),
// lambda_t the clock from the segment start and G_t the inclusive sum of log alpha
// from the segment start (App. B, the carried-state recurrence unrolled from a
// zero state).  G_end - G_t <= 0, so every weight lies in [0, 1].
//
// Wave w owns the 32 slot columns 32w .. 32w+31 of both contributions and builds
// its own part of the decayed write matrix directly in MFMA operand registers:
// lane l holds column 32w + l%32 at the 8 tokens 16ks + 8h + p (h = l/32), which
// is the B operand of Kbar^T += K^T A_dec and the A operand of
// Vbar += A_dec^T V alike.  K^T and V come from swizzled tiles through the
// transpose read, double-buffered so that a chunk needs one barrier.  Each wave
// runs the chunk's clock and decay scans itself (lane = token) and passes the
// per-token phase and amplitude through a private LDS row.
// kMix (layer forward): 0 the plain operator; otherwise the gates come from their
// projections, and with kMix = 1 the staged k and v rows are the raw projections,
// which the mixer's ShortConv and k's RMSNorm turn into the operator's k and v in
// LDS first (kMix = 2: k and v are the standalone prologue's).
template <int CC, int kMix = 0>
__global__ __launch_bounds__(NT, 2) void segment_state_kernel(MfmaArgs a, float mz_scale) {
    constexpr int STILE = CC * SWS * 2;                // one swizzled K or V tile
    constexpr int KIT = CC * 16 / NT;                  // 16-byte pieces per thread per tensor
    constexpr int RPP = NT / 16;                       // tile rows per pass
    constexpr int SCB = 4 * STILE;                     // per-wave (phase, amplitude) rows
    constexpr int MIX0 = SCB + 4 * 64 * 8 + 4 * 8;     // kMix: taps, halo, RMSNorm weights
    __shared__ __attribute__((aligned(256)))
    char smem[MIX0 + (kMix == 1 ? kMixTapBytes + kMixHaloBytes + kMixNormBytes : 0)];
    const MixLds ML{MIX0, MIX0 + kMixTapBytes, MIX0 + kMixTapBytes + kMixHaloBytes};
    static_assert(SCB + 4 * 64 * 8 + 4 * 8 >= prep_lds_bytes(kPrepRows), "readout-matrix blocks fit");
    const FwdParams &p = a.p;
    const int Pm1 = a.P - 1;
    const int Hv = p.H * a.hv;                         // (virtual) heads of 128 channels
    const int bh = blockIdx.x / Pm1, seg = blockIdx.x % Pm1;
    const int b = bh / Hv, hv = bh % Hv;               // k, v column block hv
    const int h = hv / a.hv;                           // head of the per-token scalars
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hl = lane >> 5, l32 = lane & 31;
    const int m = p.m;
    const double inv_m = 1.0 / (double)m;
    {
        // blocks past the segments form 32 rows of the bf16 readout matrix each
        const int nseg = p.B * Hv * Pm1;
        if ((int)blockIdx.x >= nseg) {
            const int q = (int)blockIdx.x - nseg;
            readout_prep_rows<kPrepRows>(m, p.R, nullptr, const_cast<__bf16 *>(a.Mz), mz_scale,
                                          q / (kStoreRows / kPrepRows), q % (kStoreRows / kPrepRows), tid, smem);
            return;
        }
    }
    const int c_begin = seg * a.cps, c_end = min(c_begin + a.cps, a.nchunks);
    const int Tb = seq_tokens(p, b);
    const int t_begin = c_begin * CC, t_end = min(c_end * CC, Tb);
    if constexpr (kMix == 1) mix_setup<true>(a, ML, smem, b, h, t_begin, tid, NT);
    float2 *scw = lds_at<float2>(smem, SCB + w * 64 * 8);
    double *red = lds_at<double>(smem, SCB + 4 * 64 * 8);

    // this lane's write-matrix column: internal index cidx = 32w + l32 is the cosine
    // (even) or minus sine (odd, a quarter turn later) of pair j = cidx/2 + 1, or the
    // DC (126, amplitude 1/sqrt(2) of the pairs'), or padding / inactive pair (0)
    const int cidx = 32 * w + l32;
    const int J = (m - 1) >> 1;
    const float jf = cidx < kDC ? (float)((cidx >> 1) + 1) : 0.f;
    const float shift = (cidx < kDC && (cidx & 1)) ? 0.25f : 0.f;
    const float mult = cidx < 2 * J ? 1.f : (cidx == kDC ? 0.70710678118654752f : 0.f);
    const float amp0 = sqrtf(2.f / (float)m);

    // K, V pieces: rows tid/16 + RPP it, 16-byte column block tid%16; scalars of
    // token `lane` of the chunk on every wave
    const size_t row_el = (size_t)Hv * D;
    const unsigned loff = (unsigned)(((tid >> 4) * (int)row_el + (tid & 15) * 8) * 2);
    const unsigned pass = (unsigned)(RPP * row_el * 2);
    const int kvo = 2 * swz_elem(tid >> 4, (tid & 15) * 8);
    uint4 pk[KIT], pv[KIT];
    float dl, g, be;
    auto load = [&](int c) {
        const int t0 = c * CC;
        const size_t base = ((seq_row0(p, b) + t0) * row_el + (size_t)hv * D) * 2;
        const char *kb = reinterpret_cast<const char *>(p.k) + base;
        const char *vb = reinterpret_cast<const char *>(p.v) + base;
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            const bool in = t0 + (tid >> 4) + RPP * it < Tb;
            pk[it] = in ? *reinterpret_cast<const uint4 *>(kb + loff + it * pass) : make_uint4(0, 0, 0, 0);
            pv[it] = in ? *reinterpret_cast<const uint4 *>(vb + loff + it * pass) : make_uint4(0, 0, 0, 0);
        }
        const int t = t0 + lane;
        const size_t si = (seq_row0(p, b) + t) * p.H + h;
        const bool tin = lane < CC && t < Tb;
        if constexpr (kMix) {
            const MixIn &mx = a.mix;
            dl = tin ? mix_sigm(mx.z_delta[si] + (mx.b_delta ? mx.b_delta[h] : 0.f)) : 0.f;
            g = (tin && mx.z_alpha) ? -mx.A[h] * mix_softplus(mx.z_alpha[si] + (mx.b_alpha ? mx.b_alpha[h] : 0.f))
                                    : 0.f;
            be = tin ? (mx.z_beta ? mix_sigm(mx.z_beta[si]) : 1.f) : 0.f;
        } else {
            dl = tin ? p.delta[si] : 0.f;
            g = (tin && p.log_alpha) ? p.log_alpha[si] : 0.f;
            be = tin ? (p.beta ? p.beta[si] : 1.f) : 0.f;
        }
    };
    // the first chunk's rows are in flight while the segment total below is formed
    if (c_begin < c_end) load(c_begin);
    // segment total of log alpha (the decay reference G_end)
    double gpart = 0.0;
    if constexpr (kMix) {
        const MixIn &mx = a.mix;
        if (mx.z_alpha)
            for (int t = t_begin + tid; t < t_end; t += NT)
                gpart += (double)(-mx.A[h] * mix_softplus(mx.z_alpha[(seq_row0(p, b) + t) * p.H + h] +
                                                          (mx.b_alpha ? mx.b_alpha[h] : 0.f)));
    } else if (p.log_alpha) {
        for (int t = t_begin + tid; t < t_end; t += NT) gpart += (double)p.log_alpha[(seq_row0(p, b) + t) * p.H + h];
    }
    gpart = lane63(wave_incl_scan(gpart));
    if (lane == 0) red[w] = gpart;

    lds_barrier();                                     // (the chunk's loads stay in flight)
    const double G_end = (red[0] + red[1]) + (red[2] + red[3]);

    f32x16 kacc[4], vacc[4];
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        kacc[x] = zero_acc();
        vacc[x] = zero_acc();
    }
    double carry = 0.0, gsum = 0.0;
    const int trs = tr_off_swz(lane);
    for (int c = c_begin; c < c_end; ++c) {
        const int buf = (c - c_begin) & 1;
        char *Kt = smem + 2 * buf * STILE;
        char *Vt = Kt + STILE;
#pragma unroll
        for (int it = 0; it < KIT; ++it) {
            *reinterpret_cast<uint4 *>(Kt + kvo + it * RPP * SWS * 2) = pk[it];
            *reinterpret_cast<uint4 *>(Vt + kvo + it * RPP * SWS * 2) = pv[it];
        }
        {
            // clock (fp64, from the segment start) and decay to the segment end
            const double lam = carry + wave_incl_scan((double)dl);
            const float Gl = wave_incl_scan(g);
            const float rem = (float)(G_end - gsum);
            const double q = lam * inv_m;
            const float u = (float)(q - floor(q));
            scw[lane] = make_float2(u, be * amp0 * __expf(rem - Gl));
            carry = reduce_clock(lane63(lam), (double)m, inv_m);
            gsum += (double)lane63(Gl);
        }
        if (c + 1 < c_end) load(c + 1);
        lds_barrier();
        if constexpr (kMix == 1) {
            // raw rows -> the operator's k and v (ShortConv, k's RMSNorm), in place; the
            // raw rows CC-3 .. CC-1 become the next chunk's halo
            uint4 fk[KIT], fv[KIT];
            const int kto = 2 * buf * STILE, vto = kto + STILE;
            mix_conv_rows<CC>(a, ML, smem, kto, 1, tid, c * CC, Tb, fk);
            mix_conv_rows<CC>(a, ML, smem, vto, 2, tid, c * CC, Tb, fv);
            lds_barrier();
            const int tq = opq(tid);
            const int cb = tq & 15, rq = tq >> 4;
            const int offs = 2 * swz_elem(rq, 8 * cb);
            if (rq + RPP * (KIT - 1) >= CC - 3) {
                const int hr = rq + RPP * (KIT - 1) - (CC - 3);
                const int offl = offs + RPP * (KIT - 1) * SWS * 2;
                *reinterpret_cast<uint4 *>(smem + ML.halo + ((1 * 3 + hr) * kMixHead + 8 * cb) * 2) =
                    *reinterpret_cast<const uint4 *>(smem + kto + offl);
                *reinterpret_cast<uint4 *>(smem + ML.halo + ((2 * 3 + hr) * kMixHead + 8 * cb) * 2) =
                    *reinterpret_cast<const uint4 *>(smem + vto + offl);
            }
#pragma unroll
            for (int it = 0; it < KIT; ++it) {
                *reinterpret_cast<uint4 *>(smem + kto + offs + it * RPP * SWS * 2) = fk[it];
                *reinterpret_cast<uint4 *>(smem + vto + offs + it * RPP * SWS * 2) = fv[it];
            }
            lds_barrier();
        }
        const int kt = opq(2 * buf * STILE + trs), vt = opq((2 * buf + 1) * STILE + trs);
#pragma unroll
        for (int ks = 0; ks < CC / 16; ++ks) {
            const float4 *sp = reinterpret_cast<const float4 *>(scw + 16 * ks + 8 * hl);
            bf16x8 af;
#pragma unroll
            for (int q2 = 0; q2 < 4; ++q2) {
                const float4 r = sp[q2];
                af[2 * q2] = (__bf16)(__builtin_amdgcn_cosf(__builtin_amdgcn_fractf(fmaf(jf, r.x, shift))) *
                                      (r.y * mult));
                af[2 * q2 + 1] = (__bf16)(__builtin_amdgcn_cosf(__builtin_amdgcn_fractf(fmaf(jf, r.z, shift))) *
                                          (r.w * mult));
            }
#pragma unroll
            for (int x = 0; x < 4; ++x) {
                kacc[x] = mma(lds8_tr(lds_at<__bf16>(smem, kt ^ (64 * x)) + 16 * ks * SWS, SWS), af, kacc[x]);
                vacc[x] = mma(af, lds8_tr(lds_at<__bf16>(smem, vt ^ (64 * x)) + 16 * ks * SWS, SWS), vacc[x]);
            }
        }
    }
    // dump in the accumulator order of the fused kernel: key state as written
    // (wave = slot block, x = d block); value state with the roles of wave and
    // block exchanged (the fused kernel's wave owns a d_v block)
    const size_t slot = (size_t)bh * a.P + seg;
    __bf16 *st = a.seg_state + slot * kStateFloats;
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            bf16x8 kq, vq;
#pragma unroll
            for (int v = 0; v < 8; ++v) {
                kq[v] = (__bf16)kacc[x][8 * hf + v];
                vq[v] = (__bf16)vacc[x][8 * hf + v];
            }
            *reinterpret_cast<bf16x8 *>(st + dump_off(w, x, lane, 8 * hf)) = kq;
            *reinterpret_cast<bf16x8 *>(st + 128 * 128 + dump_off(x, w, lane, 8 * hf)) = vq;
        }
    if (tid == 0) {
        a.seg_span[slot] = carry;
        a.seg_gsum[slot] = G_end;
    }
}

// ---- 2. states entering each segment ----------------------------------------
// Element pairs that a rotation U(tau) mixes, in the lane-major dump layout:
// key-state partners are adjacent lanes (offsets e, e + 16), value-state
// partners adjacent registers (offsets e, e + 1).  Pairs are numbered so that
// thread t of the scan owns pairs 4t .. 4t+3 (g < 8192 key state, else value):
//   key   t = (block wx, lane pair k, register quad q): lanes 2k, 2k+1, registers
//         4q .. 4q+3 -- one slot pair, so the four share one frequency;
//   value t = (block wx, lane, register half h8): registers 8 h8 .. 8 h8 + 7 of
//         one lane, i.e. four consecutive slot pairs of one column.
struct PairRef {
    int o0, o1;        // dump offsets of the (cos, sin) pair
    int i0;            // internal index of the first element (even)
    int col;           // state column (d for the key state, d for the value state)
    bool value;
};

__device__ __forceinline__ PairRef pair_ref(int gidx) {
    PairRef r;
    if (gidx < 8192) {                                   // key state: lanes (2k, 2k+1)
        const int t = gidx >> 2, e = gidx & 3;
        const int q = t & 3, k = (t >> 2) & 31, wx = t >> 7;
        const int w = wx >> 2, x = wx & 3, lane0 = 2 * k, h = lane0 >> 5;
        r.o0 = dump_off(w, x, lane0, 4 * q + e);
        r.o1 = r.o0 + 16;
        r.i0 = 32 * w + (lane0 & 31);
        r.col = 32 * x + 8 * q + 4 * h + e;
        r.value = false;
    } else {                                             // value state: registers (v, v+1)
        const int g = gidx - 8192;
        const int t = g >> 2, e = g & 3;
        const int h8 = t & 1, lane = (t >> 1) & 63, wx = t >> 7;
        const int w = wx >> 2, x = wx & 3, h = lane >> 5;
        const int v = 8 * h8 + 2 * e;
        r.o0 = 128 * 128 + dump_off(w, x, lane, v);
        r.o1 = r.o0 + 1;
        r.i0 = 32 * x + 8 * (v >> 2) + 4 * h + (v & 3);
        r.col = 32 * w + (lane & 31);
        r.value = true;
    }
    return r;
}

// (x0, x1) <- U(tau) (x0, x1) for the pair at internal indices (2j-2, 2j-1)
// u: the rotation angle tau in revolutions of the m-slot ring, tau / m mod 1
// (same for every pair, so computed once by the caller)
__device__ __forceinline__ double ring_rev(double tau, int m) {
    const double inv_m = 1.0 / (double)m;
    return reduce_clock(tau, (double)m, inv_m) * inv_m;
}
__device__ __forceinline__ void ring_sincos(double u, int j, float *sn, float *cs) {
    double rev = (double)j * u;
    rev -= floor(rev);
    sincos_rev((float)rev, sn, cs);
}
__device__ __forceinline__ void apply_rot(float sn, float cs, float &x0, float &x1) {
    const float y0 = cs * x0 - sn * x1;
    const float y1 = sn * x0 + cs * x1;
    x0 = y0;
    x1 = y1;
}
__device__ __forceinline__ void rotate_pair(double u, int j, float &x0, float &x1) {
    float sn, cs;
    ring_sincos(u, j, &sn, &cs);
    apply_rot(sn, cs, x0, x1);
}

// Thread = four rotation pairs moved with two 8-byte (4 x bf16) accesses per
// segment (see pair_ref): key state, four registers of each partner lane;
// value state, eight consecutive registers of one lane.  Blocks (bh, y < 16)
// of 256 threads: 2048 key and 2048 value threads per (virtual) head bh.
constexpr int kScanBlocks = 4096 / NT;                   // blocks per (virtual) head
__device__ __forceinline__ void segment_scan(const MfmaArgs &a, int bh, int y, int tid) {
    const int qi = y * NT + tid;                         // 0 .. 4095
    const int m = a.p.m;
    // ABI state [B][H][128][128 hv]: column block bh mod hv of head bh / hv
    const int dabi = 128 * a.hv;
    const size_t sbase = (size_t)(bh / a.hv) * 128 * dabi + 128 * (bh % a.hv);
    const bool value = qi >= 2048;
    PairRef pr[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) pr[k] = pair_ref(4 * qi + k);
    // key: first elements of the four pairs, then the second elements; value: the
    // four pairs' elements in register order
    const int off0 = pr[0].o0, off1 = value ? pr[2].o0 : pr[0].o1;
    int jf[4];
    bool rot[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        jf[k] = (pr[k].i0 >> 1) + 1;                     // frequency of the pair
        rot[k] = pr[k].i0 < kDC && jf[k] <= (m - 1) / 2;
    }
    const float *init = value ? a.p.V0 : a.p.K0;
    const double c0 = a.p.clock0 ? a.p.clock0[bh / a.hv] : 0.0;
    float x0[4] = {0.f, 0.f, 0.f, 0.f}, x1[4] = {0.f, 0.f, 0.f, 0.f};
    if (init) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int p0 = internal_to_paper(pr[k].i0, m), p1 = internal_to_paper(pr[k].i0 + 1, m);
            const size_t base = sbase + pr[k].col;
            x0[k] = p0 >= 0 ? init[base + (size_t)p0 * dabi] : 0.f;
            x1[k] = p1 >= 0 ? init[base + (size_t)p1 * dabi] : 0.f;
        }
    }
    {
        const double u0 = ring_rev(c0, m);               // initial state in the frame with origin clock0
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (rot[k]) rotate_pair(u0, jf[k], x0[k], x1[k]);
    }
    const double inv_m = 1.0 / (double)m;
    double origin = reduce_clock(c0, (double)m, inv_m);
    // Segment contributions, log-alpha sums and clock spans are fetched kBatch
    // segments at a time, ahead of the dependent chain through them (loaded inside
    // the chain, each segment's scalars would wait for a memory round trip behind
    // the previous segment's stores).  Every thread owns the same offsets in every
    // segment, so the loads of a batch never see this batch's stores.  The chain
    // itself runs in fp32; contributions and entering states are stored as bf16.
    constexpr int kBatch = 8;
    for (int q0 = 0; q0 < a.P; q0 += kBatch) {
        bf16x4 da[kBatch], db[kBatch];
        double gs[kBatch], sp[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int q = q0 + u;
            da[u] = bf16x4{};
            db[u] = da[u];
            gs[u] = 0.0;
            sp[u] = 0.0;
            if (q < a.P - 1) {
                const size_t slot = (size_t)bh * a.P + q;
                const __bf16 *st = a.seg_state + slot * kStateFloats;
                da[u] = *reinterpret_cast<const bf16x4 *>(st + off0);
                db[u] = *reinterpret_cast<const bf16x4 *>(st + off1);
                gs[u] = a.seg_gsum[slot];
                sp[u] = a.seg_span[slot];
            }
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int q = q0 + u;
            if (q >= a.P) break;
            const size_t slot = (size_t)bh * a.P + q;
            __bf16 *st = a.seg_state + slot * kStateFloats;
            if (qi == 0) a.seg_origin[slot] = origin;
            float d0[4], d1[4];
            bf16x4 s0, s1;
            if (!value) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    s0[k] = (__bf16)x0[k];
                    s1[k] = (__bf16)x1[k];
                    d0[k] = (float)da[u][k];
                    d1[k] = (float)db[u][k];
                }
            } else {
                s0[0] = (__bf16)x0[0]; s0[1] = (__bf16)x1[0]; s0[2] = (__bf16)x0[1]; s0[3] = (__bf16)x1[1];
                s1[0] = (__bf16)x0[2]; s1[1] = (__bf16)x1[2]; s1[2] = (__bf16)x0[3]; s1[3] = (__bf16)x1[3];
                d0[0] = (float)da[u][0]; d1[0] = (float)da[u][1]; d0[1] = (float)da[u][2]; d1[1] = (float)da[u][3];
                d0[2] = (float)db[u][0]; d1[2] = (float)db[u][1]; d0[3] = (float)db[u][2]; d1[3] = (float)db[u][3];
            }
            if (q > 0 || !a.zero_init) {
                *reinterpret_cast<bf16x4 *>(st + off0) = s0;
                *reinterpret_cast<bf16x4 *>(st + off1) = s1;
            }
            if (q < a.P - 1) {
                const float gdec = __expf((float)gs[u]);
                const double span = sp[u];               // already reduced to [0, m)
                const double u1 = span * inv_m;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    x0[k] = fmaf(gdec, x0[k], d0[k]);
                    x1[k] = fmaf(gdec, x1[k], d1[k]);
                }
                if (!value) {
                    // one slot pair: one rotation angle for all four
                    if (rot[0]) {
                        float sn, cs;
                        ring_sincos(u1, jf[0], &sn, &cs);
#pragma unroll
                        for (int k = 0; k < 4; ++k) apply_rot(sn, cs, x0[k], x1[k]);
                    }
                } else {
#pragma unroll
                    for (int k = 0; k < 4; ++k)
                        if (rot[k]) rotate_pair(u1, jf[k], x0[k], x1[k]);
                }
                origin = reduce_clock(origin + span, (double)m, inv_m);
            }
        }
    }
}

// The segment scan and, when no pre-pass formed it, the readout matrix (needed
// only by the fused kernel) in one launch: blocks [0, nscan) scan, the rest form
// 32 rows of M_h = R_h Phi each.
__global__ __launch_bounds__(NT) void scan_prep_kernel(MfmaArgs a, int nscan, float mz_scale) {
    __shared__ __attribute__((aligned(16))) char lds[prep_lds_bytes(kPrepRows)];
    const int b = blockIdx.x;
    if (b < nscan) {
        segment_scan(a, b / kScanBlocks, b % kScanBlocks, threadIdx.x);
    } else {
        const int q = b - nscan;
        readout_prep_rows<kPrepRows>(a.p.m, a.p.R, nullptr, const_cast<__bf16 *>(a.Mz), mz_scale,
                                     q / (kStoreRows / kPrepRows), q % (kStoreRows / kPrepRows), threadIdx.x, lds);
    }
}

// Transposed operand whose k index is the token s = 16 ks + 8 hl + p, times the
// right-decay factor of that token (the A_dec row scale, Eq. app-chunk-rescale);
// dw points at decw[16 ks + 8 hl].
__device__ __forceinline__ bf16x8 decay_rows(bf16x8 v, const float *dw) {
    const float4 d0 = *reinterpret_cast<const float4 *>(dw);
    const float4 d1 = *reinterpret_cast<const float4 *>(dw + 4);
    const float d[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
    bf16x8 r;
#pragma unroll
    for (int q = 0; q < 8; ++q) r[q] = (__bf16)((float)v[q] * d[q]);
    return r;
}

// ---- 3. fused chunk forward, 32-token chunks ------------------------------------
// Two workgroups share a compute unit; the readout matrix sits in LDS and the
// next chunk is prefetched into registers.
// kMix: 0 the plain operator; 1 the layer forward with the mixer prologue in the
// chunk staging and the epilogue on the output tile; 2 the layer forward after
// the standalone prologue's ShortConv and RMSNorm (gates and epilogue fused here).
// See the mixer pieces above.
template <int CC, int kMix>
__global__ __launch_bounds__(NT, 2) void chunk_forward_kernel(MfmaArgs a) {
    static_assert(CC == 32, "four-wave fused kernel: 32-token chunks");
    using Ly = Lay<CC>;
    constexpr int RB = Ly::RB;
    constexpr int SSC = Ly::SSC;
    static_assert(kMixTapBytes + kMixHaloBytes <= CC * Ly::CSW * 4, "taps and halo fit the table's place");
    static_assert(Ly::BYTES + kMixNormBytes <= 80 * 1024, "two workgroups per compute unit");
    constexpr bool kConv = kMix == 1;                // convolution in the staging; the table's
                                                     // place then holds taps and halo
    __shared__ __attribute__((aligned(256))) char smem[Ly::BYTES + (kMix != 0 ? kMixNormBytes : 0)];
    const MixLds ML{Ly::CS, Ly::CS + kMixTapBytes, Ly::BYTES};
    const Tiles s = fused_tiles<CC>(smem);
    const FwdParams &p = a.p;
    const int bh = blockIdx.x / a.P, seg = blockIdx.x % a.P;
    const int b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, l32 = lane & 31, hl = lane >> 5;
    const int m = p.m;
    const int c_begin = seg * a.cps, c_end = min(c_begin + a.cps, a.nchunks);
    const int Tb = seq_tokens(p, b);
    const int icol = 32 * w + l32;                   // this lane's slot (readout step)
    const int h4 = 4 * hl;

    // the readout matrix in LDS is M times zs = scale log2(e): slot logits come out in
    // log2 units, and the readout weights are divided by zs to compensate
    const float zs = __int_as_float(__builtin_amdgcn_readfirstlane(
        __float_as_int(p.scale * 1.4426950408889634f)));             // uniform: a scalar register
    // Per-lane bases (opaque byte offsets): every unrolled LDS access below is one
    // of these plus a compile-time offset.
    constexpr int TE = Ly::TILE / 2;                                      // padded tile size in elements
    constexpr int CSW = Ly::CSW;
    const int trs = tr_off_swz(lane);
    const float *eps_t = lds_at<float>(smem, opq(Ly::SC + 4 * (CC + l32)));          // row scale of token l32
    const int dw_off = Ly::SC + 4 * (3 * CC + 8 * hl);                                // decw, operand tokens
    // M rows (slot icol), columns 8 hl + 16 ks at byte offset Mza ^ 32 ks
    const int Mza = opq(Ly::MT + 2 * swz_elem(icol, 8 * hl));
    // transposed operands from swizzled tiles: column block w at Ly::T + trw, or block
    // x at Ly::T + (tr0 ^ 64 x) (the tile offsets are multiples of 256 bytes)
    const int trw = opq(trs ^ (64 * w));
    const int tr0 = opq(trs);
    // M columns: own base (the tile sits at 44 KiB; with the k-step offsets the sum
    // would overflow the 16-bit instruction offset)
    const __bf16 *Myt = lds_at<__bf16>(smem, opq(Ly::MT + (trs ^ (64 * w))));
    const __bf16 *Qperm = lds_at<__bf16>(smem, opq(Ly::Q + 2 * (l32 * QS + h4)));   // permuted-k A operands
    const __bf16 *Operm = Qperm + TE;
    const __bf16 *Xa = lds_at<__bf16>(smem, opq(Ly::Q + 2 * (l32 * QS + 8 * hl)));  // natural-k operands
    const __bf16 *Sa = lds_at<__bf16>(smem, opq(Ly::S + 2 * (l32 * SSC + 8 * hl)));
    const __bf16 *At = lds_at<__bf16>(smem, Ly::A + trw);
    const __bf16 *Vt = lds_at<__bf16>(smem, Ly::V + trw);
    // token-row base: row l32, columns 32w + 4hl (+ 8 v4) of the X / W and O''
    // tiles, and the matching (cos, sin) pairs (the padded tile rows and the table
    // rows are both 272 bytes)
    static_assert(QS * 2 == CSW * 4, "one token-row base for the padded tiles and the table");
    const int rowb = opq(2 * (l32 * QS + 32 * w + h4));
    __bf16 *Wrow = lds_at<__bf16>(smem, Ly::Q + rowb);
    __bf16 *O2row = Wrow + TE;
    const half2v *CSrow = lds_at<half2v>(smem, Ly::CS + rowb);
    float2 *redw = lds_at<float2>(smem, opq(Ly::RED + 8 * (w * CC + l32)));
    const float2 *redr = lds_at<float2>(smem, opq(Ly::RED + 8 * l32));

    // Issue order of the prologue's loads: the first chunk and the readout matrix
    // (needed by the first stage), then the entering states, which the first
    // chunk's products need only after its staging, scans and temporal writes.
    Prefetch<CC> pf;
    load_chunk<CC, true, NT, kMix != 0>(p, b, h, c_begin * CC, Tb, tid, pf, &a.mix);
    if constexpr (kMix != 0) mix_setup<kConv>(a, ML, smem, b, h, c_begin * CC, tid, NT);
    uint4 gpf[2];                                    // kMix: the chunk's gate rows
    {
        // readout matrix M_h (slot rows, internal basis columns), resident for the segment
        const __bf16 *Mh = a.Mz + (size_t)h * 128 * 128;
#pragma unroll
        for (int it = 0; it < 8; ++it) {
            const int e = it * NT + tid;
            const int row = e >> 4, c0 = (e & 15) * 8;
            *reinterpret_cast<uint4 *>(s.Mt + swz_elem(row, c0)) =
                *reinterpret_cast<const uint4 *>(Mh + row * 128 + c0);
        }
    }
    f32x16 kacc[4], vacc[4];
    const __bf16 *slot_state = a.seg_state + ((size_t)bh * a.P + seg) * kStateFloats;
    if (a.has_init && !(seg == 0 && a.zero_init)) {
        load_state(slot_state, w, lane, kacc, vacc);
    } else {
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            kacc[x] = f32x16{};
            vacc[x] = f32x16{};
        }
    }
    double carry = 0.0, gsum = 0.0;
    float logf = 0.f;                                // carried states are exp(logf) x registers
    __bf16 *o = static_cast<__bf16 *>(p.o);

    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * CC;
        const int n = min(CC, Tb - t0);          // <= 0 for chunks past the sequence
        // kMix: the previous chunk's epilogue, from its output tile in Q's place; each
        // thread reads exactly the positions it overwrites next
        if constexpr (kMix != 0)
            if (c > c_begin) mix_epilogue<CC>(a, ML, smem, Ly::Q, b, h, t0 - CC, Tb, tid, gpf);
        // -- A: stage the chunk, prefix sums, temporal writes; prefetch the next chunk
        store_chunk<CC, true, NT, true>(s, tid, pf);
        if (w == 0) chunk_scans<CC, NT, CC, true>(s, lane, m, pf, carry, gsum, logf);
        lds_barrier();
        if constexpr (kConv) {
            // the staged rows are raw projections: ShortConv, RMSNorm, then the
            // operator's q, k, v replace them (one more barrier: the convolution
            // reads three rows above each row)
            uint4 fq[2], fk[2], fv[2];
            mix_conv_rows<CC>(a, ML, smem, Ly::Q, 0, tid, t0, Tb, fq);
            mix_conv_rows<CC>(a, ML, smem, Ly::K, 1, tid, t0, Tb, fk);
            mix_conv_rows<CC>(a, ML, smem, Ly::V, 2, tid, t0, Tb, fv);
            lds_barrier();
            const int tq = opq(tid);
            const int cb = tq & 15, rq = tq >> 4;
            const int offq = 2 * (rq * QS + 8 * cb), offs = 2 * swz_elem(rq, 8 * cb);
            const int offq1 = offq + 2 * 16 * QS, offs1 = offs + 2 * 16 * SWS;
            if (rq + 16 >= CC - 3) {
                // raw rows CC-3 .. CC-1: the next chunk's halo
                const int hr = rq + 16 - (CC - 3);
                *reinterpret_cast<uint4 *>(smem + ML.halo + ((0 * 3 + hr) * kMixHead + 8 * cb) * 2) =
                    *reinterpret_cast<const uint4 *>(smem + Ly::Q + offq1);
                *reinterpret_cast<uint4 *>(smem + ML.halo + ((1 * 3 + hr) * kMixHead + 8 * cb) * 2) =
                    *reinterpret_cast<const uint4 *>(smem + Ly::K + offs1);
                *reinterpret_cast<uint4 *>(smem + ML.halo + ((2 * 3 + hr) * kMixHead + 8 * cb) * 2) =
                    *reinterpret_cast<const uint4 *>(smem + Ly::V + offs1);
            }
            *reinterpret_cast<uint4 *>(smem + Ly::Q + offq) = fq[0];
            *reinterpret_cast<uint4 *>(smem + Ly::Q + offq1) = fq[1];
            *reinterpret_cast<uint4 *>(smem + Ly::K + offs) = fk[0];
            *reinterpret_cast<uint4 *>(smem + Ly::K + offs1) = fk[1];
            *reinterpret_cast<uint4 *>(smem + Ly::V + offs) = fv[0];
            *reinterpret_cast<uint4 *>(smem + Ly::V + offs1) = fv[1];
        }
        if (c + 1 < c_end) load_chunk<CC, true, NT, kMix != 0>(p, b, h, t0 + CC, Tb, tid, pf, &a.mix);
        // factor applied to the carried states this chunk, and whether the chunk's
        // decay is factored (the A tile then holds A_dec); uniform: scalar registers
        const float sf = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(s.ctl[0])));
        const bool fac = __builtin_amdgcn_readfirstlane(__float_as_int(s.ctl[2])) != 0;
        build_writes_swz<CC, !kConv, NT, CSW>(s, s.As, tid, m);
        lds_barrier();
        // -- B: key pass.  O' = gamma (.) Q Kbar^T + (Q K^T (.) Gamma) A.  With the
        //    tile holding A_dec (rows times the right decay), Gamma_rs = gam_r decw_s
        //    and O' = eps (.) (Q Kbar'^T + S A_dec), S the causal Q K^T and Kbar' the
        //    state after this chunk's rescale factor (eps: row scale of the chunk
        //    scans).  A chunk that is not factored keeps A, applies Gamma in the score
        //    tile, gam to the inter-chunk term and the rescale after it.  Computed
        //    transposed: O'^T = Kbar' Q^T + A_dec^T S^T.  Wave w owns basis rows
        //    32w .. 32w+31; lane (token l32, half hl) holds 16 of them, so each
        //    (cos, sin) pair sits in two consecutive registers of one lane.
        if (fac && sf != 1.f) {
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int v = 0; v < 16; ++v) kacc[x][v] *= sf;
        }
        score_tiles<CC>(s, s.Qs, smem, Ly::K, w, lane, fac);
        f32x16 oacc = zero_acc();
#pragma unroll
        for (int ks = 0; ks < 8; ++ks)
            oacc = mma(acc_to_operand(kacc[ks >> 1], ks & 1), lds8_perm(Qperm, 16 * ks, 0), oacc);
        if (!fac) {
            const float gt = *eps_t;
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[v] *= gt;
        }
        lds_barrier();
#pragma unroll
        for (int ks = 0; ks < CC / 16; ++ks)
            oacc = mma(lds8_tr(At + 16 * ks * SWS, SWS), lds8(Sa + 16 * ks), oacc);
        if (fac) {
            const float et = *eps_t;
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[v] *= et;
        }
        {
            // key state: Kbar'^T += K^T A_dec (decay kept in L)
            if (!fac && sf != 1.f) {
#pragma unroll
                for (int x = 0; x < 4; ++x)
#pragma unroll
                    for (int v = 0; v < 16; ++v) kacc[x][v] *= sf;
            }
            const int kt = opq(tr0);
#pragma unroll
            for (int ks = 0; ks < CC / 16; ++ks) {
                bf16x8 ad_w = lds8_tr(At + 16 * ks * SWS, SWS);
                if (!fac) ad_w = decay_rows(ad_w, lds_at<float>(smem, opq(dw_off)) + 16 * ks);
#pragma unroll
                for (int x = 0; x < 4; ++x)
                    kacc[x] = mma(lds8_tr(lds_at<__bf16>(smem, Ly::K + (kt ^ (64 * x))) + 16 * ks * SWS, SWS), ad_w,
                                  kacc[x]);
            }
        }
        // -- middle step 1: X_r = U(lambda_r) O'_r -> X tile [token][basis] (reuses Q's)
        half2v csx[8];
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
            if constexpr (kConv) {
                mix_cs_pair(s.bw[l32], 4 * w + v4, 2 * hl, (m - 1) >> 1, csx[2 * v4], csx[2 * v4 + 1]);
            } else {
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) csx[2 * v4 + k2] = CSrow[4 * v4 + k2];
            }
        }
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
            bf16x4 xv;
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                const half2v cs = csx[2 * v4 + k2];
                const float c = (float)cs[0], sn = (float)cs[1];
                const float xc = oacc[4 * v4 + 2 * k2], xs = oacc[4 * v4 + 2 * k2 + 1];
                xv[2 * k2] = (__bf16)fmaf(-sn, xs, c * xc);
                xv[2 * k2 + 1] = (__bf16)fmaf(sn, xc, c * xs);
            }
            // padding column 127 (wave 3, upper lane half, last register) is set to 1:
            // the readout matrix holds kMaskLogit there on the rows of inactive slots
            if (v4 == 3 && w == 3 && hl) xv[3] = (__bf16)1.f;
            *reinterpret_cast<bf16x4 *>(Wrow + 8 * v4) = xv;
        }
        lds_barrier();
        // -- middle step 2: slot logits, transposed: Z^T = M X^T.  Wave w owns slots
        //    32w .. 32w+31; lane (token 32 nb + l32, half hl) holds 16 of them.
        f32x16 zacc[RB];
        {
#pragma unroll
            for (int nb = 0; nb < RB; ++nb) zacc[nb] = zero_acc();
            const int mz = opq(Mza);            // per chunk: the xor'ed addresses are not hoisted
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                const bf16x8 ma = lds8(lds_at<__bf16>(smem, mz ^ (32 * ks)));
#pragma unroll
                for (int nb = 0; nb < RB; ++nb)
                    zacc[nb] = mma(ma, lds8(Xa + 32 * nb * QS + 16 * ks), zacc[nb]);
            }
        }
        // -- middle step 3: softmax over the m active slots.  Per token: in-lane over
        //    16 slots, across the two lane halves, then one (max, sum) exchange
        //    between the 4 waves.
        float mwave[RB];                        // this wave's max over its slots (-inf: none active)
#pragma unroll
        for (int nb = 0; nb < RB; ++nb) {
            // inactive slots (>= m) come out of the product at about -1e30 (padding
            // column of X times the readout matrix entry): no masking here
            float mx = zacc[nb][0];
#pragma unroll
            for (int v = 1; v < 16; ++v) mx = fmaxf(mx, zacc[nb][v]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const int r = 32 * nb + l32;
            if (p.logits && r < n) {
                // the logit accumulators hold log2(e) z; report z
                float *lg = p.logits + ((seq_row0(p, b) + t0 + r) * p.H + h) * m;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int slot = icol - l32 + 8 * (v >> 2) + h4 + (v & 3);
                    if (slot < m) lg[slot] = zacc[nb][v] * 0.69314718055994531f;
                }
            }
            // a wave whose slots are all inactive (m <= 32 w) has mx about -1e30: its
            // weights and its share of the sum get the factor exp2(mx - M) = 0 below
            mwave[nb] = mx;
            const float mref = mx == -INFINITY ? 0.f : mx;
            // the accumulators now hold exp2(z - mref), reused for the weights below
#pragma unroll
            for (int v = 0; v < 16; ++v) zacc[nb][v] = __builtin_amdgcn_exp2f(zacc[nb][v] - mref);
            float t8[8];
#pragma unroll
            for (int v = 0; v < 8; ++v) t8[v] = zacc[nb][v] + zacc[nb][v + 8];
#pragma unroll
            for (int v = 0; v < 4; ++v) t8[v] += t8[v + 4];
            float sm = (t8[0] + t8[2]) + (t8[1] + t8[3]);
            sm += __shfl_xor(sm, 32);
            if (hl == 0) redw[32 * nb] = make_float2(mx, sm);
        }
        lds_barrier();
#pragma unroll
        for (int nb = 0; nb < RB; ++nb) {
            float2 pr[4];
#pragma unroll
            for (int x = 0; x < 4; ++x) pr[x] = redr[x * CC + 32 * nb];
            const float M = fmaxf(fmaxf(pr[0].x, pr[1].x), fmaxf(pr[2].x, pr[3].x));
            float Lsum = 0.f;
#pragma unroll
            for (int x = 0; x < 4; ++x) Lsum += pr[x].y * __builtin_amdgcn_exp2f(pr[x].x - M);
            // W = exp2(z - M) / L / zs = e * exp2(mwave - M) / (L zs), mwave <= M
            const float f = mwave[nb] == -INFINITY
                                ? 0.f
                                : __builtin_amdgcn_exp2f(mwave[nb] - M) * __builtin_amdgcn_rcpf(Lsum * zs);
            __bf16 *wrow = Wrow + 32 * nb * QS;
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                bf16x4 wv;
#pragma unroll
                for (int k = 0; k < 4; ++k) wv[k] = (__bf16)(zacc[nb][4 * v4 + k] * f);
                *reinterpret_cast<bf16x4 *>(wrow + 8 * v4) = wv;
            }
        }
        lds_barrier();
        // -- middle step 4: O''_r = U(-lambda_r) M^T W_r, transposed: Y^T = M^T W^T.
        //    Wave w owns basis rows 32w .. 32w+31; each (cos, sin) pair sits in two
        //    consecutive registers of one lane, so the rotation is in-lane.
        {
            // the (cos, sin) pairs are read first: they do not depend on the products
            half2v csy[8];
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                if constexpr (kConv) {
                    mix_cs_pair(s.bw[l32], 4 * w + v4, 2 * hl, (m - 1) >> 1, csy[2 * v4], csy[2 * v4 + 1]);
                } else {
#pragma unroll
                    for (int k2 = 0; k2 < 2; ++k2) csy[2 * v4 + k2] = CSrow[4 * v4 + k2];
                }
            }
            f32x16 yacc = zero_acc();
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) yacc = mma(lds8_tr(Myt + 16 * ks * SWS, SWS), lds8(Xa + 16 * ks), yacc);
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                bf16x4 ov;
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    const half2v cs = csy[2 * v4 + k2];
                    const float c = (float)cs[0], sn = (float)cs[1];
                    const float yc = yacc[4 * v4 + 2 * k2], ysn = yacc[4 * v4 + 2 * k2 + 1];
                    ov[2 * k2] = (__bf16)fmaf(sn, ysn, c * yc);
                    ov[2 * k2 + 1] = (__bf16)fmaf(-sn, yc, c * ysn);
                }
                *reinterpret_cast<bf16x4 *>(O2row + 8 * v4) = ov;
            }
        }
        lds_barrier();
        // -- D: value pass.  O = gamma (.) O'' Vbar + (O'' A^T (.) Gamma) V, as the key
        //    pass: O = eps (.) (O'' Vbar' + S2 V) with S2 the causal O'' A_dec^T (a
        //    chunk that is not factored as before); computed transposed, lane (token
        //    l32, half hl) holding 16 output columns of wave w's block 32w .. 32w+31.
        if (fac && sf != 1.f) {
#pragma unroll
            for (int x = 0; x < 4; ++x)
#pragma unroll
                for (int v = 0; v < 16; ++v) vacc[x][v] *= sf;
        }
        if constexpr (kMix != 0) mix_load_gate(a, b, h, t0, Tb, tid, gpf);
        score_tiles<CC>(s, s.Os, smem, Ly::A, w, lane, fac);
        f32x16 pacc = zero_acc();
#pragma unroll
        for (int ks = 0; ks < 8; ++ks)
            pacc = mma(acc_to_operand(vacc[ks >> 1], ks & 1), lds8_perm(Operm, 16 * ks, 0), pacc);
        if (!fac) {
            const float gt = *eps_t;
#pragma unroll
            for (int v = 0; v < 16; ++v) pacc[v] *= gt;
        }
        lds_barrier();
#pragma unroll
        for (int ks = 0; ks < CC / 16; ++ks)
            pacc = mma(lds8_tr(Vt + 16 * ks * SWS, SWS), lds8(Sa + 16 * ks), pacc);
        if (fac) {
            const float et = *eps_t;
#pragma unroll
            for (int v = 0; v < 16; ++v) pacc[v] *= et;
        }
        // output: lane (token l32, half hl) stores its 16 columns 32w + 4hl + 8 v4 ..
        // as four 8-byte pieces (uniform chunk base plus a 32-bit lane offset); the
        // four waves' pieces of a token row merge in L2
        if constexpr (kMix != 0) {
            // the operator's output tile goes to Q's place (free since the readout) for
            // the epilogue at the start of the next chunk
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                bf16x4 ov;
#pragma unroll
                for (int k = 0; k < 4; ++k) ov[k] = (__bf16)pacc[4 * v4 + k];
                *reinterpret_cast<bf16x4 *>(Wrow + 8 * v4) = ov;
            }
        } else if (l32 < n) {
            char *ob = reinterpret_cast<char *>(o + ((seq_row0(p, b) + t0) * p.H + h) * D);
            const unsigned loff = (unsigned)opq((l32 * p.H * D + 32 * w + h4) * 2);
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                bf16x4 ov;
#pragma unroll
                for (int k = 0; k < 4; ++k) ov[k] = (__bf16)pacc[4 * v4 + k];
                *reinterpret_cast<bf16x4 *>(ob + loff + 16 * v4) = ov;
            }
        }
        {
            // value state: Vbar' += A_dec^T V (decay kept in L)
            if (!fac && sf != 1.f) {
#pragma unroll
                for (int x = 0; x < 4; ++x)
#pragma unroll
                    for (int v = 0; v < 16; ++v) vacc[x][v] *= sf;
            }
            const int at = opq(tr0);
#pragma unroll
            for (int ks = 0; ks < CC / 16; ++ks) {
                bf16x8 v_w = lds8_tr(Vt + 16 * ks * SWS, SWS);
                if (!fac) v_w = decay_rows(v_w, lds_at<float>(smem, opq(dw_off)) + 16 * ks);
#pragma unroll
                for (int x = 0; x < 4; ++x)
                    vacc[x] = mma(lds8_tr(lds_at<__bf16>(smem, Ly::A + (at ^ (64 * x))) + 16 * ks * SWS, SWS), v_w,
                                  vacc[x]);
            }
        }
        lds_barrier();
    }
    if constexpr (kMix != 0)
        if (c_end > c_begin) mix_epilogue<CC>(a, ML, smem, Ly::Q, b, h, (c_end - 1) * CC, Tb, tid, gpf);
    if (a.want_final && seg == a.P - 1) {
        scale_states(kacc, vacc, __expf(s.ctl[1]));
        dump_state(a.fin_state + (size_t)bh * kStateFloats, w, lane, kacc, vacc);
        if (tid == 0) a.final_lam[bh] = carry;
    }
}

// ---- 4. final state in the ABI layout ------------------------------------------
// grid (B*H, 32): thread = one rotation pair of the key or value state.
__global__ __launch_bounds__(NT) void state_out_kernel(MfmaArgs a) {
    const int bh = blockIdx.x;                           // (virtual) head
    const int gidx = blockIdx.y * NT + threadIdx.x;
    const int m = a.p.m;
    const PairRef pr = pair_ref(gidx);
    const int j = (pr.i0 >> 1) + 1;
    const size_t slot = (size_t)bh * a.P + (a.P - 1);
    const float *st = a.fin_state + (size_t)bh * kStateFloats;
    const double origin = a.seg_origin[slot];
    // ABI state [B][H][128][128 hv]: column block bh mod hv of head bh / hv
    const int dabi = 128 * a.hv;
    const size_t base = (size_t)(bh / a.hv) * 128 * dabi + 128 * (bh % a.hv) + pr.col;
    const int p0 = internal_to_paper(pr.i0, m), p1 = internal_to_paper(pr.i0 + 1, m);
    float x0, x1;
    if (a.nchunks > 0) {
        x0 = st[pr.o0];
        x1 = st[pr.o1];
        // local frame (origin at the last segment's start) -> absolute clock: U(-origin)
        if (pr.i0 < kDC && j <= (m - 1) / 2) rotate_pair(ring_rev(-origin, m), j, x0, x1);
    } else {
        // no tokens: the final state is the initial state (zero when none is given)
        const float *init = pr.value ? a.p.V0 : a.p.K0;
        x0 = init && p0 >= 0 ? init[base + (size_t)p0 * dabi] : 0.f;
        x1 = init && p1 >= 0 ? init[base + (size_t)p1 * dabi] : 0.f;
    }
    float *out = pr.value ? a.p.V_out : a.p.K_out;
    if (out) {
        if (p0 >= 0) out[base + (size_t)p0 * dabi] = x0;
        if (p1 >= 0) out[base + (size_t)p1 * dabi] = x1;
        // padding rows m..127 of the ABI layout are written as zero (one writer per row)
        const int ip = pr.i0 >> 1;
        for (int row = m + ip; row < 128; row += 64) out[base + (size_t)row * dabi] = 0.f;
    }
    if (gidx == 0 && bh % a.hv == 0 && a.p.clock_out) {
        // with no tokens the final state is the initial one and the local clock is 0
        const double fl = a.nchunks > 0 ? a.final_lam[bh] : 0.0;
        a.p.clock_out[bh / a.hv] = reduce_clock(origin + fl, m);
    }
}

}  // namespace

// ---- host side --------------------------------------------------------------
// The matrix-core path evaluates App. B's chunk form in 32-token chunks.  A
// requested chunk length of 64 is accepted and run as two 32-token chunks: the
// chunk form is exact for any chunk length (the carried states after 64 tokens
// are those after two steps of 32), so only the rounding order differs from a
// 64-token evaluation.
constexpr int kMfmaChunk = 32;

// Head dimension 256 (both d_k and d_v): the fused chunk kernel is an eight-wave
// variant (cyfa_fwd_mfma256.hip); the pre-pass, the segment scan and the
// final-state conversion run unchanged on 128-channel virtual heads.
hipError_t launch_chunk256(const MfmaArgs &a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop);

bool mfma_supported(const FwdParams &p) {
    const bool dims = (p.dk == 128 && p.dv == 128) || (p.dk == 256 && p.dv == 256);
    return p.dtype == 1 && dims && (p.chunk == 32 || p.chunk == 64);
}

int mfma_default_chunk() { return kMfmaChunk; }

namespace {
// 128-channel column blocks per head: d = 256 states are two 128 x 128 pairs
int virtual_heads(const FwdParams &p) { return p.dk == 256 ? 2 : 1; }

struct WsLayout {
    size_t mz, state, fin, span, gsum, origin, flam, total;
};
WsLayout ws_layout(const FwdParams &p, int P) {
    auto up = [](size_t x) { return (x + 255) / 256 * 256; };
    WsLayout L{};
    const size_t BHv = (size_t)p.B * p.H * virtual_heads(p);
    size_t off = up(readout_f32_bytes(p.H));
    L.mz = off;
    off += up((size_t)p.H * 128 * 128 * 2);
    const size_t nseg = BHv * P;
    L.state = off;
    off += up(nseg * kStateFloats * 2);
    L.fin = off;
    off += up(BHv * kStateFloats * 4);
    L.span = off;
    off += up(nseg * 8);
    L.gsum = off;
    off += up(nseg * 8);
    L.origin = off;
    off += up(nseg * 8);
    L.flam = off;
    off += up(BHv * 8);
    L.total = off;
    return L;
}

// 0: the plain operator; 1, 2: the layer forward with the ShortConv in the
// staging or before it (the kernels' kMix)
int mix_mode(const MfmaArgs &a) { return a.mix.z_delta ? (a.mix.fuse_conv ? 1 : 2) : 0; }

// BHv: (virtual) heads of the pre-pass and the scan, B H hv
template <int CC>
hipError_t launch_cc(const MfmaArgs &a, int BHv, hipStream_t st, hipEvent_t ev_start,
                     hipEvent_t ev_stop) {
    hipError_t e;
    // the bf16 readout matrix carries the logit scale in log2 units, scale log2(e)
    const float mz_scale = a.p.scale * 1.4426950408889634f;
    const bool prepass = a.P > 1 && a.nchunks > 0;
    if (prepass) {
        // Only each segment's total contribution is needed, so the pre-pass may
        // step through a segment in 64-token chunks (fewer barriers and per-chunk
        // costs) whenever its length is a whole number of them.  Every segment but
        // the last is full, and the last one is not pre-passed.  Extra blocks of
        // the same launch form the bf16 readout matrix, 32 rows each.
        const int nblk = BHv * (a.P - 1) + a.p.H * (kStoreRows / kPrepRows);
        const int mode = mix_mode(a);
        auto pre = [&](auto kern, const MfmaArgs &args) {
            hipLaunchKernelGGL(kern, dim3(nblk), dim3(NT), 0, st, args, mz_scale);
        };
        if (CC == 32 && a.cps % 2 == 0) {
            MfmaArgs a64 = a;
            a64.chunk = 64;
            a64.cps = a.cps / 2;
            a64.nchunks = (a.p.T + 63) / 64;
            if (mode == 1) pre(segment_state_kernel<64, 1>, a64);
            else if (mode == 2) pre(segment_state_kernel<64, 2>, a64);
            else pre(segment_state_kernel<64, 0>, a64);
        } else {
            if (mode == 1) pre(segment_state_kernel<CC, 1>, a);
            else if (mode == 2) pre(segment_state_kernel<CC, 2>, a);
            else pre(segment_state_kernel<CC, 0>, a);
        }
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (a.has_init) {
        const int nscan = BHv * kScanBlocks;
        const int nprep = prepass ? 0 : a.p.H * (kStoreRows / kPrepRows);
        hipLaunchKernelGGL(scan_prep_kernel, dim3(nscan + nprep), dim3(NT), 0, st, a, nscan, mz_scale);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else if ((e = launch_readout_prep(a.p.H, a.p.m, a.p.R, nullptr, const_cast<__bf16 *>(a.Mz),
                                        mz_scale, st)) != hipSuccess) {
        return e;
    }
    // Timing events, when given, are taken by the fused kernel's own dispatch: they
    // bracket the kernel alone and add no gap between launches.
    if (a.nchunks > 0 && a.hv == 2) {
        if ((e = launch_chunk256(a, st, ev_start, ev_stop)) != hipSuccess) return e;
    } else if (a.nchunks > 0) {
        const int mode = mix_mode(a);
        auto fused = [&](auto kern) {
            hipExtLaunchKernelGGL(kern, dim3(BHv * a.P), dim3(NT), 0, st, ev_start, ev_stop, 0, a);
        };
        if (mode == 1) fused(chunk_forward_kernel<CC, 1>);
        else if (mode == 2) fused(chunk_forward_kernel<CC, 2>);
        else fused(chunk_forward_kernel<CC, 0>);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else {
        if (ev_start && (e = hipEventRecord(ev_start, st)) != hipSuccess) return e;
        if (ev_stop && (e = hipEventRecord(ev_stop, st)) != hipSuccess) return e;
    }
    return hipSuccess;
}
}  // namespace

size_t mfma_workspace_bytes(const FwdParams &p, int segments) {
    // bytes beyond the float readout block the host API reserves first
    return ws_layout(p, segments).total - (readout_f32_bytes(p.H) + 255) / 256 * 256;
}

int mfma_auto_segments(const FwdParams &p) {
    // two workgroups of the four-wave kernel are resident per compute unit, one of
    // the eight-wave kernel (d = 256): split sequences until B*H*P fills the 256
    // compute units with them
    const int C = kMfmaChunk;
    const int slots = p.dk == 256 ? 256 : 256 * 2;
    const int seqs = p.B * p.H;
    int P = (slots + seqs - 1) / seqs;
    const int nchunks = (p.T + C - 1) / C;
    if (P > nchunks) P = nchunks;
    return P < 1 ? 1 : P;
}

hipError_t launch_fwd_mfma(const FwdParams &p, int P, void *ws, hipStream_t st,
                           hipEvent_t ev_start, hipEvent_t ev_stop, const MixIn *mix) {
    char *base = static_cast<char *>(ws);
    const WsLayout L = ws_layout(p, P);
    const int C = kMfmaChunk;
    MfmaArgs a{};
    a.p = p;
    a.chunk = C;
    a.nchunks = (p.T + C - 1) / C;
    a.P = P;
    a.cps = (a.nchunks + P - 1) / P;
    if (a.nchunks > 0) a.P = (a.nchunks + a.cps - 1) / a.cps;   // no empty trailing segment
    if (a.P < 1) a.P = 1;
    a.Mz = reinterpret_cast<const __bf16 *>(base + L.mz);
    a.seg_state = reinterpret_cast<__bf16 *>(base + L.state);
    a.fin_state = reinterpret_cast<float *>(base + L.fin);
    a.seg_span = reinterpret_cast<double *>(base + L.span);
    a.seg_gsum = reinterpret_cast<double *>(base + L.gsum);
    a.seg_origin = reinterpret_cast<double *>(base + L.origin);
    a.final_lam = reinterpret_cast<double *>(base + L.flam);
    a.want_final = (p.K_out || p.V_out || p.clock_out) ? 1 : 0;
    a.has_init = (a.P > 1 || p.K0 || p.V0 || p.clock0 || a.want_final) ? 1 : 0;
    a.zero_init = (p.K0 || p.V0) ? 0 : 1;
    a.hv = virtual_heads(p);
    if (mix) a.mix = *mix;
    const int BHv = p.B * p.H * a.hv;

    hipError_t e = launch_cc<32>(a, BHv, st, ev_start, ev_stop);
    if (e != hipSuccess) return e;
    if (a.want_final) {
        hipLaunchKernelGGL(state_out_kernel, dim3(BHv, 2 * 64 * 128 / NT), dim3(NT), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace cyfa
