// Matrix-core (bf16 MFMA) chunk-wise CyFA forward for head dimension 256
// (d_k = d_v = 256, the paper's head size), 32-token chunks, m <= 127.
//
// The same computation as the 128-channel fused kernel (App. B: clock and
// log-decay prefix sums, temporal writes, key pass Eq. app-cyfa-key-chunk,
// token-wise softmax readout Eq. cyfa-two-pass (middle line), value pass
// Eq. app-cyfa-value-chunk), on one eight-wave workgroup per segment.  Both
// 256 x 128 carried states stay in MFMA accumulators:
//   wave w = (slot block sb = w mod 4, channel half dh = w div 4) holds
//     Kbar^T[d in 128 dh .. + 127][slots 32 sb .. + 31]   (4 accumulators), and
//     Vbar[all slots][d_v in 32 w .. + 31]                (4 accumulators),
// 128 registers per lane as in the 128-channel kernel.  The key pass's
// inter-chunk product contracts over all 256 channels: each wave forms the part
// of its own channel half and the high-half waves pass theirs to the low-half
// waves through LDS.  The causal score blocks (over 256 channels), the readout
// (128-dim, channel-independent) and the value-pass score blocks run on the four
// low-half waves; every wave updates its own part of both states and writes its
// own 32 output channels.
//
// Layout in LDS: q, k, v of a chunk as two 128-channel tiles each (low, high);
// the temporal writes, the (cos, sin) table, the readout matrix, X / W and O''
// exactly as in the 128-channel kernel (they live in the 128-dim slot / basis
// space).  One workgroup per compute unit (~118 KB of LDS); a sequence is cut
// into segments of whole chunks as in the 128-channel path.
//
// Segments: the states of a 256-channel head are two independent 128 x 128
// pairs (one per 128-channel block of k and v; the clock, the gates and the
// writes are shared), so the segment pre-pass, the scan of the entering states
// and the final-state conversion of the 128-channel path run on "virtual heads"
// of 128 channels, and this kernel reads and writes those heads' pairs.  Wave
// (sb, dh) holds what wave sb of the 128-channel kernel holds for block dh.
#include "cyfa_mfma_chunk.h"
#include "cyfa_prep.h"

#include <hip/hip_ext.h>

namespace cyfa {

using namespace mfma;

namespace {

constexpr int kNT8 = 512;                              // eight waves
constexpr int kCC = 32;                                // chunk length
constexpr int kD2 = 256;                               // head dimension

struct Lay2 {
    static constexpr int SSC = kCC + 8;                // score tile row stride
    static constexpr int CSW = 68;                     // (cos, sin) table row stride (half2 words)
    static constexpr int PTILE = kCC * QS * 2;         // padded [32][136] bf16 tile
    static constexpr int STILE = kCC * SWS * 2;        // swizzled [32][128] bf16 tile
    static constexpr int Q0 = 0;                       // Q channels 0..127 -> X -> W (padded)
    static constexpr int Q1 = Q0 + PTILE;              // Q channels 128..255 (padded)
    static constexpr int K0 = Q1 + PTILE;              // K low (swizzled) -> O'' (padded)
    static constexpr int K1 = K0 + PTILE;              // K high (swizzled)
    static constexpr int V0 = K1 + STILE;              // V low (swizzled)
    static constexpr int V1 = V0 + STILE;              // V high (swizzled)
    static constexpr int A = V1 + STILE;               // temporal writes (swizzled)
    static constexpr int S = A + STILE;                // score tile [32][SSC] bf16 / softmax partials
    static constexpr int RED = S;
    static constexpr int CS = S + kCC * SSC * 2;       // (cos, sin) table [32][CSW]
    static constexpr int MT = CS + kCC * CSW * 4;      // readout matrix [128][128] (swizzled)
    static constexpr int XB = MT + 128 * SWS * 2;      // high-half key-pass parts [4][64 lanes][16] fp32
    static constexpr int SC = XB + 4 * 64 * 16 * 4;    // per-token scalars
    static constexpr int BYTES = SC + scalar_bytes(kCC);
    static_assert(K0 % 256 == 0 && K1 % 256 == 0 && V0 % 256 == 0 && V1 % 256 == 0 && A % 256 == 0 &&
                      MT % 256 == 0,
                  "swizzled tiles start on a bank-window boundary");
    static_assert(QS * 2 == CSW * 4, "one token-row base for the padded tiles and the table");
    static_assert(4 * kCC * 8 <= kCC * SSC * 2, "softmax partials fit the score tile");
    static_assert(BYTES <= 160 * 1024, "one workgroup per compute unit");
};

// chunk staging: thread t holds row t/16, 16-byte column block t%16 of both
// channel halves of q, k and v
struct Pf2 {
    uint4 q[2], k[2], v[2];
    float g, dl, be;
};

__device__ __forceinline__ void load2(const FwdParams &p, int b, int h, int t0, int Tb, int tid, Pf2 &pf) {
    const size_t row_el = (size_t)p.H * kD2;
    const size_t base = (seq_row0(p, b) + t0) * row_el + (size_t)h * kD2;
    const int avail = Tb - t0;                          // rows of this chunk inside the sequence (uniform)
    const int r = tid >> 4;
    // rows past the sequence re-read its last row (always inside the tensor) and
    // are zeroed below: no load is predicated per lane
    const int rr = min(r, max(avail - 1, 0));
    const unsigned loff = (unsigned)(rr * (int)row_el + (tid & 15) * 8) * 2u;
    const char *q = reinterpret_cast<const char *>(static_cast<const __bf16 *>(p.q) + base);
    const char *k = reinterpret_cast<const char *>(static_cast<const __bf16 *>(p.k) + base);
    const char *v = reinterpret_cast<const char *>(static_cast<const __bf16 *>(p.v) + base);
    if (avail > 0) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            pf.q[hf] = *reinterpret_cast<const uint4 *>(q + loff + 256 * hf);
            pf.k[hf] = *reinterpret_cast<const uint4 *>(k + loff + 256 * hf);
            pf.v[hf] = *reinterpret_cast<const uint4 *>(v + loff + 256 * hf);
        }
    }
    if (r >= avail) {
        const uint4 zero = make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            pf.q[hf] = zero;
            pf.k[hf] = zero;
            pf.v[hf] = zero;
        }
    }
    if (tid < 64) {
        const size_t sbase = (seq_row0(p, b) + t0) * p.H + h;
        const unsigned soff = (unsigned)opq(tid * p.H);
        if (tid < kCC && tid < avail) {
            pf.dl = (p.delta + sbase)[soff];
            pf.g = p.log_alpha ? (p.log_alpha + sbase)[soff] : 0.f;
            pf.be = p.beta ? (p.beta + sbase)[soff] : 1.f;
        } else {
            pf.dl = 0.f;
            pf.g = 0.f;
            pf.be = 0.f;
        }
    }
}

__device__ __forceinline__ void store2(char *smem, int tid, const Pf2 &pf) {
    using L = Lay2;
    const int r = tid >> 4, c = (tid & 15) * 8;
    const int po = 2 * (r * QS + c), so = 2 * swz_elem(r, c);
    *reinterpret_cast<uint4 *>(smem + L::Q0 + po) = pf.q[0];
    *reinterpret_cast<uint4 *>(smem + L::Q1 + po) = pf.q[1];
    *reinterpret_cast<uint4 *>(smem + L::K0 + so) = pf.k[0];
    *reinterpret_cast<uint4 *>(smem + L::K1 + so) = pf.k[1];
    *reinterpret_cast<uint4 *>(smem + L::V0 + so) = pf.v[0];
    *reinterpret_cast<uint4 *>(smem + L::V1 + so) = pf.v[1];
}

// One 16 x 16 block (rb, sb) of the causal score tile, contraction over the
// channels of the padded tiles (A0, A1) and the swizzled tiles at byte offsets
// (B0, B1) -- two channel halves, or one when A1 is null.  Computed transposed,
// D[s][t]; Gamma applied unless the chunk is factored; upper triangle zero.
__device__ __forceinline__ void score_block2(const __bf16 *A0, const __bf16 *A1, char *smem, int B0, int B1,
                                             __bf16 *Ss, const float *Gs, int rb, int sb, int lane, bool fac) {
    constexpr int SSC = Lay2::SSC;
    const int l16 = lane & 15, g = lane >> 4;
    f32x4 acc = zero_acc4();
    const int ao = (16 * rb + l16) * QS + 8 * g;
    const int bo = 2 * swz_elem(16 * sb + l16, 8 * g);
    const int b0 = opq(B0 + bo);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) acc = mma16(lds8(lds_at<__bf16>(smem, b0 ^ (64 * ks))), lds8(A0 + ao + 32 * ks), acc);
    if (A1) {
        const int b1 = opq(B1 + bo);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
            acc = mma16(lds8(lds_at<__bf16>(smem, b1 ^ (64 * ks))), lds8(A1 + ao + 32 * ks), acc);
    }
    const int t = 16 * rb + l16;
    const int s0 = 16 * sb + 4 * g;
    if (!fac) {
        const float Gt = Gs[t];
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] *= __expf(Gt - Gs[s0 + r]);
    }
    bf16x4 sv;
#pragma unroll
    for (int r = 0; r < 4; ++r) sv[r] = (__bf16)(s0 + r <= t ? acc[r] : 0.f);
    *reinterpret_cast<bf16x4 *>(Ss + t * SSC + s0) = sv;
}

__device__ __forceinline__ bf16x8 decay_rows2(bf16x8 v, const float *dw) {
    const float4 d0 = *reinterpret_cast<const float4 *>(dw);
    const float4 d1 = *reinterpret_cast<const float4 *>(dw + 4);
    const float d[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
    bf16x8 r;
#pragma unroll
    for (int q = 0; q < 8; ++q) r[q] = (__bf16)((float)v[q] * d[q]);
    return r;
}

__device__ __forceinline__ void scale4(f32x16 (&acc)[4], float f) {
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[x][v] *= f;
}

__global__ __launch_bounds__(kNT8, 1) void chunk_forward256_kernel(MfmaArgs a) {
    using L = Lay2;
    constexpr int SSC = L::SSC;
    constexpr int CSW = L::CSW;
    constexpr int TE = L::PTILE / 2;
    __shared__ __attribute__((aligned(256))) char smem[L::BYTES];
    Tiles s{};
    s.Qs = lds_at<__bf16>(smem, L::Q0);
    s.As = lds_at<__bf16>(smem, L::A);
    s.Ss = lds_at<__bf16>(smem, L::S);
    s.CS = lds_at<half2v>(smem, L::CS);
    s.Mt = lds_at<__bf16>(smem, L::MT);
    scalars_at(s, smem + L::SC, kCC);
    const FwdParams &p = a.p;
    const int bh = blockIdx.x / a.P, seg = blockIdx.x % a.P;
    const int b = bh / p.H, h = bh % p.H;
    const int tid = threadIdx.x, lane = tid & 63, l32 = lane & 31, hl = lane >> 5, h4 = 4 * hl;
    const int w8 = __builtin_amdgcn_readfirstlane(tid >> 6);       // wave, uniform
    const int sb = w8 & 3, dh = w8 >> 2;
    const bool low = dh == 0;
    const int m = p.m;
    const int c_begin = seg * a.cps, c_end = min(c_begin + a.cps, a.nchunks);
    const int Tb = seq_tokens(p, b);
    const float zs = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(p.scale * 1.4426950408889634f)));

    const int trs = tr_off_swz(lane);
    const float *eps_t = lds_at<float>(smem, opq(L::SC + 4 * (kCC + l32)));     // gam of token l32
    const int dw_off = L::SC + 4 * (3 * kCC + 8 * hl);                          // decw, operand tokens
    const int Mza = opq(L::MT + 2 * swz_elem(32 * sb + l32, 8 * hl));
    const int trw = opq(trs ^ (64 * sb));
    const int tr0 = opq(trs);
    const __bf16 *Myt = lds_at<__bf16>(smem, opq(L::MT + (trs ^ (64 * sb))));
    const int Qh = dh ? L::Q1 : L::Q0;                                        // this wave's q half
    const int Kh = dh ? L::K1 : L::K0;                                        // this wave's k half
    const int Vh = dh ? L::V1 : L::V0;                                        // v half of this wave's channels
    const __bf16 *Qperm = lds_at<__bf16>(smem, opq(Qh + 2 * (l32 * QS + h4)));
    const __bf16 *Operm = lds_at<__bf16>(smem, opq(L::K0 + 2 * (l32 * QS + h4)));   // O'' (K low's region)
    const __bf16 *Xa = lds_at<__bf16>(smem, opq(L::Q0 + 2 * (l32 * QS + 8 * hl)));
    const __bf16 *Sa = lds_at<__bf16>(smem, opq(L::S + 2 * (l32 * SSC + 8 * hl)));
    const __bf16 *At = lds_at<__bf16>(smem, L::A + trw);
    const __bf16 *Vt = lds_at<__bf16>(smem, Vh + trw);
    const int rowb = opq(2 * (l32 * QS + 32 * sb + h4));
    __bf16 *Wrow = lds_at<__bf16>(smem, L::Q0 + rowb);
    __bf16 *O2row = Wrow + TE * 2;                                            // K low's region (padded)
    const half2v *CSrow = lds_at<half2v>(smem, L::CS + rowb);
    float2 *redw = lds_at<float2>(smem, opq(L::RED + 8 * (sb * kCC + l32)));
    const float2 *redr = lds_at<float2>(smem, opq(L::RED + 8 * l32));
    float *xb = lds_at<float>(smem, opq(L::XB + 4 * 16 * (sb * 64 + lane)));   // part exchange, this lane
    static_assert(L::K0 == L::Q0 + 2 * L::PTILE, "O'' sits two padded tiles after X / W");

    Pf2 pf;
    load2(p, b, h, c_begin * kCC, Tb, tid, pf);
    {
        const __bf16 *Mh = a.Mz + (size_t)h * 128 * 128;
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int e = it * kNT8 + tid;
            const int row = e >> 4, c0 = (e & 15) * 8;
            *reinterpret_cast<uint4 *>(s.Mt + swz_elem(row, c0)) = *reinterpret_cast<const uint4 *>(Mh + row * 128 + c0);
        }
    }
    // Wave (sb, dh) holds exactly what wave sb of the 128-channel kernel holds for
    // the 128-channel block dh of this head: its entering and final states are
    // that virtual head's pairs (index 2 bh + dh), in the same dump layout.
    f32x16 kacc[4], vacc[4];
    const size_t vh = (size_t)bh * 2 + dh;
    if (a.has_init && !(seg == 0 && a.zero_init)) {
        load_state(a.seg_state + (vh * a.P + seg) * kStateFloats, sb, lane, kacc, vacc);
    } else {
#pragma unroll
        for (int x = 0; x < 4; ++x) {
            kacc[x] = f32x16{};
            vacc[x] = f32x16{};
        }
    }
    double carry = 0.0, gsum = 0.0;
    float logf = 0.f;
    __bf16 *o = static_cast<__bf16 *>(p.o);

    for (int c = c_begin; c < c_end; ++c) {
        const int t0 = c * kCC;
        const int n = min(kCC, Tb - t0);
        // -- A: stage, prefix sums, temporal writes; prefetch the next chunk
        store2(smem, tid, pf);
        if (w8 == 0) {
            Prefetch<kCC, kNT8> sp;
            sp.g = pf.g;
            sp.dl = pf.dl;
            sp.be = pf.be;
            chunk_scans<kCC, kNT8, kCC, true>(s, lane, m, sp, carry, gsum, logf);
        }
        lds_barrier();
        if (c + 1 < c_end) load2(p, b, h, t0 + kCC, Tb, tid, pf);
        const float sf = __int_as_float(__builtin_amdgcn_readfirstlane(__float_as_int(s.ctl[0])));
        const bool fac = __builtin_amdgcn_readfirstlane(__float_as_int(s.ctl[2])) != 0;
        build_writes_swz<kCC, true, kNT8, CSW>(s, s.As, tid, m);
        lds_barrier();
        // -- B: key pass.  O'^T = Kbar' Q^T + A_dec^T S^T (as in the 128-channel
        //    kernel), the first term summed over the two channel halves.
        if (fac && sf != 1.f) scale4(kacc, sf);
        if (low) score_block2(lds_at<__bf16>(smem, L::Q0), lds_at<__bf16>(smem, L::Q1), smem, L::K0, L::K1, s.Ss, s.Gs,
                              sb >> 1, sb & 1, lane, fac);
        f32x16 oacc = zero_acc();
#pragma unroll
        for (int ks = 0; ks < 8; ++ks)
            oacc = mma(acc_to_operand(kacc[ks >> 1], ks & 1), lds8_perm(Qperm, 16 * ks, 0), oacc);
        if (!fac) {
            const float gt = *eps_t;
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[v] *= gt;
        }
        if (!low) {
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4)
                *reinterpret_cast<float4 *>(xb + 4 * q4) =
                    make_float4(oacc[4 * q4], oacc[4 * q4 + 1], oacc[4 * q4 + 2], oacc[4 * q4 + 3]);
        }
        lds_barrier();
        if (low) {
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const float4 t = *reinterpret_cast<const float4 *>(xb + 4 * q4);
                oacc[4 * q4] += t.x;
                oacc[4 * q4 + 1] += t.y;
                oacc[4 * q4 + 2] += t.z;
                oacc[4 * q4 + 3] += t.w;
            }
#pragma unroll
            for (int ks = 0; ks < kCC / 16; ++ks) oacc = mma(lds8_tr(At + 16 * ks * SWS, SWS), lds8(Sa + 16 * ks), oacc);
            if (fac) {
                const float et = *eps_t;
#pragma unroll
                for (int v = 0; v < 16; ++v) oacc[v] *= et;
            }
        }
        {
            // key state: Kbar'^T += K^T A_dec on this wave's channel half
            if (!fac && sf != 1.f) scale4(kacc, sf);
            const int kt = opq(Kh + tr0);
#pragma unroll
            for (int ks = 0; ks < kCC / 16; ++ks) {
                bf16x8 ad_w = lds8_tr(At + 16 * ks * SWS, SWS);
                if (!fac) ad_w = decay_rows2(ad_w, lds_at<float>(smem, opq(dw_off)) + 16 * ks);
#pragma unroll
                for (int x = 0; x < 4; ++x)
                    kacc[x] = mma(lds8_tr(lds_at<__bf16>(smem, kt ^ (64 * x)) + 16 * ks * SWS, SWS), ad_w, kacc[x]);
            }
        }
        if (low) {
            // X_r = U(lambda_r) O'_r -> X tile (Q low's region)
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                bf16x4 xv;
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    const half2v cs = CSrow[4 * v4 + k2];
                    const float cc = (float)cs[0], sn = (float)cs[1];
                    const float xc = oacc[4 * v4 + 2 * k2], xs = oacc[4 * v4 + 2 * k2 + 1];
                    xv[2 * k2] = (__bf16)fmaf(-sn, xs, cc * xc);
                    xv[2 * k2 + 1] = (__bf16)fmaf(sn, xc, cc * xs);
                }
                // padding column 127 is 1: the readout matrix holds the mask logit
                // there on the rows of inactive slots
                if (v4 == 3 && sb == 3 && hl) xv[3] = (__bf16)1.f;
                *reinterpret_cast<bf16x4 *>(Wrow + 8 * v4) = xv;
            }
        }
        lds_barrier();
        // -- C: middle step on the four low-half waves (slots 32 sb ..)
        f32x16 zacc = zero_acc();
        float mwave = 0.f;
        if (low) {
            const int mz = opq(Mza);
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) zacc = mma(lds8(lds_at<__bf16>(smem, mz ^ (32 * ks))), lds8(Xa + 16 * ks), zacc);
            float mx = zacc[0];
#pragma unroll
            for (int v = 1; v < 16; ++v) mx = fmaxf(mx, zacc[v]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            if (p.logits && l32 < n) {
                float *lg = p.logits + ((seq_row0(p, b) + t0 + l32) * p.H + h) * m;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int slot = 32 * sb + 8 * (v >> 2) + h4 + (v & 3);
                    if (slot < m) lg[slot] = zacc[v] * 0.69314718055994531f;
                }
            }
            mwave = mx;
            const float mref = mx == -INFINITY ? 0.f : mx;
#pragma unroll
            for (int v = 0; v < 16; ++v) zacc[v] = __builtin_amdgcn_exp2f(zacc[v] - mref);
            float t8[8];
#pragma unroll
            for (int v = 0; v < 8; ++v) t8[v] = zacc[v] + zacc[v + 8];
#pragma unroll
            for (int v = 0; v < 4; ++v) t8[v] += t8[v + 4];
            float sm = (t8[0] + t8[2]) + (t8[1] + t8[3]);
            sm += __shfl_xor(sm, 32);
            if (hl == 0) redw[0] = make_float2(mx, sm);
        }
        lds_barrier();
        if (low) {
            float2 pr[4];
#pragma unroll
            for (int x = 0; x < 4; ++x) pr[x] = redr[x * kCC];
            const float M = fmaxf(fmaxf(pr[0].x, pr[1].x), fmaxf(pr[2].x, pr[3].x));
            float Lsum = 0.f;
#pragma unroll
            for (int x = 0; x < 4; ++x) Lsum += pr[x].y * __builtin_amdgcn_exp2f(pr[x].x - M);
            const float f = mwave == -INFINITY ? 0.f
                                               : __builtin_amdgcn_exp2f(mwave - M) * __builtin_amdgcn_rcpf(Lsum * zs);
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                bf16x4 wv;
#pragma unroll
                for (int k = 0; k < 4; ++k) wv[k] = (__bf16)(zacc[4 * v4 + k] * f);
                *reinterpret_cast<bf16x4 *>(Wrow + 8 * v4) = wv;
            }
        }
        lds_barrier();
        if (low) {
            // O''_r = U(-lambda_r) M^T W_r -> O'' tile (K low's region, padded)
            half2v csy[8];
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4)
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) csy[2 * v4 + k2] = CSrow[4 * v4 + k2];
            f32x16 yacc = zero_acc();
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) yacc = mma(lds8_tr(Myt + 16 * ks * SWS, SWS), lds8(Xa + 16 * ks), yacc);
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                bf16x4 ov;
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                    const half2v cs = csy[2 * v4 + k2];
                    const float cc = (float)cs[0], sn = (float)cs[1];
                    const float yc = yacc[4 * v4 + 2 * k2], ysn = yacc[4 * v4 + 2 * k2 + 1];
                    ov[2 * k2] = (__bf16)fmaf(sn, ysn, cc * yc);
                    ov[2 * k2 + 1] = (__bf16)fmaf(-sn, yc, cc * ysn);
                }
                *reinterpret_cast<bf16x4 *>(O2row + 8 * v4) = ov;
            }
        }
        lds_barrier();
        // -- D: value pass.  O^T = Vbar'^T O''^T + V^T S2^T for this wave's 32
        //    output channels 32 w8 ..; S2 = O'' A_dec^T (low-half waves)
        if (fac && sf != 1.f) scale4(vacc, sf);
        if (low) score_block2(lds_at<__bf16>(smem, L::K0), nullptr, smem, L::A, 0, s.Ss, s.Gs, sb >> 1, sb & 1, lane,
                              fac);
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
        for (int ks = 0; ks < kCC / 16; ++ks) pacc = mma(lds8_tr(Vt + 16 * ks * SWS, SWS), lds8(Sa + 16 * ks), pacc);
        if (fac) {
            const float et = *eps_t;
#pragma unroll
            for (int v = 0; v < 16; ++v) pacc[v] *= et;
        }
        if (l32 < n) {
            char *ob = reinterpret_cast<char *>(o + ((seq_row0(p, b) + t0) * p.H + h) * kD2);
            const unsigned loff = (unsigned)opq((l32 * p.H * kD2 + 32 * w8 + h4) * 2);
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
                bf16x4 ov;
#pragma unroll
                for (int k = 0; k < 4; ++k) ov[k] = (__bf16)pacc[4 * v4 + k];
                *reinterpret_cast<bf16x4 *>(ob + loff + 16 * v4) = ov;
            }
        }
        {
            // value state: Vbar' += A_dec^T V on this wave's channels
            if (!fac && sf != 1.f) scale4(vacc, sf);
            const int at = opq(L::A + tr0);
#pragma unroll
            for (int ks = 0; ks < kCC / 16; ++ks) {
                bf16x8 v_w = lds8_tr(Vt + 16 * ks * SWS, SWS);
                if (!fac) v_w = decay_rows2(v_w, lds_at<float>(smem, opq(dw_off)) + 16 * ks);
#pragma unroll
                for (int x = 0; x < 4; ++x)
                    vacc[x] = mma(lds8_tr(lds_at<__bf16>(smem, at ^ (64 * x)) + 16 * ks * SWS, SWS), v_w, vacc[x]);
            }
        }
        lds_barrier();
    }
    if (a.want_final && seg == a.P - 1) {
        const float f = __expf(s.ctl[1]);
        scale4(kacc, f);
        scale4(vacc, f);
        dump_state(a.fin_state + vh * kStateFloats, sb, lane, kacc, vacc);
        if (tid == 0) {
            // the clock runs on wave 0; both virtual heads carry it
            a.final_lam[2 * bh] = carry;
            a.final_lam[2 * bh + 1] = carry;
        }
    }
}

}  // namespace

hipError_t launch_chunk256(const MfmaArgs &a, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
    hipExtLaunchKernelGGL(chunk_forward256_kernel, dim3(a.p.B * a.p.H * a.P), dim3(kNT8), 0, st, ev_start,
                          ev_stop, 0, a);
    return hipGetLastError();
}

}  // namespace cyfa
