// Mixer prologue and epilogue around the CyFA operator (Sec. 4, network design).
//
// Prologue, per token t and head h:
//   ShortConv  y_t[c] = sum_{j<K} w[c][j] x_{t-K+1+j}[c]   (causal, depthwise; zero
//              before the sequence start), optionally SiLU, on q, k and v;
//   QK RMSNorm q_t <- q_t / sqrt(mean(q_t^2) + eps) * g_q  (and k);
//   gates      delta = sigmoid(z_delta + b_delta)           (Eq. clock_gradient_stabilization)
//              log alpha = -A softplus(z_alpha + b_alpha)   (the forget-gate parameterization)
//              beta = sigmoid(z_beta)
// Epilogue: out_t = RMSNorm(o_t) * g_o * sigmoid(gate_t)     (head-wise RMSNorm, output gate)
//
// Both are streaming kernels bound by HBM bandwidth; the gates are computed by
// extra workgroups of the convolution launch.  Thread layout: each thread
// owns eight consecutive channels (one 16-byte bf16 load or two float4 loads per
// token) of one head; the D / 8 threads of a head are consecutive lanes, so the
// RMSNorm sum is a shuffle reduction inside the wave.  A workgroup walks a run of
// kTokens consecutive tokens of one sequence, keeping the convolution's K - 1
// previous inputs in registers.
#include <algorithm>
#include "cyfa_mixer.h"

namespace cyfa {

namespace {

constexpr int kThreads = 256;
constexpr int kCh = 8;              // channels per thread
constexpr int kTokens = 16;         // tokens per workgroup
static_assert(kMixMaxConv % 4 == 0, "16-byte tap loads");

__device__ __forceinline__ float sigm(float x) { return mix_sigm(x); }
__device__ __forceinline__ float softplus_f(float x) { return mix_softplus(x); }

__device__ __forceinline__ int mix_tokens(const int *lens, int b, int T) {
    return lens ? min(max(lens[b], 0), T) : T;
}

__device__ __forceinline__ void load8(const float *p, float *x) {
    const float4 a = *reinterpret_cast<const float4 *>(p);
    const float4 b = *reinterpret_cast<const float4 *>(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ __forceinline__ void load8(const __hip_bfloat16 *p, float *x) {
    const uint4 u = *reinterpret_cast<const uint4 *>(p);
    const unsigned w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = __uint_as_float(w[i] << 16);
        x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}
__device__ __forceinline__ void store8(float *p, const float *y) {
    *reinterpret_cast<float4 *>(p) = make_float4(y[0], y[1], y[2], y[3]);
    *reinterpret_cast<float4 *>(p + 4) = make_float4(y[4], y[5], y[6], y[7]);
}
__device__ __forceinline__ void store8(__hip_bfloat16 *p, const float *y) {
    *reinterpret_cast<uint4 *>(p) = mix_pack_bf16x8(y);            // round to nearest even
}
// The same as nontemporal (streaming) stores.  The prologue's outputs are whole
// 16-byte pieces of consecutive lanes, read back only by a later launch; streaming
// them measured ~15 % faster than ordinary stores for that kernel (the epilogue,
// which reads two tensors per written one, measured no gain).
typedef unsigned u32x4_nt __attribute__((ext_vector_type(4)));
typedef float f32x4_nt __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store8_stream(float *p, const float *y) {
    const f32x4_nt a = {y[0], y[1], y[2], y[3]}, b = {y[4], y[5], y[6], y[7]};
    __builtin_nontemporal_store(a, reinterpret_cast<f32x4_nt *>(p));
    __builtin_nontemporal_store(b, reinterpret_cast<f32x4_nt *>(p + 4));
}
__device__ __forceinline__ void store8_stream(__hip_bfloat16 *p, const float *y) {
    const uint4 u = mix_pack_bf16x8(y);                               // round to nearest even
    const u32x4_nt v = {u.x, u.y, u.z, u.w};
    __builtin_nontemporal_store(v, reinterpret_cast<u32x4_nt *>(p));
}

// sum over the D / 8 consecutive lanes of one head
template <int D>
__device__ __forceinline__ float head_sum(float s) {
#pragma unroll
    for (int o = 1; o < D / kCh; o <<= 1) s += __shfl_xor(s, o);
    return s;
}

// Up to three [B, T, H, D] tensors (q, k, v) in one launch: blockIdx.z = tensor * B + b.
struct ConvSet {
    const void *x[3];
    const float *w[3];
    const float *g[3];
    void *y[3];
    int n;                          // tensors in the set; blockIdx.z >= n B runs the gates
    const float *z_delta, *b_delta, *z_alpha, *b_alpha, *A, *z_beta;
    float *delta, *log_alpha, *beta;
};


// ShortConv (+ SiLU) (+ RMSNorm) of the tensors of a ConvSet.
template <int D, int KMAX, typename Tin>
__global__ __launch_bounds__(kThreads) void conv_norm_kernel(ConvSet cs, int B, int T, int H, int K, int act,
                                                             float eps, const int *__restrict__ lens) {
    const int tensor = blockIdx.z / B, b = blockIdx.z % B, t_begin = blockIdx.y * kTokens;
    if (tensor >= cs.n) {
        // the scalar gates of tokens [t_begin, t_begin + kTokens) of sequence b, all heads
        if (blockIdx.x != 0) return;
        const int Tg = mix_tokens(lens, b, T);
        for (int e = threadIdx.x; e < kTokens * H; e += kThreads) {
            const int t = t_begin + e / H, h = e % H;
            if (t >= T) continue;
            const size_t i = ((size_t)b * T + t) * H + h;
            const bool live = t < Tg;
            if (cs.z_delta) cs.delta[i] = live ? sigm(cs.z_delta[i] + (cs.b_delta ? cs.b_delta[h] : 0.f)) : 0.f;
            if (cs.z_alpha) {
                const float za = cs.z_alpha[i] + (cs.b_alpha ? cs.b_alpha[h] : 0.f);
                cs.log_alpha[i] = live ? -cs.A[h] * softplus_f(za) : 0.f;
            }
            if (cs.z_beta) cs.beta[i] = live ? sigm(cs.z_beta[i]) : 0.f;
        }
        return;
    }
    const Tin *__restrict__ x = static_cast<const Tin *>(cs.x[tensor]);
    const float *__restrict__ w = cs.w[tensor];
    const float *__restrict__ g = cs.g[tensor];
    Tin *__restrict__ y = static_cast<Tin *>(cs.y[tensor]);
    const int c0 = (blockIdx.x * kThreads + threadIdx.x) * kCh;    // first channel of this thread
    const int HD = H * D;
    const bool active = c0 < HD;                                    // whole heads are active or not
    const int Tb = mix_tokens(lens, b, T);
    const int t_end = min(t_begin + kTokens, T);
    // wr[i][s]: weight of x_{t-s} (tap K - 1 - s), zero for s >= K; win[s] = x_{t-s}
    float wr[kCh][KMAX], gr[kCh], win[KMAX][kCh];
    if (w && active && K == KMAX) {
        // the eight channels' taps are KMAX * 8 consecutive floats: 16-byte loads
        const float4 *w4 = reinterpret_cast<const float4 *>(w + (size_t)c0 * KMAX);
#pragma unroll
        for (int i = 0; i < kCh; ++i) {
            float tap[KMAX];
#pragma unroll
            for (int q = 0; q < KMAX / 4; ++q) {
                const float4 f = w4[i * (KMAX / 4) + q];
                tap[4 * q] = f.x; tap[4 * q + 1] = f.y; tap[4 * q + 2] = f.z; tap[4 * q + 3] = f.w;
            }
#pragma unroll
            for (int s = 0; s < KMAX; ++s) wr[i][s] = tap[KMAX - 1 - s];
        }
    } else {
#pragma unroll
        for (int i = 0; i < kCh; ++i)
#pragma unroll
            for (int s = 0; s < KMAX; ++s)
                wr[i][s] = (w && active && s < K) ? w[(size_t)(c0 + i) * K + (K - 1 - s)] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kCh; ++i) gr[i] = (g && active) ? g[(c0 + i) % D] : 1.f;
    // inputs before the run, zero before the sequence start
#pragma unroll
    for (int s = 1; s < KMAX; ++s) {
        const int t = t_begin - s;
        if (w && active && s < K && t >= 0 && t < Tb) {
            load8(x + ((size_t)b * T + t) * HD + c0, win[s]);
        } else {
#pragma unroll
            for (int i = 0; i < kCh; ++i) win[s][i] = 0.f;
        }
    }
    // four tokens per step: their loads are issued together
    constexpr int kU = 4;
    for (int t0 = t_begin; t0 < t_end; t0 += kU) {
        float xin[kU][kCh];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int t = t0 + u;
            if (active && t < t_end && t < Tb) {
                load8(x + ((size_t)b * T + t) * HD + c0, xin[u]);
            } else {
#pragma unroll
                for (int i = 0; i < kCh; ++i) xin[u][i] = 0.f;
            }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int t = t0 + u;
            if (t >= t_end) break;
            const bool live = t < Tb;
            float yt[kCh];
#pragma unroll
            for (int i = 0; i < kCh; ++i) win[0][i] = xin[u][i];
#pragma unroll
            for (int i = 0; i < kCh; ++i) {
                float acc = w ? 0.f : win[0][i];
                if (w)
#pragma unroll
                    for (int s = 0; s < KMAX; ++s) acc = fmaf(wr[i][s], win[s][i], acc);
                yt[i] = act ? acc * sigm(acc) : acc;
            }
            if (g) {
                float ss = 0.f;
#pragma unroll
                for (int i = 0; i < kCh; ++i) ss = fmaf(yt[i], yt[i], ss);
                const float r = rsqrtf(head_sum<D>(ss) / (float)D + eps);
#pragma unroll
                for (int i = 0; i < kCh; ++i) yt[i] *= r * gr[i];
            }
            if (!live)
#pragma unroll
                for (int i = 0; i < kCh; ++i) yt[i] = 0.f;
            if (active) store8_stream(y + ((size_t)b * T + t) * HD + c0, yt);
            // slide the window: win[s] <- win[s - 1]
#pragma unroll
            for (int s = KMAX - 1; s >= 1; --s)
#pragma unroll
                for (int i = 0; i < kCh; ++i) win[s][i] = win[s - 1][i];
        }
    }
}

// Epilogue: head-wise RMSNorm and sigmoid output gate.
template <int D, typename Tin>
__global__ __launch_bounds__(kThreads) void norm_gate_kernel(const Tin *__restrict__ o, const Tin *__restrict__ gate,
                                                             const float *__restrict__ g, Tin *__restrict__ out,
                                                             int T, int H, float eps, const int *__restrict__ lens) {
    const int b = blockIdx.z, t_begin = blockIdx.y * kTokens;
    const int c0 = (blockIdx.x * kThreads + threadIdx.x) * kCh;
    const int HD = H * D;
    const bool active = c0 < HD;
    const int Tb = mix_tokens(lens, b, T);
    const int t_end = min(t_begin + kTokens, T);
    float gr[kCh];
#pragma unroll
    for (int i = 0; i < kCh; ++i) gr[i] = (g && active) ? g[(c0 + i) % D] : 1.f;
    for (int t = t_begin; t < t_end; ++t) {
        const bool live = t < Tb;
        const size_t base = ((size_t)b * T + t) * HD + c0;
        float yt[kCh], gt[kCh];
        if (active && live) {
            load8(o + base, yt);
            if (gate) load8(gate + base, gt);
        } else {
#pragma unroll
            for (int i = 0; i < kCh; ++i) yt[i] = 0.f;
        }
        float ss = 0.f;
#pragma unroll
        for (int i = 0; i < kCh; ++i) ss = fmaf(yt[i], yt[i], ss);
        const float r = rsqrtf(head_sum<D>(ss) / (float)D + eps);
#pragma unroll
        for (int i = 0; i < kCh; ++i) {
            float v = yt[i] * r * gr[i];
            if (gate && active && live) v *= sigm(gt[i]);
            yt[i] = live ? v : 0.f;
        }
        if (active) store8(out + base, yt);
    }
}

template <int D, typename Tin>
hipError_t launch_conv(const MixParams &p, const ConvSet &cs, int n, hipStream_t s) {
    (void)n;
    const int HD = p.H * D;
    const bool gates = p.z_delta || p.z_alpha || p.z_beta;
    const dim3 grid((HD / kCh + kThreads - 1) / kThreads, (p.T + kTokens - 1) / kTokens,
                    (cs.n + (gates ? 1 : 0)) * p.B);
    hipLaunchKernelGGL((conv_norm_kernel<D, kMixMaxConv, Tin>), grid, dim3(kThreads), 0, s, cs, p.B, p.T, p.H,
                       p.K, p.act, p.eps, p.lens);
    return hipGetLastError();
}

template <typename Tin>
hipError_t launch_conv_d(const MixParams &p, int D, const ConvSet &cs, int n, hipStream_t s) {
    if (D == 64) return launch_conv<64, Tin>(p, cs, n, s);
    if (D == 128) return launch_conv<128, Tin>(p, cs, n, s);
    return launch_conv<256, Tin>(p, cs, n, s);
}

// q, k and v in one launch when d_k = d_v, else q and k together and v alone
template <typename Tin>
hipError_t launch_qkv(const MixParams &p, hipStream_t s) {
    // the gates ride along with the launch that carries q and k
    ConvSet qkv{{p.q_in, p.k_in, p.v_in}, {p.wq, p.wk, p.wv}, {p.gq, p.gk, nullptr}, {p.q_out, p.k_out, p.v_out},
                p.dk == p.dv ? 3 : 2, p.z_delta, p.b_delta, p.z_alpha, p.b_alpha, p.A, p.z_beta,
                p.delta, p.log_alpha, p.beta};
    if (p.dk == p.dv) return launch_conv_d<Tin>(p, p.dk, qkv, 3, s);
    hipError_t e = launch_conv_d<Tin>(p, p.dk, qkv, 2, s);
    if (e != hipSuccess) return e;
    ConvSet v{{p.v_in, nullptr, nullptr}, {p.wv, nullptr, nullptr}, {nullptr, nullptr, nullptr},
              {p.v_out, nullptr, nullptr}, 1, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
              nullptr, nullptr, nullptr};
    MixParams pv = p;
    pv.z_delta = pv.z_alpha = pv.z_beta = nullptr;
    return launch_conv_d<Tin>(pv, p.dv, v, 1, s);
}

template <int D, typename Tin>
hipError_t launch_epi(const MixParams &p, const void *o, const void *gate, const float *g, void *out, hipStream_t s) {
    const int HD = p.H * D;
    const dim3 grid((HD / kCh + kThreads - 1) / kThreads, (p.T + kTokens - 1) / kTokens, p.B);
    hipLaunchKernelGGL((norm_gate_kernel<D, Tin>), grid, dim3(kThreads), 0, s, static_cast<const Tin *>(o),
                       static_cast<const Tin *>(gate), g, static_cast<Tin *>(out), p.T, p.H, p.eps, p.lens);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_mixer_prologue(const MixParams &p, hipStream_t s) {
    if (p.T == 0) return hipSuccess;
    return p.dtype == 0 ? launch_qkv<float>(p, s) : launch_qkv<__hip_bfloat16>(p, s);
}

hipError_t launch_mixer_epilogue(const MixParams &p, const void *o, const void *gate, const float *g, void *out,
                                 hipStream_t s) {
    if (p.T == 0) return hipSuccess;
    const int D = p.dv;
    if (p.dtype == 0) {
        if (D == 64) return launch_epi<64, float>(p, o, gate, g, out, s);
        if (D == 128) return launch_epi<128, float>(p, o, gate, g, out, s);
        return launch_epi<256, float>(p, o, gate, g, out, s);
    }
    if (D == 64) return launch_epi<64, __hip_bfloat16>(p, o, gate, g, out, s);
    if (D == 128) return launch_epi<128, __hip_bfloat16>(p, o, gate, g, out, s);
    return launch_epi<256, __hip_bfloat16>(p, o, gate, g, out, s);
}

}  // namespace cyfa
