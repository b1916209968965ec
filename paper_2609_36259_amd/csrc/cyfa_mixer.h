// Internal declarations of the mixer prologue / epilogue (not part of the public ABI).
#pragma once

#include "cyfa_internal.h"

namespace cyfa {

constexpr int kMixMaxConv = 4;      // longest ShortConv supported

struct MixParams {
    int B, T, H, dk, dv;
    int K;                          // ShortConv width (1 .. kMixMaxConv)
    int act;                        // 1: SiLU after the convolution
    float eps;                      // RMSNorm epsilon
    int dtype;                      // cyfa_dtype of q, k, v (and o, gate, out)
    const void *q_in, *k_in, *v_in;
    const float *wq, *wk, *wv;      // [H*d][K] or NULL (no convolution)
    const float *gq, *gk;           // [d_k] RMSNorm weights or NULL (no normalisation)
    const float *z_delta, *b_delta, *z_alpha, *b_alpha, *A, *z_beta;
    const int *lens;
    void *q_out, *k_out, *v_out;
    float *delta, *log_alpha, *beta;
};

// Gate activations of the prologue (Eq. clock_gradient_stabilization and the
// forget-gate parameterisation); shared by the standalone prologue and the
// matrix-core forward that runs the prologue inside its chunk staging, so that
// both produce the same bits.
// (the reciprocal is the hardware one, within 1 ulp; the fused and the standalone
// paths both use this function, so they agree bit for bit)
__device__ __forceinline__ float mix_sigm(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }
// fp32 -> bf16, round to nearest even (the hardware conversion)
__device__ __forceinline__ uint4 mix_pack_bf16x8(const float *y) {
    typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
    bf16x8_t t;
#pragma unroll
    for (int i = 0; i < 8; ++i) t[i] = (__bf16)y[i];
    return *reinterpret_cast<const uint4 *>(&t);
}
__device__ __forceinline__ float mix_softplus(float x) { return x > 20.f ? x : log1pf(__expf(x)); }

// Mixer inputs of the fused layer forward (cyfa_forward_mixer): the raw
// projections come in through FwdParams q, k, v; these are the rest.
struct MixIn {
    const float *wq, *wk, *wv;      // [H*128][K] ShortConv taps or NULL (no convolution)
    const float *gq, *gk;           // [128] RMSNorm weights or NULL (no normalisation)
    const float *z_delta, *b_delta; // delta = sigmoid(z_delta + b_delta); z_delta required
    const float *z_alpha, *b_alpha, *A;  // log alpha = -A softplus(z_alpha + b_alpha); NULL: 0
    const float *z_beta;            // beta = sigmoid(z_beta); NULL: 1
    const void *gate;               // [B, T, H, 128] output gate or NULL
    const float *g_o;               // [128] output RMSNorm weights or NULL (unit)
    int K, act;                     // ShortConv width 1..kMixMaxConv, SiLU after it
    float eps;                      // RMSNorm epsilon
    int fuse_conv;                  // 1: ShortConv and QK RMSNorm in the forward kernels' staging;
                                    // 0: q, k, v arrive already through them (standalone prologue)
};

hipError_t launch_mixer_prologue(const MixParams &p, hipStream_t s);
hipError_t launch_mixer_epilogue(const MixParams &p, const void *o, const void *gate, const float *g, void *out,
                                 hipStream_t s);

}  // namespace cyfa
