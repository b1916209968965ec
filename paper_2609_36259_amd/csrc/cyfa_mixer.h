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

hipError_t launch_mixer_prologue(const MixParams &p, hipStream_t s);
hipError_t launch_mixer_epilogue(const MixParams &p, const void *o, const void *gate, const float *g, void *out,
                                 hipStream_t s);

}  // namespace cyfa
