// Internal declarations shared by the HIP translation units of libcyfa.
// Not part of the public ABI (include/cyfa.h).
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <stdint.h>

namespace cyfa {

constexpr int kStoreRows = 128;     // m* storage rows of every state (App. A.7)
constexpr int kMaxActive = 127;     // largest supported active slot count m

// Problem parameters handed from the host API to the launchers.
struct FwdParams {
    int B, T, H, dk, dv, m, chunk, segments;
    float scale;
    int dtype;                      // cyfa_dtype
    const void *q, *k, *v;
    const float *delta, *log_alpha, *beta, *R;
    const float *K0, *V0;
    const double *clock0;
    void *o;
    float *K_out, *V_out;
    double *clock_out;
    float *logits;
    const int *lens;                // [B] tokens of each sequence (clamped to [0, T]); NULL: all T
    const int *cu;                  // [B+1] packed sequences: sequence b is rows cu[b] .. cu[b+1]-1 of
                                    // [total, H, d] tensors (count clamped to [0, T]); NULL: [B, T, H, d]
};

struct DecParams {
    int N, H, dk, dv, m;
    float scale;
    int dtype;
    const void *q, *k, *v;
    const float *delta, *log_alpha, *beta, *R;
    float *K, *V;
    double *clock;
    void *o;
    float *logits;
};

// ---- workspace layout ----------------------------------------------------
// Readout matrices M_h = R_h Phi as float [H][128][128] (slot row, basis column
// in the basis order of App. A.1, zero padded).
inline size_t readout_f32_bytes(int H) { return (size_t)H * kStoreRows * kStoreRows * 4; }

// ---- launchers (return hipSuccess or the launch error) -------------------
hipError_t launch_readout_prep(int H, int m, const float *R, float *M, __bf16 *Mz, float mz_scale,
                               hipStream_t s);
hipError_t launch_fwd_valu(const FwdParams &p, const float *M, hipStream_t s);
hipError_t launch_decode(const DecParams &p, const float *M, hipStream_t s);

// ---- device helpers --------------------------------------------------------
// Tokens of sequence b: lens[b] clamped to [0, T], or T without lengths.  Tokens
// t >= that count are treated like the tail past the end of a sequence: no
// write, no decay, no clock shift, and their output rows are not written.
__device__ __forceinline__ int seq_tokens(const FwdParams &p, int b) {
    if (p.cu) return min(max(p.cu[b + 1] - p.cu[b], 0), p.T);
    return p.lens ? min(max(p.lens[b], 0), p.T) : p.T;
}
// Row (token index over the whole [rows, H, ...] tensor) of token 0 of sequence b:
// b T for the padded layout, cu[b] for packed sequences.
__device__ __forceinline__ size_t seq_row0(const FwdParams &p, int b) {
    return p.cu ? (size_t)p.cu[b] : (size_t)b * p.T;
}
__device__ __forceinline__ float load_as_float(const float *p, size_t i) { return p[i]; }
__device__ __forceinline__ float load_as_float(const __hip_bfloat16 *p, size_t i) {
    return __bfloat162float(p[i]);
}
__device__ __forceinline__ void store_from_float(float *p, size_t i, float x) { p[i] = x; }
__device__ __forceinline__ void store_from_float(__hip_bfloat16 *p, size_t i, float x) {
    p[i] = __float2bfloat16(x);   // round to nearest even
}

// lambda reduced to [0, m): exact up to the rounding of the subtraction, and
// harmless because U(tau + m) = U(tau).
__device__ __forceinline__ double reduce_clock(double lam, int m) {
    double r = lam - (double)m * floor(lam / (double)m);
    return (r >= (double)m) ? r - (double)m : r;
}
// Same with a multiply by inv_m = 1/m in place of the division: the quotient
// may round across an integer, which the two-sided correction undoes.
__device__ __forceinline__ double reduce_clock(double lam, double m, double inv_m) {
    double r = lam - m * floor(lam * inv_m);
    r = (r >= m) ? r - m : r;
    return (r < 0.0) ? r + m : r;
}

// cos and sin of theta_j = 2 pi j lam / m for a clock already reduced to
// [0, m).  The angle is reduced in revolutions in double precision first, so
// the float evaluation sees an argument in [0, 2) half-turns.
__device__ __forceinline__ void clock_phase(double lam_red, int j, int m, float *c, float *s) {
    double rev = (double)j * lam_red / (double)m;
    rev -= floor(rev);
    sincospif((float)(2.0 * rev), s, c);
}

}  // namespace cyfa
