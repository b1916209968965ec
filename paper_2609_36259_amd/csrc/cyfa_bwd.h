// Internal declarations of the backward pass (not part of the public ABI).
#pragma once

#include "cyfa_internal.h"

namespace cyfa {

constexpr int kBwdChunk = 16;       // tokens per chunk of the vector-ALU backward kernels
constexpr int kBwdMfmaChunk = 32;   // tokens per chunk of the matrix-core backward kernels
constexpr int kBwdFinParts = 8;     // partial sums of the final-state loss per (b, h)

// Gradients of L = sum_t <do_t, o_t> + <dK_T, Kbar_T> + <dV_T, Vbar_T>.
struct BwdParams {
    int B, T, H, dk, dv, m;
    int nc;                         // chunks per sequence, ceil(T / kBwdChunk)
    int Tpad;                       // nc * kBwdChunk: rows of the per-token workspace arrays
    int groups, cpg;                // chunk groups per sequence and chunks per group
    float scale;
    int dtype;
    const void *q, *k, *v, *dout;
    const float *delta, *log_alpha, *beta, *R;
    const int *lens;
    const int *cu;                  // packed sequences (the forward's group pre-pass only; see FwdParams)
    const float *K0, *V0;
    const double *clock0;
    const float *dK_T, *dV_T;
    void *gq, *gk, *gv;             // dtype of q
    float *gdelta, *glog_alpha, *gbeta, *gR, *gK0, *gV0;
    double *gclock0;
    // workspace (see bwd_workspace_bytes)
    const float *M;                 // [H][128][128] readout matrix R Phi
    // States entering chunk c of group g: Kst[c] + exp(Gin[c]) Ecar[g] (Kst from
    // the group's own tokens, Ecar the state entering the group).  Adjoint states
    // at chunk c's end: DKe[c] + exp(Gout[c]) Acar[g] (Acar: the adjoint at the
    // group's end from later groups and the final-state loss).
    float *Kst, *Vst;               // [BH][nc][128][d]
    double *clk;                    // [BH][nc] clock entering each chunk (reduced mod m)
    float *DKe, *DVe;               // [BH][nc][128][d]
    float *EcK, *EcV;               // [BH][groups][128][d]
    float *AcK, *AcV;               // [BH][groups][128][d]
    float *Gin, *Gout;              // [BH][nc] log decay from the group start / to the group end
    float *Gg;                      // [BH][groups] log decay over each group
    double *gclk;                   // [BH][groups] clock entering each group (reduced mod m),
                                    // written by the forward's group pre-pass only
    float *U, *dP;                  // [BH][Tpad][128] readout output u_t and key-pass adjoint dp_t
    float *udu, *dlam, *dG;         // [BH][Tpad] <u_t, du_t>, dL/dlambda_t, dL/dG_t
    float *dMp;                     // [BH][groups][128][128] partial dL/dM
    float *fin;                     // [BH][8] partial sums of <dK_T, Kbar_T> + <dV_T, Vbar_T>
};

size_t bwd_workspace_bytes(int B, int T, int H, int dk, int dv, int groups);

// The forward's chunk groups: the state entering each group of cpg 16-token
// chunks (d_k, d_v in {64, 128}, m <= 127), from the groups' own contributions
// and a combine in group order.  *EcK / *EcV point into ws at [BH][groups][128][d],
// *Eclk at [BH][groups]: the clock entering each group (reduced mod m).  The
// forward's chunk kernel reads the clock from there rather than from clock0, so
// that clock_out may alias clock0 (the last group writes it while earlier groups
// are still running).
size_t group_states_bytes(int B, int H, int dk, int dv, int groups);
hipError_t launch_group_states(const FwdParams &f, int groups, int cpg, void *ws, const float **EcK,
                               const float **EcV, const double **Eclk, hipStream_t s);
int bwd_auto_groups(int B, int T, int H);
hipError_t launch_bwd_valu(BwdParams p, void *ws, hipStream_t s);
// The last two kernels of either backward: reverse cumulative sums of p.dG and
// p.dlam (plus the final-state loss p.fin at the last token) into dlog_alpha,
// ddelta, dclock0; dR from the partial dM of every (b, h, group) in p.dMp.
hipError_t launch_bwd_tail(const BwdParams &p, hipStream_t s);

// Matrix-core backward (bf16, d_k = d_v = 128, m <= 127, 32-token chunks, p.nc and
// p.Tpad counted in those chunks).
int bwd_mfma_auto_groups(int B, int T, int H);
size_t bwd_mfma_workspace_bytes(int B, int T, int H, int groups);
hipError_t launch_bwd_mfma(BwdParams p, void *ws, hipStream_t s);

}  // namespace cyfa
