// Readout preparation: M_h = R_h Phi for every head.
//
// The absolute-clock readout (Sec. 3.2, Eq. cyfa-absolute-readout) applies
// R Phi U(lambda) to the key-pass output and U(-lambda) Phi^T R^T to the slot
// weights.  Both use the same m x m matrix M = R Phi, so it is formed once per
// call.  Phi is the real Fourier basis of App. A.1 (Eq. app-real-fourier):
// column 0 = 1/sqrt(m), column 2l-1 = sqrt(2/m) cos(2 pi l s / m), column
// 2l = sqrt(2/m) sin(2 pi l s / m).  Output [H][128][128], slot index on rows,
// basis index on columns, zero outside the active m x m block.
#pragma once

#include "cyfa_internal.h"

namespace cyfa {

constexpr float kMaskLogit = -1e30f;  // padding-column entry of inactive slots in Mz

// Block (h, rb) computes rows [ROWS rb, ROWS rb + ROWS) of M_h in LDS the caller
// provides (prep_lds_bytes(ROWS), 16-byte aligned; extra blocks of the segment
// pre-pass use the pre-pass's own, so that the readout matrix is formed while the
// pre-pass streams k and v).  256 threads: thread (j = tid % 128, g = tid / 128)
// computes paper column j of rows ROWS rb + ROWS/2 g .. + ROWS/2-1; R's rows are staged
// zero-padded to 128 columns and read four columns at a time, and Phi[s][j] comes
// from a table of the m angles 2 pi r / m (the index l s mod m advances by l per
// step, with no division).  M (fp32, paper basis order) and/or Mz (bf16, the
// matrix-core kernels' basis order: Mz[i'][j_int] = mz_scale * M[i'][paper(j_int)])
// are written when non-null.
__host__ __device__ constexpr int prep_lds_bytes(int rows) { return (256 + rows * 128) * 4; }
template <int ROWS>
__device__ __forceinline__ void readout_prep_rows(int m, const float *__restrict__ R, float *__restrict__ M,
                                                  __bf16 *__restrict__ Mz, float mz_scale, int h,
                                                  int rb, int tid, char *lds) {
    constexpr int RPT = ROWS / 2;                           // rows per thread
    float *tab = reinterpret_cast<float *>(lds);            // [2][128] cos, sin of 2 pi r / m
    float *Rr = tab + 256;                                  // [ROWS][128]
    const int row0 = ROWS * rb;
    if (tid < m) {
        double sn, cs;
        sincospi(2.0 * (double)tid / (double)m, &sn, &cs);
        tab[tid] = (float)cs;
        tab[128 + tid] = (float)sn;
    }
    const float *Rh = R ? R + (size_t)h * m * m : nullptr;
    for (int e = tid; e < ROWS * 128; e += 256) {
        const int r = e >> 7, sc = e & 127, i = row0 + r;
        Rr[e] = (i < m && sc < m) ? (Rh ? Rh[(size_t)i * m + sc] : (sc == i ? 1.f : 0.f)) : 0.f;
    }
    __syncthreads();
    const int j = tid & 127, g = tid >> 7;
    // column j: DC (j = 0: constant 1), cosine (odd j) or sine (even j > 0) of
    // frequency l = (j + 1) / 2; the table index l s mod m advances by l per step
    const float *t = (j == 0 || (j & 1)) ? tab : tab + 128;
    const int l = (j + 1) >> 1;
    float acc[RPT];
#pragma unroll
    for (int r = 0; r < RPT; ++r) acc[r] = 0.f;
    if (j < m) {
        int idx = 0;
        for (int s0 = 0; s0 < 128; s0 += 4) {
            float ph[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                ph[q] = t[idx];
                idx += l;
                if (idx >= m) idx -= m;
            }
#pragma unroll
            for (int r = 0; r < RPT; ++r) {
                const float4 rv = *reinterpret_cast<const float4 *>(Rr + (RPT * g + r) * 128 + s0);
                acc[r] = fmaf(rv.x, ph[0], fmaf(rv.y, ph[1], fmaf(rv.z, ph[2], fmaf(rv.w, ph[3], acc[r]))));
            }
        }
    }
    const float cscale = j == 0 ? (float)(1.0 / sqrt((double)m)) : (float)sqrt(2.0 / (double)m);
    const int jint = j == 0 ? kStoreRows - 2 : (j == kStoreRows - 1 ? kStoreRows - 1 : j - 1);
#pragma unroll
    for (int r = 0; r < RPT; ++r) {
        const int i = row0 + RPT * g + r;
        const float val = (j < m && i < m) ? acc[r] * cscale : 0.f;
        if (M) M[((size_t)h * kStoreRows + i) * kStoreRows + j] = val;
        if (Mz) {
            // inactive slots (rows >= m) carry kMaskLogit in the padding column: a kernel
            // that sets that column of its operand to 1 gets their logits at about
            // kMaskLogit, i.e. softmax weights of exactly 0, without masking code
            const float z = (j == kStoreRows - 1 && i >= m) ? kMaskLogit : mz_scale * val;
            Mz[((size_t)h * kStoreRows + i) * kStoreRows + jint] = (__bf16)z;
        }
    }
}

}  // namespace cyfa
