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

constexpr int kPrepRows = 4;          // rows of M_h per workgroup (two per thread)
constexpr float kMaskLogit = -1e30f;  // padding-column entry of inactive slots in Mz

// Block (h, rb) of the grid (H, 128 / kPrepRows) computes rows [4 rb, 4 rb + 4) of M_h.
// Thread (j = tid % 128, g = tid / 128) owns paper basis column j and rows
// 4 rb + 2 g, 4 rb + 2 g + 1.  Phi[s][j] is read from a table of the m angles
// 2 pi r / m: the index (l s) mod m advances by l per step, with no division.
// M (fp32, paper basis order) and/or Mz (bf16, the matrix-core kernels' basis
// order: Mz[i'][j_int] = mz_scale * M[i'][paper(j_int)]) are written when non-null.
// 256 threads; (h, rb) is the block's head and row block.
__device__ __forceinline__ void readout_prep_block(int m, const float *__restrict__ R,
                                                   float *__restrict__ M, __bf16 *__restrict__ Mz,
                                                   float mz_scale, int h, int rb, int tid) {
    __shared__ float tab[2][kMaxActive];                     // cos, sin of 2 pi r / m
    __shared__ float Rrows[kPrepRows][kMaxActive + 1];
    const int row0 = rb * kPrepRows;
    if (tid < m) {
        double sn, cs;
        sincospi(2.0 * (double)tid / (double)m, &sn, &cs);
        tab[0][tid] = (float)cs;
        tab[1][tid] = (float)sn;
    }
    const float *Rh = R ? R + (size_t)h * m * m : nullptr;
    for (int e = tid; e < kPrepRows * m; e += 256) {
        const int r = e / m, s = e % m;
        const int i = row0 + r;
        Rrows[r][s] = i < m ? (Rh ? Rh[(size_t)i * m + s] : (s == i ? 1.f : 0.f)) : 0.f;
    }
    __syncthreads();
    const int j = tid & 127, r0 = 2 * (tid >> 7);
    float acc0 = 0.f, acc1 = 0.f;
    if (j == 0) {
        for (int s = 0; s < m; ++s) {
            acc0 += Rrows[r0][s];
            acc1 += Rrows[r0 + 1][s];
        }
        const float dc = (float)(1.0 / sqrt((double)m));
        acc0 *= dc;
        acc1 *= dc;
    } else if (j < m) {
        const int l = (j + 1) >> 1;                          // frequency of the column
        const float *t = tab[(j & 1) ? 0 : 1];               // odd columns cos, even sin
        int idx = 0;
#pragma unroll 4
        for (int s = 0; s < m; ++s) {
            const float ph = t[idx];
            acc0 = fmaf(Rrows[r0][s], ph, acc0);
            acc1 = fmaf(Rrows[r0 + 1][s], ph, acc1);
            idx += l;
            if (idx >= m) idx -= m;
        }
        const float ac = (float)sqrt(2.0 / (double)m);
        acc0 *= ac;
        acc1 *= ac;
    }
    const bool live = j < m;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int i = row0 + r0 + k;
        const float val = (live && i < m) ? (k ? acc1 : acc0) : 0.f;
        if (M) M[((size_t)h * kStoreRows + i) * kStoreRows + j] = val;
        if (Mz) {
            const int jint = j == 0 ? kStoreRows - 2 : (j == kStoreRows - 1 ? kStoreRows - 1 : j - 1);
            // inactive slots (rows >= m) carry kMaskLogit in the padding column: a kernel
            // that sets that column of its operand to 1 gets their logits at about
            // kMaskLogit, i.e. softmax weights of exactly 0, without masking code
            const float z = (j == kStoreRows - 1 && i >= m) ? kMaskLogit : mz_scale * val;
            Mz[((size_t)h * kStoreRows + i) * kStoreRows + jint] = (__bf16)z;
        }
    }
}

// Rows [32 rb, 32 rb + 32) of the bf16 matrix Mz of head h (the matrix-core
// kernels' copy only), in LDS the caller provides (at least 17 KiB, 16-byte
// aligned): extra blocks of the segment pre-pass run this, so that the readout
// matrix is formed while the pre-pass streams k and v.  Thread (j = tid % 128,
// g = tid / 128) computes paper column j of rows 32 rb + 16 g .. + 15; R's rows
// are staged zero-padded to 128 columns and read four columns at a time.
constexpr int kPrepRows32 = 32;
__device__ __forceinline__ void readout_prep_rows32(int m, const float *__restrict__ R,
                                                    __bf16 *__restrict__ Mz, float mz_scale, int h,
                                                    int rb, int tid, char *lds) {
    float *tab = reinterpret_cast<float *>(lds);            // [2][128] cos, sin of 2 pi r / m
    float *Rr = tab + 256;                                  // [32][128]
    const int row0 = kPrepRows32 * rb;
    if (tid < m) {
        double sn, cs;
        sincospi(2.0 * (double)tid / (double)m, &sn, &cs);
        tab[tid] = (float)cs;
        tab[128 + tid] = (float)sn;
    }
    const float *Rh = R ? R + (size_t)h * m * m : nullptr;
    for (int e = tid; e < kPrepRows32 * 128; e += 256) {
        const int r = e >> 7, sc = e & 127, i = row0 + r;
        Rr[e] = (i < m && sc < m) ? (Rh ? Rh[(size_t)i * m + sc] : (sc == i ? 1.f : 0.f)) : 0.f;
    }
    __syncthreads();
    const int j = tid & 127, g = tid >> 7;
    // column j: DC (j = 0: constant 1), cosine (odd j) or sine (even j > 0) of
    // frequency l = (j + 1) / 2; the table index l s mod m advances by l per step
    const float *t = (j == 0 || (j & 1)) ? tab : tab + 128;
    const int l = (j + 1) >> 1;
    float acc[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
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
            for (int r = 0; r < 16; ++r) {
                const float4 rv = *reinterpret_cast<const float4 *>(Rr + (16 * g + r) * 128 + s0);
                acc[r] = fmaf(rv.x, ph[0], fmaf(rv.y, ph[1], fmaf(rv.z, ph[2], fmaf(rv.w, ph[3], acc[r]))));
            }
        }
    }
    const float cscale = j == 0 ? (float)(1.0 / sqrt((double)m)) : (float)sqrt(2.0 / (double)m);
    const int jint = j == 0 ? kStoreRows - 2 : (j == kStoreRows - 1 ? kStoreRows - 1 : j - 1);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int i = row0 + 16 * g + r;
        const float val = (j < m && i < m) ? acc[r] * cscale : 0.f;
        const float z = (j == kStoreRows - 1 && i >= m) ? kMaskLogit : mz_scale * val;
        Mz[((size_t)h * kStoreRows + i) * kStoreRows + jint] = (__bf16)z;
    }
}

}  // namespace cyfa
