// Readout preparation: M_h = R_h Phi for every head.
//
// The absolute-clock readout (Sec. 3.2, Eq. cyfa-absolute-readout) applies
// R Phi U(lambda) to the key-pass output and U(-lambda) Phi^T R^T to the slot
// weights.  Both use the same m x m matrix M = R Phi, so it is formed once per
// call.  Phi is the real Fourier basis of App. A.1 (Eq. app-real-fourier):
// column 0 = 1/sqrt(m), column 2l-1 = sqrt(2/m) cos(2 pi l s / m), column
// 2l = sqrt(2/m) sin(2 pi l s / m).  Output: float [H][128][128], slot index
// on rows, basis index on columns, zero outside the active m x m block.
#include "cyfa_internal.h"

namespace cyfa {

constexpr int kPrepRowsPerBlock = 8;

// grid (H, 128 / 8): block (h, rb) writes rows [8 rb, 8 rb + 8) of M_h.
__global__ __launch_bounds__(256) void readout_prep_kernel(int m, const float *__restrict__ R,
                                                           float *__restrict__ M) {
    __shared__ float tab_c[kMaxActive], tab_s[kMaxActive];   // cos, sin of 2 pi r / m
    __shared__ float phi[kMaxActive][kStoreRows];            // Phi[s][j], j < 128 (zero padded)
    __shared__ float Rrows[kPrepRowsPerBlock][kMaxActive];
    const int h = blockIdx.x;
    const int row0 = blockIdx.y * kPrepRowsPerBlock;
    const int tid = threadIdx.x;
    if (tid < m) {
        double sn, cs;
        sincospi(2.0 * (double)tid / (double)m, &sn, &cs);
        tab_c[tid] = (float)cs;
        tab_s[tid] = (float)sn;
    }
    const float *Rh = R ? R + (size_t)h * m * m : nullptr;
    for (int e = tid; e < kPrepRowsPerBlock * m; e += blockDim.x) {
        const int r = e / m, s = e % m;
        const int i = row0 + r;
        Rrows[r][s] = i < m ? (Rh ? Rh[(size_t)i * m + s] : (s == i ? 1.f : 0.f)) : 0.f;
    }
    __syncthreads();
    const float dc = (float)(1.0 / sqrt((double)m));
    const float ac = (float)sqrt(2.0 / (double)m);
    {
        // thread (column j, half) fills rows s = half, half + 2, ...: the angle
        // index (l s) mod m advances by 2 l mod m without any division
        const int j = tid & 127, half = tid >> 7;
        const int l = (j + 1) >> 1;
        const int step = (2 * l) % m;
        int idx = (l * half) % m;
        for (int s = half; s < m; s += 2) {
            float val = 0.f;
            if (j == 0) {
                val = dc;
            } else if (j < m) {
                val = ac * ((j & 1) ? tab_c[idx] : tab_s[idx]);
            }
            phi[s][j] = val;
            idx += step;
            if (idx >= m) idx -= m;
        }
    }
    __syncthreads();
    // thread (j = tid % 128, half = tid / 128) computes rows 4 half .. 4 half + 3 of column j
    const int j = tid & 127, r0 = 4 * (tid >> 7);
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int s = 0; s < m; ++s) {
        const float ph = phi[s][j];
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[k] = fmaf(Rrows[r0 + k][s], ph, acc[k]);
    }
    float *Mh = M + (size_t)h * kStoreRows * kStoreRows;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int i = row0 + r0 + k;
        Mh[(size_t)i * kStoreRows + j] = (i < m && j < m) ? acc[k] : 0.f;
    }
}

hipError_t launch_readout_prep(int H, int m, const float *R, float *M, hipStream_t s) {
    hipLaunchKernelGGL(readout_prep_kernel, dim3(H, kStoreRows / kPrepRowsPerBlock), dim3(256), 0, s,
                       m, R, M);
    return hipGetLastError();
}

}  // namespace cyfa
