// Readout preparation kernel (M_h = R_h Phi for every head); the per-block
// computation is in cyfa_prep.h.
#include "cyfa_prep.h"

namespace cyfa {

// rows of M_h per workgroup of the standalone launch (H x 16 workgroups)
constexpr int kRows = 8;

__global__ __launch_bounds__(256) void readout_prep_kernel(int m, const float *__restrict__ R,
                                                           float *__restrict__ M,
                                                           __bf16 *__restrict__ Mz, float mz_scale) {
    __shared__ __attribute__((aligned(16))) char lds[prep_lds_bytes(kRows)];
    readout_prep_rows<kRows>(m, R, M, Mz, mz_scale, blockIdx.x, blockIdx.y, threadIdx.x, lds);
}

hipError_t launch_readout_prep(int H, int m, const float *R, float *M, __bf16 *Mz, float mz_scale,
                               hipStream_t s) {
    hipLaunchKernelGGL(readout_prep_kernel, dim3(H, kStoreRows / kRows), dim3(256), 0, s,
                       m, R, M, Mz, mz_scale);
    return hipGetLastError();
}

}  // namespace cyfa

// ---- 256 storage rows (127 < m <= 255) -------------------------------------
#include "cyfa_rows.h"

namespace cyfa {

constexpr int kWideRowsPerBlock = 8;

// Block (h, rb): rows 8 rb .. 8 rb + 7 of M_h; thread j computes column j of
// those rows, M[i][j] = sum_s R[i][s] Phi[s][j], with Phi[s][j] from a table of
// the m angles 2 pi n / m (index l s mod m for frequency l = (j + 1) / 2).
__global__ __launch_bounds__(256) void readout_prep_wide_kernel(int m, const float *__restrict__ R,
                                                                float *__restrict__ M) {
    __shared__ float tab[2][kWideRows];
    __shared__ float Rr[kWideRowsPerBlock][kWideRows];
    const int h = blockIdx.x, i0 = blockIdx.y * kWideRowsPerBlock, j = threadIdx.x;
    if (j < m) {
        double sn, cs;
        sincospi(2.0 * (double)j / (double)m, &sn, &cs);
        tab[0][j] = (float)cs;
        tab[1][j] = (float)sn;
    }
    const float *Rh = R ? R + (size_t)h * m * m : nullptr;
    for (int r = 0; r < kWideRowsPerBlock; ++r) {
        const int i = i0 + r;
        Rr[r][j] = (i < m && j < m) ? (Rh ? Rh[(size_t)i * m + j] : (i == j ? 1.f : 0.f)) : 0.f;
    }
    __syncthreads();
    float acc[kWideRowsPerBlock];
#pragma unroll
    for (int r = 0; r < kWideRowsPerBlock; ++r) acc[r] = 0.f;
    if (j < m) {
        const int l = (j + 1) >> 1;
        const float *t = (j == 0 || (j & 1)) ? tab[0] : tab[1];
        int idx = 0;
        for (int s = 0; s < m; ++s) {
            const float ph = t[idx];
            idx += l;
            if (idx >= m) idx -= m;
#pragma unroll
            for (int r = 0; r < kWideRowsPerBlock; ++r) acc[r] = fmaf(Rr[r][s], ph, acc[r]);
        }
    }
    const float cscale = j == 0 ? (float)(1.0 / sqrt((double)m)) : (float)sqrt(2.0 / (double)m);
#pragma unroll
    for (int r = 0; r < kWideRowsPerBlock; ++r) {
        const int i = i0 + r;
        M[((size_t)h * kWideRows + i) * kWideRows + j] = (j < m && i < m) ? acc[r] * cscale : 0.f;
    }
}

hipError_t launch_readout_prep_wide(int H, int m, const float *R, float *M, hipStream_t s) {
    hipLaunchKernelGGL(readout_prep_wide_kernel, dim3(H, kWideRows / kWideRowsPerBlock), dim3(kWideRows), 0,
                       s, m, R, M);
    return hipGetLastError();
}

}  // namespace cyfa
