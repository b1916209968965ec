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
typedef __bf16 bf16v8 __attribute__((ext_vector_type(8)));

// Block (h, rb): rows 8 rb .. 8 rb + 7 of M_h; thread j computes column j of
// those rows, M[i][j] = sum_s R[i][s] Phi[s][j], with Phi[s][j] from a table of
// the m angles 2 pi n / m (index l s mod m for frequency l = (j + 1) / 2), four
// terms per step from 16-byte reads of R's staged rows.  Writes the fp32 M (paper
// basis order) and/or, for the matrix-core kernel, Mz = zs M in its internal basis
// order (pair j at 2j-2, 2j-1, DC at 254, padding 255; kMaskLogit in the padding
// column of inactive slots) and its transpose MzT, each when non-null.
__global__ __launch_bounds__(256) void readout_prep_wide_kernel(int m, const float *__restrict__ R,
                                                                float *__restrict__ M, __bf16 *__restrict__ Mz,
                                                                __bf16 *__restrict__ MzT, float zs) {
    __shared__ float tab[2][kWideRows];
    __shared__ __attribute__((aligned(16))) float Rr[kWideRowsPerBlock][kWideRows];
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
        // R's staged rows are zero past column m, so the steps may run to a multiple of 4
        for (int s0 = 0; s0 < m; s0 += 4) {
            float ph[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                ph[q] = t[idx];
                idx += l;
                if (idx >= m) idx -= m;
            }
#pragma unroll
            for (int r = 0; r < kWideRowsPerBlock; ++r) {
                const float4 rv = *reinterpret_cast<const float4 *>(&Rr[r][s0]);
                acc[r] = fmaf(rv.x, ph[0], fmaf(rv.y, ph[1], fmaf(rv.z, ph[2], fmaf(rv.w, ph[3], acc[r]))));
            }
        }
    }
    const float cscale = j == 0 ? (float)(1.0 / sqrt((double)m)) : (float)sqrt(2.0 / (double)m);
    const int jint = j == 0 ? kWideRows - 2 : (j == kWideRows - 1 ? kWideRows - 1 : j - 1);
    bf16v8 col;
#pragma unroll
    for (int r = 0; r < kWideRowsPerBlock; ++r) {
        const int i = i0 + r;
        const float val = (j < m && i < m) ? acc[r] * cscale : 0.f;
        if (M) M[((size_t)h * kWideRows + i) * kWideRows + j] = val;
        const float zv = (j == kWideRows - 1 && i >= m) ? kMaskLogit : zs * val;
        col[r] = (__bf16)zv;
        if (Mz) Mz[((size_t)h * kWideRows + i) * kWideRows + jint] = col[r];
    }
    if (MzT) *reinterpret_cast<bf16v8 *>(MzT + ((size_t)h * kWideRows + jint) * kWideRows + i0) = col;
}

hipError_t launch_readout_prep_wide(int H, int m, const float *R, float *M, hipStream_t s) {
    hipLaunchKernelGGL(readout_prep_wide_kernel, dim3(H, kWideRows / kWideRowsPerBlock), dim3(kWideRows), 0,
                       s, m, R, M, nullptr, nullptr, 1.f);
    return hipGetLastError();
}

hipError_t launch_readout_prep_wide_bf16(int H, int m, const float *R, __bf16 *Mz, __bf16 *MzT, float zs,
                                         hipStream_t s) {
    hipLaunchKernelGGL(readout_prep_wide_kernel, dim3(H, kWideRows / kWideRowsPerBlock), dim3(kWideRows), 0,
                       s, m, R, nullptr, Mz, MzT, zs);
    return hipGetLastError();
}

}  // namespace cyfa
