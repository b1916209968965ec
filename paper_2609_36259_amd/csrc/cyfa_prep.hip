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
