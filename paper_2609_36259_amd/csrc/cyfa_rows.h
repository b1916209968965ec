// Storage rows of the states for larger slot counts (not part of the public ABI).
//
// m <= 127 active slots keep the m* = 128 storage rows of App. A.7; m up to 255
// (the largest slot count of the paper's ablation) uses m* = 256 rows, with the
// same basis order (0 = DC, 2j-1 = cos_j, 2j = sin_j) and zero padding.
#pragma once

#include "cyfa_internal.h"

namespace cyfa {

constexpr int kWideRows = 256;
constexpr int kMaxActiveWide = 255;
constexpr int kNarrowRows = 64;     // m* = 64 storage rows of the matrix-core forward for m <= 63
constexpr int kMaxActiveNarrow = 63;

__host__ __device__ inline int store_rows(int m) { return m > kMaxActive ? kWideRows : kStoreRows; }
inline size_t readout_bytes(int H, int m) {
    const size_t r = (size_t)store_rows(m);
    return (size_t)H * r * r * 4;
}

// M_h = R_h Phi as float [H][256][256] for 127 < m <= 255 (slot row, basis
// column in the order of App. A.1, zero outside the active m x m block).
hipError_t launch_readout_prep_wide(int H, int m, const float *R, float *M, hipStream_t s);
// The same matrix for the matrix-core kernel: bf16 Mz = zs M in its internal basis
// order (DC at 254, padding 255, kMaskLogit in the padding column of inactive slots)
// and its transpose MzT, [H][256][256] each.
hipError_t launch_readout_prep_wide_bf16(int H, int m, const float *R, __bf16 *Mz, __bf16 *MzT, float zs,
                                         hipStream_t s);

// Matrix-core forward for 127 < m <= 255 (bf16, d_k = d_v = 128, chunk 32 or 64 run
// as 32-token chunks, one workgroup per chunk group of a sequence).  ws
// (mfma_wide_workspace_bytes) receives the bf16 readout matrix and its transpose,
// formed from p.R, and with groups > 1 the groups' contributions; the events, when
// given, bracket the fused kernel.
bool mfma_wide_supported(const FwdParams &p);
int mfma_wide_auto_groups(const FwdParams &p);
size_t mfma_wide_workspace_bytes(const FwdParams &p, int groups);
hipError_t launch_fwd_mfma_wide(const FwdParams &p, int groups, void *ws, hipStream_t st, hipEvent_t ev_start,
                                hipEvent_t ev_stop);

// Matrix-core forward for m <= 63 on m* = 64 storage rows (bf16, d_k = d_v = 128, chunk
// 32 or 64 run as 32-token chunks, one workgroup per chunk group of a sequence, two per
// compute unit).  The state arrays keep the [B][H][128][d] layout of m <= 127; the kernel
// reads their rows 0 .. 63 and writes rows 64 .. 127 of the final states as zeros.  ws
// (mfma_narrow_workspace_bytes) receives the bf16 64 x 64 readout matrix, formed from
// p.R, and with groups > 1 the groups' contributions; the events, when given, bracket
// the fused kernel.
bool mfma_narrow_supported(const FwdParams &p);
int mfma_narrow_auto_groups(const FwdParams &p);
size_t mfma_narrow_workspace_bytes(const FwdParams &p, int groups);
hipError_t launch_fwd_mfma_narrow(const FwdParams &p, int groups, void *ws, hipStream_t st, hipEvent_t ev_start,
                                  hipEvent_t ev_stop);

// Vector-ALU forward over chunk groups (d_k, d_v <= 128 and m <= 127; other
// shapes run one group per sequence): groups > 1 forms the state entering each
// group in ws (valu_group_workspace_bytes) before the chunk kernel.
bool valu_groups_supported(const FwdParams &p);
int valu_auto_groups(const FwdParams &p);
size_t valu_group_workspace_bytes(const FwdParams &p, int groups);
hipError_t launch_fwd_valu(const FwdParams &p, const float *M, int groups, void *ws, hipStream_t s);

}  // namespace cyfa
