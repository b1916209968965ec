// Shared pieces of the matrix-core (bf16 MFMA) forward kernels.
//
// Slot/basis index order used inside these kernels (the "internal" order):
// the 63 cosine/sine pairs of the real Fourier basis (App. A.1) come first,
// pair j = 1..63 at internal indices (2j-2, 2j-1) = (cos_j, sin_j); the DC
// component sits at internal index 126 and index 127 is the storage padding
// (App. A.7).  In paper order the same coordinates are 2j-1, 2j and 0.  With
// pairs on adjacent indices, a rotation U(tau) acts on neighbouring lanes of
// an MFMA accumulator.  For m < 127 the unused pairs are zero padding too.
//
// MFMA v_mfma_f32_32x32x16_bf16 lane layouts (l = lane, h = l / 32):
//   A (32 x 16): lane l holds A[l % 32][8h + p], p = 0..7
//   B (16 x 32): lane l holds B[8h + p][l % 32]
//   D (32 x 32): lane l, register v holds D[8(v/4) + 4h + v%4][l % 32]
// A state accumulator fed back as a B operand supplies, at k-step ks, the
// k indices 16ks + {4h..4h+3, 8+4h..8+4h+3}; the other operand is read in
// that same permuted order ("perm" reads below).
//
// Operands whose k index runs down the rows of a row-major LDS tile (the
// "transposed" operands K^T, V^T, A^T) are read with ds_read_b64_tr_b16: within
// each group of 16 lanes, output lane i, element j is element (i mod 4) of the
// 8 bytes addressed by lane 4j + i/4.  When lane s of the group addresses row
// r0 + s/4, columns c0 + 4 (s mod 4) .. +3, output lane i receives column c0 + i
// of rows r0 .. r0 + 3.
#pragma once

#include "cyfa_internal.h"

namespace cyfa {
namespace mfma {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int C = 64;             // chunk length
constexpr int D = 128;            // head dim
constexpr int NT = 256;           // threads per workgroup (4 waves)
constexpr int QS = 136;           // row stride (bf16) of [64][128] tiles
constexpr int TS = 72;            // row stride (bf16) of [128][64] tiles
constexpr int SS = 72;            // row stride (bf16) of the [64][64] score tile
constexpr int ZS = 132;           // row stride (float) of the [64][128] logit tile
constexpr int kDC = 126;          // internal index of the DC coordinate
constexpr int kStateFloats = 2 * 128 * 128;   // one (b, h) segment: K then V

__device__ __forceinline__ f32x16 mma(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// v_mfma_f32_16x16x32_bf16 (l = lane, g = l / 16):
//   A (16 x 32): lane l holds A[l % 16][8g + p];  B (32 x 16): B[8g + p][l % 16]
//   D (16 x 16): lane l, register r holds D[4g + r][l % 16]
__device__ __forceinline__ f32x4 mma16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Zero accumulators: the first product of each chain then takes the inline
// constant 0 as its accumulator input, so no zero registers are held.
__device__ __forceinline__ f32x16 zero_acc() { return f32x16{}; }
__device__ __forceinline__ f32x4 zero_acc4() { return f32x4{}; }

// A lane's LDS byte offset, opaque to the compiler: accesses written as
// smem + offset + constant then keep one base register per access pattern (the
// constant folds into the instruction's offset field) instead of one register
// per (tile, row) combination held across a loop.
__device__ __forceinline__ int opq(int x) {
    asm volatile("" : "+v"(x));
    return x;
}
template <typename T>
__device__ __forceinline__ T *lds_at(char *smem, int byte_off) {
    return reinterpret_cast<T *>(smem + byte_off);
}

__device__ __forceinline__ bf16x8 lds8(const __bf16 *p) {      // 16-byte LDS read
    return *reinterpret_cast<const bf16x8 *>(p);
}
__device__ __forceinline__ bf16x8 lds8_perm(const __bf16 *row, int k0, int h) {
    // k indices k0 + {4h..4h+3} and k0 + 8 + {4h..4h+3}
    const bf16x4 lo = *reinterpret_cast<const bf16x4 *>(row + k0 + 4 * h);
    const bf16x4 hi = *reinterpret_cast<const bf16x4 *>(row + k0 + 8 + 4 * h);
    bf16x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
}
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// Four rows of one column through the transpose read (see the layout note above).
__device__ __forceinline__ bf16x4 lds4_tr(const __bf16 *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(p));
}
// Lane's base address for a transposed operand from a row-major tile with row
// stride `stride`: the operand of column n = l % 32 and k = 8h + p is then
// lds8_tr(base + k0 * stride + n0) for a tile block starting at (k0, n0).
__device__ __forceinline__ int tr_off(int stride, int lane) {
    const int s = lane & 15, g = lane >> 4;
    return (8 * (g >> 1) + (s >> 2)) * stride + 16 * (g & 1) + 4 * (s & 3);
}
__device__ __forceinline__ bf16x8 lds8_tr(const __bf16 *p, int stride) {
    const bf16x4 lo = lds4_tr(p);
    const bf16x4 hi = lds4_tr(p + 4 * stride);
    bf16x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
}

// ---- swizzled tiles -----------------------------------------------------------
// Rows of 128 bf16 with no padding (256 bytes, one pass over the 64 banks); the
// 16-byte chunk c of row r is stored at chunk c ^ 4 (r mod 4).  A transpose read
// covers 4 consecutive rows x 32 columns per half-wave: the swizzle puts those
// four 64-byte pieces in the four different quarters of the bank window, where
// a padded row stride leaves them overlapping.  Row reads and stores in which
// each group of 16 lanes covers one whole row are unaffected.  Stores of partial
// rows into a swizzled tile are slow on this LDS and are not used.
constexpr int SWS = 128;
__host__ __device__ __forceinline__ constexpr int swz_elem(int r, int col) {
    return r * SWS + ((((col >> 3) ^ ((r & 3) << 2))) << 3) + (col & 7);
}
// Byte offset, in a swizzled tile, of a lane's transposed-operand block at rows
// 0.., column block 0 (row 8 (g/2) + s/4, column 16 (g mod 2) + 4 (s mod 4), as
// tr_off).  Column block y (32 columns) is this offset ^ 64 y; the upper four
// rows of lds8_tr are 4 rows (1 KiB) further, and each 16 rows 4 KiB further.
__device__ __forceinline__ int tr_off_swz(int lane) {
    const int s = lane & 15, g = lane >> 4;
    return 2 * swz_elem(8 * (g >> 1) + (s >> 2), 16 * (g & 1) + 4 * (s & 3));
}

// registers 8*half .. 8*half+7 of an accumulator as a bf16 B operand
__device__ __forceinline__ bf16x8 acc_to_operand(const f32x16 &acc, int half) {
    bf16x8 r;
#pragma unroll
    for (int p = 0; p < 8; ++p) r[p] = (__bf16)acc[8 * half + p];
    return r;
}

// internal index -> paper-order basis index (or -1 for padding)
__host__ __device__ __forceinline__ int internal_to_paper(int i, int m) {
    if (i == kDC) return 0;
    if (i < m - 1) return i + 1;
    return -1;
}

// Segment states are stored in the "dump" layout of the fused kernel's
// accumulators, lane-major: block (w, x) of a state (wave w's accumulator x) holds
// 64 lanes x 16 registers, each lane's 16 registers consecutive, so that a lane
// moves its part of a block with two 16-byte (bf16) or four (fp32) accesses.
__host__ __device__ __forceinline__ constexpr int dump_off(int w, int x, int lane, int v) {
    return ((w * 4 + x) * 64 + lane) * 16 + v;
}
// Offsets of element (i, c) of a segment state in that layout.
// Key state: wave w = i / 32 owns columns i of Kbar^T (rows d = c), blocks db = c / 32.
__host__ __device__ __forceinline__ int dump_index_K(int i, int c) {
    const int w = i >> 5, lane_lo = i & 31;
    const int db = c >> 5, cr = c & 31;
    const int h = (cr >> 2) & 1;
    const int v = ((cr >> 3) << 2) | (cr & 3);
    return dump_off(w, db, lane_lo + 32 * h, v);
}
// Value state: wave w = c / 32 owns columns c of Vbar (rows i), blocks ib = i / 32.
__host__ __device__ __forceinline__ int dump_index_V(int i, int c) {
    const int w = c >> 5, lane_lo = c & 31;
    const int ib = i >> 5, ir = i & 31;
    const int h = (ir >> 2) & 1;
    const int v = ((ir >> 3) << 2) | (ir & 3);
    return 128 * 128 + dump_off(w, ib, lane_lo + 32 * h, v);
}

// Workgroup barrier that orders LDS accesses only.  __syncthreads() is a full
// workgroup fence: every wave first waits for all of its outstanding global loads,
// so a chunk prefetch issued just before a barrier would expose the whole memory
// latency there.  Here only the LDS operations are waited for; a prefetch stays in
// flight across the barrier and is waited for where its registers are used.  No
// wave reads another wave's global-memory results inside these kernels.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Value of lane l ^ 1 (DPP quad permutation [1,0,3,2]).
__device__ __forceinline__ float swap_pair(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), 0xB1, 0xF, 0xF, false));
}
// ---- chunk-local prefix sums on one wave (lane = token row) --------------
// DPP lane moves (no lane-address registers): row_shr:n within rows of 16 lanes
// (sources outside the row read 0), then row_bcast:15 / row_bcast:31 carry the
// row totals into the following rows.
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ int dpp0(int x) {
    return __builtin_amdgcn_update_dpp(0, x, CTRL, ROWS, 0xF, true);
}
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ float dppf(float x) {
    return __int_as_float(dpp0<CTRL, ROWS>(__float_as_int(x)));
}
template <int CTRL, int ROWS = 0xF>
__device__ __forceinline__ double dppd(double x) {
    const unsigned long long v = (unsigned long long)__double_as_longlong(x);
    const unsigned lo = (unsigned)dpp0<CTRL, ROWS>((int)(unsigned)v);
    const unsigned hi = (unsigned)dpp0<CTRL, ROWS>((int)(unsigned)(v >> 32));
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}
__device__ __forceinline__ float wave_incl_scan(float x) {
    x += dppf<0x111>(x);
    x += dppf<0x112>(x);
    x += dppf<0x114>(x);
    x += dppf<0x118>(x);
    x += dppf<0x142, 0xA>(x);
    x += dppf<0x143, 0xC>(x);
    return x;
}
__device__ __forceinline__ double wave_incl_scan(double x) {
    x += dppd<0x111>(x);
    x += dppd<0x112>(x);
    x += dppd<0x114>(x);
    x += dppd<0x118>(x);
    x += dppd<0x142, 0xA>(x);
    x += dppd<0x143, 0xC>(x);
    return x;
}
// maximum over the wave of values >= 0 (0 is the identity of the moves above)
__device__ __forceinline__ float wave_max_nonneg(float x) {
    x = fmaxf(x, dppf<0x111>(x));
    x = fmaxf(x, dppf<0x112>(x));
    x = fmaxf(x, dppf<0x114>(x));
    x = fmaxf(x, dppf<0x118>(x));
    x = fmaxf(x, dppf<0x142, 0xA>(x));
    x = fmaxf(x, dppf<0x143, 0xC>(x));
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}
__device__ __forceinline__ float lane63(float x) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 63));
}
__device__ __forceinline__ double lane63(double x) {
    const unsigned long long v = (unsigned long long)__double_as_longlong(x);
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)v, 63);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(v >> 32), 63);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}
// value of lane l ^ 16 (ds_swizzle, bitmask mode: and 0x1F, xor 0x10, within 32 lanes)
__device__ __forceinline__ float swap16(float x) {
    return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(x), 0x401F));
}

// cos / sin of 2 pi * rev (rev in revolutions, |rev| < 256) on the hardware units
__device__ __forceinline__ void sincos_rev(float rev, float *s, float *c) {
    *s = __builtin_amdgcn_sinf(rev);
    *c = __builtin_amdgcn_cosf(rev);
}

}  // namespace mfma
}  // namespace cyfa
