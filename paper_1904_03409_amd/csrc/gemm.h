// GEMM launch description shared by gemm.hip and the host library.
#pragma once
#include <stddef.h>
#include <stdint.h>

// A layouts: A(m,k) = A[m*lda+k] (MK) or A[k*lda+m] (KM); MK_F32: MK with fp32 elements,
// rounded to bf16 on load (bf16 kernels)
enum { GEMM_MK = 0, GEMM_KM = 1, GEMM_MK_F32 = 2 };
enum { GEMM_KN = 0, GEMM_NK = 1 };   // B layouts: B(k,n) = B[k*ldb+n] or B[n*ldb+k]

struct GemmArgs {
  int M, N, K;
  const void* A; int lda; int a_vec;   // a_vec: rows are 16-byte aligned vectors (ld % 4 (fp32) / % 8 (bf16) == 0)
  const void* Bm; int ldb; int b_vec;
  float* C; int ldc;                   // C[m*ldc+n] (+ split index * split_stride)
  const float* bias; int bias_H;       // + bias[caller column of n] when non-null
  int k_chunk; size_t split_stride;
  // Row gathers (null = identity). A stored row j of A (MK: j = m, KM: j = k) is row
  // a_rows[j] of the array; likewise b_rows for B (KN: j = k, NK: j = n); C row m is
  // written to row c_rows[m]. Indices must lie within the array's static extent.
  const int32_t* a_rows;
  const int32_t* b_rows;
  const int32_t* c_rows;
  // Device-side extent (null = none): M (dyn_axis 0) or K (dyn_axis 1) becomes
  // min(static extent, *dyn rounded up to a multiple of dyn_round). With a device K the
  // K range is cut into gridDim.z slices at run time (k_chunk is then ignored).
  const uint32_t* dyn; int dyn_axis; int dyn_round;
  // With a device-side M: 1 = when the tiles in use are fewer than the grid's blocks, cut each
  // tile's K range into gemm_dyn_splits() slices, written to C + z * M * ldc (the M rows in
  // use packed, c_rows must be null); k_scatter_splits then adds them into the gathered rows.
  int dyn_split;
};
// Block tile of the wide bf16 GEMM (k_gemm_wide) and its dynamic LDS (two buffers of A and B
// slices, 64 k + 8 padding per row)
constexpr int kGemmWideBM = 256, kGemmWideBN = 256;
constexpr size_t kGemmWideLds = (size_t)2 * (kGemmWideBM + kGemmWideBN) * (64 + 8) * 2;
// K slices per tile for a device-M GEMM over `active` tiles on a grid of `blocks` blocks.
__host__ __device__ inline int gemm_dyn_splits(int blocks, int active) {
  if (active <= 0) return 1;
  const int s = blocks / active;
  return s < 1 ? 1 : (s > 4 ? 4 : s);
}
