// GEMM launch description shared by gemm.hip and the host library.
#pragma once
#include <stddef.h>
#include <stdint.h>

enum { GEMM_MK = 0, GEMM_KM = 1, GEMM_KM_GATHER = 2 };  // A layouts
enum { GEMM_KN = 0, GEMM_NK = 1 };                       // B layouts

struct GemmArgs {
  int M, N, K;
  const void* A; int lda; int a_bf16; int a_vec;   // A(m,k): MK -> A[m*lda+k]; KM -> A[k*lda+m]
  const void* Bm; int ldb; int b_bf16; int b_vec;  // B(k,n): KN -> B[k*ldb+n]; NK -> B[n*ldb+k]
  float* C; int ldc;                               // C[m*ldc+n] (+ split index * split_stride)
  const float* bias; int bias_H;                   // + bias[caller column of n] when non-null
  int k_chunk; size_t split_stride;
  // KM_GATHER: row k = t*B + b of A is the state read at step t by element b
  const int32_t* gtop; const float* gh0; const void* gcell; int gcell_bf16; int gB; int gH;
};
