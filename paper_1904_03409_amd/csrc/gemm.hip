// Tiled MFMA GEMM for the non-recurrent contractions of the StackLSTM step:
//   XW  = x Wp + b          (input projection for all T steps at once; paper, Algorithm 1's
//                            LSTM(x_t, .) has an x_t part independent of the recurrence)
//   dx  = dA Wp^T           (input gradient)
//   dW  = x^T dA            (weight gradients, split over K = T*B with fixed-order reduction)
//   dU  = Hprev^T dA        (Hprev rows gathered through the producer table)
// C[M][N] = sum_k A(m, k) B(k, n). 128x128 block tile, 32-deep K slices staged in LDS,
// four waves of 64x64, v_mfma_f32_16x16x4f32 (fp32) or v_mfma_f32_16x16x32_bf16.
#include "common.h"
#include "gemm.h"

namespace {

constexpr int BM = 128, BN = 128, BK = 32;

template <int PREC> struct Lds;
template <> struct Lds<0> { using T = float; static constexpr int PAD = 4; };
template <> struct Lds<1> { using T = bf16_t; static constexpr int PAD = 8; };

__device__ __forceinline__ float ld_any(const void* p, size_t i, int src_bf16) {
  return src_bf16 ? bf16_bits_to_f32(((const bf16_t*)p)[i]) : ((const float*)p)[i];
}

template <int PREC>
__device__ __forceinline__ void st_lds(typename Lds<PREC>::T* s, float v) {
  if constexpr (PREC == 0) *s = v; else *s = f32_to_bf16_bits(v);
}

// Loads 4 consecutive elements p[i..i+3] (bounded by lim) as floats.
__device__ __forceinline__ void ld4(const void* p, size_t i, size_t lim, int src_bf16, bool vec_ok, float v[4]) {
  if (vec_ok && i + 3 < lim) {
    if (src_bf16) {
      uint2 r = *(const uint2*)((const bf16_t*)p + i);
      v[0] = __uint_as_float(r.x << 16); v[1] = __uint_as_float(r.x & 0xffff0000u);
      v[2] = __uint_as_float(r.y << 16); v[3] = __uint_as_float(r.y & 0xffff0000u);
    } else {
      float4 r = *(const float4*)((const float*)p + i);
      v[0] = r.x; v[1] = r.y; v[2] = r.z; v[3] = r.w;
    }
  } else {
    for (int j = 0; j < 4; ++j) v[j] = (i + j < lim) ? ld_any(p, i + j, src_bf16) : 0.f;
  }
}

// Base of row tb of Hprev: the state read at step t = tb / B by element b = tb % B.
__device__ __forceinline__ const void* gather_row(const GemmArgs& g, int tb, int* is_bf16) {
  int t = tb / g.gB, b = tb - t * g.gB;
  int src = (t == 0) ? -1 : g.gtop[(size_t)(t - 1) * g.gB + b];
  if (src >= t) src = -1;                       // a producer precedes its reader; guard bad tables
  if (src < 0) { *is_bf16 = 0; return g.gh0 + (size_t)b * g.gH; }
  *is_bf16 = g.gcell_bf16;
  return g.gcell_bf16 ? (const void*)((const bf16_t*)g.gcell + ((size_t)src * g.gB + b) * g.gH)
                      : (const void*)((const float*)g.gcell + ((size_t)src * g.gB + b) * g.gH);
}

// Stage A(m0.., k0..) into As[m][k] and B(k0.., n0..) into Bs[n][k].
template <int PREC, int AL, int BL>
__device__ __forceinline__ void stage(const GemmArgs& g, int m0, int n0, int k0, int kend,
                                      typename Lds<PREC>::T* As, typename Lds<PREC>::T* Bs) {
  constexpr int LD = BK + Lds<PREC>::PAD;
  const int tid = threadIdx.x;
  // A
  for (int e = tid; e < BM * BK / 4; e += 256) {
    float v[4];
    if (AL == GEMM_MK) {
      int m = e / (BK / 4), k4 = (e % (BK / 4)) * 4;
      int gm = m0 + m, gk = k0 + k4;
      if (gm < g.M && gk < kend) {
        ld4(g.A, (size_t)gm * g.lda + gk, (size_t)gm * g.lda + kend, g.a_bf16, g.a_vec, v);
      } else { v[0] = v[1] = v[2] = v[3] = 0.f; }
      for (int j = 0; j < 4; ++j) st_lds<PREC>(&As[m * LD + k4 + j], v[j]);
    } else {
      int k = e / (BM / 4), m4 = (e % (BM / 4)) * 4;
      int gk = k0 + k, gm = m0 + m4;
      if (gk < kend && gm < g.M) {
        if (AL == GEMM_KM) {
          ld4(g.A, (size_t)gk * g.lda + gm, (size_t)gk * g.lda + g.M, g.a_bf16, g.a_vec, v);
        } else {
          int rb;
          const void* row = gather_row(g, gk, &rb);
          ld4(row, (size_t)gm, (size_t)g.M, rb, g.a_vec, v);
        }
      } else { v[0] = v[1] = v[2] = v[3] = 0.f; }
      for (int j = 0; j < 4; ++j) st_lds<PREC>(&As[(m4 + j) * LD + k], v[j]);
    }
  }
  // B
  for (int e = tid; e < BN * BK / 4; e += 256) {
    float v[4];
    if (BL == GEMM_NK) {
      int n = e / (BK / 4), k4 = (e % (BK / 4)) * 4;
      int gn = n0 + n, gk = k0 + k4;
      if (gn < g.N && gk < kend) {
        ld4(g.Bm, (size_t)gn * g.ldb + gk, (size_t)gn * g.ldb + kend, g.b_bf16, g.b_vec, v);
      } else { v[0] = v[1] = v[2] = v[3] = 0.f; }
      for (int j = 0; j < 4; ++j) st_lds<PREC>(&Bs[n * LD + k4 + j], v[j]);
    } else {
      int k = e / (BN / 4), n4 = (e % (BN / 4)) * 4;
      int gk = k0 + k, gn = n0 + n4;
      if (gk < kend && gn < g.N) {
        ld4(g.Bm, (size_t)gk * g.ldb + gn, (size_t)gk * g.ldb + g.N, g.b_bf16, g.b_vec, v);
      } else { v[0] = v[1] = v[2] = v[3] = 0.f; }
      for (int j = 0; j < 4; ++j) st_lds<PREC>(&Bs[(n4 + j) * LD + k], v[j]);
    }
  }
}

}  // namespace

template <int PREC, int AL, int BL>
__global__ void __launch_bounds__(256) k_gemm(GemmArgs g) {
  using T = typename Lds<PREC>::T;
  constexpr int LD = BK + Lds<PREC>::PAD;
  __shared__ __align__(16) T As[BM * LD];
  __shared__ __align__(16) T Bs[BN * LD];
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int kz = blockIdx.z;
  const int kbeg = kz * g.k_chunk;
  const int kend = min(g.K, kbeg + g.k_chunk);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l16 = lane & 15, lq = lane >> 4;
  f32x4 acc[4][4];
  for (int i = 0; i < 4; ++i)
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    __syncthreads();
    stage<PREC, AL, BL>(g, m0, n0, k0, kend, As, Bs);
    __syncthreads();
    if constexpr (PREC == 0) {
      for (int kc = 0; kc < BK / 16; ++kc) {
        float4 a4[4], b4[4];
        for (int i = 0; i < 4; ++i) a4[i] = *(const float4*)&As[(wm * 64 + i * 16 + l16) * LD + kc * 16 + 4 * lq];
        for (int j = 0; j < 4; ++j) b4[j] = *(const float4*)&Bs[(wn * 64 + j * 16 + l16) * LD + kc * 16 + 4 * lq];
        for (int i = 0; i < 4; ++i)
          for (int j = 0; j < 4; ++j) {
            acc[i][j] = mfma_f32_16x16x4(a4[i].x, b4[j].x, acc[i][j]);
            acc[i][j] = mfma_f32_16x16x4(a4[i].y, b4[j].y, acc[i][j]);
            acc[i][j] = mfma_f32_16x16x4(a4[i].z, b4[j].z, acc[i][j]);
            acc[i][j] = mfma_f32_16x16x4(a4[i].w, b4[j].w, acc[i][j]);
          }
      }
    } else {
      bf16x8 a8[4], b8[4];
      for (int i = 0; i < 4; ++i) a8[i] = *(const bf16x8*)&As[(wm * 64 + i * 16 + l16) * LD + 8 * lq];
      for (int j = 0; j < 4; ++j) b8[j] = *(const bf16x8*)&Bs[(wn * 64 + j * 16 + l16) * LD + 8 * lq];
      for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma_bf16_16x16x32(a8[i], b8[j], acc[i][j]);
    }
  }

  // epilogue: lane holds rows 4*lq + r, column l16 of each 16x16 tile
  float* C = g.C + (size_t)kz * g.split_stride;
  for (int i = 0; i < 4; ++i)
    for (int j = 0; j < 4; ++j) {
      int n = n0 + wn * 64 + j * 16 + l16;
      if (n >= g.N) continue;
      float bv = g.bias ? g.bias[perm_to_orig(n, g.bias_H)] : 0.f;
      for (int r = 0; r < 4; ++r) {
        int m = m0 + wm * 64 + i * 16 + 4 * lq + r;
        if (m < g.M) C[(size_t)m * g.ldc + n] = acc[i][j][r] + bv;
      }
    }
}

// out[m][col(n)] = sum_z P[z][m][n] in increasing z (deterministic), col = caller order.
__global__ void __launch_bounds__(256) k_reduce_splits(const float* __restrict__ P, int splits, size_t split_stride,
                                                       int M, int N, int unperm_H, float* __restrict__ out) {
  const size_t n_el = (size_t)M * N;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_el; i += (size_t)gridDim.x * blockDim.x) {
    float s = 0.f;
    for (int z = 0; z < splits; ++z) s += P[(size_t)z * split_stride + i];
    size_t m = i / N;
    int n = (int)(i - m * N);
    int col = unperm_H ? perm_to_orig(n, unperm_H) : n;
    out[m * N + col] = s;
  }
}

#define INST(P, A, B) template __global__ void k_gemm<P, A, B>(GemmArgs);
INST(0, GEMM_MK, GEMM_KN)
INST(0, GEMM_MK, GEMM_NK)
INST(0, GEMM_KM, GEMM_KN)
INST(0, GEMM_KM_GATHER, GEMM_KN)
INST(1, GEMM_MK, GEMM_KN)
INST(1, GEMM_MK, GEMM_NK)
INST(1, GEMM_KM, GEMM_KN)
INST(1, GEMM_KM_GATHER, GEMM_KN)
