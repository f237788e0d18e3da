// Persistent forward kernel of the parallelised StackLSTM (paper, Algorithm 1):
// for every step t and every batch element, read the state at the stack pointer,
// run one LSTM cell, write its result as the state of step t (slot p+1), move the
// pointer by op and return the state at the new pointer. No branch depends on op.
//
// Work split: the batch is cut into G groups of 16*NT rows. A group runs on the NW
// workgroups of one XCC (one shared L2); workgroup w of the group owns hidden units
// [16w, 16w+16), i.e. 64 gate-interleaved columns of U, which sit in VGPRs for the
// whole kernel (one 16-column MFMA tile per wave). Per step each workgroup gathers
// the group's h_prev rows into LDS, runs h_prev U on MFMA (gates^T = U^T h_prev^T so
// one lane holds the four gates of one (unit, row) pair), applies the gate
// nonlinearities and the cell update in registers, writes h, c, the bf16 copy of h
// and the gate activations, and meets the group at a barrier. Workgroup 0 of the
// group also keeps the integer stack: stack[b][p+1] <- t, p <- p + op, top <- stack[b][p].
#include "common.h"
#include "recurrent.h"
#include "rec_config.h"

template <int PREC, int NT, int NTB, int KS, int OCC>
__global__ void __launch_bounds__(256, OCC) k_fwd(RecArgs a) {
  constexpr int KC = PREC ? 32 : 16;               // K per chunk
  constexpr int KP = KS * KC;                      // K capacity of the U registers
  constexpr int LDS_LD = KP + (PREC ? 8 : 4);      // LDS row stride (elements)
  constexpr int ROWS_B = NTB * 16;                 // rows staged per pass
  constexpr int BG = NT * 16;                      // rows per group
  using elem_t = typename std::conditional<PREC == 1, bf16_t, float>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  elem_t* hs = reinterpret_cast<elem_t*>(smem);
  __shared__ int s_src[BG];
  __shared__ int s_g, s_w, s_flag;

  claim_group_slot(a.ctl + CTL_XCC_SLOT, a.G, a.NW, &s_g, &s_w);
  const int g = s_g, w = s_w;
  if (g < 0) return;

  const int T = a.T, B = a.B, H = a.H, H4 = 4 * H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, lq = lane >> 4;
  const int row0 = g * BG;
  const int unit_base = w * 16 + wave * 4;
  const int ks_eff = a.ks_eff;
  const size_t TBH = (size_t)T * B * H;
  const rsrc_t r_top = make_rsrc(a.top, (size_t)T * B * 4);
  const rsrc_t r_h = PREC ? make_rsrc(a.hx, TBH * 2) : make_rsrc(a.hcell, TBH * 4);

  // ---- U slice into registers: A operand, row m = l16 -> (unit_base + m/4, gate m%4), K permuted per chunk
  const int a_unit = unit_base + (l16 >> 2), a_gate = l16 & 3;
  const bool a_ok = a_unit < H;
  const float* Ucol = a.U + (size_t)a_gate * H + a_unit;
  float ureg32[PREC ? 1 : KS][4];
  bf16x8 ureg16[PREC ? KS : 1];
#pragma unroll
  for (int c = 0; c < KS; ++c) {
    if constexpr (PREC == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int k = c * 16 + 4 * lq + j;
        ureg32[c][j] = (a_ok && k < H) ? Ucol[(size_t)k * H4] : 0.f;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        int k = c * 32 + 8 * lq + j;
        ureg16[c][j] = f32_to_bf16((a_ok && k < H) ? Ucol[(size_t)k * H4] : 0.f);
      }
    }
  }

  const bool tracer = (w == 0) && ((int)threadIdx.x < BG) && (row0 + (int)threadIdx.x < B);
  const int my_row = row0 + (int)threadIdx.x;
  const bool row_thread = ((int)threadIdx.x < BG) && (my_row < B);
  const size_t stk_base = (size_t)my_row * (T + 1);
  const int kmax = ks_eff * KC;                    // staged K (>= H, zero beyond H)
  const bool vec_ok = PREC ? (H % 8 == 0) : (H % 4 == 0);

  // Integer stack of the group's rows, kept by workgroup 0 one step ahead of the floats:
  // step t's trace is written during step t-1, so every workgroup can fetch the producer
  // it reads at step t+1 while step t is still running.
  int my_p = 0, my_top = -1, op_next = 0;
  if (tracer) {
    int op0 = a.ops[my_row];
    op_next = (T > 1) ? a.ops[(size_t)B + my_row] : 0;
    a.stack[stk_base] = -1;                       // slot 0: the initial state
    a.stack[stk_base + 1] = 0;
    my_p = max(0, op0);
    my_top = (op0 == 1) ? 0 : -1;                 // a pop at step 0 is rejected by the scan
    a.top[my_row] = my_top;
  }
  if ((int)threadIdx.x < BG) s_src[threadIdx.x] = -1;
  if (group_barrier(&a.ctl[CTL_BAR_F + g * 16], (uint32_t)a.NW, a.ctl, a.spin_limit, &s_flag)) return;

  long long* clk = a.clk ? a.clk + (size_t)blockIdx.x * T * 4 : nullptr;
  for (int t = 0; t < T; ++t) {
    if (clk && threadIdx.x == 0) clk[t * 4 + 0] = wall_clock64();
    // producer of the state each row reads at step t+1 (= top[t], written one step ago)

    int src_next = -1, tp_next = 0;

    for (int nb = 0; nb < NT / NTB; ++nb) {
      // ---- gather h_prev rows of this pass into LDS (zero beyond H and for rows past B)
      if (vec_ok) {
        // every thread issues all of its loads before the first LDS write, so the
        // latency of the L2 round trip is paid once per step, not once per vector
        constexpr int VW = PREC ? 8 : 4;
        constexpr int NLD = (ROWS_B * (KP / VW) + 255) / 256;
        const int per_row = kmax / VW;
        const int n_el = ROWS_B * per_row;
        uint4 buf[NLD];
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
          const int e = threadIdx.x + 256 * i;
          buf[i] = uint4{0u, 0u, 0u, 0u};
          if (e >= n_el) continue;
          const int r = e / per_row, k = (e - r * per_row) * VW;
          const int rr = nb * ROWS_B + r, b = row0 + rr;
          if (b >= B || k >= H) continue;
          const int src = s_src[rr];
          const size_t e2 = ((size_t)src * B + b) * H + k;
          if constexpr (PREC == 0) {
            if (src < 0) buf[i] = *(const uint4*)(a.h0 + (size_t)b * H + k);
            else if (a.coh_rows) buf[i] = ld_coh_b128(r_h, (uint32_t)(e2 * 4));
            else buf[i] = *(const uint4*)(a.hcell + e2);
          } else {
            if (src < 0) {
              const float* p = a.h0 + (size_t)b * H + k;
              float4 v0 = *(const float4*)p, v1 = *(const float4*)(p + 4);
              bf16_t o[8] = {f32_to_bf16_bits(v0.x), f32_to_bf16_bits(v0.y), f32_to_bf16_bits(v0.z),
                             f32_to_bf16_bits(v0.w), f32_to_bf16_bits(v1.x), f32_to_bf16_bits(v1.y),
                             f32_to_bf16_bits(v1.z), f32_to_bf16_bits(v1.w)};
              buf[i] = *(const uint4*)o;
            } else if (a.coh_rows) {
              buf[i] = ld_coh_b128(r_h, (uint32_t)(e2 * 2));
            } else {
              buf[i] = *(const uint4*)(a.hx + e2);
            }
          }
        }
#pragma unroll
        for (int i = 0; i < NLD; ++i) {
          const int e = threadIdx.x + 256 * i;
          if (e >= n_el) continue;
          const int r = e / per_row, k = (e - r * per_row) * VW;
          *(uint4*)(hs + r * LDS_LD + k) = buf[i];
        }
      } else {
        for (int e = threadIdx.x; e < ROWS_B * kmax; e += 256) {
          int r = e / kmax, k = e - r * kmax;
          int rr = nb * ROWS_B + r, b = row0 + rr;
          float v = 0.f;
          if (b < B && k < H) {
            int src = s_src[rr];
            size_t e2 = ((size_t)src * B + b) * H + k;
            if (src < 0) v = a.h0[(size_t)b * H + k];
            else if constexpr (PREC == 0) v = __uint_as_float(ld_coh_b32(r_h, (uint32_t)(e2 * 4)));
            else v = bf16_bits_to_f32(ld_coh_b16(r_h, (uint32_t)(e2 * 2)));
          }
          if constexpr (PREC == 0) hs[r * LDS_LD + k] = v;
          else hs[r * LDS_LD + k] = f32_to_bf16_bits(v);
        }
      }
      __syncthreads();
      if (clk && threadIdx.x == 0 && nb == 0) clk[t * 4 + 1] = wall_clock64();
      if (nb == 0 && row_thread && t + 1 < T) {
        const size_t o = (size_t)t * B + my_row;
        src_next = a.coh_top ? (int)ld_coh_b32(r_top, (uint32_t)(o * 4)) : a.top[o];
      }
      // trace for step t+1: stack[p+1] <- t+1, p <- p + op, top <- stack[p]; issued after the
      // h_prev loads so that their wait does not include it, consumed before the barrier
      if (nb == 0 && tracer && t + 1 < T) {
        int op = op_next;
        op_next = (t + 2 < T) ? a.ops[(size_t)(t + 2) * B + my_row] : 0;
        a.stack[stk_base + my_p + 1] = t + 1;
        my_p = max(0, my_p + op);
        tp_next = (op == 1) ? t + 1 : (op == 0 ? my_top : a.stack[stk_base + my_p]);
      }

      // ---- epilogue operands, fetched before the MFMA loop so their latency overlaps it
      const int u = unit_base + lq;
      float4 xw4[NTB];
      float cprev[NTB];
#pragma unroll
      for (int nt = 0; nt < NTB; ++nt) {
        int rr = nb * ROWS_B + nt * 16 + l16, b = row0 + rr;
        xw4[nt] = float4{0.f, 0.f, 0.f, 0.f};
        cprev[nt] = 0.f;
        if (b < B && u < H) {
          xw4[nt] = *(const float4*)(a.xw + ((size_t)t * B + b) * H4 + 4 * u);
          int src = s_src[rr];
          cprev[nt] = (src < 0) ? a.c0[(size_t)b * H + u] : a.ccell[((size_t)src * B + b) * H + u];
        }
      }

      // ---- gates^T (16 cols x 16 rows per tile) = U^T h_prev^T
      f32x4 acc[NTB];
#pragma unroll
      for (int nt = 0; nt < NTB; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < KS; ++c) {
        if (c < ks_eff) {
#pragma unroll
          for (int nt = 0; nt < NTB; ++nt) {
            if constexpr (PREC == 0) {
              float4 bv = *(const float4*)&hs[(nt * 16 + l16) * LDS_LD + c * 16 + 4 * lq];
              acc[nt] = mfma_f32_16x16x4(ureg32[c][0], bv.x, acc[nt]);
              acc[nt] = mfma_f32_16x16x4(ureg32[c][1], bv.y, acc[nt]);
              acc[nt] = mfma_f32_16x16x4(ureg32[c][2], bv.z, acc[nt]);
              acc[nt] = mfma_f32_16x16x4(ureg32[c][3], bv.w, acc[nt]);
            } else {
              bf16x8 bv = *(const bf16x8*)&hs[(nt * 16 + l16) * LDS_LD + c * 32 + 8 * lq];
              acc[nt] = mfma_bf16_16x16x32(ureg16[c], bv, acc[nt]);
            }
          }
        }
      }

      if (clk && threadIdx.x == 0 && nb == 0) clk[t * 4 + 2] = wall_clock64();
      // ---- fused LSTM cell: lane holds gates i, f, g, o of unit u for row l16 of each tile
#pragma unroll
      for (int nt = 0; nt < NTB; ++nt) {
        int rr = nb * ROWS_B + nt * 16 + l16, b = row0 + rr;
        if (b >= B || u >= H) continue;
        float gi = sigmoidf_(acc[nt][0] + xw4[nt].x);
        float gf = sigmoidf_(acc[nt][1] + xw4[nt].y);
        float gg = tanhf(acc[nt][2] + xw4[nt].z);
        float go = sigmoidf_(acc[nt][3] + xw4[nt].w);
        float c = gf * cprev[nt] + gi * gg;
        float h = go * tanhf(c);
        size_t o = ((size_t)t * B + b) * H + u;
        a.hcell[o] = h;
        a.ccell[o] = c;
        if constexpr (PREC == 1) a.hx[o] = f32_to_bf16_bits(h);
        *(float4*)(a.stash + ((size_t)t * B + b) * H4 + 4 * u) = float4{gi, gf, gg, go};
      }
      if (NT / NTB > 1) __syncthreads();
    }

    if (clk && threadIdx.x == 0) clk[t * 4 + 3] = wall_clock64();
    if (tracer && t + 1 < T) {
      a.top[(size_t)(t + 1) * B + my_row] = tp_next;
      my_top = tp_next;
    }
    if (group_barrier(&a.ctl[CTL_BAR_F + g * 16], (uint32_t)(a.NW * (t + 2)), a.ctl, a.spin_limit, &s_flag)) break;
    if (src_next < -1 || src_next > t) src_next = -1;   // only a valid producer is ever indexed
    if ((int)threadIdx.x < BG) s_src[threadIdx.x] = src_next;
    __syncthreads();
  }
}

// ---- instantiations and launcher: one kernel per (precision, row tiles per group, K chunks)
template <int P, int NT, int KS>
static hipError_t launch_fwd_t(const RecArgs& a, dim3 grid, hipStream_t st, int* occ_out) {
  constexpr int NTB = rec_ntb(P, NT, KS);
  constexpr int OCC = rec_occ(P, KS);
  auto kern = k_fwd<P, NT, NTB, KS, OCC>;
  size_t shm = rec_lds_bytes(P, NTB, KS);
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
  if (e != hipSuccess) return e;
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 256, shm);
  if (e != hipSuccess) return e;
  if (occ_out) *occ_out = occ;
  if (!grid.x) return hipSuccess;  // occupancy query only
  RecArgs args = a;
  void* kargs[] = {&args};
  return hipLaunchCooperativeKernel((const void*)kern, grid, dim3(256), kargs, (unsigned)shm, st);
}

hipError_t launch_fwd(const RecArgs& a, int prec, int NT, int KS, dim3 grid, hipStream_t st, int* occ_out) {
#define CASE(P, NT_, KS_) if (prec == P && NT == NT_ && KS == KS_) return launch_fwd_t<P, NT_, KS_>(a, grid, st, occ_out);
  REC_CASES(CASE)
#undef CASE
  return hipErrorInvalidValue;
}
