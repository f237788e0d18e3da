// Device pieces shared by the forward recurrent kernels (plain and pipelined).
#pragma once
#include "common.h"
#include "recurrent.h"

// Source of one staged h_prev granule: the state produced at step src (h0 for src = -1) of
// batch row b, columns from k. fp32 mode reads h_cell or h0; bf16 mode reads the bf16 state
// copy, whose slot 0 holds h0 and slot s+1 the state of step s.
template <int PREC>
__device__ __forceinline__ const void* staged_src(const RecArgs& a, int src, int b, int k) {
  if constexpr (PREC == 0)
    return (src < 0) ? (const void*)(a.h0 + (size_t)b * a.H + k)
                     : (const void*)(a.hcell + ((size_t)src * a.B + b) * a.H + k);
  else return (const void*)(a.hx + ((size_t)(src + 1) * a.B + b) * a.H + k);
}

// U slice of a forward workgroup in registers, the MFMA A operand: row m = l16 of the
// wave's tile is (unit unit_base + m/4, gate m%4); chunk c holds K rows c*16 + 4lq .. +3
// (fp32) or c*32 + 8lq .. +7 (bf16). Zero past H, so every chunk can always run.
template <int PREC, int KS>
__device__ __forceinline__ void fwd_load_u(const RecArgs& a, int unit_base, int l16, int lq,
                                           float (&u32)[PREC ? 1 : KS][4], bf16x8 (&u16)[PREC ? KS : 1]) {
  const int H = a.H, H4 = 4 * H;
  const int a_unit = unit_base + (l16 >> 2), a_gate = l16 & 3;
  const bool a_ok = a_unit < H;
  const float* Ucol = a.U + (size_t)a_gate * H + a_unit;
#pragma unroll
  for (int c = 0; c < KS; ++c) {
    if constexpr (PREC == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int k = c * 16 + 4 * lq + j;
        u32[c][j] = (a_ok && k < H) ? Ucol[(size_t)k * H4] : 0.f;
      }
    } else {
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = c * 32 + 8 * lq + j;
        v[j] = (a_ok && k < H) ? Ucol[(size_t)k * H4] : 0.f;
      }
      u16[c] = pack_bf16x8(v);
    }
  }
}

// Fused LSTM cell of one (step t, row b, unit u) pair from the MFMA output (gates i, f, g,
// o of the pair in acc) and the input projection: writes h, c, the bf16 copy of h and, when
// `keep` (a push step: the backward reads the gate activations of push steps only), the
// gate activations; returns c. h is never stored as the all-ones fill pattern.
template <int PREC>
__device__ __forceinline__ float fwd_cell(const RecArgs& a, const f32x4& acc, const float4& xw, float cp, int t,
                                          int b, int u, bool keep) {
  const float gi = sigmoidf_(acc[0] + xw.x);
  const float gf = sigmoidf_(acc[1] + xw.y);
  const float gg = tanhf_(acc[2] + xw.z);
  const float go = sigmoidf_(acc[3] + xw.w);
  const float c = gf * cp + gi * gg;
  const float h = canon_nan(go * tanhf_(c));
  const size_t o = ((size_t)t * a.B + b) * a.H + u;
  a.hcell[o] = h;
  a.ccell[o] = c;
  if constexpr (PREC == 1) a.hx[o + (size_t)a.B * a.H] = f32_to_bf16_bits(h);
  // (the gate stash is read only by the backward: a non-temporal store)
  if (keep) __builtin_nontemporal_store(f32x4{gi, gf, gg, go}, (f32x4*)(a.stash + ((size_t)t * a.B + b) * (4 * a.H) + 4 * u));
  return c;
}
