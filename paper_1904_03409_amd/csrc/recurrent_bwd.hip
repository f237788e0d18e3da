// Persistent backward kernel of the parallelised StackLSTM: back-propagation through
// time over the stack (paper, section 5: the gradient keeps reaching states that were
// popped and later overwritten, because every produced state is kept once).
//
// The state read at step t is the one produced at step src[t] (src[t] = top[t-1]), and
// the state returned at step t is the one produced at step top[t]. Reverse sweep, with
// dh_acc/dc_acc[s+1] the gradient w.r.t. the state produced at step s (slot 0 = h0/c0):
//   non-push t:  dh_acc[top+1] += dh_top[t], dc_acc[top+1] += dc_top[t]; dA[t] = 0
//   push t:      dh = dh_acc[t+1] + dh_top[t], dc = dc_acc[t+1] + dc_top[t] + dh o (1 - tanh^2 c)
//                dA = (dc g i(1-i), dc c_prev f(1-f), dc i (1-g^2), dh tanh(c) o(1-o))
//                dc_acc[src+1] += dc f;   [group barrier]   dh_acc[src+1] += dA U^T
// Same work split as the forward: group of 16*NT rows on one XCC, workgroup w owns
// hidden units [16w, 16w+16). dA U^T needs all 4H gate columns, so dA is exchanged
// through L2 at the barrier; wave q contracts gate columns [qH, (q+1)H) against its
// register-resident slice of U and the four partial sums are added in LDS in a fixed
// order. Every dh_acc/dc_acc element is owned by one thread, so there are no atomics.
#include "common.h"
#include "recurrent.h"
#include "rec_config.h"

template <int PREC, int NT, int KS, int OCC>
__global__ void __launch_bounds__(256, OCC) k_bwd(RecArgs a) {
  constexpr int KC = PREC ? 32 : 16;
  constexpr int BG = NT * 16;
  constexpr int PAIRS = BG * 16 / 256;            // (row, unit) pairs per thread
  __shared__ float red[4][BG][17];
  __shared__ int s_op[BG], s_top[BG], s_src[BG];
  __shared__ float s_db[16][16][4];
  __shared__ int s_g, s_w, s_flag;

  claim_group_slot(a.ctl + CTL_XCC_SLOT_B, a.G, a.NW, &s_g, &s_w);
  const int g = s_g, w = s_w;
  if (g < 0) return;

  const int T = a.T, B = a.B, H = a.H, H4 = 4 * H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, lq = lane >> 4;
  const int row0 = g * BG;
  const int ks_eff = a.ks_eff;
  constexpr int ESZ = PREC ? 2 : 4;
  const rsrc_t r_dA = make_rsrc(a.dA, (size_t)T * B * H4 * ESZ);

  // ---- U^T slice: A(m = unit 16w + l16, k = gate column q*H + kk) = U[unit][caller column]
  const int a_unit = w * 16 + l16;
  const bool a_ok = a_unit < H;
  const float* Urow = a.U + (size_t)(a_ok ? a_unit : 0) * H4;
  float ureg32[PREC ? 1 : KS][4];
  bf16x8 ureg16[PREC ? KS : 1];
#pragma unroll
  for (int c = 0; c < KS; ++c) {
    if constexpr (PREC == 0) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        int kk = c * 16 + 4 * lq + j;
        ureg32[c][j] = (a_ok && kk < H) ? Urow[perm_to_orig(wave * H + kk, H)] : 0.f;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        int kk = c * 32 + 8 * lq + j;
        ureg16[c][j] = f32_to_bf16((a_ok && kk < H) ? Urow[perm_to_orig(wave * H + kk, H)] : 0.f);
      }
    }
  }

  // ---- this thread's (row, unit) pairs: unit fixed per thread, rows r = tid/16 + 16 i
  const int uu = threadIdx.x & 15;
  const int u = w * 16 + uu;
  int prow[PAIRS];
  bool pok[PAIRS];
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    prow[i] = (threadIdx.x >> 4) + 16 * i;
    pok[i] = (row0 + prow[i] < B) && (u < H);
  }
  // zero the accumulator slots that can receive gradient: slot 0 and the slots of push steps
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    if (!pok[i]) continue;
    int b = row0 + prow[i];
    a.dh_acc[(size_t)b * H + u] = 0.f;
    a.dc_acc[(size_t)b * H + u] = 0.f;
    for (int s = 0; s < T; ++s) {
      if (a.ops[(size_t)s * B + b] == 1) {
        size_t o = ((size_t)(s + 1) * B + b) * H + u;
        a.dh_acc[o] = 0.f;
        a.dc_acc[o] = 0.f;
      }
    }
  }
  float dbacc[4] = {0.f, 0.f, 0.f, 0.f};
  const bool vec_ok = PREC ? (H % 8 == 0) : (H % 4 == 0);
  __syncthreads();

  long long* clk = a.clk ? a.clk + (size_t)blockIdx.x * T * 4 : nullptr;
  for (int t = T - 1; t >= 0; --t) {
    if (clk && threadIdx.x == 0) clk[t * 4 + 0] = wall_clock64();
    if ((int)threadIdx.x < BG) {
      int b = row0 + (int)threadIdx.x;
      int op = 0, tp = -1, sp = -1;
      if (b < B) {
        op = a.ops[(size_t)t * B + b];
        tp = a.top[(size_t)t * B + b];
        sp = (t == 0) ? -1 : a.top[(size_t)(t - 1) * B + b];
        // guard against a producer table that is not the forward's: no access outside [-1, t]
        if (tp < -1 || tp > t || (op == 1 && tp != t)) { tp = -1; op = (op == 1) ? 0 : op; }
        if (sp < -1 || sp >= t) sp = -1;
      }
      s_op[threadIdx.x] = op; s_top[threadIdx.x] = tp; s_src[threadIdx.x] = sp;
    }
    __syncthreads();

    // ---- cell backward for this workgroup's (row, unit) pairs
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      if (!pok[i]) continue;
      const int r = prow[i], b = row0 + r;
      const size_t o = ((size_t)t * B + b) * H + u;
      const int op = s_op[r];
      float gh = a.dh_top[o];
      float gc = a.dc_top ? a.dc_top[o] : 0.f;
      float4 dA4 = float4{0.f, 0.f, 0.f, 0.f};
      if (op == 1) {
        const int src = s_src[r];
        const size_t so = ((size_t)(t + 1) * B + b) * H + u;
        float dh = a.dh_acc[so] + gh;
        float dcin = a.dc_acc[so] + gc;
        float4 act = *(const float4*)(a.stash + ((size_t)t * B + b) * H4 + 4 * u);
        float c = a.ccell[o];
        float cp = (src < 0) ? a.c0[(size_t)b * H + u] : a.ccell[((size_t)src * B + b) * H + u];
        float tc = tanhf(c);
        float dc = dcin + dh * act.w * (1.f - tc * tc);
        dA4.x = dc * act.z * act.x * (1.f - act.x);
        dA4.y = dc * cp * act.y * (1.f - act.y);
        dA4.z = dc * act.x * (1.f - act.z * act.z);
        dA4.w = dh * tc * act.w * (1.f - act.w);
        const size_t po = ((size_t)(src + 1) * B + b) * H + u;
        a.dc_acc[po] += dc * act.y;
        dbacc[0] += dA4.x; dbacc[1] += dA4.y; dbacc[2] += dA4.z; dbacc[3] += dA4.w;
      } else {
        const size_t io = ((size_t)(s_top[r] + 1) * B + b) * H + u;
        a.dh_acc[io] += gh;
        if (a.dc_top) a.dc_acc[io] += gc;
      }
      const size_t ao = ((size_t)t * B + b) * H4 + 4 * u;
      if constexpr (PREC == 0) {
        *(float4*)((float*)a.dA + ao) = dA4;
      } else {
        bf16_t q[4] = {f32_to_bf16_bits(dA4.x), f32_to_bf16_bits(dA4.y), f32_to_bf16_bits(dA4.z),
                       f32_to_bf16_bits(dA4.w)};
        *(uint2*)((bf16_t*)a.dA + ao) = *(const uint2*)q;
      }
    }

    if (clk && threadIdx.x == 0) clk[t * 4 + 1] = wall_clock64();
    if (group_barrier(&a.ctl[CTL_BAR_B + g * 16], (uint32_t)(a.NW * (T - t)), a.ctl, a.spin_limit, &s_flag)) break;
    if (clk && threadIdx.x == 0) clk[t * 4 + 2] = wall_clock64();

    // ---- dh_prev^T (16 units x 16 rows per tile) = U^T-slice x dA^T over this wave's gate columns
    // B fragments are fetched one group of CG chunks ahead of the MFMAs that use them
    constexpr int CG = (NT >= 8) ? 1 : (8 / NT);
    constexpr int NG = (KS + CG - 1) / CG;
    f32x4 acc[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
    bool live[NT];
    size_t rowo[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int r = nt * 16 + l16, b = row0 + r;
      live[nt] = (b < B) && (s_op[r] == 1);              // dA rows of non-push steps are zero
      rowo[nt] = ((size_t)t * B + (live[nt] ? b : 0)) * H4 + (size_t)wave * H;
    }
    // Branch-free fragment loads through the bounds-checked descriptor: a lane whose row
    // is not a push (its dA row is exactly 0) or whose k is past H gets an offset beyond
    // the buffer, which returns 0 without a memory access.
    const uint32_t kOOB = 0xffffffffu;
    auto fetch = [&](int c, int nt) -> uint4 {
      const int kk = c * KC + (PREC ? 8 : 4) * lq;
      const size_t el = rowo[nt] + kk;
      if (vec_ok) {
        const uint32_t off = (live[nt] && kk < H) ? (uint32_t)(el * ESZ) : kOOB;
        if (a.coh_rows) return ld_coh_b128(r_dA, off);
        return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r_dA, off, 0, 0));
      }
      uint4 raw;
      uint32_t* rw = (uint32_t*)&raw;
      if constexpr (PREC == 0) {
        for (int j = 0; j < 4; ++j)
          rw[j] = ld_coh_b32(r_dA, (live[nt] && kk + j < H) ? (uint32_t)((el + j) * 4) : kOOB);
      } else {
        for (int j = 0; j < 4; ++j) {
          uint32_t lo = ld_coh_b16(r_dA, (live[nt] && kk + 2 * j < H) ? (uint32_t)((el + 2 * j) * 2) : kOOB);
          uint32_t hi = ld_coh_b16(r_dA, (live[nt] && kk + 2 * j + 1 < H) ? (uint32_t)((el + 2 * j + 1) * 2) : kOOB);
          rw[j] = lo | (hi << 16);
        }
      }
      return raw;
    };
    uint4 bufA[CG][NT], bufB[CG][NT];
#pragma unroll
    for (int j = 0; j < CG; ++j)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) bufA[j][nt] = fetch(j, nt);
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) {
      uint4 (&cur)[CG][NT] = (gi & 1) ? bufB : bufA;
      uint4 (&nxt)[CG][NT] = (gi & 1) ? bufA : bufB;
      if (gi + 1 < NG) {
#pragma unroll
        for (int j = 0; j < CG; ++j)
#pragma unroll
          for (int nt = 0; nt < NT; ++nt) nxt[j][nt] = fetch((gi + 1) * CG + j, nt);
      }
#pragma unroll
      for (int j = 0; j < CG; ++j) {
        const int c = gi * CG + j;
        if (c >= KS) continue;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          if constexpr (PREC == 0) {
            const float4 bv = __builtin_bit_cast(float4, cur[j][nt]);
            acc[nt] = mfma_f32_16x16x4(ureg32[c][0], bv.x, acc[nt]);
            acc[nt] = mfma_f32_16x16x4(ureg32[c][1], bv.y, acc[nt]);
            acc[nt] = mfma_f32_16x16x4(ureg32[c][2], bv.z, acc[nt]);
            acc[nt] = mfma_f32_16x16x4(ureg32[c][3], bv.w, acc[nt]);
          } else {
            acc[nt] = mfma_bf16_16x16x32(ureg16[c], __builtin_bit_cast(bf16x8, cur[j][nt]), acc[nt]);
          }
        }
      }
    }
    // lane holds units 4*lq + j of row l16 of each tile
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
      for (int j = 0; j < 4; ++j) red[wave][nt * 16 + l16][4 * lq + j] = acc[nt][j];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      if (!pok[i]) continue;
      const int r = prow[i], b = row0 + r;
      if (s_op[r] != 1) continue;
      float s = red[0][r][uu] + red[1][r][uu] + red[2][r][uu] + red[3][r][uu];
      a.dh_acc[((size_t)(s_src[r] + 1) * B + b) * H + u] += s;
    }
    __syncthreads();
    if (clk && threadIdx.x == 0) clk[t * 4 + 3] = wall_clock64();
  }

  // ---- outputs of this workgroup: dh0, dc0 for its pairs; per-group bias gradient
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    if (!pok[i]) continue;
    int b = row0 + prow[i];
    a.dh0[(size_t)b * H + u] = a.dh_acc[(size_t)b * H + u];
    a.dc0[(size_t)b * H + u] = a.dc_acc[(size_t)b * H + u];
  }
  const int rgrp = threadIdx.x >> 4;                 // 16 row groups share a unit
  for (int j = 0; j < 4; ++j) s_db[rgrp][uu][j] = dbacc[j];
  __syncthreads();
  if (threadIdx.x < 64) {
    int uu2 = threadIdx.x >> 2, j = threadIdx.x & 3;
    float s = 0.f;
    for (int q = 0; q < 16; ++q) s += s_db[q][uu2][j];
    int u2 = w * 16 + uu2;
    if (u2 < H) a.db_part[(size_t)g * H4 + 4 * u2 + j] = s;
  }
}

template <int P, int NT, int KS>
static hipError_t launch_bwd_t(const RecArgs& a, dim3 grid, hipStream_t st, int* occ_out) {
  constexpr int OCC = rec_occ(P, KS);
  auto kern = k_bwd<P, NT, KS, OCC>;
  int occ = 0;
  hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 256, 0);
  if (e != hipSuccess) return e;
  if (occ_out) *occ_out = occ;
  if (!grid.x) return hipSuccess;
  RecArgs args = a;
  void* kargs[] = {&args};
  return hipLaunchCooperativeKernel((const void*)kern, grid, dim3(256), kargs, 0, st);
}

hipError_t launch_bwd(const RecArgs& a, int prec, int NT, int KS, dim3 grid, hipStream_t st, int* occ_out) {
#define CASE(P, NT_, KS_) if (prec == P && NT == NT_ && KS == KS_) return launch_bwd_t<P, NT_, KS_>(a, grid, st, occ_out);
  REC_CASES(CASE)
#undef CASE
  return hipErrorInvalidValue;
}
