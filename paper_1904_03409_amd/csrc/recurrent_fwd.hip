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
// and (for push steps, the only ones the backward reads) the gate activations, and meets
// the group at a barrier. The producer of every state read comes from top[], which the op
// scan filled before the kernel (the integer stack stack[p+1] <- t, p <- p + op,
// top <- stack[p] depends on the ops alone).
//
// Latency schedule of one step: the h_prev rows go straight from L2 into LDS
// (global_load_lds, whole 1 KB row segments per wave instruction) when the row length
// allows it; the input projection of the next step, the producer indices of the next
// step and, once those are known, the c_prev values of the next step are fetched
// while this step computes, so the epilogue works from registers only.
#include "common.h"
#include "recurrent.h"
#include "rec_config.h"
#include "rec_device.h"

template <int PREC, int NT, int NTB, int KS, int OCC>
__global__ void __launch_bounds__(256, OCC) k_fwd(RecArgs a, FxArgs f) {
  constexpr int KC = PREC ? 32 : 16;               // K per chunk
  constexpr int KP = KS * KC;                      // K capacity of the U registers
  constexpr int ESZ = PREC ? 2 : 4;                // bytes per staged element
  constexpr int LDS_LD = rec_lds_ld(PREC, KS);     // LDS row stride (elements), padded
  constexpr int ROWS_B = NTB * 16;                 // rows staged per pass
  constexpr int NPASS = NT / NTB;
  constexpr int BG = NT * 16;                      // rows per group
  typedef __attribute__((address_space(3))) void* lds_ptr_t;
  using elem_t = typename std::conditional<PREC == 1, bf16_t, float>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  elem_t* hs = reinterpret_cast<elem_t*>(smem);
  __shared__ int s_src[BG];
  __shared__ int s_g, s_w;
  __shared__ int s_abort[2];   // [0]: a staging wait gave up, [1]: a group barrier gave up

  claim_group_slot(a.ctl + CTL_XCC_SLOT, a.G, a.NW, &s_g, &s_w);
  const int g = s_g, w = s_w;
  if (g < 0) return;

  const int T = a.T, B = a.B, H = a.H, H4 = 4 * H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, lq = lane >> 4;
  const int row0 = g * BG;
  const int unit_base = w * 16 + wave * 4;
  const int u = unit_base + lq;                    // epilogue unit of this lane
  const int ks_eff = a.ks_eff;
  const size_t TBH = (size_t)T * B * H;
  // staged rows: fp32 mode reads h_cell (src >= 0) or h0; bf16 mode reads the bf16 copy
  // whose slot 0 holds h0 and slot s+1 the state of step s
  const rsrc_t r_h = PREC ? make_rsrc(a.hx, TBH * 2 + (size_t)B * H * 2) : make_rsrc(a.hcell, TBH * 4);

  // ---- U slice into registers (MFMA A operand), resident for the whole kernel
  float ureg32[PREC ? 1 : KS][4];
  bf16x8 ureg16[PREC ? KS : 1];
  fwd_load_u<PREC, KS>(a, unit_base, l16, lq, ureg32, ureg16);

  const int kmax = ks_eff * KC;                    // staged K (>= H)
  const bool vec_ok = PREC ? (H % 8 == 0) : (H % 4 == 0);
  const bool direct = vec_ok && kmax == KP && (KP * ESZ) % 1024 == 0;

  // ---- fused input projection (bf16, one pass per step, I <= 256): x_t W is contracted in
  // the step itself. The W slice (this wave's 16 gate columns x I, bf16) sits in registers
  // like the U slice. The x rows of a step are copied (fp32, by LDS DMA, one row per wave
  // instruction, 1 KB + 16 B per row) into a ring of three LDS buffers two steps ahead: the
  // copy of step t+2 is issued right after step t's row wait, so the next wait that covers it
  // is step t+1's, one step later, and the data is in LDS for step t+2. The bias is added in
  // the cell update.
  constexpr bool FX_BUILT = rec_fx_built(PREC, KS);
  constexpr int XLD = 260;                         // LDS row stride of x (fp32): 1 KB + 16 B
  const bool fx = FX_BUILT && f.fuse_x && NPASS == 1;
  const int I = a.I, kx = f.kx;
  float* xsb = reinterpret_cast<float*>(smem + (size_t)ROWS_B * LDS_LD * ESZ);   // [3][ROWS_B][XLD]
  float4 bias4 = float4{0.f, 0.f, 0.f, 0.f};
  bf16x8 wreg[FX_BUILT ? 8 : 1];
  const rsrc_t r_x = make_rsrc(f.x, fx ? (size_t)T * B * I * 4 : 0);
  const uint32_t x_voff = (fx && lane * 4 < I) ? (uint32_t)lane * 16u : kOOB;   // k >= I reads 0
  auto dma_x = [&](int tt, int buf) {
    for (int r = wave; r < ROWS_B; r += 4) {
      const int b = row0 + r;
      if (b >= B) break;                            // rows past the batch: outputs are masked
      bdma16(r_x, x_voff, (uint32_t)(((size_t)tt * B + b) * I * 4),
             lds_addr(xsb + ((size_t)buf * ROWS_B + r) * XLD));
    }
  };
  // x_t W for every tile of the pass: A = W^T slice rows (unit, gate) of this wave, B = x rows
  // (fp32 in LDS, rounded to bf16 as they are read)
  auto xpart = [&](f32x4* acc, int buf) {
    if constexpr (FX_BUILT) {
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        if (c < kx) {
#pragma unroll
          for (int nt = 0; nt < NTB; ++nt) {
            const float* xp = xsb + ((size_t)buf * ROWS_B + nt * 16 + l16) * XLD + c * 32 + 8 * lq;
            const float4 x0 = *(const float4*)xp, x1 = *(const float4*)(xp + 4);
            bf16x8 xv;
            xv[0] = f32_to_bf16(x0.x); xv[1] = f32_to_bf16(x0.y); xv[2] = f32_to_bf16(x0.z); xv[3] = f32_to_bf16(x0.w);
            xv[4] = f32_to_bf16(x1.x); xv[5] = f32_to_bf16(x1.y); xv[6] = f32_to_bf16(x1.z); xv[7] = f32_to_bf16(x1.w);
            acc[nt] = mfma_bf16_16x16x32(wreg[c], xv, acc[nt]);
          }
        }
      }
    }
  };
  if (fx) {
    // W slice: row m = l16 of this wave's tile is gate m % 4 of unit unit_base + m / 4 (the U
    // slice's order); chunk c holds inputs c*32 + 8lq .. +7, zero past I
    const int unit = unit_base + (l16 >> 2), gate = l16 & 3;
#pragma unroll
    for (int c = 0; c < (FX_BUILT ? 8 : 1); ++c)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int k = c * 32 + 8 * lq + j;
        wreg[c][j] = f32_to_bf16((unit < H && k < I) ? f.W[(size_t)k * H4 + gate * H + unit] : 0.f);
      }
    if (u < H) bias4 = float4{f.bias[u], f.bias[H + u], f.bias[2 * H + u], f.bias[3 * H + u]};
    dma_x(0, 0);
    if (T > 1) dma_x(1, 1);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  // rows of this lane in the MFMA output layout: tile ti covers rows ti*16 .. ti*16+15
  int lrow[NT];
  bool lok[NT];
#pragma unroll
  for (int ti = 0; ti < NT; ++ti) {
    lrow[ti] = row0 + ti * 16 + l16;
    lok[ti] = (lrow[ti] < B) && (u < H);
  }
  auto xw_at = [&](int t, int ti) -> float4 {
    const int b = lok[ti] ? lrow[ti] : 0, uu = lok[ti] ? u : 0;
    // read once: non-temporal, so the stream does not push the exchanged rows out of L2
    const f32x4 v = __builtin_nontemporal_load((const f32x4*)(a.xw + ((size_t)t * B + b) * H4 + 4 * uu));
    return float4{v[0], v[1], v[2], v[3]};
  };
  auto top_at = [&](int t, int ti) -> int {
    const int b = lrow[ti] < B ? lrow[ti] : 0;
    return a.top[(size_t)t * B + b];
  };
  if ((int)threadIdx.x < BG) s_src[threadIdx.x] = -1;
  if (threadIdx.x < 2) s_abort[threadIdx.x] = 0;
  constexpr int NV = (BG + 63) / 64;
  int vsrc[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) vsrc[j] = -1;
  for (int i = threadIdx.x; i < ROWS_B * LDS_LD * ESZ / 16; i += 256) ((uint4*)smem)[i] = uint4{0u, 0u, 0u, 0u};
  // operands of step 0's epilogue
  float4 xw_cur[NT];
  float cp_cur[NT];
#pragma unroll
  for (int ti = 0; ti < NT; ++ti) {
    xw_cur[ti] = fx ? bias4 : xw_at(0, ti);
    cp_cur[ti] = lok[ti] ? a.c0[(size_t)lrow[ti] * H + u] : 0.f;
  }
  if (!a.poll) {
    if (group_barrier(&a.ctl[CTL_BAR_F + g * 16], (uint32_t)a.NW, a.ctl, a.spin_limit, &s_abort[1])) return;
  } else {
    __syncthreads();
  }

  // Direct staging: one wave instruction moves one 1 KB segment of one row into LDS, 16 bytes
  // per lane. Segment i of this wave is row segment wave + 4 i of the pass; the row's producer
  // comes from lane rr of vsrc (wave-uniform), no LDS round trip.
  constexpr int SEG = (KP * ESZ) / 1024 > 0 ? (KP * ESZ) / 1024 : 1;
  constexpr int NSEG_W = (ROWS_B * SEG + 3) / 4;
  static_assert(NSEG_W <= 32, "segment mask is 32 bits");
  long long* clk = a.clk ? a.clk + (size_t)blockIdx.x * T * 4 : nullptr;
  bool stop = false;
  for (int t = 0; t < T; ++t) {
    if (clk && threadIdx.x == 0) clk[t * 4 + 0] = wall_clock64();
    const bool more = t + 1 < T;
    float4 xw_nxt[NT];
    int src_nxt[NT];
    float cp_nxt[NT];

    if constexpr (PREC == 1) {
      // bf16 steps are short: the next step's input projection (HBM) and producer indices are
      // requested before the staging loads, so their latency overlaps the staging instead of
      // following it (vector loads complete in issue order)
#pragma unroll
      for (int ti = 0; ti < NT; ++ti) src_nxt[ti] = top_at(t, ti);
      if (fx) {
#pragma unroll
        for (int ti = 0; ti < NT; ++ti) xw_nxt[ti] = bias4;
      } else {
#pragma unroll
        for (int ti = 0; ti < NT; ++ti) xw_nxt[ti] = xw_at(more ? t + 1 : t, ti);
      }
      asm volatile("" ::: "memory");
    }
#pragma unroll
    for (int nb = 0; nb < NPASS; ++nb) {
      f32x4 acc[NTB];
#pragma unroll
      for (int nt = 0; nt < NTB; ++nt) acc[nt] = f32x4{0.f, 0.f, 0.f, 0.f};
      // ---- gather this pass's h_prev rows into LDS; granules that still hold the fill are
      // fetched again until their producers' stores have arrived. With the fused input
      // projection, its MFMAs run while the rows are in flight.
      if (fx && !direct) xpart(acc, t % 3);
      if (direct) {
#pragma unroll
        for (int i = 0; i < NSEG_W; ++i) {
          const int sgi = wave + 4 * i;
          if (sgi < ROWS_B * SEG) {
            const int r = sgi / SEG, sj = sgi % SEG, rr = nb * ROWS_B + r;
            const int src = __builtin_amdgcn_readlane(vsrc[rr >> 6], rr & 63);
            int k = sj * (1024 / ESZ) + lane * (16 / ESZ);
            if (k >= H) k = 0;                    // finite filler; the U registers are 0 there
            elem_t* lp = hs + r * LDS_LD + sj * (1024 / ESZ);
            // rows past B: any finite row (their columns are masked)
            const void* gp = staged_src<PREC>(a, src, min(row0 + rr, B - 1), k);
            if (a.coh_rows) __builtin_amdgcn_global_load_lds(gp, (lds_ptr_t)lp, 16, 0, kSc1);
            else __builtin_amdgcn_global_load_lds(gp, (lds_ptr_t)lp, 16, 0, 0);
          }
        }
        if (fx) xpart(acc, t % 3);
      } else {
        constexpr int VW = PREC ? 8 : 4;
        if (vec_ok) {
          // batches of four vector loads per thread: latency paid once per batch
          const int per_row = kmax / VW;
          const int n_el = ROWS_B * per_row;
          for (int e0 = 0; e0 < n_el; e0 += 4 * 256) {
            uint4 buf[4];
            const void* pp[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int e = e0 + threadIdx.x + 256 * i;
              buf[i] = uint4{0u, 0u, 0u, 0u};
              pp[i] = nullptr;
              if (e >= n_el) continue;
              const int r = e / per_row, k = (e - r * per_row) * VW;
              const int rr = nb * ROWS_B + r, b = row0 + rr;
              if (b >= B || k >= H) continue;
              const int src = s_src[rr];
              if constexpr (PREC == 0) {
                if (src < 0) {
                  buf[i] = *(const uint4*)(a.h0 + (size_t)b * H + k);
                  continue;
                }
                const size_t e2 = ((size_t)src * B + b) * H + k;
                pp[i] = a.hcell + e2;
                if (a.coh_rows) buf[i] = ld_coh_b128(r_h, (uint32_t)(e2 * 4));
                else buf[i] = *(const uint4*)(a.hcell + e2);
              } else {
                const size_t e2 = ((size_t)(src + 1) * B + b) * H + k;
                if (src >= 0) pp[i] = a.hx + e2;
                if (a.coh_rows) buf[i] = ld_coh_b128(r_h, (uint32_t)(e2 * 2));
                else buf[i] = *(const uint4*)(a.hx + e2);
              }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              int spins = 0;
              while (pp[i] && pending_granule<PREC>(buf[i])) {
                if (spin_out(spins, a.ctl, a.spin_limit)) {
                  s_abort[0] = 1;
                  break;
                }
                buf[i] = ld_poll_b128(pp[i]);
              }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int e = e0 + threadIdx.x + 256 * i;
              if (e >= n_el) continue;
              const int r = e / per_row, k = (e - r * per_row) * VW;
              *(uint4*)(hs + r * LDS_LD + k) = buf[i];
            }
          }
        } else {
          for (int e = threadIdx.x; e < ROWS_B * kmax; e += 256) {
            const int r = e / kmax, k = e - r * kmax;
            const int rr = nb * ROWS_B + r, b = row0 + rr;
            float v = 0.f;
            if (b < B && k < H) {
              const int src = s_src[rr];
              int spins = 0;
              if constexpr (PREC == 0) {
                if (src < 0) {
                  v = a.h0[(size_t)b * H + k];
                } else {
                  const size_t e2 = ((size_t)src * B + b) * H + k;
                  uint32_t bits = ld_coh_b32(r_h, (uint32_t)(e2 * 4));
                  while (bits == 0xffffffffu) {
                    if (spin_out(spins, a.ctl, a.spin_limit)) {
                      s_abort[0] = 1;
                      break;
                    }
                    bits = __hip_atomic_load((uint32_t*)(a.hcell + e2), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                  }
                  v = __uint_as_float(bits);
                }
              } else {
                const size_t e2 = ((size_t)(src + 1) * B + b) * H + k;
                uint32_t bits = ld_coh_b16(r_h, (uint32_t)(e2 * 2));
                while (src >= 0 && bits == 0xffffu) {
                  if (spin_out(spins, a.ctl, a.spin_limit)) {
                    s_abort[0] = 1;
                    break;
                  }
                  // the aligned word that holds the element
                  const uint32_t wv = __hip_atomic_load((uint32_t*)(a.hx + (e2 & ~(size_t)1)), __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT);
                  bits = (e2 & 1) ? (wv >> 16) : (wv & 0xffffu);
                }
                v = bf16_bits_to_f32((bf16_t)bits);
              }
            }
            if constexpr (PREC == 0) hs[r * LDS_LD + k] = v;
            else hs[r * LDS_LD + k] = f32_to_bf16_bits(v);
          }
        }
      }
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      if (direct && a.poll) {
        // granules that still hold the fill are fetched again (only the lanes that hold one take
        // part in the copy), bypassing L1, until every producer's store has arrived
        uint32_t bad = 0;
#pragma unroll
        for (int i = 0; i < NSEG_W; ++i) {
          const int sgi = wave + 4 * i;
          if (sgi < ROWS_B * SEG) {
            const int r = sgi / SEG, sj = sgi % SEG, rr = nb * ROWS_B + r;
            const int src = __builtin_amdgcn_readlane(vsrc[rr >> 6], rr & 63);
            const elem_t* lp = hs + r * LDS_LD + sj * (1024 / ESZ);
            if (src >= 0 && pending_granule<PREC>(*(const uint4*)(lp + lane * (16 / ESZ)))) bad |= 1u << i;
          }
        }
        int spins = 0;
        while (__builtin_amdgcn_ballot_w64(bad != 0u)) {
          if (spin_out(spins, a.ctl, a.spin_limit)) {
            s_abort[0] = 1;
            break;
          }
#pragma unroll
          for (int i = 0; i < NSEG_W; ++i) {
            const int sgi = wave + 4 * i;
            if (sgi < ROWS_B * SEG && ((bad >> i) & 1u)) {
              const int r = sgi / SEG, sj = sgi % SEG, rr = nb * ROWS_B + r;
              const int src = __builtin_amdgcn_readlane(vsrc[rr >> 6], rr & 63);
              int k = sj * (1024 / ESZ) + lane * (16 / ESZ);
              if (k >= H) k = 0;                      // finite filler; the U registers are 0 there
              elem_t* lp = hs + r * LDS_LD + sj * (1024 / ESZ);
              const void* gp = staged_src<PREC>(a, src, min(row0 + rr, B - 1), k);
              __builtin_amdgcn_global_load_lds(gp, (lds_ptr_t)lp, 16, 0, kSc1);
            }
          }
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
          for (int i = 0; i < NSEG_W; ++i) {
            const int sgi = wave + 4 * i;
            if (sgi < ROWS_B * SEG && ((bad >> i) & 1u)) {
              const int r = sgi / SEG, sj = sgi % SEG;
              const elem_t* lp = hs + r * LDS_LD + sj * (1024 / ESZ);
              if (!pending_granule<PREC>(*(const uint4*)(lp + lane * (16 / ESZ)))) bad &= ~(1u << i);
            }
          }
        }
      }
      __syncthreads();
      if (s_abort[0]) {
        stop = true;
        break;
      }
      if (clk && threadIdx.x == 0 && nb == 0) clk[t * 4 + 1] = wall_clock64();
      // x rows of step t+2 into the buffer step t-1 used (read before step t-1 ended)
      if (fx && t + 2 < T) dma_x(t + 2, (t + 2) % 3);
      if (PREC == 0 && nb == 0) {
        // fp32 steps are long: the producer indices read at step t+1 (top[t], published one
        // step ago) and the next step's input projection are in flight during the MFMAs
#pragma unroll
        for (int ti = 0; ti < NT; ++ti) src_nxt[ti] = top_at(t, ti);
#pragma unroll
        for (int ti = 0; ti < NT; ++ti) xw_nxt[ti] = xw_at(more ? t + 1 : t, ti);
      }

      // ---- gates^T (16 cols x 16 rows per tile) += U^T h_prev^T; B fragments read one chunk ahead
      // all KS chunks run: U registers and staged LDS columns are zero beyond H
      if constexpr (PREC == 0) {
        float4 bcur[NTB], bnxt[NTB];
#pragma unroll
        for (int nt = 0; nt < NTB; ++nt) bcur[nt] = *(const float4*)&hs[(nt * 16 + l16) * LDS_LD + 4 * lq];
#pragma unroll
        for (int c = 0; c < KS; ++c) {
          if (c + 1 < KS) {
#pragma unroll
            for (int nt = 0; nt < NTB; ++nt)
              bnxt[nt] = *(const float4*)&hs[(nt * 16 + l16) * LDS_LD + (c + 1) * 16 + 4 * lq];
          }
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int nt = 0; nt < NTB; ++nt) acc[nt] = mfma_f32_16x16x4(ureg32[c][j], bcur[nt][j], acc[nt]);
#pragma unroll
          for (int nt = 0; nt < NTB; ++nt) bcur[nt] = bnxt[nt];
        }
      } else {
        bf16x8 bcur[NTB], bnxt[NTB];
#pragma unroll
        for (int nt = 0; nt < NTB; ++nt) bcur[nt] = *(const bf16x8*)&hs[(nt * 16 + l16) * LDS_LD + 8 * lq];
#pragma unroll
        for (int c = 0; c < KS; ++c) {
          if (c + 1 < KS) {
#pragma unroll
            for (int nt = 0; nt < NTB; ++nt)
              bnxt[nt] = *(const bf16x8*)&hs[(nt * 16 + l16) * LDS_LD + (c + 1) * 32 + 8 * lq];
          }
#pragma unroll
          for (int nt = 0; nt < NTB; ++nt) acc[nt] = mfma_bf16_16x16x32(ureg16[c], bcur[nt], acc[nt]);
#pragma unroll
          for (int nt = 0; nt < NTB; ++nt) bcur[nt] = bnxt[nt];
        }
      }
      if (clk && threadIdx.x == 0 && nb == 0) clk[t * 4 + 2] = wall_clock64();

      // ---- fused LSTM cell: lane holds gates i, f, g, o of unit u for row l16 of each tile
#pragma unroll
      for (int nt = 0; nt < NTB; ++nt) {
        const int ti = nb * NTB + nt;
        if (!lok[ti]) continue;
        // the state this step produced; gate activations kept for a push (top[t] = t)
        cp_cur[ti] = fwd_cell<PREC>(a, acc[nt], xw_cur[ti], cp_cur[ti], t, lrow[ti], u, src_nxt[ti] == t);
      }
      if (NPASS > 1) __syncthreads();
    }
    if (stop) break;

    // c_prev of step t+1: the state produced now (push at t) or an older one of this workgroup
#pragma unroll
    for (int ti = 0; ti < NT; ++ti) {
      const int s = more ? checked_src(src_nxt[ti], t, a.ctl) : -1;
      src_nxt[ti] = s;
      cp_nxt[ti] = cp_cur[ti];
      if (lok[ti] && s != t) {
        const int b = lrow[ti];
        cp_nxt[ti] = (s < 0) ? a.c0[(size_t)b * H + u] : a.ccell[((size_t)s * B + b) * H + u];
      }
    }
    if (clk && threadIdx.x == 0) clk[t * 4 + 3] = wall_clock64();
    if (wave == 0 && lq == 0) {
#pragma unroll
      for (int ti = 0; ti < NT; ++ti) s_src[ti * 16 + l16] = src_nxt[ti];
    }
#pragma unroll
    for (int ti = 0; ti < NT; ++ti) { xw_cur[ti] = xw_nxt[ti]; cp_cur[ti] = cp_nxt[ti]; }
    if (!a.poll) {
      // barrier mode: every state of step t is complete past this point
      if (group_barrier(&a.ctl[CTL_BAR_F + g * 16], (uint32_t)(a.NW * (t + 2)), a.ctl, a.spin_limit, &s_abort[1]))
        break;
    } else {
      __syncthreads();
    }
    if (s_abort[1]) break;
#pragma unroll
    for (int j = 0; j < NV; ++j) vsrc[j] = (64 * j + lane < BG) ? s_src[64 * j + lane] : -1;
  }
}

// ---- instantiations and launcher: one kernel per (precision, row tiles per group, K chunks)
template <int P, int NT, int KS>
static hipError_t launch_fwd_t(const RecArgs& a, const FxArgs& f, dim3 grid, hipStream_t st, int* occ_out) {
  constexpr int NTB = rec_ntb(P, NT, KS);
  constexpr int OCC = rec_occ(P, KS);
  auto kern = k_fwd<P, NT, NTB, KS, OCC>;
  size_t shm = rec_lds_bytes(P, NTB, KS);
  if (f.fuse_x) {
    // the fused projection: built variants, one pass per step, x rows within the staging registers
    if (!rec_fx_built(P, KS) || NTB != NT || !rec_fx_fits(16 * NT, f.kx)) return hipErrorInvalidValue;
    shm += rec_fx_lds_bytes(16 * NTB);
  }
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
  if (e != hipSuccess) return e;
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 256, shm);
  if (e != hipSuccess) return e;
  if (occ_out) *occ_out = occ;
  if (!grid.x) return hipSuccess;  // occupancy query only
  RecArgs args = a;
  FxArgs fargs = f;
  void* kargs[] = {&args, &fargs};
  return hipLaunchCooperativeKernel((const void*)kern, grid, dim3(256), kargs, (unsigned)shm, st);
}

hipError_t launch_fwd(const RecArgs& a, const FxArgs& f, int prec, int NT, int KS, dim3 grid, hipStream_t st,
                      int* occ_out) {
#define CASE(P, NT_, KS_) \
  if (prec == P && NT == NT_ && KS == KS_) return launch_fwd_t<P, NT_, KS_>(a, f, grid, st, occ_out);
  REC_CASES(CASE)
#undef CASE
  return hipErrorInvalidValue;
}
