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
//                dc_acc[src+1] += dc f;   dh_acc[src+1] += dA U^T
// Same work split as the forward: group of 16*NT rows on one XCC, workgroup w owns
// hidden units [16w, 16w+16). dA U^T needs all 4H gate columns, so dA is exchanged
// through L2 without a group barrier: dA starts filled with all-one bits, and a reader
// fetches again every granule that still holds them. Wave q contracts gate columns
// [qH, (q+1)H) against its register-resident slice of U and the four partial sums are
// added in LDS in a fixed order. Every dh_acc/dc_acc element is owned by one thread, so
// there are no atomics.
#include "common.h"
#include "recurrent.h"
#include "rec_config.h"

template <int PREC, int NT, int KS, int OCC>
__global__ void __launch_bounds__(256, OCC) k_bwd(RecArgs a) {
  constexpr int KC = PREC ? 32 : 16;
  constexpr int BG = NT * 16;
  constexpr int PAIRS = BG * 16 / 256;            // (row, unit) pairs per thread
  // staged dA rows (direct path): per wave 16 compacted rows of its H gate columns
  constexpr int QLD = KS * KC + (PREC ? 8 : 4);         // row stride (elements), 16-byte pad
  extern __shared__ __align__(16) unsigned char dsm[];
  __shared__ float red[4][BG][17];
  __shared__ int s_op[BG], s_top[BG], s_src[BG], s_crow[BG], s_cidx[BG], s_nlive;
  __shared__ float s_db[16][16][4];
  __shared__ int s_g, s_w;
  __shared__ int s_abort;                          // a wait for dA rows gave up

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
  const int ul = (u < H) ? u : 0;                   // unit used in load addresses (in bounds)
  int prow[PAIRS];
  bool pok[PAIRS];
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    prow[i] = (threadIdx.x >> 4) + 16 * i;
    pok[i] = (row0 + prow[i] < B) && (u < H);
  }
  // zero this workgroup's accumulator slots ([T+1] slots x group rows x its 16 units) with
  // 16-byte stores; slot 0 is the initial state
  {
    const int n4 = (T + 1) * BG * 4;
    for (int i = threadIdx.x; i < n4; i += 256) {
      const int slot = i / (BG * 4), rem = i - slot * (BG * 4);
      const int r = rem >> 2, q = rem & 3;
      const int b = row0 + r, u0 = w * 16 + 4 * q;
      if (b >= B) continue;
      const size_t o = ((size_t)slot * B + b) * H + u0;
      if (u0 + 3 < H && (H & 3) == 0) {
        *(float4*)(a.dh_acc + o) = float4{0.f, 0.f, 0.f, 0.f};
        *(float4*)(a.dc_acc + o) = float4{0.f, 0.f, 0.f, 0.f};
      } else {
        for (int j = 0; j < 4; ++j)
          if (u0 + j < H) { a.dh_acc[o + j] = 0.f; a.dc_acc[o + j] = 0.f; }
      }
    }
  }
  float dbacc[4] = {0.f, 0.f, 0.f, 0.f};
  const bool vec_ok = PREC ? (H % 8 == 0) : (H % 4 == 0);
  const bool direct = a.bwd_direct != 0;
  typedef __attribute__((address_space(3))) void* lds_ptr_t;
  using elem_t = typename std::conditional<PREC == 1, bf16_t, float>::type;
  elem_t* wbuf = reinterpret_cast<elem_t*>(dsm) + (size_t)wave * 16 * QLD;
  if (direct)
    for (int i = threadIdx.x; i < 4 * 16 * QLD * ESZ / 16; i += 256) ((uint4*)dsm)[i] = uint4{0u, 0u, 0u, 0u};
  if (threadIdx.x == 0) s_abort = 0;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // Loads are issued a step (or at least a phase) before their values are used. Per pair:
  //   cur_*  operands of the current step t, fetched during step t+1;
  //   slot_* gradient of the state produced at step t (dh_acc/dc_acc slot t+1), fetched at the
  //          start of step t+1 and updated in registers by step t+1's contributions to it;
  //   tg_*   the slot this step adds into (src+1 for a push, top+1 otherwise), fetched at the
  //          start of step t and written back with the contribution.
  auto valid = [&](int t, int op, int& tp, int& sp) {
    // guard against a producer table that is not the forward's: no access outside [-1, t]
    if (tp < -1 || tp > t || (op == 1 && tp != t)) tp = -1;
    if (sp < -1 || sp >= t) sp = -1;
  };
  int c_op[PAIRS], c_tp[PAIRS], c_sp[PAIRS];            // step t row info
  int n_op[PAIRS], n_sp[PAIRS];                          // step t-1 (top[t-1] = c_sp)
  float c_gh[PAIRS], c_gc[PAIRS], c_c[PAIRS], c_cp[PAIRS];
  float4 c_act[PAIRS];
  float n_gh[PAIRS], n_gc[PAIRS], n_c[PAIRS], n_cp[PAIRS];
  float4 n_act[PAIRS];
  float slot_dh[PAIRS], slot_dc[PAIRS], nx_dh[PAIRS], nx_dc[PAIRS], tg_dh[PAIRS], tg_dc[PAIRS];
  auto ld_row = [&](int t, int b, int& op, int& sp) {
    op = a.ops[(size_t)t * B + b];
    sp = (t == 0) ? -1 : a.top[(size_t)(t - 1) * B + b];
  };
  auto ld_ops = [&](int t, int b, float& gh, float& gc, float4& act, float& c) {
    const size_t o = ((size_t)t * B + b) * H + ul;
    gh = a.dh_top[o];
    gc = a.dc_top ? a.dc_top[o] : 0.f;
    act = *(const float4*)(a.stash + ((size_t)t * B + b) * H4 + 4 * ul);
    c = a.ccell[o];
  };
  auto ld_cp = [&](int sp, int b) -> float {
    return (sp < 0) ? a.c0[(size_t)b * H + ul] : a.ccell[((size_t)sp * B + b) * H + ul];
  };
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    const int b = pok[i] ? row0 + prow[i] : 0;
    int op, sp;
    ld_row(T - 1, b, op, sp);
    int tp = a.top[(size_t)(T - 1) * B + b];
    valid(T - 1, op, tp, sp);
    c_op[i] = op; c_tp[i] = tp; c_sp[i] = sp;
    ld_ops(T - 1, b, c_gh[i], c_gc[i], c_act[i], c_c[i]);
    c_cp[i] = ld_cp(sp, b);
    slot_dh[i] = 0.f; slot_dc[i] = 0.f;                // slot T was zeroed and nothing adds to it later
  }

  long long* clk = a.clk ? a.clk + (size_t)blockIdx.x * T * 4 : nullptr;
  for (int t = T - 1; t >= 0; --t) {
    if (clk && threadIdx.x == 0) clk[t * 4 + 0] = wall_clock64();
    // row tables of step t for the compaction (from the registers of the unit-0 threads)
    if (uu == 0) {
#pragma unroll
      for (int i = 0; i < PAIRS; ++i) {
        s_op[prow[i]] = pok[i] ? c_op[i] : 0;
        s_src[prow[i]] = c_sp[i];
        s_top[prow[i]] = c_tp[i];
      }
    }
    // loads, in the order they are needed (vector loads complete in issue order, so the
    // epilogue's wait for the target slot does not include the HBM prefetch behind it):
    // this step's target slot, slot t, then row info and operands of step t-1
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      const int b = pok[i] ? row0 + prow[i] : 0;
      const int tgt = (c_op[i] == 1) ? c_sp[i] : c_tp[i];
      const size_t to = ((size_t)(tgt + 1) * B + b) * H + ul;
      tg_dh[i] = a.dh_acc[to];
      tg_dc[i] = a.dc_acc[to];
    }
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      const int b = pok[i] ? row0 + prow[i] : 0;
      if (t > 0) {
        const size_t no = ((size_t)t * B + b) * H + ul;
        nx_dh[i] = a.dh_acc[no];
        nx_dc[i] = a.dc_acc[no];
      }
    }
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      const int b = pok[i] ? row0 + prow[i] : 0;
      if (t > 0) {
        ld_row(t - 1, b, n_op[i], n_sp[i]);
        ld_ops(t - 1, b, n_gh[i], n_gc[i], n_act[i], n_c[i]);
      }
    }
    __syncthreads();
    if (wave == 0) {
      // list the push rows in row order (wave-wide ballot + prefix count)
      int base = 0;
#pragma unroll
      for (int r0 = 0; r0 < BG; r0 += 64) {
        const int r = r0 + lane;
        const bool live = (r < BG) && (s_op[r] == 1);
        const unsigned long long m = __ballot(live);
        const int ci = base + __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
        if (live) { s_cidx[r] = ci; s_crow[ci] = r; }
        base += __popcll(m);
      }
      if (lane == 0) s_nlive = base;
    }

    // ---- cell backward for this workgroup's (row, unit) pairs
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      float4 dA4 = float4{0.f, 0.f, 0.f, 0.f};
      const int b = row0 + prow[i];
      const int tgt = (c_op[i] == 1) ? c_sp[i] : c_tp[i];
      const bool fwd_slot = (t > 0) && (tgt + 1 == t);   // contribution lands in next step's slot
      float add_dh = 0.f, add_dc = 0.f;
      if (c_op[i] == 1) {
        const float4 act = c_act[i];
        const float dh = slot_dh[i] + c_gh[i];
        const float dcin = slot_dc[i] + c_gc[i];
        const float tc = tanhf_(c_c[i]);
        const float dc = dcin + dh * act.w * (1.f - tc * tc);
        // never the all-ones fill pattern: a NaN is stored as the canonical quiet NaN
        dA4.x = canon_nan(dc * act.z * act.x * (1.f - act.x));
        dA4.y = canon_nan(dc * c_cp[i] * act.y * (1.f - act.y));
        dA4.z = canon_nan(dc * act.x * (1.f - act.z * act.z));
        dA4.w = canon_nan(dh * tc * act.w * (1.f - act.w));
        add_dc = dc * act.y;
        if (pok[i]) { dbacc[0] += dA4.x; dbacc[1] += dA4.y; dbacc[2] += dA4.z; dbacc[3] += dA4.w; }
      } else {
        add_dh = c_gh[i];
        add_dc = c_gc[i];
      }
      if (fwd_slot) {
        nx_dh[i] += add_dh;
        nx_dc[i] += add_dc;
      } else if (pok[i]) {
        const size_t to = ((size_t)(tgt + 1) * B + b) * H + u;
        tg_dh[i] += add_dh;
        tg_dc[i] += add_dc;
        if (c_op[i] != 1) a.dh_acc[to] = tg_dh[i];   // a push's dh contribution comes after the GEMM
        a.dc_acc[to] = tg_dc[i];
      }
      if (pok[i]) {
        const size_t ao = ((size_t)t * B + b) * H4 + 4 * u;
        if constexpr (PREC == 0) {
          *(float4*)((float*)a.dA + ao) = dA4;
        } else {
          bf16_t q[4] = {f32_to_bf16_bits(dA4.x), f32_to_bf16_bits(dA4.y), f32_to_bf16_bits(dA4.z),
                         f32_to_bf16_bits(dA4.w)};
          *(uint2*)((bf16_t*)a.dA + ao) = *(const uint2*)q;
        }
      }
    }

    if (clk && threadIdx.x == 0) clk[t * 4 + 1] = wall_clock64();
    if (a.poll) {
      __syncthreads();
    } else if (group_barrier(&a.ctl[CTL_BAR_B + g * 16], (uint32_t)(a.NW * (T - t)), a.ctl, a.spin_limit, &s_abort)) {
      break;
    }
    if (clk && threadIdx.x == 0) clk[t * 4 + 2] = wall_clock64();
    // c_prev of step t-1 (its producer index arrived with the prefetch above)
    if (t > 0) {
#pragma unroll
      for (int i = 0; i < PAIRS; ++i) {
        int op = n_op[i], tp = c_sp[i], sp = n_sp[i];
        valid(t - 1, op, tp, sp);
        n_sp[i] = sp;
        n_cp[i] = ld_cp(sp, pok[i] ? row0 + prow[i] : 0);
      }
    }

    // Only push rows have non-zero dA. They are listed (in row order) in s_crow and run as
    // compacted 16-row MFMA tiles; each tile's K loop fetches its fragments one group of CG
    // chunks ahead, through the bounds-checked descriptor (a lane past the list or k past H
    // gets an out-of-range offset: value 0, no memory access). Two accumulators per tile
    // keep two independent MFMA chains.
    constexpr int CG = 8;
    constexpr int NG = (KS + CG - 1) / CG;
    const uint32_t kOOB = 0xffffffffu;
    const int nlive = s_nlive;
    if (direct) {
      // Each wave copies its own H gate columns of the compacted rows straight into its LDS
      // slice (global_load_lds, 1 KB row segments), waits for its own loads only, and runs
      // the tile's MFMAs from LDS with the fragments of the next chunk read ahead.
      constexpr int SEGQ = KS * KC * ESZ / 1024;          // 1 KB segments per staged row
      for (int jt = 0; jt < NT; ++jt) {
        if (jt * 16 >= nlive) break;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ci = jt * 16 + r;
          if (ci < nlive) {
            const int b = row0 + s_crow[ci];
            const elem_t* rowp = (const elem_t*)a.dA + ((size_t)t * B + b) * H4 + (size_t)wave * H;
#pragma unroll
            for (int sj = 0; sj < SEGQ; ++sj) {
              const elem_t* gp = rowp + sj * (1024 / ESZ) + lane * (16 / ESZ);
              lds_ptr_t dst = (lds_ptr_t)(wbuf + r * QLD + sj * (1024 / ESZ));
              if (a.coh_rows) __builtin_amdgcn_global_load_lds((const void*)gp, dst, 16, 0, kSc1);
              else __builtin_amdgcn_global_load_lds((const void*)gp, dst, 16, 0, 0);
            }
          }
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        if (a.poll) {
          // granules whose producer's store has not arrived yet are fetched again (only the lanes
          // that hold one take part in the copy), bypassing L1, until complete
          static_assert(16 * SEGQ <= 32, "segment mask is 32 bits");
          uint32_t bad = 0;
#pragma unroll
          for (int r = 0; r < 16; ++r)
#pragma unroll
            for (int sj = 0; sj < SEGQ; ++sj)
              if (jt * 16 + r < nlive &&
                  pending_granule<PREC>(*(const uint4*)(wbuf + r * QLD + sj * (1024 / ESZ) + lane * (16 / ESZ))))
                bad |= 1u << (r * SEGQ + sj);
          int spins = 0;
          while (__builtin_amdgcn_ballot_w64(bad != 0u)) {
            if (spin_out(spins, a.ctl, a.spin_limit)) {
              s_abort = 1;
              break;
            }
#pragma unroll
            for (int r = 0; r < 16; ++r)
#pragma unroll
              for (int sj = 0; sj < SEGQ; ++sj) {
                if ((bad >> (r * SEGQ + sj)) & 1u) {
                  const int b = row0 + s_crow[jt * 16 + r];
                  const elem_t* gp = (const elem_t*)a.dA + ((size_t)t * B + b) * H4 + (size_t)wave * H +
                                     sj * (1024 / ESZ) + lane * (16 / ESZ);
                  __builtin_amdgcn_global_load_lds((const void*)gp, (lds_ptr_t)(wbuf + r * QLD + sj * (1024 / ESZ)),
                                                   16, 0, kSc1);
                }
              }
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
            for (int r = 0; r < 16; ++r)
#pragma unroll
              for (int sj = 0; sj < SEGQ; ++sj)
                if (((bad >> (r * SEGQ + sj)) & 1u) &&
                    !pending_granule<PREC>(*(const uint4*)(wbuf + r * QLD + sj * (1024 / ESZ) + lane * (16 / ESZ))))
                  bad &= ~(1u << (r * SEGQ + sj));
          }
        }
        f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f}, acc1 = f32x4{0.f, 0.f, 0.f, 0.f};
        if constexpr (PREC == 0) {
          float4 bcur = *(const float4*)&wbuf[l16 * QLD + 4 * lq], bnxt = bcur;
#pragma unroll
          for (int c = 0; c < KS; ++c) {
            if (c + 1 < KS) bnxt = *(const float4*)&wbuf[l16 * QLD + (c + 1) * 16 + 4 * lq];
            f32x4& acc = (c & 1) ? acc1 : acc0;
            acc = mfma_f32_16x16x4(ureg32[c][0], bcur.x, acc);
            acc = mfma_f32_16x16x4(ureg32[c][1], bcur.y, acc);
            acc = mfma_f32_16x16x4(ureg32[c][2], bcur.z, acc);
            acc = mfma_f32_16x16x4(ureg32[c][3], bcur.w, acc);
            bcur = bnxt;
          }
        } else {
          bf16x8 bcur = *(const bf16x8*)&wbuf[l16 * QLD + 8 * lq], bnxt = bcur;
#pragma unroll
          for (int c = 0; c < KS; ++c) {
            if (c + 1 < KS) bnxt = *(const bf16x8*)&wbuf[l16 * QLD + (c + 1) * 32 + 8 * lq];
            f32x4& acc = (c & 1) ? acc1 : acc0;
            acc = mfma_bf16_16x16x32(ureg16[c], bcur, acc);
            bcur = bnxt;
          }
        }
        const int ci = jt * 16 + l16;
        if (ci < nlive) {
#pragma unroll
          for (int j = 0; j < 4; ++j) red[wave][ci][4 * lq + j] = acc0[j] + acc1[j];
        }
      }
    } else
    for (int jt = 0; jt < NT; ++jt) {
      if (jt * 16 >= nlive) break;
      const int ci = jt * 16 + l16;
      const bool lv = ci < nlive;
      const int r = lv ? s_crow[ci] : 0;
      const size_t rowo = ((size_t)t * B + row0 + r) * H4 + (size_t)wave * H;
      auto fetch = [&](int c) -> uint4 {
        const int kk = c * KC + (PREC ? 8 : 4) * lq;
        const size_t el = rowo + kk;
        if (vec_ok) {
          const uint32_t off = (lv && kk < H) ? (uint32_t)(el * ESZ) : kOOB;
          if (a.coh_rows) return ld_coh_b128(r_dA, off);
          return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r_dA, off, 0, 0));
        }
        uint4 raw;
        uint32_t* rw = (uint32_t*)&raw;
        if constexpr (PREC == 0) {
          for (int j = 0; j < 4; ++j) rw[j] = ld_coh_b32(r_dA, (lv && kk + j < H) ? (uint32_t)((el + j) * 4) : kOOB);
        } else {
          for (int j = 0; j < 4; ++j) {
            uint32_t lo = ld_coh_b16(r_dA, (lv && kk + 2 * j < H) ? (uint32_t)((el + 2 * j) * 2) : kOOB);
            uint32_t hi = ld_coh_b16(r_dA, (lv && kk + 2 * j + 1 < H) ? (uint32_t)((el + 2 * j + 1) * 2) : kOOB);
            rw[j] = lo | (hi << 16);
          }
        }
        return raw;
      };
      // the same granule through agent-scope atomic loads (re-read on every call, L1 bypassed)
      auto fetch_poll = [&](int c) -> uint4 {
        const int kk = c * KC + (PREC ? 8 : 4) * lq;
        const size_t el = rowo + kk;
        const char* base = (const char*)a.dA;
        uint4 raw = uint4{0u, 0u, 0u, 0u};
        if (!lv) return raw;
        if (vec_ok) {
          if (kk < H) raw = ld_poll_b128(base + el * ESZ);
          return raw;
        }
        uint32_t* rw = (uint32_t*)&raw;
        if constexpr (PREC == 0) {
          for (int j = 0; j < 4; ++j)
            if (kk + j < H)
              rw[j] = __hip_atomic_load((uint32_t*)(base + (el + j) * 4), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        } else {
          for (int j = 0; j < 8; ++j) {
            if (kk + j >= H) continue;
            const size_t e = el + j;
            const uint32_t wv = __hip_atomic_load((uint32_t*)(base + (e & ~(size_t)1) * 2), __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
            const uint32_t hv = (e & 1) ? (wv >> 16) : (wv & 0xffffu);
            rw[j >> 1] |= hv << (16 * (j & 1));
          }
        }
        return raw;
      };
      f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f}, acc1 = f32x4{0.f, 0.f, 0.f, 0.f};
      uint4 bufA[CG], bufB[CG];
#pragma unroll
      for (int j = 0; j < CG; ++j) bufA[j] = (j < KS) ? fetch(j) : uint4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        uint4 (&cur)[CG] = (gi & 1) ? bufB : bufA;
        uint4 (&nxt)[CG] = (gi & 1) ? bufA : bufB;
        if (gi + 1 < NG) {
#pragma unroll
          for (int j = 0; j < CG; ++j) nxt[j] = ((gi + 1) * CG + j < KS) ? fetch((gi + 1) * CG + j) : uint4{0u, 0u, 0u, 0u};
        }
        if (a.poll) {
          // granules whose producer's store has not arrived yet are fetched again
          bool any = false;
#pragma unroll
          for (int j = 0; j < CG; ++j)
            if (gi * CG + j < KS && pending_granule<PREC>(cur[j])) any = true;
          if (__builtin_amdgcn_ballot_w64(any)) {
#pragma unroll
            for (int j = 0; j < CG; ++j) {
              const int c = gi * CG + j;
              if (c >= KS) continue;
              int spins = 0;
              while (pending_granule<PREC>(cur[j])) {
                if (spin_out(spins, a.ctl, a.spin_limit)) {
                  s_abort = 1;
                  break;
                }
                cur[j] = fetch_poll(c);
              }
            }
          }
        }
#pragma unroll
        for (int j = 0; j < CG; ++j) {
          const int c = gi * CG + j;
          if (c >= KS) continue;
          f32x4& acc = (j & 1) ? acc1 : acc0;
          if constexpr (PREC == 0) {
            const float4 bv = __builtin_bit_cast(float4, cur[j]);
            acc = mfma_f32_16x16x4(ureg32[c][0], bv.x, acc);
            acc = mfma_f32_16x16x4(ureg32[c][1], bv.y, acc);
            acc = mfma_f32_16x16x4(ureg32[c][2], bv.z, acc);
            acc = mfma_f32_16x16x4(ureg32[c][3], bv.w, acc);
          } else {
            acc = mfma_bf16_16x16x32(ureg16[c], __builtin_bit_cast(bf16x8, cur[j]), acc);
          }
        }
      }
      // lane holds units 4*lq + j of compacted row ci
      if (lv) {
#pragma unroll
        for (int j = 0; j < 4; ++j) red[wave][ci][4 * lq + j] = acc0[j] + acc1[j];
      }
    }
    __syncthreads();
    if (s_abort) break;
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      if (c_op[i] == 1) {
        const int r = prow[i], b = row0 + r;
        const int ci = s_cidx[r];
        const float sdh = red[0][ci][uu] + red[1][ci][uu] + red[2][ci][uu] + red[3][ci][uu];
        if (t > 0 && c_sp[i] + 1 == t) {
          nx_dh[i] += sdh;
        } else if (pok[i]) {
          tg_dh[i] += sdh;
          a.dh_acc[((size_t)(c_sp[i] + 1) * B + b) * H + u] = tg_dh[i];
        }
      }
    }
    if (clk && threadIdx.x == 0) clk[t * 4 + 3] = wall_clock64();
    // rotate: step t-1 becomes current
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      slot_dh[i] = nx_dh[i]; slot_dc[i] = nx_dc[i];
      c_tp[i] = c_sp[i];
      c_op[i] = n_op[i]; c_sp[i] = n_sp[i];
      {
        int op = c_op[i], tp = c_tp[i], sp = c_sp[i];
        valid(t - 1, op, tp, sp);
        c_tp[i] = tp;
      }
      c_gh[i] = n_gh[i]; c_gc[i] = n_gc[i]; c_act[i] = n_act[i]; c_c[i] = n_c[i]; c_cp[i] = n_cp[i];
    }
    __syncthreads();
  }

  // ---- outputs of this workgroup: dh0, dc0 for its pairs; per-group bias gradient
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
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
  const size_t shm = a.bwd_direct ? rec_bwd_lds_bytes(P, KS) : 0;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
  if (e != hipSuccess) return e;
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 256, shm);
  if (e != hipSuccess) return e;
  if (occ_out) *occ_out = occ;
  if (!grid.x) return hipSuccess;
  RecArgs args = a;
  void* kargs[] = {&args};
  return hipLaunchCooperativeKernel((const void*)kern, grid, dim3(256), kargs, (unsigned)shm, st);
}

hipError_t launch_bwd(const RecArgs& a, int prec, int NT, int KS, dim3 grid, hipStream_t st, int* occ_out) {
#define CASE(P, NT_, KS_) if (prec == P && NT == NT_ && KS == KS_) return launch_bwd_t<P, NT_, KS_>(a, grid, st, occ_out);
  REC_CASES(CASE)
#undef CASE
  return hipErrorInvalidValue;
}
