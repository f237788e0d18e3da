// Persistent backward kernel of the parallelised StackLSTM: back-propagation through
// time over the stack (paper, section 5: the gradient keeps reaching states that were
// popped and later overwritten, because every produced state is kept once).
//
// The reverse sweep walks the stack backwards. Per (row, unit) pair the gradient of the
// state at the top (after step t) is kept in registers, (Gh, Gc); step t's upstream
// gradient dh_top[t], dc_top[t] is added to it. Then, by the op of step t:
//   hold: nothing more (the same state was on top before the step);
//   pop:  the state below came back to the top in forward order, so in reverse the popped
//         state comes back: (Gh, Gc) is stored at the depth of the top, S[p], and the popped
//         state's gradient starts at 0;
//   push: (Gh, Gc) is the produced state's whole gradient. The cell backward gives
//         dA = (dc g i(1-i), dc c_prev f(1-f), dc i (1-g^2), dh tanh(c) o(1-o)) and the
//         parent (depth p-1) becomes the top: (Gh, Gc) = S[p-1] + (dA U^T, dc f).
// S[d] of a state that stays on the stack to the end is 0 (zeroed before the sweep); every
// other S[d] read was stored by the pop of the state above it, at a later step. The most
// recent store is forwarded in registers, older ones are prefetched a step ahead (the lean
// variant below loads the slot at the step instead); no accumulator is read and written in
// the same step.
//
// Same work split as the forward: group of 16*NT rows on one XCC, workgroup w owns
// hidden units [16w, 16w+16) (the lean variant: [32w, 32w+32)). dA U^T needs all 4H gate
// columns, so dA is exchanged
// through L2, with a group barrier per step (each workgroup stores its push rows' dA, arrives,
// waits for the others, then reads every push row of the group). Wave q contracts
// gate columns [qH, (q+1)H) (lean: the q-th eighth of the 4H) against its register-resident
// slice of U and the wave partial sums are added in LDS in a fixed order. Every gradient element is owned by one thread,
// so there are no atomics. Workgroup barriers that only order LDS accesses do not wait for
// outstanding global loads.
//
// Gate-split variant (GS): the contraction is cut over gate columns instead. Workgroup w
// holds U[:, its own 64 gate columns] (the columns its cell backward produces), contracts
// its own dA rows (kept in LDS, no exchange of dA) into partial sums for every unit, stores
// them, and after the group barrier adds the NW partials of its own 16 units in a fixed order
// (quarters of the workgroups, each in workgroup order). Per push row a workgroup then reads
// NW*16 floats (2 KB at H = 512) instead of the row's 4H dA values (8 KB fp32, 4 KB bf16).
// The partials are double-buffered by step parity: a workgroup can be at most one step ahead
// of the slowest reader, since the next barrier waits for it.
#include "common.h"
#include "recurrent.h"
#include "rec_config.h"

#pragma clang diagnostic ignored "-Winline-asm"   // M0 is written by the LDS DMA blocks

namespace {
// Workgroup barrier for LDS data only: it does not wait for global loads or stores.
__device__ __forceinline__ void lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
}  // namespace

// Threads per workgroup: 512 for the lean variant (compiled for OCC = 2, see below), else 256.
constexpr int bwd_threads(int occ) { return occ == 2 ? 512 : 256; }

template <int PREC, int NT, int KS, int OCC, bool GS>
__global__ void __launch_bounds__(bwd_threads(OCC), OCC == 2 ? 1 : OCC) k_bwd(RecArgs a) {
  constexpr int KC = PREC ? 32 : 16;
  constexpr int BG = NT * 16;
  // Lean variant (bf16, K = 32 chunks, i.e. H up to 1024): 256 registers per lane, half of
  // them for the U slice. One workgroup of 512 threads per CU owns 32 hidden units (eight
  // waves; wave q contracts the q-th eighth of the 4H gate columns for both 16-unit halves),
  // so a CU reads every exchanged dA row once (two 256-thread workgroups of 16 units would
  // each read it). It keeps per pair only the top state's gradient in registers; the row
  // state (op and producer of the step, depth), the same for the threads of a row, sits in
  // LDS; each step's operands, and the spill slot a push reads, are loaded at the step (in
  // batches of LB pairs), after every earlier store of the same thread, so the slot's last
  // spill needs no forwarding. The wave partials of each 16-row tile are added in LDS right
  // after the tile, into one sum per (row, unit).
  constexpr bool LEAN = OCC == 2;
  constexpr int NTH = bwd_threads(OCC);           // threads
  constexpr int UPW = LEAN ? 32 : 16;             // hidden units per workgroup
  constexpr int NWV = NTH / 64;                   // waves
  constexpr int MTW = LEAN ? 2 : 1;               // 16-unit M tiles per wave
  constexpr int KW = LEAN ? KS / 2 : KS;          // K chunks per wave (a wave's gate columns)
  constexpr int PAIRS = BG * UPW / NTH;           // (row, unit) pairs per thread
  static_assert(NTH / UPW == 16, "rows r = tid / UPW + 16 i");
  static_assert(!LEAN || (PREC == 1 && KS % 2 == 0 && !GS), "lean: bf16, whole K halves");
  static_assert(BG <= NTH, "one row-info thread per row");
  constexpr int LB = PAIRS < 2 ? PAIRS : 2;
  static_assert(PAIRS % LB == 0, "whole load batches");
  // staged dA rows (direct path): per wave 16 compacted rows of its H gate columns
  constexpr int QLD = rec_lds_ld(PREC, KS);             // row stride (elements), padded
  extern __shared__ __align__(16) unsigned char dsm[];
  __shared__ float red[LEAN ? 1 : 4][LEAN ? 1 : BG][17];
  // lean: the wave partials of a tile (two tiles in turn) and the per-(row, unit) sums
  __shared__ float red_t[LEAN ? 2 : 1][LEAN ? NWV : 1][16][LEAN ? UPW + 1 : 1];
  __shared__ float s_dh[LEAN ? BG : 1][LEAN ? UPW + 1 : 1];
  __shared__ int s_op[BG], s_crow[BG], s_cidx[BG], s_nlive;
  __shared__ float s_db[16][UPW][4];
  __shared__ int s_g, s_w;
  __shared__ int s_abort;                          // a wait for dA rows gave up
  // lean variant: op and producer of each row by step parity, depth of each row
  __shared__ int s_rop[LEAN ? 2 : 1][LEAN ? BG : 1], s_rsp[LEAN ? 2 : 1][LEAN ? BG : 1], s_rdep[LEAN ? BG : 1];
  // GS: this workgroup's dA rows (its 64 gate columns, by row of the group), fp32 or bf16
  constexpr int SDL = PREC ? 72 : 68;                 // row stride (elements): 16-byte pad
  using sd_t = typename std::conditional<PREC == 1, bf16_t, float>::type;
  __shared__ __align__(16) sd_t s_dA[GS ? BG : 1][GS ? SDL : 1];

  claim_group_slot(a.ctl + CTL_XCC_SLOT_B, a.G, a.NW, &s_g, &s_w);
  const int g = s_g, w = s_w;
  if (g < 0) return;

  const int T = a.T, B = a.B, H = a.H, H4 = 4 * H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, lq = lane >> 4;
  const int row0 = g * BG;
  constexpr int ESZ = PREC ? 2 : 4;
  const rsrc_t r_dA = make_rsrc(a.dA, (size_t)T * B * H4 * ESZ);

  // ---- U^T slice: A(m = unit 16w + l16, k = gate column q*H + kk) = U[unit][caller column]
  // (GS: A(m = unit wave*H/4 + mt*16 + l16, k = this workgroup's gate column 64w + kk); the
  // same number of registers: H/64 M tiles of 64 / KC chunks per wave)
  const int a_unit = w * UPW + l16;
  const bool a_ok = a_unit < H;
  const float* Urow = a.U + (size_t)(a_ok ? a_unit : 0) * H4;
  float ureg32[PREC ? 1 : KS][4];
  bf16x8 ureg16[PREC && !LEAN ? KS : 1];
  // lean: wave q's gate columns [kcb, kcb + kspan) of the 4H (an eighth), M tile mt = units
  // w*32 + 16 mt + l16; chunk c holds columns kcb + c*32 + 8lq .. +7
  const int kcb = LEAN ? (wave * H4) / NWV : wave * H;
  const int kspan = LEAN ? ((wave + 1) * H4) / NWV - kcb : H;
  bf16x8 uw[LEAN ? MTW : 1][LEAN ? KW : 1];
  if constexpr (LEAN) {
#pragma unroll
    for (int mt = 0; mt < MTW; ++mt) {
      const int unit = w * UPW + mt * 16 + l16;
      const float* Ur = a.U + (size_t)(unit < H ? unit : 0) * H4;
#pragma unroll
      for (int c = 0; c < KW; ++c) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int kk = c * 32 + 8 * lq + j;
          v[j] = (unit < H && kk < kspan) ? Ur[perm_to_orig(kcb + kk, H)] : 0.f;
        }
        uw[mt][c] = pack_bf16x8(v);
      }
    }
  }
  constexpr int GCH = 64 / KC;                      // GS: K chunks of the own gate columns
  if constexpr (GS) {
    static_assert(KS % GCH == 0 && (KS / GCH) % 2 == 0, "GS: whole M tiles, two at a time");
#pragma unroll
    for (int e = 0; e < KS; ++e) {
      const int mt = e / GCH, ch = e % GCH;
      const int unit = wave * (KS / GCH) * 16 + mt * 16 + l16;
      const float* Ur = a.U + (size_t)(unit < H ? unit : 0) * H4;
      if constexpr (PREC == 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          ureg32[e][j] = unit < H ? Ur[perm_to_orig(w * 64 + ch * 16 + 4 * lq + j, H)] : 0.f;
      } else {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = unit < H ? Ur[perm_to_orig(w * 64 + ch * 32 + 8 * lq + j, H)] : 0.f;
        ureg16[e] = pack_bf16x8(v);
      }
    }
  }
  if constexpr (!GS && !LEAN) {
#pragma unroll
    for (int c = 0; c < KS; ++c) {
      if constexpr (PREC == 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          int kk = c * 16 + 4 * lq + j;
          ureg32[c][j] = (a_ok && kk < H) ? Urow[perm_to_orig(wave * H + kk, H)] : 0.f;
        }
      } else {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          int kk = c * 32 + 8 * lq + j;
          v[j] = (a_ok && kk < H) ? Urow[perm_to_orig(wave * H + kk, H)] : 0.f;
        }
        ureg16[c] = pack_bf16x8(v);
      }
    }
  }

  // ---- this thread's (row, unit) pairs: unit fixed per thread, rows r = tid/UPW + 16 i
  const int uu = threadIdx.x % UPW;
  const int u = w * UPW + uu;
  const int ul = (u < H) ? u : 0;                   // unit used in load addresses (in bounds)
  int prow[PAIRS];
  bool pok[PAIRS];
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    prow[i] = threadIdx.x / UPW + 16 * i;
    pok[i] = (row0 + prow[i] < B) && (u < H);
  }
  // depth after the last step, per pair; the spill slots S[0 .. depth) of the states that
  // stay on the stack to the end start at 0
  int dep[LEAN ? 1 : PAIRS];
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    const int b = pok[i] ? row0 + prow[i] : 0;
    const int d0 = pok[i] ? min(max(a.depth_end[b], 0), T) : 0;
    if constexpr (!LEAN) dep[i] = d0;
    for (int d = 0; d < d0; ++d) {
      const size_t o = ((size_t)d * B + b) * H + u;
      a.dh_acc[o] = 0.f;
      a.dc_acc[o] = 0.f;
    }
  }
  float dbacc[4] = {0.f, 0.f, 0.f, 0.f};
  // 16-byte fetches: whole vectors in every row (lean: also at each wave's first column)
  const bool vec_ok = LEAN ? (H % 16 == 0) : PREC ? (H % 8 == 0) : (H % 4 == 0);
  const bool direct = rec_bwd_direct_built(PREC, NT, KS) && !GS && a.bwd_direct != 0;
  using elem_t = typename std::conditional<PREC == 1, bf16_t, float>::type;
  elem_t* wbuf = reinterpret_cast<elem_t*>(dsm) + (size_t)wave * 16 * QLD;
  if (direct)
    for (int i = threadIdx.x; i < 4 * 16 * QLD * ESZ / 16; i += NTH) ((uint4*)dsm)[i] = uint4{0u, 0u, 0u, 0u};
  if (threadIdx.x == 0) s_abort = 0;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();

  // Loads are issued a step before their values are used. Per pair:
  //   c_*  row info and operands of the current step t;
  //   n_*  row info of step t-1 (fetched during step t+1) and its operands (during step t);
  //   nn_* row info of step t-2 (fetched during step t).
  // The operands are fetched after the step's last wait for dA rows, so no wait of the
  // step includes them.
  auto valid_sp = [&](int t, int& sp) {
    // a producer table that is not the forward's is reported (no access outside [-1, t))
    sp = checked_src(sp, t - 1, a.ctl);
  };
  constexpr int PR = LEAN ? 1 : PAIRS;                   // pairs with row info in registers
  int c_op[PR], c_sp[PR];                                // step t row info
  int n_op[PR], n_sp[PR], nn_op[PR], nn_sp[PR];
  float c_gh[PR], c_gc[PR], c_c[PR], c_cp[PR];
  float4 c_act[PAIRS];
  float n_gh[PR], n_gc[PR], n_c[PR], n_cp[PR];
  float4 n_act[PAIRS];
  // gradient of the top state; last spill (value and depth); spill slot prefetched for a push
  float gh[PAIRS], gc[PAIRS], lh[PR], lc[PR], ph[PR], pc[PR];
  int ld[PR];
  auto ld_row = [&](int t, int b, int& op, int& sp) {
    op = a.ops[(size_t)t * B + b];
    sp = (t == 0) ? -1 : a.top[(size_t)(t - 1) * B + b];
  };
  // the cell operands (gates, c, c_prev) are read for push steps only
  auto ld_ops = [&](int t, int b, int ul, int op, int sp, float& gh_, float& gc_, float4& act, float& c, float& cp) {
    const size_t o = ((size_t)t * B + b) * H + ul;
    // (GS: the operands read once and the dA rows kept for the post-loop GEMMs go through
    // non-temporal accesses, which leaves more of the XCC's L2 to the partial sums that
    // every step rewrites: large fp32 1.41 -> 1.375 ms, 0.88 -> 0.69 GB written per launch)
    if constexpr (GS) {
      gh_ = __builtin_nontemporal_load(a.dh_top + o);
      gc_ = a.dc_top ? __builtin_nontemporal_load(a.dc_top + o) : 0.f;
    } else {
      gh_ = a.dh_top[o];
      gc_ = a.dc_top ? a.dc_top[o] : 0.f;
    }
    if (op == 1) {
      if constexpr (GS) {
        const f32x4 v = __builtin_nontemporal_load((const f32x4*)(a.stash + ((size_t)t * B + b) * H4 + 4 * ul));
        act = float4{v[0], v[1], v[2], v[3]};
      }
      else act = *(const float4*)(a.stash + ((size_t)t * B + b) * H4 + 4 * ul);
      c = a.ccell[o];
      cp = (sp < 0) ? a.c0[(size_t)b * H + ul] : a.ccell[((size_t)sp * B + b) * H + ul];
    }
  };
  // operands of step t-1 and row info of step t-2; the spill slot a push at step t-1 reads
  // (depth dep-1 after this step's update)
  auto prefetch = [&](int t) {
    if constexpr (!LEAN) {
#pragma unroll
      for (int i = 0; i < PAIRS; ++i) {
        const int b = pok[i] ? row0 + prow[i] : 0;
        if (t > 0) {
          ld_ops(t - 1, b, ul, n_op[i], n_sp[i], n_gh[i], n_gc[i], n_act[i], n_c[i], n_cp[i]);
          const size_t so = ((size_t)max(dep[i] - 1, 0) * B + b) * H + ul;
          ph[i] = a.dh_acc[so];
          pc[i] = a.dc_acc[so];
        }
        if (t > 1) ld_row(t - 2, b, nn_op[i], nn_sp[i]);   // validated at the rotation
      }
    }
  };
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    gh[i] = gc[i] = 0.f;
    if constexpr (!LEAN) {
      const int b = pok[i] ? row0 + prow[i] : 0;
      ld_row(T - 1, b, c_op[i], c_sp[i]);
      valid_sp(T - 1, c_sp[i]);
      ld_ops(T - 1, b, ul, c_op[i], c_sp[i], c_gh[i], c_gc[i], c_act[i], c_c[i], c_cp[i]);
      if (T > 1) {
        ld_row(T - 2, b, n_op[i], n_sp[i]);
        valid_sp(T - 2, n_sp[i]);
      }
      lh[i] = lc[i] = 0.f;
      ld[i] = -1;
      // spill slot for a push at step T-1 (the parent sits at depth dep-1): stays-on-stack, 0
      ph[i] = pc[i] = 0.f;
    }
  }
  // lean variant: thread r < BG keeps row r's info of the next step in registers and writes
  // the LDS row state; rows outside the batch hold at depth 0 (no op, nothing stored)
  const int rr = threadIdx.x;
  const bool rr_ok = LEAN && rr < BG && row0 + rr < B;
  int r_nop = 0, r_nsp = -1;
  if constexpr (LEAN) {
    if (rr < BG) {
      int op = 0, sp = -1;
      if (rr_ok) {
        ld_row(T - 1, row0 + rr, op, sp);
        valid_sp(T - 1, sp);
        if (T > 1) ld_row(T - 2, row0 + rr, r_nop, r_nsp);
      }
      s_rop[(T - 1) & 1][rr] = op;
      s_rsp[(T - 1) & 1][rr] = sp;
      s_rdep[rr] = rr_ok ? min(max(a.depth_end[row0 + rr], 0), T) : 0;
    }
    __syncthreads();
  }

  long long* clk = a.clk ? a.clk + (size_t)blockIdx.x * T * 4 : nullptr;
  for (int t = T - 1; t >= 0; --t) {
    if (clk && threadIdx.x == 0) clk[t * 4 + 0] = wall_clock64();
    // lean variant: the pairs' rows and unit come from a copy of the thread index that the
    // compiler cannot see through, so their address terms are recomputed at each step rather
    // than held in registers (spilled) through the loop
    int tq = threadIdx.x;
    if constexpr (LEAN) asm volatile("" : "+v"(tq));
    const int uq = LEAN ? w * UPW + tq % UPW : u;
    const int ulq = uq < H ? uq : 0;
    auto prw = [&](int i) { return LEAN ? tq / UPW + 16 * i : prow[i]; };
    auto pk = [&](int i) { return LEAN ? (row0 + tq / UPW + 16 * i < B) && (uq < H) : pok[i]; };
    // row tables of step t for the compaction (from the registers of the unit-0 threads)
    if (uu == 0 && !LEAN) {
#pragma unroll
      for (int i = 0; i < PR; ++i) {
        s_op[prow[i]] = pok[i] ? c_op[i] : 0;
      }
    }
    lds_sync();
    const int* const op_now = LEAN ? s_rop[t & 1] : s_op;
    if (wave == 0) {
      // list the push rows in row order (wave-wide ballot + prefix count)
      int base = 0;
#pragma unroll
      for (int r0 = 0; r0 < BG; r0 += 64) {
        const int r = r0 + lane;
        const bool live = (r < BG) && (op_now[r] == 1);
        const unsigned long long m = __ballot(live);
        const int ci = base + __builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
        if (live) { s_cidx[r] = ci; s_crow[ci] = r; }
        base += __popcll(m);
      }
      if (lane == 0) s_nlive = base;
    }

    // ---- cell backward for this workgroup's (row, unit) pairs
    // lean variant: the row state and operands of LB pairs (and the spill slot a push reads)
    // are loaded together, then used
    float e_gh[LEAN ? LB : 1], e_gc[LEAN ? LB : 1], e_c[LEAN ? LB : 1], e_cp[LEAN ? LB : 1];
    float e_ph[LEAN ? LB : 1], e_pc[LEAN ? LB : 1];
    float4 e_act[LEAN ? LB : 1];
    int e_op[LEAN ? LB : 1], e_dep[LEAN ? LB : 1];
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      if constexpr (LEAN) {
        if (i % LB == 0) {
#pragma unroll
          for (int j = 0; j < LB; ++j) {
            const int r = prw(i + j);
            const int bl = pk(i + j) ? row0 + r : 0;
            e_op[j] = s_rop[t & 1][r];
            e_dep[j] = s_rdep[r];
            ld_ops(t, bl, ulq, e_op[j], s_rsp[t & 1][r], e_gh[j], e_gc[j], e_act[j], e_c[j], e_cp[j]);
            const size_t so = ((size_t)max(e_dep[j] - 1, 0) * B + bl) * H + ulq;
            e_ph[j] = a.dh_acc[so];
            e_pc[j] = a.dc_acc[so];
          }
        }
      }
      int op_i, dp;
      float o_gh, o_gc, o_c, o_cp, sh, sc;
      float4 o_act;
      if constexpr (LEAN) {
        const int j = i % LB;
        op_i = e_op[j]; dp = e_dep[j];
        o_gh = e_gh[j]; o_gc = e_gc[j]; o_c = e_c[j]; o_cp = e_cp[j]; o_act = e_act[j];
        sh = e_ph[j]; sc = e_pc[j];
      } else {
        op_i = c_op[i]; dp = dep[i];
        o_gh = c_gh[i]; o_gc = c_gc[i]; o_c = c_c[i]; o_cp = c_cp[i]; o_act = c_act[i];
        sh = ph[i]; sc = pc[i];
      }
      float4 dA4 = float4{0.f, 0.f, 0.f, 0.f};
      const int b = row0 + prw(i);
      const bool okp = pk(i);
      // dh_top[t], dc_top[t] belong to the state at the top after step t
      gh[i] += o_gh;
      gc[i] += o_gc;
      if (op_i == 1) {
        // the state produced at step t: its whole gradient is (gh, gc)
        const float4 act = o_act;
        const float dh = gh[i];
        const float tc = tanhf_(o_c);
        const float dc = gc[i] + dh * act.w * (1.f - tc * tc);
        dA4.x = dc * act.z * act.x * (1.f - act.x);
        dA4.y = dc * o_cp * act.y * (1.f - act.y);
        dA4.z = dc * act.x * (1.f - act.z * act.z);
        dA4.w = dh * tc * act.w * (1.f - act.w);
        if (okp) { dbacc[0] += dA4.x; dbacc[1] += dA4.y; dbacc[2] += dA4.z; dbacc[3] += dA4.w; }
        // the parent (depth dep-1) comes back to the top with its spilled gradient plus dc f;
        // dA U^T follows. (Register variants: the last spill if it was to that depth, else
        // the slot prefetched before that spill's store.)
        if constexpr (LEAN) {
          gh[i] = sh;
          gc[i] = sc + dc * act.y;
        } else {
          const bool fwd = ld[i] == dp - 1;
          gh[i] = fwd ? lh[i] : sh;
          gc[i] = (fwd ? lc[i] : sc) + dc * act.y;
        }
        dp -= 1;
      } else if (op_i == -1) {
        // the popped state comes back: the state below is spilled, the popped one starts at 0.
        // The depth stays in [0, T] for the forward's ops; ops that are not the forward's are
        // reported, with no store outside the spill slots. (Pairs outside the batch or the
        // units store nothing.)
        if (dp < 0 || dp > T) {
          if (okp) raise_badidx(a.ctl);
          dp = 0;
        }
        if (okp) {
          const size_t o = ((size_t)dp * B + b) * H + uq;
          a.dh_acc[o] = gh[i];
          a.dc_acc[o] = gc[i];
        }
        if constexpr (!LEAN) {
          lh[i] = gh[i];
          lc[i] = gc[i];
          ld[i] = dp;
        }
        gh[i] = gc[i] = 0.f;
        dp += 1;
      }
      // (lean: every thread of the row computed the same depth; one of them keeps it)
      if constexpr (LEAN) {
        if (uu == 0 && op_i != 0) s_rdep[prw(i)] = dp;
      } else {
        dep[i] = dp;
      }
      if constexpr (GS) {
        // the contraction's operand: this row's dA of the thread's unit (rows the list does
        // not name are never read)
        if constexpr (PREC == 0) {
          *(float4*)&s_dA[prw(i)][4 * uu] = dA4;
        } else {
          bf16_t q[4] = {f32_to_bf16_bits(dA4.x), f32_to_bf16_bits(dA4.y), f32_to_bf16_bits(dA4.z),
                         f32_to_bf16_bits(dA4.w)};
          *(uint2*)&s_dA[prw(i)][4 * uu] = *(const uint2*)q;
        }
      }
      if (okp && op_i == 1) {                   // only push rows are read (exchange, post-loop GEMMs)
        const size_t ao = ((size_t)t * B + b) * H4 + 4 * uq;
        if constexpr (PREC == 0) {
          if constexpr (GS) __builtin_nontemporal_store(f32x4{dA4.x, dA4.y, dA4.z, dA4.w}, (f32x4*)((float*)a.dA + ao));
          else *(float4*)((float*)a.dA + ao) = dA4;
        } else {
          bf16_t q[4] = {f32_to_bf16_bits(dA4.x), f32_to_bf16_bits(dA4.y), f32_to_bf16_bits(dA4.z),
                         f32_to_bf16_bits(dA4.w)};
          *(uint2*)((bf16_t*)a.dA + ao) = *(const uint2*)q;
        }
      }
    }

    if (clk && threadIdx.x == 0) clk[t * 4 + 1] = wall_clock64();
    // byte offset (this wave's gate columns) of the dA row of compacted row r of tile 0, in
    // lane r: computed while the group barrier is in flight
    uint32_t soff0 = 0;
    auto row_offsets0 = [&]() {
      const int cr = lane & 15;
      const int crow0 = cr < s_nlive ? s_crow[cr] : 0;
      soff0 = (((uint32_t)t * B + row0 + crow0) * H4 + wave * H) * ESZ;
    };
    if constexpr (GS) {
      // own dA rows and the row list complete; partial sums of every unit for the listed rows
      lds_sync();
      const int nl = s_nlive;
      // partials of compacted row ci: P[step parity][group][ci][workgroup][unit] (only the listed
      // rows' slots are touched, so a step's partials stay small enough for the XCC's L2)
      float* Pp = a.gs_part + (size_t)((t & 1) * a.G + g) * BG * a.NW * H;
      for (int jt = 0; jt * 16 < nl; ++jt) {
        const int ci = jt * 16 + l16;
        const bool lv = ci < nl;
        const int r = lv ? s_crow[ci] : 0;
        constexpr int MT = KS / GCH;                // M tiles of this wave
        float* prow_p = Pp + ((size_t)ci * a.NW + w) * H + wave * MT * 16 + 4 * lq;
        if constexpr (PREC == 0) {
          float4 bf[GCH];
#pragma unroll
          for (int ch = 0; ch < GCH; ++ch)
            bf[ch] = lv ? *(const float4*)&s_dA[r][ch * 16 + 4 * lq] : float4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int mt = 0; mt < MT; mt += 2) {
            f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
#pragma unroll
            for (int ch = 0; ch < GCH; ++ch) {
              acc0 = mfma_f32_16x16x4(ureg32[mt * GCH + ch][0], bf[ch].x, acc0);
              acc1 = mfma_f32_16x16x4(ureg32[(mt + 1) * GCH + ch][0], bf[ch].x, acc1);
              acc0 = mfma_f32_16x16x4(ureg32[mt * GCH + ch][1], bf[ch].y, acc0);
              acc1 = mfma_f32_16x16x4(ureg32[(mt + 1) * GCH + ch][1], bf[ch].y, acc1);
              acc0 = mfma_f32_16x16x4(ureg32[mt * GCH + ch][2], bf[ch].z, acc0);
              acc1 = mfma_f32_16x16x4(ureg32[(mt + 1) * GCH + ch][2], bf[ch].z, acc1);
              acc0 = mfma_f32_16x16x4(ureg32[mt * GCH + ch][3], bf[ch].w, acc0);
              acc1 = mfma_f32_16x16x4(ureg32[(mt + 1) * GCH + ch][3], bf[ch].w, acc1);
            }
            mfma_drain(acc0, acc1);
            // lane: units 4*lq .. 4*lq+3 of M tiles mt and mt+1, row ci
            if (lv) {
              *(float4*)(prow_p + mt * 16) = float4{acc0[0], acc0[1], acc0[2], acc0[3]};
              *(float4*)(prow_p + (mt + 1) * 16) = float4{acc1[0], acc1[1], acc1[2], acc1[3]};
            }
          }
        } else {
          bf16x8 bf[GCH];
#pragma unroll
          for (int ch = 0; ch < GCH; ++ch) {
            uint4 z = uint4{0u, 0u, 0u, 0u};
            if (lv) z = *(const uint4*)&s_dA[r][ch * 32 + 8 * lq];
            bf[ch] = __builtin_bit_cast(bf16x8, z);
          }
#pragma unroll
          for (int mt = 0; mt < MT; mt += 2) {
            f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
#pragma unroll
            for (int ch = 0; ch < GCH; ++ch) {
              acc0 = mfma_bf16_16x16x32(ureg16[mt * GCH + ch], bf[ch], acc0);
              acc1 = mfma_bf16_16x16x32(ureg16[(mt + 1) * GCH + ch], bf[ch], acc1);
            }
            mfma_drain(acc0, acc1);
            if (lv) {
              *(float4*)(prow_p + mt * 16) = float4{acc0[0], acc0[1], acc0[2], acc0[3]};
              *(float4*)(prow_p + (mt + 1) * 16) = float4{acc1[0], acc1[1], acc1[2], acc1[3]};
            }
          }
        }
      }
      group_arrive(&a.ctl[CTL_BAR_B + g * 16]);
      prefetch(t);
      if (group_wait(&a.ctl[CTL_BAR_B + g * 16], (uint32_t)(a.NW * (T - t)), a.ctl, a.spin_limit, &s_abort)) break;
    } else {
      group_arrive(&a.ctl[CTL_BAR_B + g * 16]);
      if (direct) row_offsets0();
      if (group_wait(&a.ctl[CTL_BAR_B + g * 16], (uint32_t)(a.NW * (T - t)), a.ctl, a.spin_limit, &s_abort)) break;
    }
    if (clk && threadIdx.x == 0) clk[t * 4 + 2] = wall_clock64();
    // Only push rows have non-zero dA. They are listed (in row order) in s_crow and run as
    // compacted 16-row MFMA tiles; each tile's K loop fetches its fragments one group of CG
    // chunks ahead, through the bounds-checked descriptor (a lane past the list or k past H
    // gets an out-of-range offset: value 0, no memory access). Two accumulators per tile
    // keep two independent MFMA chains.
    constexpr int CG = LEAN ? 4 : 8;                // lean: measured fastest (fewer spills)
    constexpr int NG = (KW + CG - 1) / CG;
    const int nlive = s_nlive;
    if (!GS && (!direct || nlive == 0)) prefetch(t);
    // whole 1 KB row segments, at most two per staged row (H of at most 512 fp32 / 1024 bf16);
    // not at two workgroups per CU, where the staged rows do not fit beside the other
    // workgroup's LDS (the host then never asks for it)
    constexpr bool kDirectOk = rec_bwd_direct_built(PREC, NT, KS) && !GS;
    if constexpr (GS) {
      // (the contraction ran before the barrier) The NW workgroups' partial sums of this
      // workgroup's 16 units, per listed row: item (row, quarter q of the workgroups, 4 units)
      // adds its NW/4 partials in workgroup order into red[q]; the four quarters are added as
      // in the other variants. Every item's loads are issued together (one round trip).
      const int NWr = a.NW, WPG = NWr / 4;          // at most 8 (NW <= 32)
      const rsrc_t r_p = make_rsrc(a.gs_part + (size_t)((t & 1) * a.G + g) * BG * NWr * H, (size_t)BG * NWr * H * 4);
      for (int it = threadIdx.x; it < nlive * 16; it += NTH) {
        const int ci = it >> 4, qg = (it >> 2) & 3, q4 = it & 3;
        const uint32_t base = (uint32_t)((((size_t)ci * NWr + qg * WPG) * H + w * 16 + 4 * q4) * 4);
        uint4 v[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = ld_coh_b128(r_p, k < WPG ? base + (uint32_t)(k * H * 4) : kOOB);
        float4 sum = float4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float4 f = __builtin_bit_cast(float4, v[k]);
          sum.x += f.x; sum.y += f.y; sum.z += f.z; sum.w += f.w;
        }
        red[qg][ci][4 * q4] = sum.x;
        red[qg][ci][4 * q4 + 1] = sum.y;
        red[qg][ci][4 * q4 + 2] = sum.z;
        red[qg][ci][4 * q4 + 3] = sum.w;
      }
    } else if (kDirectOk && direct) {
     if constexpr (kDirectOk) {
      // Each wave copies its own H gate columns of the compacted rows straight into its LDS
      // slice (buffer LDS DMA, 1 KB row segments, segment-major: segment s of the tile's rows
      // before segment s+1), waits for its own loads only, and runs the MFMAs of segment s
      // while the later segments are still arriving. Only listed rows are copied: an LDS DMA
      // costs about the same whether its lanes are in range or not. Slots of the rows past
      // the list keep an earlier tile's values, which only reach the MFMA output columns of
      // those rows (discarded). Fragments of the next chunks are read ahead.
      constexpr int SEGQ = KS * KC * ESZ / 1024;          // 1 KB segments per staged row
      constexpr int CPS = 1024 / (KC * ESZ);               // K chunks per segment (16)
      static_assert(SEGQ * CPS == KS && SEGQ <= 2, "whole segments");
      for (int jt = 0; jt < NT; ++jt) {
        if (jt * 16 >= nlive) break;
        // lane r holds the byte offset of the dA row of compacted row jt*16 + r (broadcast per row)
        uint32_t soffv = soff0;
        if (jt > 0) {
          const int crow = (jt * 16 + (lane & 15) < nlive) ? s_crow[jt * 16 + (lane & 15)] : 0;
          soffv = (((uint32_t)t * B + row0 + crow) * H4 + wave * H) * ESZ;
        }
        const int nrows = min(16, nlive - jt * 16);
        const uint32_t lds0 = lds_addr(wbuf);
        // every workgroup of the group reads the same rows in the same order (measured faster
        // than starting each at another row)
#pragma unroll
        for (int sj = 0; sj < SEGQ; ++sj)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            if (r < nrows) {
              const uint32_t soff = (uint32_t)__builtin_amdgcn_readlane((int)soffv, r) + sj * 1024;
              bdma16(r_dA, lane * 16u, soff, lds0 + (uint32_t)((r * QLD + sj * (1024 / ESZ)) * ESZ));
            }
          }
        // segment sj is in LDS once at most nrows * (SEGQ - 1 - sj) DMAs are outstanding; the
        // next step's operands are fetched after the tile's last wait (tile 0 only)
        auto seg_ready = [&](int sj) {
          if (sj == SEGQ - 1) wait_vm<0>();
          else wait_vm_upto16(nrows);   // SEGQ == 2: the second segment's nrows DMAs may be in flight
          if (sj == SEGQ - 1 && jt == 0) prefetch(t);
        };
        f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f}, acc1 = f32x4{0.f, 0.f, 0.f, 0.f};
        // fragments read PD chunks ahead (the scheduler is held to that order); the wait for
        // a segment comes before the first read ahead into it
        constexpr int PD = PREC ? 6 : 3;
        // MFMAs over chunks [C0, C1): its own read-ahead ring, so no read crosses a segment
        // boundary ahead of that segment's wait
        auto run = [&](auto c0_, auto c1_) {
          constexpr int C0 = decltype(c0_)::value, C1 = decltype(c1_)::value, N = C1 - C0;
          if constexpr (PREC == 0) {
            float4 fr[PD + 1];
#pragma unroll
            for (int c = 0; c < PD && c < N; ++c) fr[c] = *(const float4*)&wbuf[l16 * QLD + (C0 + c) * 16 + 4 * lq];
            __builtin_amdgcn_sched_group_barrier(0x100, PD < N ? PD : N, 0);
#pragma unroll
            for (int c = 0; c < N; ++c) {
              if (c + PD < N) fr[(c + PD) % (PD + 1)] = *(const float4*)&wbuf[l16 * QLD + (C0 + c + PD) * 16 + 4 * lq];
              f32x4& acc = (c & 1) ? acc1 : acc0;
              const float4 bcur = fr[c % (PD + 1)];
              acc = mfma_f32_16x16x4(ureg32[C0 + c][0], bcur.x, acc);
              acc = mfma_f32_16x16x4(ureg32[C0 + c][1], bcur.y, acc);
              acc = mfma_f32_16x16x4(ureg32[C0 + c][2], bcur.z, acc);
              acc = mfma_f32_16x16x4(ureg32[C0 + c][3], bcur.w, acc);
              if (c + PD < N) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
            }
          } else {
            bf16x8 fr[PD + 1];
#pragma unroll
            for (int c = 0; c < PD && c < N; ++c) fr[c] = *(const bf16x8*)&wbuf[l16 * QLD + (C0 + c) * 32 + 8 * lq];
            __builtin_amdgcn_sched_group_barrier(0x100, PD < N ? PD : N, 0);
#pragma unroll
            for (int c = 0; c < N; ++c) {
              if (c + PD < N) fr[(c + PD) % (PD + 1)] = *(const bf16x8*)&wbuf[l16 * QLD + (C0 + c + PD) * 32 + 8 * lq];
              f32x4& acc = (c & 1) ? acc1 : acc0;
              acc = mfma_bf16_16x16x32(ureg16[C0 + c], fr[c % (PD + 1)], acc);
              if (c + PD < N) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            }
          }
        };
        seg_ready(0);
        if constexpr (SEGQ == 1) {
          run(std::integral_constant<int, 0>{}, std::integral_constant<int, KS>{});
        } else {
          run(std::integral_constant<int, 0>{}, std::integral_constant<int, CPS>{});
          seg_ready(1);
          run(std::integral_constant<int, CPS>{}, std::integral_constant<int, KS>{});
        }
        const int ci = jt * 16 + l16;
        if (ci < nlive) {
#pragma unroll
          for (int j = 0; j < 4; ++j) red[wave][ci][4 * lq + j] = acc0[j] + acc1[j];
        }
      }
     }
    } else
    for (int jt = 0; jt < NT && !GS; ++jt) {
      if (jt * 16 >= nlive) break;
      const int ci = jt * 16 + l16;
      const bool lv = ci < nlive;
      const int r = lv ? s_crow[ci] : 0;
      const size_t rowo = ((size_t)t * B + row0 + r) * H4 + (size_t)kcb;
      // k bound of this lane (0 past the list): an element at k >= klim gets offset all-ones (out
      // of range: value 0, no access), computed arithmetically so that no per-chunk condition
      // masks are held in scalar registers
      const int klim = lv ? kspan : 0;
      auto oob = [&](int k) -> uint32_t { return (uint32_t)((klim - 1 - k) >> 31); };
      auto fetch = [&](int c) -> uint4 {
        const int kk = c * KC + (PREC ? 8 : 4) * lq;
        const uint32_t el = (uint32_t)(rowo + kk);
        if (vec_ok) {
          const uint32_t off = el * ESZ | oob(kk);
          if (a.coh_rows) return ld_coh_b128(r_dA, off);
          return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r_dA, off, 0, 0));
        }
        uint4 raw;
        uint32_t* rw = (uint32_t*)&raw;
        if constexpr (PREC == 0) {
          for (int j = 0; j < 4; ++j) rw[j] = ld_coh_b32(r_dA, (el + j) * 4 | oob(kk + j));
        } else {
          for (int j = 0; j < 4; ++j) {
            const uint32_t lo = ld_coh_b16(r_dA, (el + 2 * j) * 2 | oob(kk + 2 * j));
            const uint32_t hi = ld_coh_b16(r_dA, (el + 2 * j + 1) * 2 | oob(kk + 2 * j + 1));
            rw[j] = lo | (hi << 16);
          }
        }
        return raw;
      };
      f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f}, acc1 = f32x4{0.f, 0.f, 0.f, 0.f};
      f32x4 accl[LEAN ? MTW : 1][2];
#pragma unroll
      for (int mt = 0; mt < (LEAN ? MTW : 1); ++mt) accl[mt][0] = accl[mt][1] = acc0;
      uint4 bufA[CG], bufB[CG];
#pragma unroll
      for (int j = 0; j < CG; ++j) bufA[j] = (j < KW) ? fetch(j) : uint4{0u, 0u, 0u, 0u};
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
        uint4 (&cur)[CG] = (gi & 1) ? bufB : bufA;
        uint4 (&nxt)[CG] = (gi & 1) ? bufA : bufB;
        if (gi + 1 < NG) {
#pragma unroll
          for (int j = 0; j < CG; ++j) nxt[j] = ((gi + 1) * CG + j < KW) ? fetch((gi + 1) * CG + j) : uint4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int j = 0; j < CG; ++j) {
          const int c = gi * CG + j;
          if (c >= KW) continue;
          f32x4& acc = (j & 1) ? acc1 : acc0;
          if constexpr (LEAN) {
            // one fragment of 16 rows feeds both 16-unit M tiles
#pragma unroll
            for (int mt = 0; mt < MTW; ++mt)
              accl[mt][j & 1] = mfma_bf16_16x16x32(uw[mt][c], __builtin_bit_cast(bf16x8, cur[j]), accl[mt][j & 1]);
          } else if constexpr (PREC == 0) {
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
      if constexpr (LEAN) {
        // lane holds units 16 mt + 4*lq + j of tile row l16; the tile's wave partials (tiles
        // alternate between two buffers: a buffer is written again two tiles later, after the
        // barrier that follows the next tile's writes, by when every thread has summed it)
        const int pb = jt & 1;
        if (lv) {
#pragma unroll
          for (int mt = 0; mt < MTW; ++mt)
#pragma unroll
            for (int j = 0; j < 4; ++j) red_t[pb][wave][l16][mt * 16 + 4 * lq + j] = accl[mt][0][j] + accl[mt][1][j];
        }
        lds_sync();
        const int rs = threadIdx.x / UPW, cs = jt * 16 + rs;
        if (cs < nlive) {
          float sum = 0.f;
#pragma unroll
          for (int q = 0; q < NWV; ++q) sum += red_t[pb][q][rs][uu];
          s_dh[cs][uu] = sum;
        }
      } else if (lv) {
        // lane holds units 4*lq + j of compacted row ci
#pragma unroll
        for (int j = 0; j < 4; ++j) red[wave][ci][4 * lq + j] = acc0[j] + acc1[j];
      }
    }
    lds_sync();
    if (s_abort) break;
    // dA U^T of the push rows: the parent's dh (the parent is now the top)
#pragma unroll
    for (int i = 0; i < PAIRS; ++i) {
      if (pk(i) && (LEAN ? op_now[prw(i)] : c_op[LEAN ? 0 : i]) == 1) {
        const int ci = s_cidx[prw(i)];
        if constexpr (LEAN) gh[i] += s_dh[ci][uu];
        else gh[i] += red[0][ci][uu] + red[1][ci][uu] + red[2][ci][uu] + red[3][ci][uu];
      }
    }
    if (clk && threadIdx.x == 0) clk[t * 4 + 3] = wall_clock64();
    // rotate: step t-1 becomes current
    if constexpr (LEAN) {
      // row info of step t-1 into the other parity's LDS slots (last read during step t+1),
      // then the loads of step t-2's
      if (rr < BG && t > 0) {
        int sp = r_nsp;
        if (rr_ok) valid_sp(t - 1, sp);
        s_rop[(t - 1) & 1][rr] = rr_ok ? r_nop : 0;
        s_rsp[(t - 1) & 1][rr] = rr_ok ? sp : -1;
        if (rr_ok && t > 1) ld_row(t - 2, row0 + rr, r_nop, r_nsp);
      }
    } else {
#pragma unroll
      for (int i = 0; i < PAIRS; ++i) {
        c_op[i] = n_op[i]; c_sp[i] = n_sp[i];
        n_op[i] = nn_op[i]; n_sp[i] = nn_sp[i];
        if (t > 2) valid_sp(t - 2, n_sp[i]);
        c_gh[i] = n_gh[i]; c_gc[i] = n_gc[i]; c_act[i] = n_act[i]; c_c[i] = n_c[i]; c_cp[i] = n_cp[i];
      }
    }
    lds_sync();
  }

  // ---- outputs of this workgroup: dh0, dc0 for its pairs; per-group bias gradient
  // after step 0 the initial state is the top: its gradient is dh0, dc0
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < PAIRS; ++i) {
    if (!pok[i]) continue;
    int b = row0 + prow[i];
    a.dh0[(size_t)b * H + u] = gh[i];
    a.dc0[(size_t)b * H + u] = gc[i];
  }
  const int rgrp = threadIdx.x / UPW;                // 16 row groups share a unit
  for (int j = 0; j < 4; ++j) s_db[rgrp][uu][j] = dbacc[j];
  __syncthreads();
  if (threadIdx.x < UPW * 4) {
    int uu2 = threadIdx.x >> 2, j = threadIdx.x & 3;
    float s = 0.f;
    for (int q = 0; q < 16; ++q) s += s_db[q][uu2][j];
    int u2 = w * UPW + uu2;
    if (u2 < H) a.db_part[(size_t)g * H4 + 4 * u2 + j] = s;
  }
}

template <int P, int NT, int KS, bool GS>
static hipError_t launch_bwd_k(const RecArgs& a, dim3 grid, hipStream_t st, int* occ_out) {
  constexpr int OCC = rec_occ(P, KS);
  auto kern = k_bwd<P, NT, KS, OCC, GS>;
  const size_t shm = (!GS && a.bwd_direct) ? rec_bwd_lds_bytes(P, KS) : 0;
  hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)shm);
  if (e != hipSuccess) return e;
  int occ = 0;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, bwd_threads(OCC), shm);
  if (e != hipSuccess) return e;
  if (occ_out) *occ_out = occ;
  if (!grid.x) return hipSuccess;
  RecArgs args = a;
  void* kargs[] = {&args};
  return hipLaunchCooperativeKernel((const void*)kern, grid, dim3(bwd_threads(OCC)), kargs, (unsigned)shm, st);
}

template <int P, int NT, int KS>
static hipError_t launch_bwd_t(const RecArgs& a, dim3 grid, hipStream_t st, int* occ_out) {
  if constexpr (rec_bwd_gs_built(P, NT, KS)) {
    if (a.bwd_gs) return launch_bwd_k<P, NT, KS, true>(a, grid, st, occ_out);
  } else {
    if (a.bwd_gs) return hipErrorInvalidValue;
  }
  return launch_bwd_k<P, NT, KS, false>(a, grid, st, occ_out);
}

hipError_t launch_bwd(const RecArgs& a, int prec, int NT, int KS, dim3 grid, hipStream_t st, int* occ_out) {
#define CASE(P, NT_, KS_) if (prec == P && NT == NT_ && KS == KS_) return launch_bwd_t<P, NT_, KS_>(a, grid, st, occ_out);
  REC_CASES(CASE)
#undef CASE
  return hipErrorInvalidValue;
}
