// Wide pipelined forward kernel of the parallelised StackLSTM (paper, Algorithm 1) for
// bf16 GEMM operands and hidden sizes above 512 (up to 1024), where a workgroup that owns
// 16 hidden units would need two workgroups per CU and could not keep its U slice in
// registers. Same arithmetic as the other forward kernels; a different work split and
// schedule.
//
// Work split: a group of 16*NT batch rows runs on the NW = ceil(H/32) workgroups of one
// XCC, one workgroup per CU. Workgroup w owns hidden units [32w, 32w+32): wave v owns the
// eight units ub = 32w + 8v .. ub+7, as two 16-row MFMA A tiles of U^T (A tile j, row m =
// unit ub + 2(m/4) + j, gate m%4), so lane (l16, lq) of the output holds all four gates of
// the adjacent units ub + 2lq and ub + 2lq + 1 for batch row l16 of the tile. The U slice
// (128 gate columns x K) stays in registers for the whole kernel; one B fragment read from
// LDS feeds two MFMAs.
//
// Schedule: the NT tiles of a step are independent batch rows and run one pass each; pass
// q = t*NT + p computes tile p of step t from LDS buffer q%3 while the h_prev rows of tile
// q+2 are copied into buffer (q+2)%3 (global_load_lds, 1 KB row segments, L1 bypassed).
// A tile's cell update runs at the start of the next pass (its stores complete under that
// pass's MFMAs). The
// copy of tile q is complete when at most kAfter vector loads are outstanding: every pass
// issues the same sequence of loads, at least kAfter of them after the copy of tile q,
// and loads complete in issue order. No barrier waits for memory: workgroup barriers are
// bare s_barrier instructions (after lgkmcnt(0) where LDS stores must be visible).
//
// Exchange: the bf16 state rows (slot s+1 = step s, slot 0 = h0) start filled with all-one
// bits; a copied granule that still holds them is copied again until the producer's store
// has arrived (see common.h). Producer indices come from the op scan before the kernel, so
// no workgroup keeps the integer stack; they are staged in LDS three steps at a time.
//
// Registers hold the U slice (128 gate columns x K in bf16: 256 per lane at K = 1024,
// pinned to AGPRs) and little else: every per-pass load goes into LDS by DMA (the h_prev
// tiles, the input projection of tiles q+1 and q+2, the c of the state at the top after a
// tile's next update, the producer indices of step t+2), and the per-tile recurrence state
// (c_prev) lives there too. So no register load is pending across passes, and the only
// vector-memory waits are the counted ones.
#include "common.h"
#include "recurrent.h"
#include "rec_config.h"

#pragma clang diagnostic ignored "-Winline-asm"   // M0 is written by the LDS DMA blocks below

typedef unsigned v2u __attribute__((ext_vector_type(2)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));

namespace {

__device__ __forceinline__ void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// Workgroup barrier for LDS data only: it does not wait for global loads or stores.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ void order() { asm volatile("" ::: "memory"); }

__device__ __forceinline__ uint32_t f2u(float f) { return __float_as_uint(f); }
__device__ __forceinline__ void dma4(const void* gp, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off" ::"s"(lds), "v"(gp) : "memory", "m0");
}
__device__ __forceinline__ uint32_t umax3(uint32_t a, uint32_t b, uint32_t c) { return max(max(a, b), c); }


}  // namespace

template <int NT, int KS>
__global__ void __launch_bounds__(256, 1) k_fwd_wide(RecArgs a) {
  constexpr int KC = 32;                          // K per MFMA chunk (bf16)
  constexpr int KP = KS * KC;                     // K capacity of the U registers
  constexpr int LDS_LD = KP + rec_wide_pad;       // LDS row stride (elements), padded
  constexpr int SEG = KP * 2 / 1024;              // 1 KB segments per staged row
  constexpr int BUF = 16 * LDS_LD;                // elements per tile buffer
  constexpr int NBUF = 3, DIST = 2;               // tile buffers; copies run DIST passes ahead
  constexpr int NXS = 3;                          // input-projection slots (tile q in slot q % 3)
  constexpr int CPW = 16 * SEG / 4;               // copy instructions per wave and tile
  constexpr int BG = 16 * NT;                     // rows per group
  constexpr int PD = 6;                           // B fragments read ahead in the MFMA loop
  // Every pass issues, in this order: the copy of tile q+2 (CPW loads), the next update's
  // c source (2 loads) and the input projection of tile q+2 (2 loads); the last pass of a
  // step also fetches producer indices before its copy. The copy of tile q is complete once
  // no more than the loads after it (rest of pass q-2, pass q-1) are pending.
  constexpr int kTail = 4, kPass = kTail + CPW;
  constexpr int kAfter = kTail + (DIST - 1) * kPass;
  static_assert(SEG == 2 && NT >= DIST + 4 && BG <= 256, "wide forward: 2 KB rows, 6+ tiles");
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* hs = reinterpret_cast<bf16_t*>(smem);
  // per tile and lane: c_prev of the tile's next update ([0] x, [1] y) and the c of the state
  // at the top after that update when the update does not produce it ([2] x, [3] y)
  float* st = reinterpret_cast<float*>(smem + (size_t)NBUF * BUF * 2);
  auto stp = [&](int p, int k) -> float* { return st + ((size_t)(p * 4 + k) << 8); };
  // input projection slots: [slot][j][lane] float4 (gates of unit u0 + j)
  float4* xs = reinterpret_cast<float4*>(st + (size_t)NT * 4 * 256);
  auto xsp = [&](int sl, int j) -> float4* { return xs + ((size_t)(sl * 2 + j) << 8); };
  __shared__ int s_top[3][BG];                    // top[s] of the group's rows in slot (s+3)%3
  __shared__ int s_g, s_w, s_abort;

  claim_group_slot(a.ctl + CTL_XCC_SLOT, a.G, a.NW, &s_g, &s_w);
  const int g = uni(s_g), w = uni(s_w);
  if (g < 0) return;

  const int T = a.T, B = a.B, H = a.H, H4 = 4 * H;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = uni(tid >> 6);
  const int l16 = lane & 15, lq = lane >> 4;
  const int row0 = g * BG;
  const int ub = w * 32 + wave * 8;
  const int u0 = ub + 2 * lq;                     // epilogue units u0, u0 + 1 of this lane
  const bool uok = u0 < H;                        // H % 8 == 0: u0 < H implies u0 + 1 < H
  const int uc = uok ? u0 : 0;
  const size_t BH = (size_t)B * H;

  // ---- U^T slice: A tile j, row m = unit ub + 2(m/4) + j, gate m%4; chunk c holds K rows
  // c*32 + 8lq .. +7. Zero past H, so every chunk runs without a branch.
  bf16x8 ureg[2][KS];
  {
    const int gate = l16 & 3;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int unit = ub + 2 * (l16 >> 2) + j;
      const bool ok = unit < H;
      const float* col = a.U + (size_t)gate * H + (ok ? unit : 0);
#pragma unroll
      for (int c = 0; c < KS; ++c) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int k = c * KC + 8 * lq + e;
          ureg[j][c][e] = f32_to_bf16((ok && k < H) ? col[(size_t)k * H4] : 0.f);
        }
        {
          // pinned to AGPRs (MFMA A operands can come from there), which leaves the VGPRs to
          // everything else
          typedef int i32x4 __attribute__((ext_vector_type(4)));
          i32x4 v = __builtin_bit_cast(i32x4, ureg[j][c]);
          asm volatile("" : "+a"(v));
          ureg[j][c] = __builtin_bit_cast(bf16x8, v);
        }
        if ((c & 3) == 3) order();                // bounded number of U loads in flight
      }
    }
  }

  auto slot = [](int s) { return (s + 3) % 3; };

  // producer indices of steps -1 (the initial state), 0 and 1; initial recurrence state
  for (int i = tid; i < BG; i += 256) {
    const int b = min(row0 + i, B - 1);
    s_top[slot(-1)][i] = -1;
    s_top[slot(0)][i] = a.top[b];
    s_top[slot(1)][i] = T > 1 ? a.top[(size_t)B + b] : -1;
  }
  for (int p = 0; p < NT; ++p) {
    const int b = min(row0 + 16 * p + l16, B - 1);
    const float2 c0v = *(const float2*)(a.c0 + (size_t)b * H + uc);
    stp(p, 0)[tid] = c0v.x; stp(p, 1)[tid] = c0v.y;
    stp(p, 2)[tid] = c0v.x; stp(p, 3)[tid] = c0v.y;   // top after step 0: produced there or initial
  }
  if (tid == 0) s_abort = 0;

  // ---- descriptors and per-lane constant offsets
  const rsrc_t r_hx = make_rsrc(a.hx, (size_t)(T + 1) * BH * 2);
  // copy segment i of this wave: row (wave >> 1) + 2i, half wave & 1 of the 2 KB row; the
  // lane's 16 bytes (a column past H reads column 0: finite filler, U registers are 0 there)
  const int sj = wave & 1;
  const uint32_t koff = (uint32_t)((sj * 512 + lane * 8 < H) ? (sj * 512 + lane * 8) * 2 : 0);
  const int rbase = wave >> 1;
  auto copy_tile = [&](int tc, int ptile, int bi) {
    // row r's producer (src = top[tc-1], -1 at tc = 0 and past the last step) in lane r
    const int srcv = (tc == 0 || tc >= T) ? -1 : s_top[slot(tc - 1)][16 * ptile + l16];
    const uint32_t lbuf = lds_addr(hs + bi * BUF + sj * 512);
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int r = rbase + 2 * i;
      const int src = __builtin_amdgcn_readlane(srcv, r);
      const int b = min(row0 + 16 * ptile + r, B - 1);
      const uint32_t soff = (uint32_t)(((src + 1) * B + b) * H) * 2u;
      bdma16_sc1(r_hx, koff, soff, lbuf + (uint32_t)(r * LDS_LD * 2));
    }
  };
  // granules of tile (tc, ptile) in buffer bi that still hold the fill are copied again
  // until every producer's store has arrived; false when the wait gave up. A produced word
  // (two bf16 written by one 4-byte store) is never all-ones, so a granule is pending when
  // its largest word is.
  auto granule = [&](int bi, int i) -> uint4 {
    return *(const uint4*)(hs + bi * BUF + (rbase + 2 * i) * LDS_LD + sj * 512 + lane * 8);
  };
  auto gmax = [](uint4 v) -> uint32_t { return max(umax3(v.x, v.y, v.z), v.w); };
  auto complete_tile = [&](int tc, int ptile, int bi) -> bool {
    uint32_t m = 0;
#pragma unroll
    for (int i = 0; i < CPW; ++i) m = max(m, gmax(granule(bi, i)));
    if (!__builtin_amdgcn_ballot_w64(m == 0xffffffffu)) return true;   // the usual case
    const int srcv = tc == 0 ? -1 : s_top[slot(tc - 1)][16 * ptile + l16];
    const uint32_t lbuf = lds_addr(hs + bi * BUF + sj * 512);
    uint32_t bad = 0;
#pragma unroll
    for (int i = 0; i < CPW; ++i)
      if (gmax(granule(bi, i)) == 0xffffffffu && __builtin_amdgcn_readlane(srcv, rbase + 2 * i) >= 0) bad |= 1u << i;
    int spins = 0;
    while (__builtin_amdgcn_ballot_w64(bad != 0u)) {
      if (spin_out(spins, a.ctl, a.spin_limit)) return false;
#pragma unroll
      for (int i = 0; i < CPW; ++i) {
        if ((bad >> i) & 1u) {
          const int r = rbase + 2 * i;
          const int src = __builtin_amdgcn_readlane(srcv, r);
          const int b = min(row0 + 16 * ptile + r, B - 1);
          bdma16_sc1(r_hx, koff, (uint32_t)(((src + 1) * B + b) * H) * 2u, lbuf + (uint32_t)(r * LDS_LD * 2));
        }
      }
      wait_vm0();
#pragma unroll
      for (int i = 0; i < CPW; ++i)
        if (((bad >> i) & 1u) && gmax(granule(bi, i)) != 0xffffffffu) bad &= ~(1u << i);
    }
    return true;
  };

  // input projection of tile (t, p) into slot sl: this lane's 8 gate pre-activations
  auto xw_fetch = [&](int t, int p, int sl) {
    const int tt = min(t, T - 1);
    const rsrc_t rx = make_rsrc(a.xw + (size_t)tt * B * H4, (size_t)B * H4 * 4);
    const int b = min(row0 + 16 * p + l16, B - 1);
    const uint32_t vo = (uint32_t)(b * H4 + 4 * uc) * 4u;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // earlier reads of the slot have returned
    bdma16(rx, vo, 0u, lds_addr(xsp(sl, 0) + wave * 64));
    bdma16(rx, vo + 16u, 0u, lds_addr(xsp(sl, 1) + wave * 64));
  };
  // the c of the state at the top after step ts+1 when that step does not produce it:
  // produced at a step <= ts by this lane (already stored) or the initial state
  auto c_fetch = [&](int ts, int pe, int topn) {
    const int bc = min(row0 + 16 * pe + l16, B - 1);
    // topn = ts + 1: step ts+1 produces its top itself (a push); the c fetched is unused
    const int sc = checked_src(topn, ts + 1, a.ctl);
    const int sn = sc > ts ? -1 : sc;
    const float* cs = (sn < 0 ? a.c0 : a.ccell) + (uint32_t)((max(sn, 0) * B + bc) * H + uc);
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // earlier reads of the slot have returned
    dma4(cs, lds_addr(stp(pe, 2) + wave * 64));
    dma4(cs + 1, lds_addr(stp(pe, 3) + wave * 64));
  };

  // ---- cell update of tile (te, pe) from its gates; stores through bounds-checked
  // descriptors (a lane outside the batch or the units stores nothing). Returns top[te+1]
  // of the lane's row for the fetch of the next update's state.
  const rsrc_t r_h = make_rsrc(a.hcell, (size_t)T * BH * 4);
  const rsrc_t r_c = make_rsrc(a.ccell, (size_t)T * BH * 4);
  const rsrc_t r_ht = make_rsrc(a.htop, a.htop ? (size_t)T * BH * 4 : 0);
  const rsrc_t r_ct = make_rsrc(a.ctop, a.ctop ? (size_t)T * BH * 4 : 0);
  auto epilogue = [&](int te, int pe, const f32x4 (&acc)[2], int sl, bool live) -> int {
    const int b = row0 + 16 * pe + l16;
    const bool ok = live && uok && b < B;
    const int topv = s_top[slot(te)][16 * pe + l16];
    const int topn = s_top[slot(te + 1)][16 * pe + l16];
    float cp[2] = {stp(pe, 0)[tid], stp(pe, 1)[tid]};
    float pc[2] = {stp(pe, 2)[tid], stp(pe, 3)[tid]};
    // materialised here: a load feeding only a select would become a branch around the load,
    // which would cut the MFMA loop's scheduling region
    asm volatile("" : "+v"(pc[0]), "+v"(pc[1]));
    const float4 xw[2] = {xsp(sl, 0)[tid], xsp(sl, 1)[tid]};
    float hv[2], cv[2], act[2][4];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      act[j][0] = sigmoidf_(acc[j][0] + xw[j].x);
      act[j][1] = sigmoidf_(acc[j][1] + xw[j].y);
      act[j][2] = tanhf_(acc[j][2] + xw[j].z);
      act[j][3] = sigmoidf_(acc[j][3] + xw[j].w);
      cv[j] = act[j][1] * cp[j] + act[j][0] * act[j][2];
      hv[j] = canon_nan(act[j][3] * tanhf_(cv[j]));
    }
    const uint32_t e0 = (uint32_t)b * (uint32_t)H + (uint32_t)u0;   // element of (b, u0) within a step
    const uint32_t o4 = ok ? e0 * 4u : kOOB;
    const uint32_t so4 = (uint32_t)te * (uint32_t)BH * 4u;         // step offsets (< 4 GB)
    const rsrc_t rx = make_rsrc(a.hx + (size_t)(te + 1) * BH, BH * 2);
    const rsrc_t rs = make_rsrc(a.stash + (size_t)te * BH * 4, BH * 16);
    __builtin_amdgcn_raw_buffer_store_b64(v2u{f2u(hv[0]), f2u(hv[1])}, r_h, o4, so4, 0);
    __builtin_amdgcn_raw_buffer_store_b64(v2u{f2u(cv[0]), f2u(cv[1])}, r_c, o4, so4, 0);
    __builtin_amdgcn_raw_buffer_store_b32((uint32_t)f32_to_bf16_bits(hv[0]) | ((uint32_t)f32_to_bf16_bits(hv[1]) << 16),
                                          rx, ok ? e0 * 2u : kOOB, 0, 0);
    // Algorithm 1's return value: the state at the pointer after step te. c_top here; h_top
    // of a push here, of the other steps by a gather after the kernel. The gate activations
    // are kept for a push only (the backward reads no others).
    const bool push = topv == te;
    __builtin_amdgcn_raw_buffer_store_b128(v4u{f2u(act[0][0]), f2u(act[0][1]), f2u(act[0][2]), f2u(act[0][3])}, rs,
                                           ok && push ? e0 * 16u : kOOB, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b128(v4u{f2u(act[1][0]), f2u(act[1][1]), f2u(act[1][2]), f2u(act[1][3])}, rs,
                                           ok && push ? e0 * 16u + 16u : kOOB, 0, 0);
    const float ct0 = push ? cv[0] : pc[0], ct1 = push ? cv[1] : pc[1];
    __builtin_amdgcn_raw_buffer_store_b64(v2u{f2u(hv[0]), f2u(hv[1])}, r_ht, push ? o4 : kOOB, so4, 0);
    __builtin_amdgcn_raw_buffer_store_b64(v2u{f2u(ct0), f2u(ct1)}, r_ct, o4, so4, 0);
    stp(pe, 0)[tid] = live ? ct0 : cp[0];           // step te+1 reads the state at the top
    stp(pe, 1)[tid] = live ? ct1 : cp[1];
    return topn;
  };

  // prologue: copies and input projections of tiles 0 .. DIST-1 of step 0
#pragma unroll
  for (int p = 0; p < DIST; ++p) {
    copy_tile(0, p, p);
    xw_fetch(0, p, p % NXS);
  }

  f32x4 acc_pend[2];
  acc_pend[0] = acc_pend[1] = f32x4{0.f, 0.f, 0.f, 0.f};
  long long* clk = a.clk ? a.clk + (size_t)blockIdx.x * T * 4 : nullptr;
  // One pass per tile, not unrolled: every per-tile value lives in LDS, so the pass body is
  // the same code for every tile.
  const int nq = T * NT;
  int q = 0;
#pragma unroll 1
  for (; q < nq; ++q) {
    const int t = q / NT, p = q - t * NT;
    // ---- tile (t, p) in LDS: loads issued after its copy bound what may still be pending
    if (q < DIST) wait_vm0();
    else wait_vm<kAfter>();
    if (!complete_tile(t, p, q % NBUF)) s_abort = 1;
    lds_barrier();
    if (s_abort) break;
    if (clk && tid == 0 && p == 1) clk[t * 4 + 0] = wall_clock64();
    // producer indices of step t+2 into slot t-1, whose last readers (the copies of this
    // step's tiles and the check above) are done once the last pass of the step starts
    if (p == NT - 1 && tid < BG) {
      const int b = min(row0 + tid, B - 1);
      dma4(a.top + (size_t)min(t + 2, T - 1) * B + b, lds_addr(&s_top[slot(t + 2)][wave * 64]));
    }
    // ---- copy of tile q + DIST into the buffer that tile q-1 used
    {
      const int qn = q + DIST, tn = qn / NT;
      copy_tile(tn, qn - tn * NT, qn % NBUF);
    }
    if (clk && tid == 0 && p == 1) clk[t * 4 + 1] = wall_clock64();
    // ---- gates^T = U^T h_prev^T for tile (t, p), two A tiles per B fragment, interleaved
    // with the cell update of the previous tile (its gates are in acc_pend)
    const bf16_t* buf = hs + (q % NBUF) * BUF;
    f32x4 acc[2];
    acc[0] = acc[1] = f32x4{0.f, 0.f, 0.f, 0.f};
    bf16x8 fr[PD + 1];
#pragma unroll
    for (int c = 0; c < PD; ++c) fr[c] = *(const bf16x8*)&buf[l16 * LDS_LD + c * KC + 8 * lq];
    // (the first pass runs it on the initial values with every store dropped: no branch, so
    // the scheduler can interleave it with the MFMAs)
    const bool live = q > 0;
    const int qe = live ? q - 1 : NT - 1, te = qe / NT, pe = qe - te * NT;
    const int topn = epilogue(te, pe, acc_pend, qe % NXS, live);
    // the scheduler keeps PD fragment reads in flight: PD reads, then one read per MFMA pair
    __builtin_amdgcn_sched_group_barrier(0x100, PD, 0);
#pragma unroll
    for (int c = 0; c < KS; ++c) {
      if (c + PD < KS) fr[(c + PD) % (PD + 1)] = *(const bf16x8*)&buf[l16 * LDS_LD + (c + PD) * KC + 8 * lq];
      const bf16x8 bv = fr[c % (PD + 1)];
      acc[0] = mfma_bf16_16x16x32(ureg[0][c], bv, acc[0]);
      acc[1] = mfma_bf16_16x16x32(ureg[1][c], bv, acc[1]);
      if (c + PD < KS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);   // cell-update ALU work between MFMAs
    }
    acc_pend[0] = acc[0];
    acc_pend[1] = acc[1];
    if (clk && tid == 0 && p == 1) clk[t * 4 + 2] = wall_clock64();
    // ---- the next update's c source for the tile just updated, then the input projection
    // of tile q + DIST (its slot held tile q-1, read by the update above)
    c_fetch(te, pe, live ? topn : -1);            // the first pass fetches the initial c (unused)
    {
      const int qn = q + DIST, tn = qn / NT;
      xw_fetch(tn, qn - tn * NT, qn % NXS);
    }
    if (clk && tid == 0 && p == 1) clk[t * 4 + 3] = wall_clock64();
  }
  if (q == nq && nq > 0) {
    wait_vm0();
    epilogue(T - 1, NT - 1, acc_pend, (nq - 1) % NXS, true);
  }
  // loads started for passes past the last step are never read; let them land
  wait_vm0();
}

template <int NT, int KS>
static hipError_t launch_fwd_wide_t(const RecArgs& a, dim3 grid, hipStream_t st, int* occ_out) {
  auto kern = k_fwd_wide<NT, KS>;
  const size_t shm = rec_wide_lds_bytes(KS, NT);
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

hipError_t launch_fwd_wide(const RecArgs& a, int NT, int KS, dim3 grid, hipStream_t st, int* occ_out) {
  if (NT == 8 && KS == 32) return launch_fwd_wide_t<8, 32>(a, grid, st, occ_out);
  return hipErrorInvalidValue;
}
