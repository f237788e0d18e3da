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
// A tile's cell update runs in the next pass, interleaved with that pass's MFMAs. The
// copy of tile q is complete when at most kAfter vector loads are outstanding: every pass
// issues the same sequence of loads, at least kAfter of them after the copy of tile q,
// and loads complete in issue order. No barrier waits for memory: workgroup barriers are
// bare s_barrier instructions (after lgkmcnt(0) where LDS stores must be visible).
//
// Exchange: the bf16 state rows (slot s+1 = step s, slot 0 = h0) start filled with all-one
// bits; a copied granule that still holds them is copied again until the producer's store
// has arrived (see common.h). Producer indices come from k_trace before the kernel, so no
// workgroup keeps the integer stack; they are staged in LDS three steps at a time.
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

// Waits until at most N vector memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N <= 63, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
  asm volatile("" ::: "memory");
}
__device__ __forceinline__ void wait_vm0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// Workgroup barrier for LDS data only: it does not wait for global loads or stores.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
__device__ __forceinline__ void order() { asm volatile("" ::: "memory"); }

__device__ __forceinline__ uint32_t f2u(float f) { return __float_as_uint(f); }
// LDS DMA written as inline assembly: the compiler then does not order every later LDS
// read behind it with a vmcnt(0) wait (this kernel counts its own waits). M0 holds the
// wave's LDS destination; lane i writes at M0 + i * size. Writing M0 needs one wait state
// before the DMA.
__device__ __forceinline__ void dma16_sc1(const void* gp, const void* lds) {
  const uint32_t m = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off sc1" ::"s"(m), "v"(gp) : "memory", "m0");
}
__device__ __forceinline__ void dma16(const void* gp, const void* lds) {
  const uint32_t m = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(m), "v"(gp) : "memory", "m0");
}
__device__ __forceinline__ void dma4(const void* gp, const void* lds) {
  const uint32_t m = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dword %1, off" ::"s"(m), "v"(gp) : "memory", "m0");
}
// An opaque copy of v: addresses derived from it are computed where they are used instead
// of being hoisted out of the step loop for every unrolled pass (register pressure).
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

constexpr uint32_t kOOB = 0xffffffffu;   // buffer offset past every record: the store is dropped

}  // namespace

template <int NT, int KS>
__global__ void __launch_bounds__(256, 1) k_fwd_wide(RecArgs a) {
  constexpr int KC = 32;                          // K per MFMA chunk (bf16)
  constexpr int KP = KS * KC;                     // K capacity of the U registers
  constexpr int LDS_LD = KP + 8;                  // LDS row stride (elements): 16-byte pad
  constexpr int SEG = KP * 2 / 1024;              // 1 KB segments per staged row
  constexpr int BUF = 16 * LDS_LD;                // elements per tile buffer
  constexpr int NBUF = 3, DIST = 2;               // tile buffers; copies run DIST passes ahead
  constexpr int NXS = 3;                          // input-projection slots (tile q in slot q % 3)
  constexpr int CPW = 16 * SEG / 4;               // copy instructions per wave and tile
  constexpr int BG = 16 * NT;                     // rows per group
  constexpr int PD = 2;                           // B fragments read ahead in the MFMA loop
  // Every pass issues, in this order: the copy of tile q+2 (CPW loads), the next update's
  // c source (2 loads, inside the cell update) and the input projection of tile q+2 (2
  // loads); the first pass of a step also fetches producer indices before its copy. The copy
  // of tile q is complete once no more than the loads after it (rest of pass q-2, pass q-1)
  // are pending.
  constexpr int kTail = 4, kPass = kTail + CPW;
  constexpr int kAfter = kTail + (DIST - 1) * kPass;
  static_assert(SEG >= 1 && NT >= DIST + 4 && BG <= 256, "wide forward: 1 KB segments, 6+ tiles");
  static_assert(16 * SEG <= 32 && CPW <= 32, "segment mask");
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
  const int g = s_g, w = s_w;
  if (g < 0) return;

  const int T = a.T, B = a.B, H = a.H, H4 = 4 * H;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
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

  // rows of this lane: tile p covers rows row0 + 16p .. +15; lane row l16
  auto lrow = [&](int p) { return opaque(row0 + 16 * p + l16); };
  auto slot = [](int s) { return (s + 3) % 3; };

  // producer indices of steps -1 (the initial state), 0 and 1; initial recurrence state
  for (int i = tid; i < BG; i += 256) {
    const int b = min(row0 + i, B - 1);
    s_top[slot(-1)][i] = -1;
    s_top[slot(0)][i] = a.top[b];
    s_top[slot(1)][i] = T > 1 ? a.top[(size_t)B + b] : -1;
  }
  for (int p = 0; p < NT; ++p) {
    const int b = min(lrow(p), B - 1);
    const float2 c0v = *(const float2*)(a.c0 + (size_t)b * H + uc);
    stp(p, 0)[tid] = c0v.x; stp(p, 1)[tid] = c0v.y;
    stp(p, 2)[tid] = c0v.x; stp(p, 3)[tid] = c0v.y;   // top after step 0: produced there or initial
  }
  if (tid == 0) s_abort = 0;

  // input projection of tile (t, p) into slot sl: this lane's 8 gate pre-activations
  auto xw_fetch = [&](int t, int p, int sl) {
    const int tt = min(t, T - 1), b = min(lrow(p), B - 1);
    const float* src = a.xw + ((size_t)tt * B + b) * H4 + 4 * uc;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // earlier reads of the slot have returned
    dma16(src, xsp(sl, 0) + wave * 64);
    dma16(src + 4, xsp(sl, 1) + wave * 64);
  };
#pragma unroll
  for (int p = 0; p < DIST; ++p) xw_fetch(0, p, p % NXS);

  // ---- copy of tile (tc, ptile) into buffer bi: segment i of this wave is row segment
  // wave + 4i; the row's producer comes from the staged trace (src = top[tc-1], -1 at tc = 0;
  // a copy for a step past the end reads the initial rows and is never used)
  auto seg_src = [&](int tc, int ptile, int r) -> int {
    return (tc == 0 || tc >= T) ? -1 : s_top[slot(tc - 1)][16 * ptile + r];
  };
  auto seg_copy = [&](int src, int ptile, int r, int sj, bf16_t* buf) {
    int k = sj * 512 + lane * 8;
    if (k >= H) k = 0;                            // finite filler; U registers are 0 there
    const int b = min(opaque(row0 + 16 * ptile + r), B - 1);
    const bf16_t* gp = a.hx + ((size_t)(src + 1) * B + b) * H + k;
    dma16_sc1(gp, buf + r * LDS_LD + sj * 512);
  };
  auto copy_tile = [&](int tc, int ptile, int bi) {
    bf16_t* buf = hs + bi * BUF;
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int sgi = wave + 4 * i;
      const int r = sgi / SEG, sj = sgi % SEG;
      seg_copy(seg_src(tc, ptile, r), ptile, r, sj, buf);
    }
  };
  // granules of tile (tc, ptile) in buffer bi that still hold the fill are copied again
  // until every producer's store has arrived; false when the wait gave up
  auto complete_tile = [&](int tc, int ptile, int bi) -> bool {
    bf16_t* buf = hs + bi * BUF;
    uint32_t bad = 0;
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int sgi = wave + 4 * i;
      const int r = sgi / SEG, sj = sgi % SEG;
      const uint4 v = *(const uint4*)(buf + r * LDS_LD + sj * 512 + lane * 8);
      if (pending_bf16x8(v) && seg_src(tc, ptile, r) >= 0) bad |= 1u << i;
    }
    int spins = 0;
    while (__builtin_amdgcn_ballot_w64(bad != 0u)) {
      if (spin_out(spins, a.ctl, a.spin_limit)) return false;
#pragma unroll
      for (int i = 0; i < CPW; ++i) {
        if ((bad >> i) & 1u) {
          const int sgi = wave + 4 * i;
          const int r = sgi / SEG, sj = sgi % SEG;
          seg_copy(seg_src(tc, ptile, r), ptile, r, sj, buf);
        }
      }
      wait_vm0();
#pragma unroll
      for (int i = 0; i < CPW; ++i) {
        if ((bad >> i) & 1u) {
          const int sgi = wave + 4 * i;
          const int r = sgi / SEG, sj = sgi % SEG;
          if (!pending_bf16x8(*(const uint4*)(buf + r * LDS_LD + sj * 512 + lane * 8))) bad &= ~(1u << i);
        }
      }
    }
    return true;
  };

  // the c of the state at the top after step ts+1 when that step does not produce it:
  // produced at a step <= ts by this lane (already stored) or the initial state
  auto c_fetch = [&](int ts, int pe, int topn) {
    const int bc = min(lrow(pe), B - 1);
    const int sn = (topn < -1 || topn > ts) ? -1 : topn;
    const size_t off = (size_t)bc * H + uc;
    const float* cs = sn < 0 ? a.c0 + off : a.ccell + (size_t)sn * BH + off;
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // earlier reads of the slot have returned
    dma4(cs, stp(pe, 2) + wave * 64);
    dma4(cs + 1, stp(pe, 3) + wave * 64);
  };

  // ---- cell update of tile (te, pe) from its gates; stores through bounds-checked
  // descriptors (a lane outside the batch or the units stores nothing)
  auto epilogue = [&](int te, int pe, const f32x4 (&acc)[2], int sl) {
    const int b = lrow(pe);
    const bool ok = uok && b < B;
    const int topv = s_top[slot(te)][16 * pe + l16];
    const int topn = s_top[slot(te + 1)][16 * pe + l16];
    const float cp[2] = {stp(pe, 0)[tid], stp(pe, 1)[tid]};
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
    const uint32_t e0 = (uint32_t)b * (uint32_t)H + (uint32_t)u0;   // element of (b, u0)
    const uint32_t o4 = ok ? e0 * 4u : kOOB;
    const uint32_t o2 = ok ? e0 * 2u : kOOB;
    const uint32_t o16 = ok ? e0 * 16u : kOOB;
    const rsrc_t rh = make_rsrc(a.hcell + (size_t)te * BH, BH * 4);
    const rsrc_t rc = make_rsrc(a.ccell + (size_t)te * BH, BH * 4);
    const rsrc_t rx = make_rsrc(a.hx + (size_t)(te + 1) * BH, BH * 2);
    const rsrc_t rs = make_rsrc(a.stash + (size_t)te * BH * 4, BH * 16);
    __builtin_amdgcn_raw_buffer_store_b64(v2u{f2u(hv[0]), f2u(hv[1])}, rh, o4, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b64(v2u{f2u(cv[0]), f2u(cv[1])}, rc, o4, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b32((uint32_t)f32_to_bf16_bits(hv[0]) | ((uint32_t)f32_to_bf16_bits(hv[1]) << 16),
                                          rx, o2, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b128(v4u{f2u(act[0][0]), f2u(act[0][1]), f2u(act[0][2]), f2u(act[0][3])}, rs,
                                           o16, 0, 0);
    __builtin_amdgcn_raw_buffer_store_b128(v4u{f2u(act[1][0]), f2u(act[1][1]), f2u(act[1][2]), f2u(act[1][3])}, rs,
                                           ok ? o16 + 16u : kOOB, 0, 0);
    // Algorithm 1's return value: the state at the pointer after step te. c_top here; h_top
    // of a push here, of the other steps by a gather after the kernel
    const bool push = topv == te;
    const float ct0 = push ? cv[0] : stp(pe, 2)[tid], ct1 = push ? cv[1] : stp(pe, 3)[tid];
    if (a.htop) {
      const rsrc_t rht = make_rsrc(a.htop + (size_t)te * BH, BH * 4);
      __builtin_amdgcn_raw_buffer_store_b64(v2u{f2u(hv[0]), f2u(hv[1])}, rht, push ? o4 : kOOB, 0, 0);
    }
    if (a.ctop) {
      const rsrc_t rct = make_rsrc(a.ctop + (size_t)te * BH, BH * 4);
      __builtin_amdgcn_raw_buffer_store_b64(v2u{f2u(ct0), f2u(ct1)}, rct, o4, 0, 0);
    }
    stp(pe, 0)[tid] = ct0;                          // step te+1 reads the state at the top
    stp(pe, 1)[tid] = ct1;
    c_fetch(te, pe, topn);
  };

  // prologue: copies of tiles 0 .. DIST-1 of step 0 (initial state rows)
#pragma unroll
  for (int p = 0; p < DIST; ++p) copy_tile(0, p, p);

  f32x4 acc_pend[2];
  acc_pend[0] = acc_pend[1] = f32x4{0.f, 0.f, 0.f, 0.f};
  bool stop = false;
  long long* clk = a.clk ? a.clk + (size_t)blockIdx.x * T * 4 : nullptr;
  for (int t = 0; t < T && !stop; ++t) {
#pragma unroll
    for (int p = 0; p < NT; ++p) {
      const int q = t * NT + p;
      // ---- tile (t, p) in LDS: loads issued after its copy bound what may still be pending
      if (t == 0 && p < DIST) wait_vm0();
      else wait_vm<kAfter>();
      if (!complete_tile(t, p, q % NBUF)) s_abort = 1;
      lds_barrier();
      if (s_abort) {
        stop = true;
        break;
      }
      if (clk && tid == 0 && p < 2) clk[t * 4 + 2 * p] = wall_clock64();
      // producer indices of step t+2 into slot t-1, whose last readers (the copies of this
      // step's tiles and the check above) are done once the last pass of the step starts
      if (p == NT - 1 && tid < BG) {
        const int b = min(row0 + tid, B - 1);
        dma4(a.top + (size_t)min(t + 2, T - 1) * B + b, &s_top[slot(t + 2)][wave * 64]);
      }
      // ---- copy of tile q + DIST into the buffer that tile q-1 used
      {
        const int pn = p + DIST;
        copy_tile(pn < NT ? t : t + 1, pn % NT, (q + DIST) % NBUF);
      }
      // ---- gates^T = U^T h_prev^T for tile (t, p): two A tiles share each B fragment
      const bf16_t* buf = hs + (q % NBUF) * BUF;
      f32x4 acc[2];
      acc[0] = acc[1] = f32x4{0.f, 0.f, 0.f, 0.f};
      bf16x8 fr[PD + 1];
#pragma unroll
      for (int c = 0; c < PD; ++c) fr[c] = *(const bf16x8*)&buf[l16 * LDS_LD + c * KC + 8 * lq];
#pragma unroll
      for (int c = 0; c < KS; ++c) {
        if (c + PD < KS) fr[(c + PD) % (PD + 1)] = *(const bf16x8*)&buf[l16 * LDS_LD + (c + PD) * KC + 8 * lq];
        const bf16x8 bv = fr[c % (PD + 1)];
        acc[0] = mfma_bf16_16x16x32(ureg[0][c], bv, acc[0]);
        acc[1] = mfma_bf16_16x16x32(ureg[1][c], bv, acc[1]);
        if (c == 2) {
          // cell update of the previous tile, under this tile's matrix work
          if (p > 0) epilogue(t, p - 1, acc_pend, (q - 1) % NXS);
          else if (t > 0) epilogue(t - 1, NT - 1, acc_pend, (q - 1) % NXS);
          else c_fetch(0, NT - 1, -1);            // same loads as every pass (values unused)
        }
      }
      acc_pend[0] = acc[0];
      acc_pend[1] = acc[1];
      if (clk && tid == 0 && p < 2) clk[t * 4 + 2 * p + 1] = wall_clock64();
      // ---- input projection of tile q + DIST (its slot held tile q-1, read by the update above)
      {
        const int pn = p + DIST;
        xw_fetch(pn < NT ? t : t + 1, pn % NT, (q + DIST) % NXS);
      }
    }
  }
  if (!stop && T > 0) {
    wait_vm0();
    epilogue(T - 1, NT - 1, acc_pend, (T * NT - 1) % NXS);
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
