// Pipelined forward kernel of the parallelised StackLSTM (paper, Algorithm 1) for groups of
// two or more 16-row tiles. The arithmetic is that of the plain forward kernel (same work
// split: a group of 16*NT batch rows on the NW workgroups of one XCC, workgroup w owning
// hidden units [16w, 16w+16) with its slice of U in registers); only the schedule differs.
//
// Batch rows are independent of each other, so the tiles of a group form NT independent
// chains. A step runs the tiles one after the other (one pass per tile), and the copy of
// the next tile's h_prev rows into LDS (global_load_lds, the other of two LDS buffers) is
// started three quarters through the current tile's MFMAs: the round trip to L2 and the wait
// for the other workgroups' states overlap with matrix work instead of adding to it. The copy
// of tile 0 for step t+1 starts during the last tile of step t, by when every workgroup has
// long finished tile 0 of step t.
//
// There is no group barrier: the states a workgroup reads from the others are filled with
// all-one bits before the kernel, and a copied granule that still holds them is copied again
// (see common.h). The producer of every state read comes from top[], which the op scan
// filled before the kernel.
#include "common.h"
#include "recurrent.h"
#include "rec_config.h"
#include "rec_device.h"

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// Starts the copy of one tile's 16 h_prev rows (batch rows row_t0 ..) into an LDS buffer:
// every wave moves 16*SEG/4 whole 1 KB row segments, one per instruction (16 bytes a lane).
// The producer step of row r is lane r of srcv. Rows past B copy row B-1 and columns past H
// copy column 0: finite fillers that meet zero U registers or masked outputs.
template <int PREC, int SEG, int LDS_LD>
__device__ __forceinline__ void pipe_copy(const RecArgs& a, void* bufp, int srcv, int row_t0, int wave, int lane) {
  constexpr int ESZ = PREC ? 2 : 4;
  constexpr int NSEG_W = 16 * SEG / 4;
  using elem_t = typename std::conditional<PREC == 1, bf16_t, float>::type;
  elem_t* buf = (elem_t*)bufp;
#pragma unroll
  for (int i = 0; i < NSEG_W; ++i) {
    const int sgi = wave + 4 * i;
    const int r = sgi / SEG, sj = sgi % SEG;
    const int src = __builtin_amdgcn_readlane(srcv, r);
    int k = sj * (1024 / ESZ) + lane * (16 / ESZ);
    if (k >= a.H) k = 0;
    const void* gp = staged_src<PREC>(a, src, min(row_t0 + r, a.B - 1), k);
    __builtin_amdgcn_global_load_lds(gp, (lds_ptr_t)(buf + r * LDS_LD + sj * (1024 / ESZ)), 16, 0, kSc1);
  }
}

// After the copy has landed: every lane checks the granules it copied; a granule that still
// holds the fill is copied again by the lanes that hold one, until all have arrived.
// Returns false when the wait gave up (spin limit or abort flag).
template <int PREC, int SEG, int LDS_LD>
__device__ __forceinline__ bool pipe_complete(const RecArgs& a, void* bufp, int srcv, int row_t0, int wave,
                                              int lane) {
  constexpr int ESZ = PREC ? 2 : 4;
  constexpr int NSEG_W = 16 * SEG / 4;
  static_assert(NSEG_W <= 32, "segment mask is 32 bits");
  using elem_t = typename std::conditional<PREC == 1, bf16_t, float>::type;
  elem_t* buf = (elem_t*)bufp;
  uint32_t bad = 0;
#pragma unroll
  for (int i = 0; i < NSEG_W; ++i) {
    const int sgi = wave + 4 * i;
    const int r = sgi / SEG, sj = sgi % SEG;
    const int src = __builtin_amdgcn_readlane(srcv, r);
    const elem_t* lp = buf + r * LDS_LD + sj * (1024 / ESZ) + lane * (16 / ESZ);
    if (src >= 0 && pending_granule<PREC>(*(const uint4*)lp)) bad |= 1u << i;
  }
  int spins = 0;
  while (__builtin_amdgcn_ballot_w64(bad != 0u)) {
    if (spin_out(spins, a.ctl, a.spin_limit)) return false;
#pragma unroll
    for (int i = 0; i < NSEG_W; ++i) {
      if ((bad >> i) & 1u) {
        const int sgi = wave + 4 * i;
        const int r = sgi / SEG, sj = sgi % SEG;
        const int src = __builtin_amdgcn_readlane(srcv, r);
        int k = sj * (1024 / ESZ) + lane * (16 / ESZ);
        if (k >= a.H) k = 0;
        const void* gp = staged_src<PREC>(a, src, min(row_t0 + r, a.B - 1), k);
        __builtin_amdgcn_global_load_lds(gp, (lds_ptr_t)(buf + r * LDS_LD + sj * (1024 / ESZ)), 16, 0, kSc1);
      }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
    for (int i = 0; i < NSEG_W; ++i) {
      if ((bad >> i) & 1u) {
        const int sgi = wave + 4 * i;
        const int r = sgi / SEG, sj = sgi % SEG;
        const elem_t* lp = buf + r * LDS_LD + sj * (1024 / ESZ) + lane * (16 / ESZ);
        if (!pending_granule<PREC>(*(const uint4*)lp)) bad &= ~(1u << i);
      }
    }
  }
  return true;
}

template <int PREC, int NT, int KS, int OCC>
__global__ void __launch_bounds__(256, OCC) k_fwd_pipe(RecArgs a) {
  constexpr int KC = PREC ? 32 : 16;               // K per chunk
  constexpr int KP = KS * KC;                      // K capacity of the U registers
  constexpr int ESZ = PREC ? 2 : 4;
  constexpr int LDS_LD = rec_lds_ld(PREC, KS);     // LDS row stride (elements), padded
  constexpr int SEG = KP * ESZ / 1024;             // 1 KB segments per row
  constexpr int BUF = 16 * LDS_LD;                 // elements per tile buffer
  constexpr int BG = NT * 16;                      // rows per group
  constexpr int COPY_AT = 3 * KS / 4;              // MFMA chunk at which the next tile's copy starts (measured best of 0, 1/2, 3/4)
  static_assert(SEG >= 1 && NT >= 2 && NT % 2 == 0, "pipelined forward: whole 1 KB segments, an even tile count");
  using elem_t = typename std::conditional<PREC == 1, bf16_t, float>::type;
  extern __shared__ __align__(16) unsigned char smem[];
  elem_t* hs = reinterpret_cast<elem_t*>(smem);  // two tile buffers; tile p of a step uses buffer p % 2
  __shared__ int s_g, s_w;
  // wait failures of the copies of even/odd tiles. Each flag is read right after the barrier
  // that follows its writes, and written again only after a later one.
  __shared__ int s_abort[2];

  claim_group_slot(a.ctl + CTL_XCC_SLOT, a.G, a.NW, &s_g, &s_w);
  const int g = s_g, w = s_w;
  if (g < 0) return;

  const int T = a.T, B = a.B, H = a.H, H4 = 4 * H;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int l16 = lane & 15, lq = lane >> 4;
  const int row0 = g * BG;
  const int unit_base = w * 16 + wave * 4;
  const int u = unit_base + lq;                    // epilogue unit of this lane

  float ureg32[PREC ? 1 : KS][4];
  bf16x8 ureg16[PREC ? KS : 1];
  fwd_load_u<PREC, KS>(a, unit_base, l16, lq, ureg32, ureg16);

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

  // c_prev of tile ti at step ts+1 given its producer s and the state c just produced
  auto next_cp = [&](int ti, int s, int ts, float c) -> float {
    if (s == ts || !lok[ti]) return c;
    const int b = lrow[ti];
    return (s < 0) ? a.c0[(size_t)b * H + u] : a.ccell[((size_t)s * B + b) * H + u];
  };

  // per lane and tile: producer step of row l16, input projection and c_prev of the step
  // whose MFMAs run next (cp_cur of a tile moves to the next step once its cell update ran)
  int src_cur[NT];
  float4 xw_cur[NT];
  float cp_cur[NT];
#pragma unroll
  for (int ti = 0; ti < NT; ++ti) {
    src_cur[ti] = -1;
    xw_cur[ti] = xw_at(0, ti);
    cp_cur[ti] = lok[ti] ? a.c0[(size_t)lrow[ti] * H + u] : 0.f;
  }
  // The cell update of a tile runs one pass after its MFMAs, before the next tile's MFMAs,
  // so that its stores and c_prev loads complete under matrix work: acc_pend holds the gates
  // of the tile waiting for it, xw_last / cp_last the operands of the last tile of a step.
  f32x4 acc_pend = f32x4{0.f, 0.f, 0.f, 0.f};
  float4 xw_last = float4{0.f, 0.f, 0.f, 0.f};
  float cp_last = 0.f;
  bool keep_last = false;                          // the last tile's pending step was a push
  long long stamp[4] = {0, 0, 0, 0};
  if (threadIdx.x < 2) s_abort[threadIdx.x] = 0;
  __syncthreads();
  pipe_copy<PREC, SEG, LDS_LD>(a, hs, src_cur[0], row0, wave, lane);

  long long* clk = a.clk ? a.clk + (size_t)blockIdx.x * T * 4 : nullptr;
  bool stop = false;
  int t = 0;
  for (; t < T && !stop; ++t) {
    const bool more = t + 1 < T;
    float4 xw_nxt[NT];
    int src_nxt[NT];
#pragma unroll
    for (int p = 0; p < NT; ++p) {
      elem_t* buf = hs + (p & 1) * BUF;
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      if (!pipe_complete<PREC, SEG, LDS_LD>(a, buf, src_cur[p], row0 + 16 * p, wave, lane)) s_abort[p & 1] = 1;
      __syncthreads();
      if (s_abort[p & 1]) {
        stop = true;
        break;
      }
      if (clk && threadIdx.x == 0) {
        // profiling stamps: tiles 0 and 1 copied and checked ([0], [2]), their MFMAs done ([1], [3]);
        // the previous step's are stored here, where the MFMAs that follow cover the stores
        if (p == 0 && t > 0) {
#pragma unroll
          for (int k = 0; k < 4; ++k) clk[(t - 1) * 4 + k] = stamp[k];
        }
        if (p < 2) stamp[2 * p] = wall_clock64();
      }
      if (p == 0) {
        // producer indices of step t+1 (top[t]) and the next step's input projection: in
        // flight during this step
#pragma unroll
        for (int ti = 0; ti < NT; ++ti) src_nxt[ti] = top_at(t, ti);
#pragma unroll
        for (int ti = 0; ti < NT; ++ti) xw_nxt[ti] = xw_at(more ? t + 1 : t, ti);
        // deferred cell update of the last tile of step t-1
        if (t > 0) {
          float c = 0.f;
          if (lok[NT - 1]) c = fwd_cell<PREC>(a, acc_pend, xw_last, cp_last, t - 1, lrow[NT - 1], u, keep_last);
          cp_cur[NT - 1] = next_cp(NT - 1, src_cur[NT - 1], t - 1, c);
        }
      } else {
        // deferred cell update of tile p-1 of this step; its producers at step t+1 are needed now
        const int q = p - 1;
        float c = 0.f;
        if (lok[q]) c = fwd_cell<PREC>(a, acc_pend, xw_cur[q], cp_cur[q], t, lrow[q], u, src_nxt[q] == t);
        const int s = more ? checked_src(src_nxt[q], t, a.ctl) : -1;
        src_nxt[q] = s;
        cp_cur[q] = next_cp(q, s, t, c);
      }
      // next copy: tile p+1 of this step, or tile 0 of the next step (harmless after the last step)
      const int nsrc = (p + 1 < NT) ? src_cur[(p + 1) % NT] : src_nxt[0];
      elem_t* nbuf = hs + ((p + 1) & 1) * BUF;
      const int nrow0 = row0 + 16 * ((p + 1) % NT);

      // ---- gates^T (16 cols x 16 rows) = U^T h_prev^T: B fragments read PD chunks ahead, two
      // accumulator chains (even and odd chunks). The fragments of the chunks from COPY_AT on
      // are read into registers first and the next tile's copy is issued right after them: no
      // LDS read of this pass follows the copy, so nothing waits for it before the next pass.
      constexpr int PD = PREC ? 4 : 2;
      constexpr int NPRE = KS - COPY_AT;
      static_assert(COPY_AT >= PD && NPRE >= 1, "copy issued after the read-ahead ring has started");
      f32x4 acc0 = f32x4{0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
      if constexpr (PREC == 0) {
        float4 fr[PD + 1], pre[NPRE];
#pragma unroll
        for (int c = 0; c < PD; ++c) fr[c] = *(const float4*)&buf[l16 * LDS_LD + c * 16 + 4 * lq];
#pragma unroll
        for (int c = 0; c < KS; ++c) {
          if (c + PD < COPY_AT) fr[(c + PD) % (PD + 1)] = *(const float4*)&buf[l16 * LDS_LD + (c + PD) * 16 + 4 * lq];
          if (c == COPY_AT - PD) {
#pragma unroll
            for (int j = 0; j < NPRE; ++j) pre[j] = *(const float4*)&buf[l16 * LDS_LD + (COPY_AT + j) * 16 + 4 * lq];
            pipe_copy<PREC, SEG, LDS_LD>(a, nbuf, nsrc, nrow0, wave, lane);
          }
          f32x4& acc = (c & 1) ? acc1 : acc0;
          const float4 bv = c < COPY_AT ? fr[c % (PD + 1)] : pre[c < COPY_AT ? 0 : c - COPY_AT];
          acc = mfma_f32_16x16x4(ureg32[c][0], bv.x, acc);
          acc = mfma_f32_16x16x4(ureg32[c][1], bv.y, acc);
          acc = mfma_f32_16x16x4(ureg32[c][2], bv.z, acc);
          acc = mfma_f32_16x16x4(ureg32[c][3], bv.w, acc);
        }
      } else {
        bf16x8 fr[PD + 1], pre[NPRE];
#pragma unroll
        for (int c = 0; c < PD; ++c) fr[c] = *(const bf16x8*)&buf[l16 * LDS_LD + c * 32 + 8 * lq];
#pragma unroll
        for (int c = 0; c < KS; ++c) {
          if (c + PD < COPY_AT) fr[(c + PD) % (PD + 1)] = *(const bf16x8*)&buf[l16 * LDS_LD + (c + PD) * 32 + 8 * lq];
          if (c == COPY_AT - PD) {
#pragma unroll
            for (int j = 0; j < NPRE; ++j) pre[j] = *(const bf16x8*)&buf[l16 * LDS_LD + (COPY_AT + j) * 32 + 8 * lq];
            pipe_copy<PREC, SEG, LDS_LD>(a, nbuf, nsrc, nrow0, wave, lane);
          }
          f32x4& acc = (c & 1) ? acc1 : acc0;
          acc = mfma_bf16_16x16x32(ureg16[c], c < COPY_AT ? fr[c % (PD + 1)] : pre[c < COPY_AT ? 0 : c - COPY_AT], acc);
        }
      }
      mfma_drain(acc0, acc1);
      acc_pend = acc0 + acc1;
      if (clk && threadIdx.x == 0 && p < 2) stamp[2 * p + 1] = wall_clock64();
    }
    if (stop) break;

    // producers of the last tile at step t+1, needed by its cell update in the next step's first pass
    keep_last = src_nxt[NT - 1] == t;
    src_nxt[NT - 1] = more ? checked_src(src_nxt[NT - 1], t, a.ctl) : -1;
    xw_last = xw_cur[NT - 1];
    cp_last = cp_cur[NT - 1];
#pragma unroll
    for (int ti = 0; ti < NT; ++ti) {
      xw_cur[ti] = xw_nxt[ti];
      src_cur[ti] = src_nxt[ti];
    }
  }
  if (!stop && T > 0) {
    // the last tile of the last step
    if (lok[NT - 1]) (void)fwd_cell<PREC>(a, acc_pend, xw_last, cp_last, T - 1, lrow[NT - 1], u, keep_last);
    if (clk && threadIdx.x == 0) {
#pragma unroll
      for (int k = 0; k < 4; ++k) clk[(T - 1) * 4 + k] = stamp[k];
    }
  }
  // the copy started for the step after the last one is never read; let it land
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

template <int P, int NT, int KS>
static hipError_t launch_fwd_pipe_t(const RecArgs& a, dim3 grid, hipStream_t st, int* occ_out) {
  constexpr int OCC = rec_occ(P, KS);
  auto kern = k_fwd_pipe<P, NT, KS, OCC>;
  const size_t shm = rec_pipe_lds_bytes(P, KS);
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

hipError_t launch_fwd_pipe(const RecArgs& a, int prec, int NT, int KS, dim3 grid, hipStream_t st, int* occ_out) {
#define CASE(P, NT_, KS_) \
  if (prec == P && NT == NT_ && KS == KS_) return launch_fwd_pipe_t<P, NT_, KS_>(a, grid, st, occ_out);
  REC_PIPE_CASES(CASE)
#undef CASE
  return hipErrorInvalidValue;
}
