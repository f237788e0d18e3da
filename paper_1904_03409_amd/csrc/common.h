// Shared device helpers for the StackLSTM HIP library (gfx950 / CDNA4).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;  // raw bfloat16 bits in memory

// Status codes shared with the C-ABI (values fixed by include/stacklstm.h).
enum {
  ST_OK = 0, ST_EINVAL = 1, ST_EOPS = 2, ST_EUNDERFLOW = 3, ST_EWORKSPACE = 4,
  ST_ENORESIDENT = 5, ST_EDEVICE = 6, ST_ETIMEOUT = 7, ST_EINDEX = 8
};

// CTL_STATUS while every op is valid.
constexpr uint32_t kStatusOk = 0x7fffffffu;

// Work-space word offsets (uint32 units) of the control block at the start of the work space.
enum {
  CTL_STATUS = 0,        // lowest (element * 8 + code) of a failing element, or 0x7fffffff
  CTL_MAXDEPTH = 1,
  CTL_ABORT = 2,         // set when a wait ran out of spins: every workgroup leaves its loop
  CTL_TIMEOUT = 3,       // set when a wait ran out of spins (reported as SLSTM_ETIMEOUT)
  CTL_NPUSH = 4,         // number of push rows (written by k_push_rows in the backward)
  CTL_NPUSHF = 5,        // number of push rows (counted by k_scan in the forward)
  CTL_BADIDX = 6,        // set when a kernel read a producer index outside its valid range
  CTL_XCC_SLOT = 16,     // 16 per-XCC slot counters (forward kernel)
  CTL_XCC_SLOT_B = 32,   // 16 per-XCC slot counters (backward kernel)
  CTL_BAR_F = 64,        // forward group barrier counters, one 64-byte line per group
  CTL_BAR_B = 64 + 16 * 64,   // backward group barrier counters
  CTL_WORDS = 64 + 2 * 16 * 64
};
#define MAX_GROUPS 64

// Gate-interleaved ("permuted") column order used inside the library: column 4*u + k
// holds gate k (0=i, 1=f, 2=g, 3=o) of hidden unit u. The caller's order is k*H + u.
__device__ __forceinline__ int perm_to_orig(int np, int H) { return (np & 3) * H + (np >> 2); }

__device__ __forceinline__ float bf16_bits_to_f32(bf16_t v) {
  return __uint_as_float(((uint32_t)v) << 16);
}
// Round to bfloat16, nearest-even (the hardware conversion on gfx950).
__device__ __forceinline__ __bf16 f32_to_bf16(float f) { return static_cast<__bf16>(f); }
__device__ __forceinline__ bf16_t f32_to_bf16_bits(float f) {
  __bf16 h = static_cast<__bf16>(f);
  return __builtin_bit_cast(bf16_t, h);
}

// Eight floats rounded to bf16 (nearest-even) in pairs, packed as they are converted.
__device__ __forceinline__ bf16x8 pack_bf16x8(const float (&v)[8]) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  u32x4 w;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    w[j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{v[2 * j], v[2 * j + 1]}, bf16x2));
  // (an empty asm on the packed words keeps the compiler from sinking the conversions to the
  // first use, which would keep all the fp32 values live through the set-up)
  asm volatile("" : "+v"(w));
  return __builtin_bit_cast(bf16x8, w);
}

__device__ __forceinline__ f32x4 mfma_f32_16x16x4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_bf16_16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
// Results of an MFMA chain in AGPRs may be read only some wait states after its last
// instruction (10 for the fp32 16x16x4 form, 8 for the bf16 16x16x32 form: the counts the
// compiler itself inserts in straight-line code). The compiler's hazard pass misses them on
// a branch edge that leaves the MFMA's block (measured: 3 wait states on the taken path
// round a conditional store, and the fourth accumulator read stale). This drain issues 12
// wait states after the chain, as an asm statement that takes the accumulators as operands
// and so runs after the chain's last MFMA and before any read of its results; the compiler
// sees the asm, not an MFMA, as their last writer.
__device__ __forceinline__ void mfma_drain(f32x4& a, f32x4& b) {
  asm volatile("s_nop 7\n\ts_nop 3" : "+a"(a), "+a"(b));
}

// Gate nonlinearities from the hardware base-2 exponential and reciprocal (about one ulp
// each): sigma(z) = 1 / (1 + 2^(-z log2 e)); tanh(x) = 2 sigma(2x) - 1. Absolute error is
// a few 1e-7 over the whole range; both saturate correctly (2^(+inf) = inf gives 0, 2^(-inf)
// = 0 gives 1) and need no branch.
__device__ __forceinline__ float sigmoidf_(float z) {
  return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-1.4426950408889634f * z));
}
__device__ __forceinline__ float tanhf_(float x) {
  return 2.f * __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-2.8853900817779268f * x)) - 1.f;
}

__device__ __forceinline__ unsigned xcc_id() {
  unsigned v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 0xf;
}

// Loads of data that another CU wrote earlier in the same kernel. They go through a
// buffer descriptor (bounds-checked: an offset past `bytes` reads 0 instead of faulting)
// with the sc1 cache policy, which bypasses this CU's L1 and reads the XCC's L2, so a
// line that L1 cached before the other CU's write is never returned stale.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
__device__ __forceinline__ rsrc_t make_rsrc(const void* base, size_t bytes) {
  uint32_t n = bytes > 0xffffffffu ? 0xffffffffu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}
constexpr int kSc1 = 16;  // cache-policy bit SC1 of gfx94x/gfx950 memory instructions
__device__ __forceinline__ uint4 ld_coh_b128(rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kSc1));
}
__device__ __forceinline__ uint32_t ld_coh_b32(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kSc1);
}
__device__ __forceinline__ uint16_t ld_coh_b16(rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, kSc1);
}

// Barrier-free exchange of states between the workgroups of one XCC. Before the kernel
// the exchanged rows are filled with all-one bits (a NaN no producer ever stores: produced
// NaNs are stored as the canonical quiet NaN); a consumer reads a row, and re-reads every
// 16-byte granule that still holds the fill, with agent-scope atomic loads (never hoisted
// or merged by the compiler, and they miss in this CU's L1), until the producer's store has
// reached the XCC's L2.
__device__ __forceinline__ bool pending_f32x4(uint4 v) {
  return v.x == 0xffffffffu || v.y == 0xffffffffu || v.z == 0xffffffffu || v.w == 0xffffffffu;
}
__device__ __forceinline__ bool pending_bf16_word(uint32_t w) {
  return (w & 0xffffu) == 0xffffu || (w >> 16) == 0xffffu;
}
__device__ __forceinline__ bool pending_bf16x8(uint4 v) {
  return pending_bf16_word(v.x) || pending_bf16_word(v.y) || pending_bf16_word(v.z) || pending_bf16_word(v.w);
}
template <int PREC>
__device__ __forceinline__ bool pending_granule(uint4 v) {
  if constexpr (PREC == 0) return pending_f32x4(v);
  else return pending_bf16x8(v);
}
__device__ __forceinline__ uint4 ld_poll_b128(const void* p) {
  const uint64_t* q = (const uint64_t*)p;
  uint64_t lo = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  uint64_t hi = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return uint4{(uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32)};
}
__device__ __forceinline__ float canon_nan(float h) { return h == h ? h : __builtin_nanf(""); }

// A producer index s read at step t must lie in [-1, t) (the state read at step t) or
// [-1, t] (the state at the top after step t). An index outside its range means that the
// producer table passed in was not the forward's, or that a read returned stale data: the
// kernel raises CTL_BADIDX (the call then reports SLSTM_EINDEX), and uses -1 so that every
// access stays inside the arrays.
__device__ __forceinline__ void raise_badidx(uint32_t* ctl) {
  __hip_atomic_store(&ctl[CTL_BADIDX], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int checked_src(int s, int hi, uint32_t* ctl) {
  if (s < -1 || s > hi) {
    raise_badidx(ctl);
    return -1;
  }
  return s;
}

// Bounded wait: counts failed polls of one wait; gives up (returns true) when the count
// reaches the limit, raising the abort and time-out flags, or when another workgroup has
// raised the abort flag.
__device__ __forceinline__ bool spin_out(int& spins, uint32_t* ctl, int spin_limit) {
  ++spins;
  if (spins >= spin_limit) {
    __hip_atomic_store(&ctl[CTL_ABORT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&ctl[CTL_TIMEOUT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return true;
  }
  return (spins & 255) == 0 && __hip_atomic_load(&ctl[CTL_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Group barrier for workgroups that all run on one XCC (one shared L2).
// Each wave waits until its own stores are acknowledged by L2, the workgroup meets at
// s_barrier, one lane adds to the group counter and polls it with L1-bypassing loads.
// Data written by other workgroups before the barrier must then be read with the
// ld_coh_* loads above. Returns true when the spin limit ran out (or another group's
// did): the caller must then leave its loop so that every wave of the grid exits.
// Arrival half: stores acknowledged, workgroup met, the group counter incremented.
__device__ __forceinline__ void group_arrive(uint32_t* ctr) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Waiting half: one lane polls the counter up to target; returns true when the spin limit
// ran out or another workgroup gave up. Work that needs no other workgroup's data can run
// between the two halves.
__device__ __forceinline__ bool group_wait(uint32_t* ctr, uint32_t target, uint32_t* ctl, int spin_limit,
                                           int* s_flag) {
  if (threadIdx.x == 0) {
    int spins = 0, bad = 0;
    while (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      ++spins;
      if ((spins & 255) == 0 && __hip_atomic_load(&ctl[CTL_ABORT], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        bad = 1;
        break;
      }
      if (spins > spin_limit) {
        __hip_atomic_store(&ctl[CTL_ABORT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&ctl[CTL_TIMEOUT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        bad = 1;
        break;
      }
    }
    *s_flag = bad;
  }
  __syncthreads();
  return *s_flag != 0;
}
__device__ __forceinline__ bool group_barrier(uint32_t* ctr, uint32_t target, uint32_t* ctl, int spin_limit,
                                              int* s_flag) {
  group_arrive(ctr);
  return group_wait(ctr, target, ctl, spin_limit, s_flag);
}

// Claims this workgroup's (group, member) slot from the XCC it runs on, so that every
// group's members share one XCC. Groups are dealt to XCCs round-robin (group g on XCC
// g % 8); a workgroup with nothing to do gets group -1 and must exit.
__device__ __forceinline__ void claim_group_slot(uint32_t* slot_ctrs, int G, int NW, int* s_g, int* s_w) {
  if (threadIdx.x == 0) {
    unsigned x = xcc_id();
    int g = -1, w = 0;
    if (x < 8) {
      unsigned slot = __hip_atomic_fetch_add(&slot_ctrs[x], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      int per_xcc = NW * ((G + 7) / 8);
      if ((int)slot < per_xcc) {
        int lg = (int)slot / NW;
        w = (int)slot % NW;
        g = lg * 8 + (int)x;
        if (g >= G) g = -1;
      }
    }
    *s_g = g;
    *s_w = w;
  }
  __syncthreads();
}

// LDS DMA (global memory -> LDS, 16 bytes or 4 bytes per lane) written as inline assembly:
// the compiler then does not order every later LDS read behind it with a vmcnt(0) wait; a
// kernel that uses these counts its own waits. M0 holds the wave's LDS destination (lane i
// writes at M0 + i * size); writing M0 needs one wait state before the DMA. The buffer
// forms address descriptor base + soff (wave-uniform) + voff (the lane's offset, the only
// part the descriptor's range check covers).
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }
// Buffer form: address = descriptor base + soff (wave-uniform) + voff (the lane's offset,
// the only part the descriptor's range check covers: a lane given kOOB reads no memory and
// writes zeros to its 16 LDS bytes). sc1 bypasses this CU's L1. An instruction immediate
// offset would move the LDS address as well (M0 + immediate + 16 * lane); these forms use none.
constexpr uint32_t kOOB = 0xffffffffu;
__device__ __forceinline__ void bdma16_sc1(rsrc_t r, uint32_t voff, uint32_t soff, uint32_t lds) {
  lds = __builtin_amdgcn_readfirstlane(lds);   // wave-uniform by contract: kept in SGPRs
  soff = __builtin_amdgcn_readfirstlane(soff);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen sc1 lds"
               ::"s"(lds), "v"(voff), "s"(r), "s"(soff) : "memory", "m0");
}
__device__ __forceinline__ void bdma16(rsrc_t r, uint32_t voff, uint32_t soff, uint32_t lds) {
  lds = __builtin_amdgcn_readfirstlane(lds);   // wave-uniform by contract: kept in SGPRs
  soff = __builtin_amdgcn_readfirstlane(soff);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               ::"s"(lds), "v"(voff), "s"(r), "s"(soff) : "memory", "m0");
}
// Waits until at most N vector memory operations of this wave are outstanding (they
// complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N <= 63, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
  asm volatile("" ::: "memory");
}
// The same for a wave-uniform count n in [0, 16] (n outside it waits for all).
__device__ __forceinline__ void wait_vm_upto16(int n) {
  switch (n) {
#define SLSTM_WAIT_CASE(k) case k: wait_vm<k>(); break;
    SLSTM_WAIT_CASE(1) SLSTM_WAIT_CASE(2) SLSTM_WAIT_CASE(3) SLSTM_WAIT_CASE(4) SLSTM_WAIT_CASE(5)
    SLSTM_WAIT_CASE(6) SLSTM_WAIT_CASE(7) SLSTM_WAIT_CASE(8) SLSTM_WAIT_CASE(9) SLSTM_WAIT_CASE(10)
    SLSTM_WAIT_CASE(11) SLSTM_WAIT_CASE(12) SLSTM_WAIT_CASE(13) SLSTM_WAIT_CASE(14) SLSTM_WAIT_CASE(15)
    SLSTM_WAIT_CASE(16)
#undef SLSTM_WAIT_CASE
    default: wait_vm<0>(); break;
  }
}
// Wave-uniform value kept in a scalar register.
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ void dma16_global(const void* gp, uint32_t lds, bool sc1) {
  lds = __builtin_amdgcn_readfirstlane(lds);   // wave-uniform by contract; keeps it in an SGPR
  if (sc1)
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off sc1" ::"s"(lds), "v"(gp) : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(gp) : "memory", "m0");
}
