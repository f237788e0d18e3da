// Host side of the StackLSTM library: argument checks, work-space layout, launch
// configuration and the launch order of the forward and backward passes.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>
#include <algorithm>
#include <mutex>

#include "../../include/stacklstm.h"
#include "common.h"
#include "gemm.h"
#include "rec_config.h"
#include "recurrent.h"

__global__ void k_init_ctl(uint32_t* ctl, int keep_errors);
template <bool LDS>
__global__ void k_scan(const int8_t* ops, int T, int B, int cap, int32_t* ptr, int32_t* top, int32_t* depth_end,
                       int32_t* gstack, uint32_t* ctl);
__global__ void k_gather_top(const int32_t* top, const float* cellv, const float* init, float* out, int T, int B,
                             int H, int skip_push, uint32_t* ctl);
__global__ void k_gather_top4(const int32_t* top, const float* hcell, const float* h0, float* htop, const float* ccell,
                              const float* c0, float* ctop, int T, int B, int H, int skip_h, uint32_t* ctl);
__global__ void k_permute_w(const float* W, float* Wp32, bf16_t* Wp16, bf16_t* WpT16, int I, int H);
__global__ void k_fill_f32(float* p, size_t n, float v);
__global__ void k_zero_u32(uint32_t* p, int n);
__global__ void k_zero_ctl_bwd(uint32_t* ctl, int keep_errors);
__global__ void k_fill_pattern(unsigned char* p, size_t bytes, uint32_t v);
__global__ void k_h0_bf16(const float* h0, bf16_t* hx, size_t n);
__global__ void k_to_bf16x8(const float* in, bf16_t* out, size_t n8);
__global__ void k_push_rows(const int8_t* ops, int n, int32_t* rows, uint32_t* count);
__global__ void k_zero_nonpush_rows(const int8_t* ops, float* out, size_t n, int cols);
__global__ void k_gather_hprev(const int32_t* top, const float* hcell, const float* h0, const int32_t* prow,
                               const uint32_t* count, float* out, int T, int B, int H, uint32_t* ctl);
__global__ void k_transpose_bf16(const void* src, int src_f32, int ld, int cols, const int32_t* prow,
                                 const uint32_t* count, int ldo, const int32_t* gtop, int B, bf16_t* out, uint32_t* ctl);
template <int PREC, int AL, int BL> __global__ void k_gemm(GemmArgs g);
__global__ void k_gemm_wide(GemmArgs g);
__global__ void k_gemm_ring(GemmArgs g);
__global__ void k_reduce_splits(const float* P, int splits, size_t split_stride, int M, int N, int unperm_H,
                                float* out);
__global__ void k_scatter_splits(const float* P, const int32_t* rows, const uint32_t* count, size_t max_rows, int N,
                                 int grid_blocks, int n_tiles, float* dst);

namespace {

constexpr int kDefaultSpin = 1 << 22;
constexpr int kGemmBM = 128, kGemmBN = 128, kGemmBK = 64;

struct DevInfo { int cus; bool ok; };

int device_cus() {
  static std::mutex mu;
  static DevInfo info[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  std::lock_guard<std::mutex> lk(mu);
  if (!info[dev].ok) {
    hipDeviceProp_t p;
    if (hipGetDeviceProperties(&p, dev) != hipSuccess) return 0;
    info[dev].cus = p.multiProcessorCount;
    info[dev].ok = true;
  }
  return info[dev].cus;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
bool al16(const void* q) { return ((uintptr_t)q & 15u) == 0; }

// Rows per group are chosen per kernel (forward and backward differ in register use and so
// in how many workgroups share a CU): NT/G/per_xcc for the forward, NTb/Gb/per_xcc_b for
// the backward.
struct Plan {
  int prec, KS, ks_eff, NW;
  int NT, G, per_xcc, pipe;   // pipe: the forward runs the pipelined kernel
  int fuse, kx;               // fuse: the plain bf16 forward contracts x_t W itself (kx chunks of 32)
  int wide, NWw;              // wide: the forward runs the 32-unit kernel (NWw workgroups per group)
  int NTb, Gb, per_xcc_b, NWb; // NWb: backward workgroups per group (32 units each in the lean variant)
  int gs;                     // the backward runs the gate-split contraction
  int splits_w, splits_u;
};

struct Layout {
  size_t ctl, stack, dep, wp, r1, stash, hx, fwd_end, xbt, hp, dat, dh, dc, dbp, part, prow, total;
};

Layout layout(const slstm_dims* d);

// Push-row count padded to the K tile: leading dimension of the transposed bf16 operands
size_t padded_rows(const slstm_dims* d) { return ((size_t)d->T * d->B + 63) / 64 * 64; }

bool dims_ok(const slstm_dims* d) {
  if (!d) return false;
  if (d->T < 0 || d->B < 1 || d->I < 1 || d->H < 1) return false;
  if (d->precision != SLSTM_FP32 && d->precision != SLSTM_BF16_GEMM) return false;
  if (d->H > (d->precision == SLSTM_FP32 ? 512 : 1024)) return false;
  if ((int64_t)d->T * d->B > ((int64_t)1 << 28)) return false;
  // the persistent kernels address T*B*4H fp32 (fp32 mode) or bf16 values with 32-bit byte offsets
  const int64_t esz = d->precision == SLSTM_FP32 ? 4 : 2;
  if ((int64_t)d->T * d->B * 4 * d->H * esz >= ((int64_t)1 << 32)) return false;
  if ((int64_t)d->T * d->B * d->H * 4 >= ((int64_t)1 << 32)) return false;
  return true;
}

int ks_bucket(int prec, int ks_eff) {
  const int lo = prec ? 2 : 4;
  int ks = lo;
  while (ks < ks_eff) ks *= 2;
  return ks <= 32 ? ks : -1;
}

// Split-K slices of dW / dU: about 512 blocks, one round of the GEMM's two workgroups per CU
// on 256 CUs (measured at large: 1024 blocks 0.26 / 0.37 ms fp32 dW + db / dU, 512 blocks
// 0.24 / 0.36 ms, 384 or 256 blocks slower; bf16 0.13 / 0.09 -> 0.12 / 0.07 ms)
int splits_for(int M, int N, int K) {
  int tiles = ((M + kGemmBM - 1) / kGemmBM) * ((N + kGemmBN - 1) / kGemmBN);
  int s = std::max(1, 512 / std::max(1, tiles));
  int max_s = std::max(1, (K + kGemmBK - 1) / kGemmBK);
  return std::min(std::min(s, 64), max_s);
}

// Chooses rows per group (16*NT) so that every group's workgroups fit on one XCC.
int make_plan(const slstm_dims* d, Plan* p) {
  if (!dims_ok(d)) return SLSTM_EINVAL;
  const int prec = d->precision;
  const int KC = rec_kc(prec);
  p->prec = prec;
  p->ks_eff = (d->H + KC - 1) / KC;
  p->KS = ks_bucket(prec, p->ks_eff);
  if (p->KS < 0) return SLSTM_EINVAL;
  p->NW = (d->H + 15) / 16;
  // the backward compiled for K = 32 bf16 chunks (lean variant) runs 512-thread workgroups
  // of 32 units, one per CU; the others 256-thread workgroups of 16 units
  p->NWb = rec_occ(prec, p->KS) == 2 ? (d->H + 31) / 32 : p->NW;
  const int cus = device_cus();
  const int cu_per_xcc = cus > 0 ? cus / 8 : 32;
  // smallest row tile count per group whose workgroups (NW per group, groups dealt to the 8
  // XCCs round-robin) are co-resident on one XCC at the kernel's occupancy
  // the pipelined forward needs whole 1 KB row segments (vector rows, every K chunk in use)
  const bool pipe_ok = d->H % (prec ? 8 : 4) == 0 && p->ks_eff == p->KS && p->KS >= 16;
  p->kx = (d->I + 31) / 32;
  p->fuse = 0;
  p->gs = 0;
  // the backward's gate-split contraction covers exactly H units with whole M tiles; its
  // partial sums (two step buffers of G x 16*NT rows x NW x H fp32) use the post-loop GEMMs'
  // partials area
  const Layout Lp = layout(d);
  const bool gs_ok = p->ks_eff == p->KS && p->KS * KC == d->H;
  auto pick = [&](bool bwd, int* NT_out, int* G_out, int* per_out, int* pipe_out) -> int {
    for (int NT = 1; NT <= 8; NT *= 2) {
      int G = (d->B + 16 * NT - 1) / (16 * NT);
      if (G > MAX_GROUPS) continue;
      int per_xcc = (bwd ? p->NWb : p->NW) * ((G + 7) / 8);
      int occ = 0;
      const bool pipe = !bwd && pipe_ok && NT >= 2 && rec_pipe_built(prec, NT, p->KS);
      // the plain bf16 forward fuses the input projection when one pass covers the group
      // (x rows copied whole: I % 4 == 0, byte offsets within 32 bits)
      const bool fuse = !bwd && !pipe && rec_fx_built(prec, p->KS) && rec_ntb(prec, NT, p->KS) == NT &&
                        rec_fx_fits(16 * NT, p->kx) && d->I % 4 == 0 &&
                        (int64_t)d->T * d->B * d->I * 4 < ((int64_t)1 << 32) &&
                        rec_lds_bytes(prec, NT, p->KS) + rec_fx_lds_bytes(16 * NT) <= (size_t)160 * 1024;
      RecArgs dummy;
      memset(&dummy, 0, sizeof(dummy));
      FxArgs fdummy;
      memset(&fdummy, 0, sizeof(fdummy));
      fdummy.fuse_x = fuse ? 1 : 0;
      fdummy.kx = p->kx;
      const bool gs = bwd && gs_ok && rec_bwd_gs_built(prec, NT, p->KS) &&
                      (size_t)2 * G * 16 * NT * p->NW * d->H * 4 <= Lp.prow - Lp.part;
      dummy.bwd_gs = gs ? 1 : 0;
      hipError_t e = bwd    ? launch_bwd(dummy, prec, NT, p->KS, dim3(0), nullptr, &occ)
                     : pipe ? launch_fwd_pipe(dummy, prec, NT, p->KS, dim3(0), nullptr, &occ)
                            : launch_fwd(dummy, fdummy, prec, NT, p->KS, dim3(0), nullptr, &occ);
      if (e != hipSuccess) {
        (void)hipGetLastError();                  // a failed query leaves no error for later calls
        return SLSTM_EDEVICE;
      }
      if (per_xcc <= cu_per_xcc * occ) {
        *NT_out = NT;
        *G_out = G;
        *per_out = per_xcc;
        if (pipe_out) *pipe_out = pipe ? 1 : 0;
        if (!bwd) p->fuse = fuse ? 1 : 0;
        if (bwd) p->gs = gs ? 1 : 0;
        return SLSTM_OK;
      }
    }
    return SLSTM_ENORESIDENT;
  };
  // bf16 with H > 512: 16-unit workgroups would need two per CU and spill their U slice;
  // the wide forward gives each CU one workgroup of 32 units (groups of 128 rows, one per XCC)
  p->wide = 0;
  p->NWw = (d->H + 31) / 32;
  if (prec == SLSTM_BF16_GEMM && d->H > 512 && d->H % 8 == 0 && p->KS == 32 && p->NWw <= cu_per_xcc &&
      (d->B + 127) / 128 <= 8) {
    int occ = 0;
    RecArgs dummy;
    memset(&dummy, 0, sizeof(dummy));
    if (launch_fwd_wide(dummy, 8, 32, dim3(0), nullptr, &occ) != hipSuccess) return SLSTM_EDEVICE;
    if (occ >= 1) {
      p->wide = 1;
      p->NT = 8;
      p->G = (d->B + 127) / 128;
      p->per_xcc = p->NWw;
      p->pipe = 0;
    }
  }
  int rc = p->wide ? SLSTM_OK : pick(false, &p->NT, &p->G, &p->per_xcc, &p->pipe);
  if (rc) return rc;
  if ((rc = pick(true, &p->NTb, &p->Gb, &p->per_xcc_b, nullptr))) return rc;
  int64_t K = (int64_t)d->T * d->B;
  p->splits_w = splits_for(d->I, 4 * d->H, (int)std::min<int64_t>(K, 1 << 30));
  p->splits_u = splits_for(d->H, 4 * d->H, (int)std::min<int64_t>(K, 1 << 30));
  return SLSTM_OK;
}

// Work-space layout; splits are bounded by 64 so the layout does not depend on the device.
Layout layout(const slstm_dims* d) {
  const size_t T = d->T, B = d->B, I = d->I, H = d->H;
  const bool bf = d->precision == SLSTM_BF16_GEMM;
  const size_t KP = padded_rows(d);
  Layout L;
  size_t o = 0;
  L.ctl = o; o += align256(CTL_WORDS * 4);
  L.stack = o; o += align256(B * (T + 1) * 4);                        // op scan: stacks that do not fit in LDS
  L.dep = o; o += align256(B * 4);                                     // pointer after the last step
  L.wp = o; o += align256(I * 4 * H * 4);                             // Wp fp32, or Wp and Wp^T in bf16
  L.r1 = o; o += align256(std::max<size_t>(T * B * 4 * H * 4, 16));   // XW (forward), dA (backward)
  L.stash = o; o += align256(std::max<size_t>(T * B * 4 * H * 4, 16));
  L.hx = o; o += bf ? align256((T + 1) * B * H * 2) : 0;
  L.fwd_end = o;                                                       // the forward uses [0, fwd_end)
  // post-loop operands over the push rows (at most T*B of them; KP with the K-tile padding)
  L.xbt = o; o += bf ? align256(KP * I * 2) : 0;                      // x^T in bf16 (bf16 mode)
  L.hp = o; o += align256(std::max<size_t>(bf ? KP * H * 2 : T * B * H * 4, 16));   // Hprev (bf16 mode: Hprev^T)
  L.dat = o; o += bf ? align256(KP * 4 * H * 2) : 0;                  // dA^T in bf16 (bf16 mode)
  L.dh = o; o += align256((T + 1) * B * H * 4);
  L.dc = o; o += align256((T + 1) * B * H * 4);
  L.dbp = o; o += align256((size_t)MAX_GROUPS * 4 * H * 4);
  // split-K partials of dW / dU (at most min(64, ceil(T*B / 64)) slices: the split counts never
  // exceed the GEMM's 64-row K steps over the T*B rows), the K-slice partials of dx (at most the
  // rows of the grid's whole tiles: padded T*B x I), and the fp32 backward's gate-split partial
  // sums (two step buffers of the groups' rows, at most B + 127, x H/16 workgroups x H)
  const size_t max_splits = std::min<size_t>(64, std::max<size_t>(1, (T * B + 63) / 64));
  L.part = o; o += align256(std::max({max_splits * std::max(I, H) * 4 * H, (T * B + 127) / 128 * 128 * I,
                                      bf ? 0 : 2 * (B + 127) * ((H + 15) / 16) * H}) * 4);
  L.prow = o; o += align256(std::max<size_t>(T * B * 4, 16));         // push-row list
  L.total = o;
  return L;
}

int hip_status(hipError_t e) {
  if (e == hipSuccess) return SLSTM_OK;
  if (e == hipErrorCooperativeLaunchTooLarge) return SLSTM_ENORESIDENT;
  return SLSTM_EDEVICE;
}

void mark(const slstm_dims* d, int i, hipStream_t st) {
  if (d->phase_events) (void)hipEventRecord(((hipEvent_t*)d->phase_events)[i], st);
}

int grid1d(size_t n) { return (int)std::min<size_t>((n + 255) / 256, 8192); }

int launch_gemm(int prec, int AL, int BL, const GemmArgs& g, int splits, hipStream_t st) {
  dim3 grid((g.N + kGemmBN - 1) / kGemmBN, (g.M + kGemmBM - 1) / kGemmBM, splits);
#define GCASE(P, A, B_)                                                       \
  if (prec == P && AL == A && BL == B_) {                                     \
    hipLaunchKernelGGL((k_gemm<P, A, B_>), grid, dim3(256), 0, st, g);        \
    return hip_status(hipGetLastError());                                     \
  }
  GCASE(0, GEMM_MK, GEMM_KN) GCASE(0, GEMM_MK, GEMM_NK) GCASE(0, GEMM_KM, GEMM_KN)
  GCASE(1, GEMM_MK, GEMM_NK) GCASE(1, GEMM_MK_F32, GEMM_NK)
#undef GCASE
  return SLSTM_EINVAL;
}

// The wide-tile bf16 GEMM takes MK x NK bf16 operands with 16-byte rows, no row gathers and
// no device-side M.
bool gemm_wide_ok(int prec, int AL, int BL, const GemmArgs& g) {
  return prec == SLSTM_BF16_GEMM && AL == GEMM_MK && BL == GEMM_NK && g.a_vec && g.b_vec && !g.a_rows && !g.b_rows &&
         !g.c_rows && !(g.dyn && g.dyn_axis == 0) && g.K % 8 == 0;
}
int wide_tiles(int M, int N) { return ((M + kGemmWideBM - 1) / kGemmWideBM) * ((N + kGemmWideBN - 1) / kGemmWideBN); }
// split K of a wide-tile GEMM: one round of one workgroup per CU (256 blocks), at most 64
// slices and one 64-deep K tile per slice
int wide_splits(int M, int N, int K) {
  const int s = std::max(1, 256 / std::max(1, wide_tiles(M, N)));
  return std::min(std::min(s, 64), std::max(1, (K + 63) / 64));
}
int launch_gemm_wide(const GemmArgs& g, int splits, hipStream_t st) {
  if (hipFuncSetAttribute((const void*)k_gemm_wide, hipFuncAttributeMaxDynamicSharedMemorySize, (int)kGemmWideLds) !=
      hipSuccess)
    return SLSTM_EDEVICE;
  dim3 grid((g.N + kGemmWideBN - 1) / kGemmWideBN, (g.M + kGemmWideBM - 1) / kGemmWideBM, splits);
  hipLaunchKernelGGL(k_gemm_wide, grid, dim3(256), kGemmWideLds, st, g);
  return hip_status(hipGetLastError());
}

// K slice per split, a multiple of the GEMM's K tile (64 covers both precisions)
int k_chunk_for(int K, int splits) { return ((K + splits - 1) / splits + 63) / 64 * 64; }

// The call's one host synchronisation: reads the control words its kernels set and maps them
// to a status (op errors first, then a wait that gave up, then a producer index out of range).
int read_status(const uint32_t* ctl, hipStream_t st) {
  uint32_t v[CTL_BADIDX + 1] = {};
  if (hipMemcpyAsync(v, ctl, sizeof(v), hipMemcpyDeviceToHost, st) != hipSuccess) return SLSTM_EDEVICE;
  if (hipStreamSynchronize(st) != hipSuccess) return SLSTM_EDEVICE;
  if (v[CTL_STATUS] != kStatusOk) return (int)(v[CTL_STATUS] & 7u);
  if (v[CTL_TIMEOUT]) return SLSTM_ETIMEOUT;
  if (v[CTL_BADIDX]) return SLSTM_EINDEX;
  return SLSTM_OK;
}

// The status a call returns: its control words read back (one host synchronisation), or,
// for a deferred call, OK once its kernels are queued (sync_status reads the words later).
int call_status(const slstm_dims* d, const uint32_t* ctl, hipStream_t st) {
  if (hipGetLastError() != hipSuccess) return SLSTM_EDEVICE;
  return d->defer_status ? SLSTM_OK : read_status(ctl, st);
}

// Backward direct staging: a variant built with it, whole 1 KB row segments, K range equal
// to the register capacity, and the LDS slice plus static LDS within one CU (one workgroup
// per CU).
bool bwd_direct_for(const slstm_dims* d, const Plan& p) {
  const int esz = d->precision == SLSTM_BF16_GEMM ? 2 : 4;
  return !p.gs && rec_bwd_direct_built(d->precision, p.NTb, p.KS) && ((size_t)d->H * esz) % 1024 == 0 &&
         p.KS * rec_kc(d->precision) == d->H &&
         rec_bwd_lds_bytes(d->precision, p.KS) + rec_bwd_static_lds(p.NTb) <= 160 * 1024 &&
         p.per_xcc_b <= std::max(1, device_cus() / 8);
}

RecArgs rec_args(const slstm_dims* d, const Plan& p, char* ws, const Layout& L, bool bwd) {
  RecArgs a;
  memset(&a, 0, sizeof(a));
  a.T = d->T; a.B = d->B; a.I = d->I; a.H = d->H;
  a.G = bwd ? p.Gb : p.G; a.NW = bwd ? p.NWb : p.NW; a.ks_eff = p.ks_eff;
  a.spin_limit = d->spin_limit > 0 ? d->spin_limit : kDefaultSpin;
  a.ctl = (uint32_t*)(ws + L.ctl);
  a.stash = (float*)(ws + L.stash);
  a.hx = d->precision == SLSTM_BF16_GEMM ? (uint16_t*)(ws + L.hx) : nullptr;
  a.clk = (long long*)d->step_clock;
  // Exchange protocol (measured on the large parser workload): the bf16 forward's step is
  // short and a group barrier's fixed cost (store acknowledgement, then an atomic and a poll
  // round trip) dominates it, so its workgroups poll the fill-marked rows instead; the fp32
  // forward's rows are twice as long and checking a staged tile for the fill pattern costs
  // more than the barrier. The backward uses the barrier in both precisions: it stores and
  // exchanges only push rows, its barrier's arrival overlaps the row-offset set-up, and a
  // fill of dA before it would be a large write (bf16 large: 1.24 ms with the barrier,
  // 1.32 ms polling).
  a.poll = (d->precision == SLSTM_BF16_GEMM && !bwd) ? 1 : 0;
  // the pipelined forward has no barrier: it always polls
  if (!bwd && p.pipe) a.poll = 1;
  const int esz = d->precision == SLSTM_BF16_GEMM ? 2 : 4;
  a.coh_rows = ((size_t)d->H * esz) % 128 != 0;
  a.bwd_direct = bwd_direct_for(d, p) ? 1 : 0;
  if (bwd && p.gs) {
    a.bwd_gs = 1;
    a.gs_part = (float*)(ws + L.part);   // free until the post-loop GEMMs
  }
  return a;
}

}  // namespace

extern "C" {

size_t stacklstm_workspace_bytes(const slstm_dims* d) {
  if (!dims_ok(d)) return 0;
  return layout(d).total;
}

const char* stacklstm_status_string(int s) {
  switch (s) {
    case SLSTM_OK: return "ok";
    case SLSTM_EINVAL: return "invalid argument (dims, null pointer or unsupported size)";
    case SLSTM_EOPS: return "op outside {-1, 0, 1}";
    case SLSTM_EUNDERFLOW: return "pop with only the initial state on the stack";
    case SLSTM_EWORKSPACE: return "work space too small";
    case SLSTM_ENORESIDENT: return "persistent kernels cannot be co-resident";
    case SLSTM_EDEVICE: return "HIP runtime error";
    case SLSTM_ETIMEOUT: return "a wait for another workgroup's data exceeded the spin limit";
    case SLSTM_EINDEX: return "a producer index or stack depth outside its valid range (top or ops not the forward's)";
    default: return "unknown status";
  }
}

int stacklstm_plan(const slstm_dims* d, slstm_plan* out) {
  Plan p;
  int rc = make_plan(d, &p);
  if (rc) return rc;
  if (!out) return SLSTM_EINVAL;
  memset(out, 0, sizeof(*out));
  out->groups = p.G;
  out->wg_per_group = p.wide ? p.NWw : p.NW;
  out->rows_per_group = 16 * p.NT;
  out->k_chunks = p.ks_eff;
  out->fwd_kernel = p.wide ? 2 : (p.pipe ? 1 : 0);
  out->fwd_tiles = p.NT;
  out->k_chunk_cap = p.KS;
  out->occupancy = rec_occ(p.prec, p.KS);
  out->bwd_groups = p.Gb;
  out->bwd_tiles = p.NTb;
  out->bwd_direct = bwd_direct_for(d, p) ? 1 : 0;
  out->fused_x = p.fuse;
  out->bwd_split = p.gs;
  return SLSTM_OK;
}

}  // extern "C"

namespace {

// The forward pass on a work space that the caller checked (at least layout(d).fwd_end bytes).
int fwd_impl(const slstm_dims* d, const Plan& p, const Layout& L, const float* x, const int8_t* ops, const float* W,
             const float* U, const float* b, const float* h0, const float* c0, float* h_cell, float* c_cell,
             float* h_top, float* c_top, int32_t* ptr, int32_t* top, char* ws, hipStream_t st) {
  int rc = SLSTM_OK;
  uint32_t* ctl = (uint32_t*)(ws + L.ctl);
  const int T = d->T, B = d->B, I = d->I, H = d->H;
  const bool bf = p.prec == SLSTM_BF16_GEMM;

  // a1: op validation, pointer scan and producer trace. One thread per element; its stack of
  // T + 1 step indices in LDS when a few elements' stacks fit in 64 KB, else in the work space
  mark(d, 0, st);
  hipLaunchKernelGGL(k_init_ctl, dim3(1), dim3(256), 0, st, ctl, d->defer_status ? 1 : 0);
  {
    const int cap = (T + 1) | 1;                  // odd: neighbouring stacks start in other banks
    int R = (int)std::min<size_t>(64, 65536 / ((size_t)cap * 4));
    const int lds = R >= 1 ? 1 : 0;
    if (!lds) R = 64;
    if (lds)
      hipLaunchKernelGGL(k_scan<true>, dim3((B + R - 1) / R), dim3(R), (size_t)R * cap * 4, st, ops, T, B, cap, ptr, top,
                         (int32_t*)(ws + L.dep), (int32_t*)(ws + L.stack), ctl);
    else
      hipLaunchKernelGGL(k_scan<false>, dim3((B + R - 1) / R), dim3(R), 0, st, ops, T, B, cap, ptr, top,
                         (int32_t*)(ws + L.dep), (int32_t*)(ws + L.stack), ctl);
  }
  if ((rc = hip_status(hipGetLastError()))) return rc;
  mark(d, 1, st);
  if (T == 0) return call_status(d, ctl, st);

  // a2: XW = x W + b for all steps on the library's MFMA GEMM, columns gate-interleaved
  // (Wp = W with permuted columns; bf16 mode: Wp and its transpose in bf16), bias added in
  // the GEMM's epilogue in fp32
  void* wp = ws + L.wp;
  bf16_t* wpt = bf ? (bf16_t*)wp + (size_t)I * 4 * H : nullptr;
  // the fused projection copies x rows by 16-byte DMA: x must be 16-byte aligned, else XW
  const bool fuse = p.fuse && al16(x);
  hipLaunchKernelGGL(k_permute_w, dim3(grid1d((size_t)I * 4 * H)), dim3(256), 0, st, W, bf ? nullptr : (float*)wp,
                     bf ? (bf16_t*)wp : nullptr, fuse ? nullptr : wpt, I, H);
  float* xw = (float*)(ws + L.r1);
  // (with the fused projection the recurrent kernel contracts x_t W itself: no XW)
  if (!fuse) {
    GemmArgs g;
    memset(&g, 0, sizeof(g));
    g.M = T * B; g.N = 4 * H; g.K = I;
    g.A = x; g.lda = I; g.a_vec = (I % 4 == 0) && al16(x);
    if (bf) { g.Bm = wpt; g.ldb = I; g.b_vec = (I % 8 == 0); }
    else    { g.Bm = wp; g.ldb = 4 * H; g.b_vec = 1; }
    g.C = xw; g.ldc = 4 * H;
    g.bias = b; g.bias_H = H;
    g.k_chunk = k_chunk_for(I, 1);
    // bf16: x rounded to bf16 once, into the gate stash's area (written by the recurrent
    // kernel only after this GEMM), then a bf16 GEMM; the GEMM that rounds fp32 x as it
    // loads it re-reads the fp32 rows once per 128-column tile (thru shape: 2.80 ms against
    // 0.16 + 2.02 ms). The same rounding (nearest even) either way.
    int al = bf ? GEMM_MK_F32 : GEMM_MK;
    const size_t nx = (size_t)T * B * I;
    if (bf && g.a_vec && I % 8 == 0 && nx * 2 <= (size_t)T * B * 4 * H * 4) {
      bf16_t* x16 = (bf16_t*)(ws + L.stash);
      hipLaunchKernelGGL(k_to_bf16x8, dim3(grid1d(nx / 8)), dim3(256), 0, st, x, x16, nx / 8);
      g.A = x16;
      al = GEMM_MK;
    }
    // (bf16 operands: the wide-tile GEMM when its 256 x 256 tiles alone fill the chip; fp32:
    // the LDS-DMA ring GEMM when its operands allow 16-byte DMAs with 32-bit offsets)
    const bool ring = !bf && g.K % 4 == 0 && g.N % 4 == 0 && al16(x) && (size_t)g.M * g.lda * 4 < ((size_t)1 << 32) &&
                      (size_t)g.K * g.ldb * 4 < ((size_t)1 << 32);
    if (ring) {
      hipLaunchKernelGGL(k_gemm_ring, dim3((g.N + kGemmBN - 1) / kGemmBN, (g.M + kGemmBM - 1) / kGemmBM), dim3(256), 0, st,
                         g);
      if ((rc = hip_status(hipGetLastError()))) return rc;
    } else if (gemm_wide_ok(p.prec, al, GEMM_NK, g) && wide_tiles(g.M, g.N) >= 256) {
      if ((rc = launch_gemm_wide(g, 1, st))) return rc;
    } else if ((rc = launch_gemm(p.prec, al, bf ? GEMM_NK : GEMM_KN, g, 1, st))) {
      return rc;
    }
  }

  // a3-a6: persistent recurrent kernel
  RecArgs a = rec_args(d, p, ws, L, false);
  if (bf) hipLaunchKernelGGL(k_h0_bf16, dim3(grid1d((size_t)B * H)), dim3(256), 0, st, h0, (bf16_t*)a.hx, (size_t)B * H);
  a.xw = fuse ? nullptr : xw; a.ops = ops; a.U = U; a.h0 = h0; a.c0 = c0; a.hcell = h_cell; a.ccell = c_cell;
  a.top = top;
  FxArgs fa;
  memset(&fa, 0, sizeof(fa));
  if (fuse) {
    fa.fuse_x = 1; fa.kx = p.kx; fa.x = x; fa.W = W; fa.bias = b;
  }
  // exchange buffers start as "not yet produced": all-one bits in the state rows the
  // workgroups read from each other
  if (a.poll || p.wide) {
    const size_t ex_bytes = (size_t)T * B * H * (bf ? 2 : 4);
    unsigned char* ex = bf ? (unsigned char*)(a.hx + (size_t)B * H) : (unsigned char*)h_cell;
    hipLaunchKernelGGL(k_fill_pattern, dim3(grid1d(ex_bytes / 16 + 1)), dim3(256), 0, st, ex, ex_bytes, 0xffffffffu);
  }
  a.htop = p.wide ? h_top : nullptr;
  a.ctop = p.wide ? c_top : nullptr;
  if (p.wide) a.NW = p.NWw;
  mark(d, 2, st);
  if ((rc = hip_status(p.wide   ? launch_fwd_wide(a, p.NT, p.KS, dim3(8 * p.per_xcc), st, nullptr)
                       : p.pipe ? launch_fwd_pipe(a, p.prec, p.NT, p.KS, dim3(8 * p.per_xcc), st, nullptr)
                                : launch_fwd(a, fa, p.prec, p.NT, p.KS, dim3(8 * p.per_xcc), st, nullptr))))
    return rc;
  mark(d, 3, st);

  // a7: Algorithm 1's return values (the wide forward writes c_top and the h_top of push steps)
  size_t n = (size_t)T * B * H;
  float* ctop_g = p.wide ? nullptr : c_top;          // the wide forward writes c_top itself
  if (H % 4 == 0 && al16(h_cell) && al16(h0) && al16(h_top) && al16(c_cell) && al16(c0) && al16(c_top)) {
    if (h_top || ctop_g)
      hipLaunchKernelGGL(k_gather_top4, dim3(grid1d(n / 4)), dim3(256), 0, st, top, h_cell, h0, h_top, c_cell, c0, ctop_g,
                         T, B, H, p.wide, ctl);
  } else {
    if (h_top)
      hipLaunchKernelGGL(k_gather_top, dim3(grid1d(n)), dim3(256), 0, st, top, h_cell, h0, h_top, T, B, H, p.wide, ctl);
    if (ctop_g)
      hipLaunchKernelGGL(k_gather_top, dim3(grid1d(n)), dim3(256), 0, st, top, c_cell, c0, ctop_g, T, B, H, 0, ctl);
  }
  if ((rc = hip_status(hipGetLastError()))) return rc;
  mark(d, 4, st);
  return call_status(d, ctl, st);
}

bool fwd_args_ok(const slstm_dims* d, const float* x, const int8_t* ops, const float* W, const float* U,
                 const float* b, const float* h0, const float* c0, const float* h_cell, const float* c_cell,
                 const int32_t* ptr, const int32_t* top) {
  return ptr && (d->T == 0 || (ops && x && W && U && b && h0 && c0 && h_cell && c_cell && top));
}

// Static work space of the allocation-free forward: one copy per GPU, held until the process
// ends. Host code uses the device address that hipGetSymbolAddress returns for the current
// device (kept per device), never the array's name.
constexpr size_t kScratchBytes = SLSTM_FWD_STATIC_MAX_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on the current device, looked up on the first call on that
// device; null if the lookup failed.
char* scratch_ptr() {
  static std::mutex mu;
  static void* addr[64] = {};
  static bool done[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  std::lock_guard<std::mutex> lk(mu);
  if (!done[dev]) {
    void* q = nullptr;
    if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    addr[dev] = q;
    done[dev] = true;
  }
  return (char*)addr[dev];
}

}  // namespace

extern "C" {

int stacklstm_fwd(const slstm_dims* d, const float* x, const int8_t* ops, const float* W, const float* U,
                  const float* b, const float* h0, const float* c0, float* h_cell, float* c_cell, float* h_top,
                  float* c_top, int32_t* ptr, int32_t* top, void* workspace, size_t ws_bytes, void* stream) {
  if (!dims_ok(d)) return SLSTM_EINVAL;
  if (!workspace || !fwd_args_ok(d, x, ops, W, U, b, h0, c0, h_cell, c_cell, ptr, top)) return SLSTM_EINVAL;
  const Layout L = layout(d);
  if (ws_bytes < L.total) return SLSTM_EWORKSPACE;
  Plan p;
  int rc = make_plan(d, &p);
  if (rc) return rc;
  return fwd_impl(d, p, L, x, ops, W, U, b, h0, c0, h_cell, c_cell, h_top, c_top, ptr, top, (char*)workspace,
                  (hipStream_t)stream);
}

int stacklstm_fwd_static(const slstm_dims* d, const float* x, const int8_t* ops, const float* W, const float* U,
                         const float* b, const float* h0, const float* c0, float* h_cell, float* c_cell, float* h_top,
                         float* c_top, int32_t* ptr, int32_t* top, void* stream) {
  if (!dims_ok(d)) return SLSTM_EINVAL;
  if (!fwd_args_ok(d, x, ops, W, U, b, h0, c0, h_cell, c_cell, ptr, top)) return SLSTM_EINVAL;
  const Layout L = layout(d);
  if (L.fwd_end > kScratchBytes) return SLSTM_EWORKSPACE;
  Plan p;
  int rc = make_plan(d, &p);
  if (rc) return rc;
  char* ws = scratch_ptr();
  if (!ws) return SLSTM_EDEVICE;
  return fwd_impl(d, p, L, x, ops, W, U, b, h0, c0, h_cell, c_cell, h_top, c_top, ptr, top, ws, (hipStream_t)stream);
}

int stacklstm_bwd(const slstm_dims* d, const float* x, const int8_t* ops, const float* W, const float* U,
                  const float* h0, const float* c0, const float* h_cell, const float* c_cell, const int32_t* top,
                  void* workspace, size_t ws_bytes, const float* dh_top, const float* dc_top, float* dx, float* dW,
                  float* dU, float* db, float* dh0, float* dc0, void* stream) {
  (void)W;
  if (!dims_ok(d)) return SLSTM_EINVAL;
  if (!workspace || !dW || !dU || !db || !dh0 || !dc0) return SLSTM_EINVAL;
  if (d->T > 0 && (!x || !ops || !U || !h0 || !c0 || !h_cell || !c_cell || !top || !dh_top || !dx))
    return SLSTM_EINVAL;
  const Layout L = layout(d);
  if (ws_bytes < L.total) return SLSTM_EWORKSPACE;
  Plan p;
  int rc = make_plan(d, &p);
  if (rc) return rc;
  hipStream_t st = (hipStream_t)stream;
  char* ws = (char*)workspace;
  uint32_t* ctl = (uint32_t*)(ws + L.ctl);
  const int T = d->T, B = d->B, I = d->I, H = d->H;
  const bool bf = p.prec == SLSTM_BF16_GEMM;
  // the backward's control words (slot and barrier counters, wait and index flags) start at 0
  hipLaunchKernelGGL(k_zero_ctl_bwd, dim3(1), dim3(256), 0, st, ctl, d->defer_status ? 1 : 0);
  if (T == 0) {
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)I * 4 * H)), dim3(256), 0, st, dW, (size_t)I * 4 * H, 0.f);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)H * 4 * H)), dim3(256), 0, st, dU, (size_t)H * 4 * H, 0.f);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)4 * H)), dim3(256), 0, st, db, (size_t)4 * H, 0.f);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)B * H)), dim3(256), 0, st, dh0, (size_t)B * H, 0.f);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)B * H)), dim3(256), 0, st, dc0, (size_t)B * H, 0.f);
    if ((rc = hip_status(hipGetLastError()))) return rc;
    return call_status(d, ctl, st);
  }

  // a8: persistent reverse loop
  RecArgs a = rec_args(d, p, ws, L, true);
  a.ops = ops; a.U = U; a.h0 = h0; a.c0 = c0;
  a.hcell = const_cast<float*>(h_cell); a.ccell = const_cast<float*>(c_cell); a.top = const_cast<int32_t*>(top);
  a.dh_top = dh_top; a.dc_top = dc_top;
  a.dA = ws + L.r1;
  a.dh_acc = (float*)(ws + L.dh); a.dc_acc = (float*)(ws + L.dc);
  a.db_part = (float*)(ws + L.dbp);
  a.depth_end = (const int32_t*)(ws + L.dep);
  a.dh0 = dh0; a.dc0 = dc0;
  if (a.clk) a.clk += (size_t)512 * T * 4;
  // rows of the push steps, for the post-loop gradients (dA is exactly zero on other rows);
  // their number stays on the device: the GEMMs below take it as their K or M extent
  int32_t* prow = (int32_t*)(ws + L.prow);
  const uint32_t* npush = ctl + CTL_NPUSH;
  hipLaunchKernelGGL(k_push_rows, dim3(1), dim3(1024), 0, st, ops, T * B, prow, ctl + CTL_NPUSH);
  mark(d, 5, st);
  if ((rc = hip_status(launch_bwd(a, p.prec, p.NTb, p.KS, dim3(8 * p.per_xcc_b), st, nullptr)))) return rc;
  mark(d, 6, st);

  // a9: post-loop gradients on the library's MFMA GEMM, contracted over the push rows only
  // (rows prow[0 .. *npush)). fp32: the GEMMs gather x and dA rows through prow, Hprev is
  // gathered first; bf16: x, dA and Hprev are written transposed and compacted (k = push
  // index contiguous, zero up to the next multiple of 64) for dW and dU.
  const int H4 = 4 * H;
  float* part = (float*)(ws + L.part);
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)H4)), dim3(256), 0, st, a.db_part, p.Gb, (size_t)H4, 1, H4,
                     H, db);
  const int K = T * B;
  const int KP = (int)padded_rows(d);
  void* hp = ws + L.hp;
  GemmArgs g;
  auto gemm_base = [&]() {
    memset(&g, 0, sizeof(g));
    g.dyn = npush;
    g.dyn_round = bf ? 64 : 1;
  };
  if (bf) {
    const dim3 tg4((H4 + 63) / 64, KP / 64), tgI((I + 63) / 64, KP / 64), tgH((H + 63) / 64, KP / 64);
    hipLaunchKernelGGL(k_transpose_bf16, tg4, dim3(256), 0, st, a.dA, 0, H4, H4, prow, npush, KP,
                       (const int32_t*)nullptr, B, (bf16_t*)(ws + L.dat), ctl);
    hipLaunchKernelGGL(k_transpose_bf16, tgI, dim3(256), 0, st, x, 1, I, I, prow, npush, KP, (const int32_t*)nullptr,
                       B, (bf16_t*)(ws + L.xbt), ctl);
    hipLaunchKernelGGL(k_transpose_bf16, tgH, dim3(256), 0, st, ws + L.hx, 0, H, H, prow, npush, KP, top, B,
                       (bf16_t*)hp, ctl);
  } else {
    hipLaunchKernelGGL(k_gather_hprev, dim3(grid1d((size_t)K * H)), dim3(256), 0, st, top, h_cell, h0, prow, npush,
                       (float*)hp, T, B, H, ctl);
  }
  // dW = x^T dA
  gemm_base();
  g.M = I; g.N = H4; g.dyn_axis = 1;
  if (bf) { g.K = KP; g.A = ws + L.xbt; g.lda = KP; g.a_vec = 1; g.Bm = ws + L.dat; g.ldb = KP; g.b_vec = 1; }
  else    { g.K = K; g.A = x; g.lda = I; g.a_vec = (I % 4 == 0) && al16(x); g.a_rows = prow;
            g.Bm = a.dA; g.ldb = H4; g.b_vec = 1; g.b_rows = prow; }
  g.C = part; g.ldc = H4;
  g.split_stride = (size_t)I * H4;
  // (bf16: the wide-tile GEMM, with its own split count, when the output has 32 or more of its
  // tiles: measured faster at the thru shape, slower at the large one, whose K slices are short)
  const bool wide_w = gemm_wide_ok(p.prec, GEMM_MK, GEMM_NK, g) && wide_tiles(g.M, g.N) >= 32;
  const int sw = wide_w ? wide_splits(g.M, g.N, g.K) : p.splits_w;
  if ((rc = wide_w ? launch_gemm_wide(g, sw, st)
                   : launch_gemm(p.prec, bf ? GEMM_MK : GEMM_KM, bf ? GEMM_NK : GEMM_KN, g, sw, st)))
    return rc;
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)I * H4)), dim3(256), 0, st, part, sw, g.split_stride, I, H4,
                     H, dW);
  mark(d, 7, st);
  // dU = Hprev^T dA
  gemm_base();
  g.M = H; g.N = H4; g.dyn_axis = 1;
  if (bf) { g.K = KP; g.A = hp; g.lda = KP; g.a_vec = 1; g.Bm = ws + L.dat; g.ldb = KP; g.b_vec = 1; }
  else    { g.K = K; g.A = hp; g.lda = H; g.a_vec = (H % 4 == 0); g.Bm = a.dA; g.ldb = H4; g.b_vec = 1;
            g.b_rows = prow; }
  g.C = part; g.ldc = H4;
  g.split_stride = (size_t)H * H4;
  const bool wide_u = gemm_wide_ok(p.prec, GEMM_MK, GEMM_NK, g) && wide_tiles(g.M, g.N) >= 32;
  const int su = wide_u ? wide_splits(g.M, g.N, g.K) : p.splits_u;
  if ((rc = wide_u ? launch_gemm_wide(g, su, st)
                   : launch_gemm(p.prec, bf ? GEMM_MK : GEMM_KM, bf ? GEMM_NK : GEMM_KN, g, su, st)))
    return rc;
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)H * H4)), dim3(256), 0, st, part, su, g.split_stride, H, H4,
                     H, dU);
  mark(d, 8, st);
  // dx = dA Wp^T on the push rows (gathered from dA); the GEMM's grid covers all T*B rows, so
  // the push rows' tiles take two or more blocks each, over K slices written as partials that
  // k_scatter_splits adds into the push rows of dx; 0 on the other rows
  gemm_base();
  g.dyn_round = 1; g.dyn_axis = 0; g.dyn_split = 1;
  g.M = K; g.N = I; g.K = H4;
  const int VE = bf ? 8 : 4;
  g.A = a.dA; g.lda = H4; g.a_vec = (H4 % VE == 0); g.a_rows = prow;
  g.Bm = ws + L.wp; g.ldb = H4; g.b_vec = (H4 % VE == 0) && (I % VE == 0);
  g.C = part; g.ldc = I;
  g.k_chunk = k_chunk_for(H4, 1);
  if ((rc = launch_gemm(p.prec, GEMM_MK, GEMM_NK, g, 1, st))) return rc;
  {
    const int ntl = (I + kGemmBN - 1) / kGemmBN, nblk = ntl * ((K + kGemmBM - 1) / kGemmBM);
    hipLaunchKernelGGL(k_scatter_splits, dim3(grid1d((size_t)K * I)), dim3(256), 0, st, (const float*)part, prow, npush,
                       (size_t)K, I, nblk, ntl, dx);
  }
  hipLaunchKernelGGL(k_zero_nonpush_rows, dim3(grid1d((size_t)K * I / 4 + 1)), dim3(256), 0, st, ops, dx, (size_t)K,
                     I);
  if ((rc = hip_status(hipGetLastError()))) return rc;
  mark(d, 9, st);
  return call_status(d, ctl, st);
}

int stacklstm_sync_status(const void* workspace, size_t ws_bytes, void* stream) {
  if (!workspace || ws_bytes < align256(CTL_WORDS * 4)) return SLSTM_EINVAL;
  return read_status((const uint32_t*)workspace, (hipStream_t)stream);
}

}  // extern "C"
