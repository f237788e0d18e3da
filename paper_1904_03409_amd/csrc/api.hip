// Host side of the StackLSTM library: argument checks, work-space layout, launch
// configuration and the launch order of the forward and backward passes.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>
#include <algorithm>
#include <mutex>
#include <unordered_map>

#include <rocblas/rocblas.h>

#include "../../include/stacklstm.h"
#include "common.h"
#include "gemm.h"
#include "rec_config.h"
#include "recurrent.h"

__global__ void k_init_ctl(uint32_t* ctl);
__global__ void k_scan(const int8_t* ops, int T, int B, int32_t* ptr, int32_t* depth_end, uint32_t* ctl);
__global__ void k_gather_top(const int32_t* top, const float* cellv, const float* init, float* out, int T, int B,
                             int H, int skip_push);
__global__ void k_trace(const int8_t* ops, int T, int B, int cap, int32_t* top);
__global__ void k_gather_top4(const int32_t* top, const float* hcell, const float* h0, float* htop, const float* ccell,
                              const float* c0, float* ctop, int T, int B, int H, int skip_h);
__global__ void k_permute_w(const float* W, float* Wp32, bf16_t* Wp16, int I, int H);
__global__ void k_fill_f32(float* p, size_t n, float v);
__global__ void k_zero_u32(uint32_t* p, int n);
__global__ void k_zero_ctl_bwd(uint32_t* ctl);
__global__ void k_fill_pattern(unsigned char* p, size_t bytes, uint32_t v);
__global__ void k_h0_bf16(const float* h0, bf16_t* hx, size_t n);
__global__ void k_to_bf16(const float* in, bf16_t* out, size_t n);
__global__ void k_augment_x(const float* x, size_t rows, int I, int KA, int nones, float* out32, bf16_t* out16);
__global__ void k_bias_rows(const float* b, int H, int nparts, int nrows, float* out32, bf16_t* out16);
__global__ void k_push_rows(const int8_t* ops, int n, int32_t* rows, uint32_t* count);
__global__ void k_zero_nonpush_rows(const int8_t* ops, float* out, size_t n, int cols);
__global__ void k_gather_rows(const float* src, const int32_t* prow, const uint32_t* count, size_t max_rows, int cols,
                              int scatter, float* dst);
__global__ void k_gather_hprev(const int32_t* top, const float* hcell, const float* h0, const int32_t* prow,
                               const uint32_t* count, float* out, int T, int B, int H);
__global__ void k_transpose_bf16(const void* src, int src_f32, int ld, int cols, const int32_t* prow,
                                 const uint32_t* count, int ldo, const int32_t* gtop, int B, bf16_t* out);
template <int PREC, int AL, int BL> __global__ void k_gemm(GemmArgs g);
__global__ void k_reduce_splits(const float* P, int splits, size_t split_stride, int M, int N, int unperm_H,
                                float* out);

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

// Rows per group are chosen per kernel (forward and backward differ in register use and so
// in how many workgroups share a CU): NT/G/per_xcc for the forward, NTb/Gb/per_xcc_b for
// the backward.
struct Plan {
  int prec, KS, ks_eff, NW;
  int NT, G, per_xcc, pipe;   // pipe: the forward runs the pipelined kernel
  int wide, NWw;              // wide: the forward runs the 32-unit kernel (NWw workgroups per group)
  int NTb, Gb, per_xcc_b;
  int splits_w, splits_u;
};

struct Layout {
  size_t ctl, stack, wp, r1, stash, hx, xb, xbt, hp, dat, dh, dc, dbp, part, prow, dep, dac, xc, total;
};

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

int splits_for(int M, int N, int K) {
  int tiles = ((M + kGemmBM - 1) / kGemmBM) * ((N + kGemmBN - 1) / kGemmBN);
  int s = std::max(1, 1024 / std::max(1, tiles));
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
  const int cus = device_cus();
  const int cu_per_xcc = cus > 0 ? cus / 8 : 32;
  // smallest row tile count per group whose workgroups (NW per group, groups dealt to the 8
  // XCCs round-robin) are co-resident on one XCC at the kernel's occupancy
  // the pipelined forward needs whole 1 KB row segments (vector rows, every K chunk in use)
  const bool pipe_ok = d->H % (prec ? 8 : 4) == 0 && p->ks_eff == p->KS && p->KS >= 16;
  auto pick = [&](bool bwd, int* NT_out, int* G_out, int* per_out, int* pipe_out) -> int {
    for (int NT = 1; NT <= 8; NT *= 2) {
      int G = (d->B + 16 * NT - 1) / (16 * NT);
      if (G > MAX_GROUPS) continue;
      int per_xcc = p->NW * ((G + 7) / 8);
      int occ = 0;
      const bool pipe = !bwd && pipe_ok && NT >= 2 && rec_pipe_built(prec, NT, p->KS);
      RecArgs dummy;
      memset(&dummy, 0, sizeof(dummy));
      hipError_t e = bwd    ? launch_bwd(dummy, prec, NT, p->KS, dim3(0), nullptr, &occ)
                     : pipe ? launch_fwd_pipe(dummy, prec, NT, p->KS, dim3(0), nullptr, &occ)
                            : launch_fwd(dummy, prec, NT, p->KS, dim3(0), nullptr, &occ);
      if (e != hipSuccess) return SLSTM_EDEVICE;
      if (per_xcc <= cu_per_xcc * occ) {
        *NT_out = NT;
        *G_out = G;
        *per_out = per_xcc;
        if (pipe_out) *pipe_out = pipe ? 1 : 0;
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

// The input projection XW = x Wp + b is one plain GEMM on the vendor BLAS: x gets columns of
// ones (one in fp32 mode; three in bf16 mode, where b is carried as the sum of three bf16
// parts, so the bias keeps fp32 precision) and Wp gets the matching bias rows; K is padded
// to a multiple of 32 with zeros (the vendor GEMM picks faster tiles for such K: measured
// 0.12 ms against 0.15 ms in bf16 at T*B = 61440, 4H = 2048, I = 256).
int xw_ones(const slstm_dims* d) { return d->precision == SLSTM_BF16_GEMM ? 3 : 1; }
size_t xw_k(const slstm_dims* d) { return ((size_t)d->I + xw_ones(d) + 31) / 32 * 32; }

// rocBLAS handles, one per (device, stream), created on first use with atomic
// (order-dependent) kernels disabled, so a GEMM's result does not depend on what runs beside
// it. A handle owns a device work space that its split-K GEMMs write, so GEMMs that run at
// once on two streams need two handles. Calls are serialised under blas_mutex().
std::mutex& blas_mutex() {
  static std::mutex mu;
  return mu;
}
// Side stream and fork/join events per device (default priority, kept for the process's
// lifetime): the producer trace runs there, beside the input projection on the caller's
// stream. Enqueued under blas_mutex(), so a join always follows the trace of the same call.
struct SideStream { hipStream_t s; hipEvent_t fork, join; bool ok; };
SideStream* side_stream() {
  static SideStream ss[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  SideStream& x = ss[dev];
  if (!x.ok) {
    if (hipStreamCreateWithFlags(&x.s, hipStreamNonBlocking) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&x.fork, hipEventDisableTiming) != hipSuccess) return nullptr;
    if (hipEventCreateWithFlags(&x.join, hipEventDisableTiming) != hipSuccess) return nullptr;
    x.ok = true;
  }
  return &x;
}
// At most kBlasHandles handles per device: past that the device is drained and its handles
// are released before a new one is made (the streams of earlier calls may be gone).
constexpr int kBlasHandles = 32;
rocblas_handle blas_handle(hipStream_t st) {
  struct Entry { hipStream_t st; rocblas_handle h; };
  static Entry tab[64][kBlasHandles] = {};
  static int used[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  Entry* e = tab[dev];
  for (int i = 0; i < used[dev]; ++i)
    if (e[i].st == st) return e[i].h;
  if (used[dev] == kBlasHandles) {
    if (hipDeviceSynchronize() != hipSuccess) return nullptr;
    for (int i = 0; i < used[dev]; ++i) rocblas_destroy_handle(e[i].h);
    used[dev] = 0;
  }
  rocblas_handle h = nullptr;
  if (rocblas_create_handle(&h) != rocblas_status_success) return nullptr;
  if (rocblas_set_atomics_mode(h, rocblas_atomics_not_allowed) != rocblas_status_success ||
      rocblas_set_stream(h, st) != rocblas_status_success) {
    rocblas_destroy_handle(h);
    return nullptr;
  }
  e[used[dev]++] = Entry{st, h};
  return h;
}

// Number of push rows per work space, read back with the forward's status: the backward's
// vendor-BLAS gradient GEMMs need it on the host. A backward without a recorded count (or
// with other T, B) runs the device-count kernels instead.
struct PushCount { int T, B; uint32_t n; };
std::mutex& push_mutex() {
  static std::mutex mu;
  return mu;
}
std::unordered_map<const void*, PushCount>& push_counts() {
  static std::unordered_map<const void*, PushCount> m;
  return m;
}

// Work-space layout; splits are bounded by 64 so the layout does not depend on the device.
Layout layout(const slstm_dims* d) {
  const size_t T = d->T, B = d->B, I = d->I, H = d->H;
  const bool bf = d->precision == SLSTM_BF16_GEMM;
  const size_t KP = padded_rows(d);
  Layout L;
  size_t o = 0;
  L.ctl = o; o += align256(CTL_WORDS * 4);
  L.stack = o; o += align256(B * (T + 1) * 4);
  const size_t KA = xw_k(d);
  L.wp = o; o += align256(KA * 4 * H * 4);                              // Wp and its bias rows
  L.r1 = o; o += align256(std::max<size_t>(T * B * 4 * H * 4, 16));   // XW (forward), dA (backward)
  L.stash = o; o += align256(std::max<size_t>(T * B * 4 * H * 4, 16));
  L.hx = o; o += bf ? align256((T + 1) * B * H * 2) : 0;
  L.xb = o; o += align256(T * B * KA * (bf ? 2 : 4));                 // [x | ones | 0] for the XW GEMM
  // post-loop operands over the push rows (at most T*B of them; KP with the K-tile padding)
  L.xbt = o; o += bf ? align256(KP * I * 2) : 0;                      // x^T in bf16 (bf16 mode)
  L.hp = o; o += align256(std::max<size_t>(bf ? KP * H * 2 : T * B * H * 4, 16));   // Hprev (bf16 mode: Hprev^T)
  L.dat = o; o += bf ? align256(KP * 4 * H * 2) : 0;                  // dA^T in bf16 (bf16 mode)
  L.dh = o; o += align256((T + 1) * B * H * 4);
  L.dc = o; o += align256((T + 1) * B * H * 4);
  L.dbp = o; o += align256((size_t)MAX_GROUPS * 4 * H * 4);
  L.part = o; o += align256((size_t)64 * std::max(I, H) * 4 * H * 4);
  L.prow = o; o += align256(std::max<size_t>(T * B * 4, 16));         // push-row list
  L.dep = o; o += align256(B * 4);                                     // pointer after the last step
  // fp32 post-loop operands on the vendor BLAS: dA and x rows of the push steps, compacted
  L.dac = o; o += bf ? 0 : align256(std::max<size_t>(T * B * 4 * H * 4, 16));
  L.xc = o; o += align256(std::max<size_t>(T * B * std::max(I, (size_t)1) * 4, 16));   // also dx rows in bf16 mode
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
  GCASE(1, GEMM_MK, GEMM_KN) GCASE(1, GEMM_MK, GEMM_NK) GCASE(1, GEMM_KM, GEMM_KN)
#undef GCASE
  return SLSTM_EINVAL;
}

// K slice per split, a multiple of the GEMM's K tile (64 covers both precisions)
int k_chunk_for(int K, int splits) { return ((K + splits - 1) / splits + 63) / 64 * 64; }

int check_timeout(const uint32_t* ctl, hipStream_t st) {
  uint32_t v = 0;
  if (hipMemcpyAsync(&v, ctl + CTL_TIMEOUT, 4, hipMemcpyDeviceToHost, st) != hipSuccess) return SLSTM_EDEVICE;
  if (hipStreamSynchronize(st) != hipSuccess) return SLSTM_EDEVICE;
  return v ? SLSTM_ETIMEOUT : SLSTM_OK;
}

RecArgs rec_args(const slstm_dims* d, const Plan& p, char* ws, const Layout& L, bool bwd) {
  RecArgs a;
  memset(&a, 0, sizeof(a));
  a.T = d->T; a.B = d->B; a.I = d->I; a.H = d->H;
  a.G = bwd ? p.Gb : p.G; a.NW = p.NW; a.ks_eff = p.ks_eff;
  a.spin_limit = d->spin_limit > 0 ? d->spin_limit : kDefaultSpin;
  a.ctl = (uint32_t*)(ws + L.ctl);
  a.stack = (int32_t*)(ws + L.stack);
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
  a.coh_top = ((size_t)d->B * 4) % 128 != 0;
  // backward direct staging: whole 1 KB row segments, K range equal to the register capacity,
  // and the LDS slice plus static LDS within one CU (one workgroup per CU)
  const int KC = rec_kc(d->precision);
  a.bwd_direct = ((size_t)d->H * esz) % 1024 == 0 && p.KS * KC == d->H && rec_occ(d->precision, p.KS) == 1 &&
                 rec_bwd_lds_bytes(d->precision, p.KS) + rec_bwd_static_lds(p.NTb) <= 160 * 1024 &&
                 p.per_xcc_b <= std::max(1, device_cus() / 8);
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
    default: return "unknown status";
  }
}

int stacklstm_plan(const slstm_dims* d, int32_t* groups, int32_t* wg_per_group, int32_t* rows_per_group,
                   int32_t* k_chunks) {
  Plan p;
  int rc = make_plan(d, &p);
  if (rc) return rc;
  if (groups) *groups = p.G;
  if (wg_per_group) *wg_per_group = p.wide ? p.NWw : p.NW;
  if (rows_per_group) *rows_per_group = 16 * p.NT;
  if (k_chunks) *k_chunks = p.ks_eff;
  return SLSTM_OK;
}

int stacklstm_fwd(const slstm_dims* d, const float* x, const int8_t* ops, const float* W, const float* U,
                  const float* b, const float* h0, const float* c0, float* h_cell, float* c_cell, float* h_top,
                  float* c_top, int32_t* ptr, int32_t* top, void* workspace, size_t ws_bytes, void* stream) {
  if (!dims_ok(d)) return SLSTM_EINVAL;
  if (!ptr || !workspace ||
      (d->T > 0 && (!ops || !x || !W || !U || !b || !h0 || !c0 || !h_cell || !c_cell || !top)))
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

  // a1: validate ops and scan the pointer (the call's one host synchronisation)
  mark(d, 0, st);
  hipLaunchKernelGGL(k_init_ctl, dim3(1), dim3(256), 0, st, ctl);
  hipLaunchKernelGGL(k_scan, dim3((B + 15) / 16), dim3(256), 0, st, ops, T, B, ptr, (int32_t*)(ws + L.dep), ctl);
  uint32_t hs[CTL_NPUSHF + 1] = {};
  if (hipMemcpyAsync(hs, ctl + CTL_STATUS, sizeof(hs), hipMemcpyDeviceToHost, st) != hipSuccess) return SLSTM_EDEVICE;
  if (hipStreamSynchronize(st) != hipSuccess) return SLSTM_EDEVICE;
  if (hs[0] != 0x7fffffffu) return (int)(hs[0] & 7u);
  {
    std::lock_guard<std::mutex> lk(push_mutex());
    if (push_counts().size() > 4096) push_counts().clear();   // bounded: work spaces are reused in practice
    push_counts()[workspace] = PushCount{T, B, hs[CTL_NPUSHF]};
  }
  // the wide and the pipelined forward read a finished producer trace (they keep no integer
  // stack of their own); the plain forward traces in-kernel
  const bool pretrace = p.wide || p.pipe;
  // producer trace from the ops: one thread per element, its stack in LDS (odd slot count:
  // no bank conflicts between neighbours); launched beside the input projection below
  const int trace_cap = (int)std::min<uint32_t>(hs[1] + 2u, (uint32_t)T + 1u) | 1;
  int trace_R = 64;
  while (trace_R > 1 && (size_t)trace_R * trace_cap * 4 > 48 * 1024) trace_R /= 2;
  if (T > 0 && pretrace && (size_t)trace_R * trace_cap * 4 > 48 * 1024) return SLSTM_EINVAL;   // deeper than 12 K slots
  mark(d, 1, st);
  if (T == 0) return SLSTM_OK;

  // a2: XW = [x | 1] [Wp ; b] for all steps (Wp = W with gate-interleaved columns), on rocBLAS
  const bool bf = p.prec == SLSTM_BF16_GEMM;
  void* wp = ws + L.wp;
  const int KA = (int)xw_k(d), NO = xw_ones(d);
  hipLaunchKernelGGL(k_permute_w, dim3(grid1d((size_t)I * 4 * H)), dim3(256), 0, st, W,
                     bf ? nullptr : (float*)wp, bf ? (bf16_t*)wp : nullptr, I, H);
  hipLaunchKernelGGL(k_bias_rows, dim3(grid1d((size_t)(KA - I) * 4 * H)), dim3(256), 0, st, b, H, NO, KA - I,
                     bf ? nullptr : (float*)wp + (size_t)I * 4 * H, bf ? (bf16_t*)wp + (size_t)I * 4 * H : nullptr);
  float* xw = (float*)(ws + L.r1);
  void* xa = ws + L.xb;
  hipLaunchKernelGGL(k_augment_x, dim3(grid1d((size_t)T * B * KA)), dim3(256), 0, st, x, (size_t)T * B, I, KA, NO,
                     bf ? nullptr : (float*)xa, bf ? (bf16_t*)xa : nullptr);
  if ((rc = hip_status(hipGetLastError()))) return rc;
  {
    // column-major view: XW^T [4H x TB] = Wp_aug^T [4H x KA] . x_aug^T [KA x TB]
    std::lock_guard<std::mutex> lk(blas_mutex());
    SideStream* side = pretrace ? side_stream() : nullptr;
    if (pretrace && !side) return SLSTM_EDEVICE;
    if (pretrace) {
      if (hipEventRecord(side->fork, st) != hipSuccess || hipStreamWaitEvent(side->s, side->fork, 0) != hipSuccess)
        return SLSTM_EDEVICE;
      hipLaunchKernelGGL(k_trace, dim3((B + trace_R - 1) / trace_R), dim3(trace_R), (size_t)trace_R * trace_cap * 4,
                         side->s, ops, T, B, trace_cap, top);
      if (hipEventRecord(side->join, side->s) != hipSuccess) return SLSTM_EDEVICE;
    }
    rocblas_handle h = blas_handle(st);
    if (!h) return SLSTM_EDEVICE;
    const float one = 1.f, zero = 0.f;
    rocblas_status bs;
    if (!bf)
      bs = rocblas_sgemm(h, rocblas_operation_none, rocblas_operation_none, 4 * H, T * B, KA, &one, (const float*)wp,
                         4 * H, (const float*)xa, KA, &zero, xw, 4 * H);
    else
      bs = rocblas_gemm_ex(h, rocblas_operation_none, rocblas_operation_none, 4 * H, T * B, KA, &one, wp,
                           rocblas_datatype_bf16_r, 4 * H, xa, rocblas_datatype_bf16_r, KA, &zero, xw,
                           rocblas_datatype_f32_r, 4 * H, xw, rocblas_datatype_f32_r, 4 * H, rocblas_datatype_f32_r,
                           rocblas_gemm_algo_standard, 0, 0);
    if (bs != rocblas_status_success) return SLSTM_EDEVICE;
    if (pretrace && hipStreamWaitEvent(st, side->join, 0) != hipSuccess) return SLSTM_EDEVICE;
  }

  // a3-a6: persistent recurrent kernel
  RecArgs a = rec_args(d, p, ws, L, false);
  if (bf) hipLaunchKernelGGL(k_h0_bf16, dim3(grid1d((size_t)B * H)), dim3(256), 0, st, h0, (bf16_t*)a.hx, (size_t)B * H);
  a.xw = xw; a.ops = ops; a.U = U; a.h0 = h0; a.c0 = c0; a.hcell = h_cell; a.ccell = c_cell; a.top = top;
  // exchange buffers start as "not yet produced": all-one bits in the state rows the
  // workgroups read from each other, kTopPending in the producer-index table
  if (a.poll || p.wide) {
    const size_t ex_bytes = (size_t)T * B * H * (bf ? 2 : 4);
    unsigned char* ex = bf ? (unsigned char*)(a.hx + (size_t)B * H) : (unsigned char*)h_cell;
    hipLaunchKernelGGL(k_fill_pattern, dim3(grid1d(ex_bytes / 16 + 1)), dim3(256), 0, st, ex, ex_bytes, 0xffffffffu);
    if (!pretrace)
      hipLaunchKernelGGL(k_fill_pattern, dim3(grid1d((size_t)T * B / 4 + 1)), dim3(256), 0, st,
                         (unsigned char*)top, (size_t)T * B * 4, kTopPending);
  }
  a.traced = pretrace ? 1 : 0;
  a.htop = p.wide ? h_top : nullptr;
  a.ctop = p.wide ? c_top : nullptr;
  if (p.wide) a.NW = p.NWw;
  mark(d, 2, st);
  if ((rc = hip_status(p.wide   ? launch_fwd_wide(a, p.NT, p.KS, dim3(8 * p.per_xcc), st, nullptr)
                       : p.pipe ? launch_fwd_pipe(a, p.prec, p.NT, p.KS, dim3(8 * p.per_xcc), st, nullptr)
                                : launch_fwd(a, p.prec, p.NT, p.KS, dim3(8 * p.per_xcc), st, nullptr))))
    return rc;
  mark(d, 3, st);

  // a7: Algorithm 1's return values (the wide forward writes c_top and the h_top of push steps)
  size_t n = (size_t)T * B * H;
  float* ctop_g = p.wide ? nullptr : c_top;          // the wide forward writes c_top itself
  const auto al16 = [](const void* q) { return ((uintptr_t)q & 15u) == 0; };
  if (H % 4 == 0 && al16(h_cell) && al16(h0) && al16(h_top) && al16(c_cell) && al16(c0) && al16(c_top)) {
    if (h_top || ctop_g)
      hipLaunchKernelGGL(k_gather_top4, dim3(grid1d(n / 4)), dim3(256), 0, st, top, h_cell, h0, h_top, c_cell, c0, ctop_g,
                         T, B, H, p.wide);
  } else {
    if (h_top)
      hipLaunchKernelGGL(k_gather_top, dim3(grid1d(n)), dim3(256), 0, st, top, h_cell, h0, h_top, T, B, H, p.wide);
    if (ctop_g)
      hipLaunchKernelGGL(k_gather_top, dim3(grid1d(n)), dim3(256), 0, st, top, c_cell, c0, ctop_g, T, B, H, 0);
  }
  if ((rc = hip_status(hipGetLastError()))) return rc;
  mark(d, 4, st);
  if (d->spin_limit > 0) return check_timeout(ctl, st);
  return SLSTM_OK;
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
  if (T == 0) {
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)I * 4 * H)), dim3(256), 0, st, dW, (size_t)I * 4 * H, 0.f);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)H * 4 * H)), dim3(256), 0, st, dU, (size_t)H * 4 * H, 0.f);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)4 * H)), dim3(256), 0, st, db, (size_t)4 * H, 0.f);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)B * H)), dim3(256), 0, st, dh0, (size_t)B * H, 0.f);
    hipLaunchKernelGGL(k_fill_f32, dim3(grid1d((size_t)B * H)), dim3(256), 0, st, dc0, (size_t)B * H, 0.f);
    return hip_status(hipGetLastError());
  }

  // a8: persistent reverse loop
  hipLaunchKernelGGL(k_zero_ctl_bwd, dim3(1), dim3(256), 0, st, ctl);
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
  // rows of the push steps, for the post-loop gradients (dA is exactly zero on other rows)
  int32_t* prow = (int32_t*)(ws + L.prow);
  const uint32_t* npush = ctl + CTL_NPUSH;
  hipLaunchKernelGGL(k_push_rows, dim3(1), dim3(1024), 0, st, ops, T * B, prow, ctl + CTL_NPUSH);
  // dA rows start as "not yet produced" (all-one bits): the workgroups read them from each other
  if (a.poll) {
    const size_t da_bytes = (size_t)T * B * 4 * H * (bf ? 2 : 4);
    hipLaunchKernelGGL(k_fill_pattern, dim3(grid1d(da_bytes / 16 + 1)), dim3(256), 0, st, (unsigned char*)a.dA,
                       da_bytes, 0xffffffffu);
  }
  mark(d, 5, st);
  if ((rc = hip_status(launch_bwd(a, p.prec, p.NTb, p.KS, dim3(8 * p.per_xcc_b), st, nullptr)))) return rc;
  mark(d, 6, st);

  // a9: post-loop gradients, contracted over the push rows only (rows prow[0 .. *npush))
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
  // dW = x^T dA and dU = Hprev^T dA over the push rows. fp32: the GEMM gathers x and dA rows
  // through prow, Hprev is gathered first; bf16: the three operands are written transposed
  // and compacted (k = push index contiguous, zero up to the next multiple of 64).
  if (bf) {
    const dim3 tg4((H4 + 63) / 64, KP / 64), tgI((I + 63) / 64, KP / 64), tgH((H + 63) / 64, KP / 64);
    hipLaunchKernelGGL(k_transpose_bf16, tg4, dim3(256), 0, st, a.dA, 0, H4, H4, prow, npush, KP,
                       (const int32_t*)nullptr, B, (bf16_t*)(ws + L.dat));
    hipLaunchKernelGGL(k_transpose_bf16, tgI, dim3(256), 0, st, x, 1, I, I, prow, npush, KP, (const int32_t*)nullptr,
                       B, (bf16_t*)(ws + L.xbt));
    hipLaunchKernelGGL(k_transpose_bf16, tgH, dim3(256), 0, st, ws + L.hx, 0, H, H, prow, npush, KP, top, B,
                       (bf16_t*)hp);
  } else {
    hipLaunchKernelGGL(k_gather_hprev, dim3(grid1d((size_t)K * H)), dim3(256), 0, st, top, h_cell, h0, prow, npush,
                       (float*)hp, T, B, H);
  }
  // fp32 with the push count known on the host (recorded by the forward on this work space):
  // the three gradient GEMMs on rocBLAS over compacted push rows
  uint32_t np_host = 0;
  {
    std::lock_guard<std::mutex> lk(push_mutex());
    auto it = push_counts().find(workspace);
    if (it != push_counts().end() && it->second.T == T && it->second.B == B && it->second.n <= (uint32_t)K)
      np_host = it->second.n;
  }
  if (bf && np_host > 0) {
    // bf16 operands are already compacted and transposed: xbt [I][KP], dat [4H][KP] (push index
    // contiguous, zero past the count); dx on rocBLAS, dW and dU on the library's kernel (faster
    // than the vendor BLAS on these transposed operands, measured at large)
    const int np = (int)np_host;
    float* xc = (float*)(ws + L.xc);
    const float one = 1.f, zero = 0.f;
    gemm_base();
    g.M = I; g.N = H4; g.dyn_axis = 1;
    g.K = KP; g.A = ws + L.xbt; g.lda = KP; g.a_vec = 1; g.Bm = ws + L.dat; g.ldb = KP; g.b_vec = 1;
    g.C = part; g.ldc = H4;
    g.split_stride = (size_t)I * H4;
    if ((rc = launch_gemm(p.prec, GEMM_MK, GEMM_NK, g, p.splits_w, st))) return rc;
    hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)I * H4)), dim3(256), 0, st, part, p.splits_w,
                       g.split_stride, I, H4, H, dW);
    mark(d, 7, st);
    gemm_base();
    g.M = H; g.N = H4; g.dyn_axis = 1;
    g.K = KP; g.A = hp; g.lda = KP; g.a_vec = 1; g.Bm = ws + L.dat; g.ldb = KP; g.b_vec = 1;
    g.C = part; g.ldc = H4;
    g.split_stride = (size_t)H * H4;
    if ((rc = launch_gemm(p.prec, GEMM_MK, GEMM_NK, g, p.splits_u, st))) return rc;
    hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)H * H4)), dim3(256), 0, st, part, p.splits_u,
                       g.split_stride, H, H4, H, dU);
    mark(d, 8, st);
    {
      std::lock_guard<std::mutex> lk(blas_mutex());
      rocblas_handle h = blas_handle(st);
      if (!h) return SLSTM_EDEVICE;
      // dx_c^T [I x np] = Wp [I x 4H] . dat [4H x np]   (Wp rows are the first I of [Wp ; b])
      if (rocblas_gemm_ex(h, rocblas_operation_transpose, rocblas_operation_transpose, I, np, H4, &one, ws + L.wp,
                          rocblas_datatype_bf16_r, H4, ws + L.dat, rocblas_datatype_bf16_r, KP, &zero, xc,
                          rocblas_datatype_f32_r, I, xc, rocblas_datatype_f32_r, I, rocblas_datatype_f32_r,
                          rocblas_gemm_algo_standard, 0, 0) != rocblas_status_success)
        return SLSTM_EDEVICE;
    }
    hipLaunchKernelGGL(k_zero_nonpush_rows, dim3(grid1d((size_t)K * I / 4 + 1)), dim3(256), 0, st, ops, dx, (size_t)K,
                       I);
    hipLaunchKernelGGL(k_gather_rows, dim3(grid1d((size_t)np * I / 4 + 1)), dim3(256), 0, st, (const float*)xc, prow,
                       npush, (size_t)K, I, 1, dx);
    if ((rc = hip_status(hipGetLastError()))) return rc;
    mark(d, 9, st);
    if (d->spin_limit > 0) return check_timeout(ctl, st);
    return SLSTM_OK;
  }
  if (!bf && np_host > 0) {
    float* dac = (float*)(ws + L.dac);
    float* xc = (float*)(ws + L.xc);
    const int np = (int)np_host;
    hipLaunchKernelGGL(k_gather_rows, dim3(grid1d((size_t)np * H4 / 4)), dim3(256), 0, st, (const float*)a.dA, prow,
                       npush, (size_t)K, H4, 0, dac);
    hipLaunchKernelGGL(k_gather_rows, dim3(grid1d((size_t)np * I / 4 + 1)), dim3(256), 0, st, x, prow, npush,
                       (size_t)K, I, 0, xc);
    if ((rc = hip_status(hipGetLastError()))) return rc;
    const float one = 1.f, zero = 0.f;
    {
      std::lock_guard<std::mutex> lk(blas_mutex());
      rocblas_handle h = blas_handle(st);
      if (!h) return SLSTM_EDEVICE;
      // column-major views: dWp^T [4H x I] = dA_c^T [4H x np] . x_c [np x I]
      if (rocblas_sgemm(h, rocblas_operation_none, rocblas_operation_transpose, H4, I, np, &one, dac, H4, xc, I, &zero,
                        part, H4) != rocblas_status_success)
        return SLSTM_EDEVICE;
    }
    hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)I * H4)), dim3(256), 0, st, part, 1, (size_t)I * H4, I, H4,
                       H, dW);
    mark(d, 7, st);
    {
      std::lock_guard<std::mutex> lk(blas_mutex());
      rocblas_handle h = blas_handle(st);
      if (!h) return SLSTM_EDEVICE;
      // dUp^T [4H x H] = dA_c^T [4H x np] . Hprev_c [np x H]
      if (rocblas_sgemm(h, rocblas_operation_none, rocblas_operation_transpose, H4, H, np, &one, dac, H4,
                        (const float*)hp, H, &zero, part, H4) != rocblas_status_success)
        return SLSTM_EDEVICE;
    }
    hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)H * H4)), dim3(256), 0, st, part, 1, (size_t)H * H4, H, H4,
                       H, dU);
    mark(d, 8, st);
    {
      std::lock_guard<std::mutex> lk(blas_mutex());
      rocblas_handle h = blas_handle(st);
      if (!h) return SLSTM_EDEVICE;
      // dx_c^T [I x np] = Wp [I x 4H] . dA_c^T [4H x np]   (Wp rows are the first I of [Wp ; b])
      if (rocblas_sgemm(h, rocblas_operation_transpose, rocblas_operation_none, I, np, H4, &one, (const float*)(ws + L.wp),
                        H4, dac, H4, &zero, xc, I) != rocblas_status_success)
        return SLSTM_EDEVICE;
    }
    hipLaunchKernelGGL(k_zero_nonpush_rows, dim3(grid1d((size_t)K * I / 4 + 1)), dim3(256), 0, st, ops, dx, (size_t)K,
                       I);
    hipLaunchKernelGGL(k_gather_rows, dim3(grid1d((size_t)np * I / 4 + 1)), dim3(256), 0, st, (const float*)xc, prow,
                       npush, (size_t)K, I, 1, dx);
    if ((rc = hip_status(hipGetLastError()))) return rc;
    mark(d, 9, st);
    if (d->spin_limit > 0) return check_timeout(ctl, st);
    return SLSTM_OK;
  }
  gemm_base();
  g.M = I; g.N = H4; g.dyn_axis = 1;
  if (bf) { g.K = KP; g.A = ws + L.xbt; g.lda = KP; g.a_vec = 1; g.Bm = ws + L.dat; g.ldb = KP; g.b_vec = 1; }
  else    { g.K = K; g.A = x; g.lda = I; g.a_vec = (I % 4 == 0); g.a_rows = prow;
            g.Bm = a.dA; g.ldb = H4; g.b_vec = 1; g.b_rows = prow; }
  g.C = part; g.ldc = H4;
  g.split_stride = (size_t)I * H4;
  if ((rc = launch_gemm(p.prec, bf ? GEMM_MK : GEMM_KM, bf ? GEMM_NK : GEMM_KN, g, p.splits_w, st))) return rc;
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)I * H4)), dim3(256), 0, st, part, p.splits_w,
                     g.split_stride, I, H4, H, dW);
  mark(d, 7, st);
  gemm_base();
  g.M = H; g.N = H4; g.dyn_axis = 1;
  if (bf) { g.K = KP; g.A = hp; g.lda = KP; g.a_vec = 1; g.Bm = ws + L.dat; g.ldb = KP; g.b_vec = 1; }
  else    { g.K = K; g.A = hp; g.lda = H; g.a_vec = (H % 4 == 0); g.Bm = a.dA; g.ldb = H4; g.b_vec = 1;
            g.b_rows = prow; }
  g.C = part; g.ldc = H4;
  g.split_stride = (size_t)H * H4;
  if ((rc = launch_gemm(p.prec, bf ? GEMM_MK : GEMM_KM, bf ? GEMM_NK : GEMM_KN, g, p.splits_u, st))) return rc;
  hipLaunchKernelGGL(k_reduce_splits, dim3(grid1d((size_t)H * H4)), dim3(256), 0, st, part, p.splits_u,
                     g.split_stride, H, H4, H, dU);
  mark(d, 8, st);
  // dx = dA Wp^T on the push rows (gathered from dA, scattered into dx); 0 on the others
  gemm_base();
  g.dyn_round = 1; g.dyn_axis = 0;
  g.M = K; g.N = I; g.K = H4;
  const int VE = bf ? 8 : 4;
  g.A = a.dA; g.lda = H4; g.a_vec = (H4 % VE == 0); g.a_rows = prow;
  g.Bm = ws + L.wp; g.ldb = H4; g.b_vec = (H4 % VE == 0) && (I % VE == 0);
  g.C = dx; g.ldc = I; g.c_rows = prow;
  g.k_chunk = k_chunk_for(H4, 1);
  if ((rc = launch_gemm(p.prec, GEMM_MK, GEMM_NK, g, 1, st))) return rc;
  hipLaunchKernelGGL(k_zero_nonpush_rows, dim3(grid1d((size_t)K * I / 4 + 1)), dim3(256), 0, st, ops, dx, (size_t)K,
                     I);
  if ((rc = hip_status(hipGetLastError()))) return rc;
  mark(d, 9, st);
  if (d->spin_limit > 0) return check_timeout(ctl, st);
  return SLSTM_OK;
}

int stacklstm_sync_status(const void* workspace, size_t ws_bytes, void* stream) {
  if (!workspace || ws_bytes < align256(CTL_WORDS * 4)) return SLSTM_EINVAL;
  return check_timeout((const uint32_t*)workspace, (hipStream_t)stream);
}

}  // extern "C"
