// Op validation and stack-pointer scan (paper, section 3: the unified update p <- p + op
// with op in {+1 push, -1 pop, 0 hold}). ptr[t][b] is the pointer before step t;
// ptr[T][b] the pointer after the last step, also kept in depth_end[b] for the backward. A pop while only the initial state is on
// the stack (p would become -1) is reported as EUNDERFLOW, an op outside {-1, 0, 1} as
// EOPS; the reported element is the lowest failing batch index, and within it the
// earliest failing step decides the code.
#include "common.h"

// Control words of a forward call at 0 (status: no error). With keep_errors (a deferred
// call) the error words keep what earlier calls on the work space set: the lowest failing
// element's op status, the time-out and the index flag.
__global__ void __launch_bounds__(256) k_init_ctl(uint32_t* ctl, int keep_errors) {
  for (int i = threadIdx.x; i < CTL_WORDS; i += blockDim.x) {
    const bool err = i == CTL_STATUS || i == CTL_TIMEOUT || i == CTL_BADIDX;
    if (keep_errors && err) continue;
    ctl[i] = (i == CTL_STATUS) ? kStatusOk : 0u;
  }
}

// Op validation, pointer scan and producer trace in one pass (section 3: the unified update
// p <- p + op on an integer stack of step indices). One thread per batch element walks its
// op stream: ptr[t+1][b] = p after step t, top[t][b] = the step that produced the state at
// the pointer after step t (-1 = the initial state). The element's stack of step indices
// has cap = T + 1 slots (slot 0 = the initial state), in LDS (LDS = true: blockDim.x stacks of
// cap ints) or in the work space (gstack [B][cap]). Each thread loads its next
// CH ops as independent byte loads (consecutive lanes read consecutive bytes), so a chunk
// costs one memory round trip. An invalid op is reported (EOPS) and walked as a hold; a pop
// at p = 0 is reported (EUNDERFLOW) and walked as a hold, so every trace value stays a valid
// producer index even then. Also: the number of pushes (CTL_NPUSHF), the deepest pointer
// (CTL_MAXDEPTH) and the pointer after the last step (depth_end, for the backward).
template <bool LDS>
__global__ void __launch_bounds__(64) k_scan(const int8_t* __restrict__ ops, int T, int B, int cap,
                                             int32_t* __restrict__ ptr, int32_t* __restrict__ top,
                                             int32_t* __restrict__ depth_end, int32_t* __restrict__ gstack,
                                             uint32_t* ctl) {
  constexpr int CH = 32;
  extern __shared__ int s_stk[];
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  // LDS stacks are indexed through s_stk itself (LDS instructions: a pop's read does not wait
  // for the pointer and trace stores in flight)
  const size_t sbase = LDS ? (size_t)threadIdx.x * cap : (size_t)b * cap;
  auto stk = [&](int i) -> int& { return LDS ? s_stk[sbase + i] : gstack[sbase + i]; };
  int p = 0, tp = -1, npush = 0, maxd = 0;
  int first_bad = 0x7fffffff, first_uf = 0x7fffffff;
  stk(0) = -1;
  ptr[b] = 0;
  for (int t0 = 0; t0 < T; t0 += CH) {
    int8_t v[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) v[i] = (t0 + i < T) ? ops[(size_t)(t0 + i) * B + b] : (int8_t)0;
    // fully unrolled (constant register index of each op); steps past T are skipped by a guard
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int t = t0 + i;
      if (t >= T) continue;
      int op = v[i];
      if (op < -1 || op > 1) {
        if (first_bad == 0x7fffffff) first_bad = t;
        op = 0;
      }
      if (op == 1) {
        ++p;
        stk(p) = t;
        tp = t;
        ++npush;
      } else if (op == -1) {
        if (p == 0) {
          if (first_uf == 0x7fffffff) first_uf = t;
        } else {
          --p;
          tp = stk(p);
        }
      }
      maxd = max(maxd, p);
      ptr[(size_t)(t + 1) * B + b] = p;
      top[(size_t)t * B + b] = tp;
    }
  }
  depth_end[b] = p;
  if (npush) atomicAdd(&ctl[CTL_NPUSHF], (uint32_t)npush);
  atomicMax(&ctl[CTL_MAXDEPTH], (uint32_t)maxd);
  if (first_bad != 0x7fffffff || first_uf != 0x7fffffff)
    atomicMin((int*)&ctl[CTL_STATUS], b * 8 + (first_uf < first_bad ? ST_EUNDERFLOW : ST_EOPS));
}
template __global__ void k_scan<true>(const int8_t*, int, int, int, int32_t*, int32_t*, int32_t*, int32_t*, uint32_t*);
template __global__ void k_scan<false>(const int8_t*, int, int, int, int32_t*, int32_t*, int32_t*, int32_t*, uint32_t*);

// h_top / c_top materialisation: the state returned at step t (Algorithm 1's return value)
// is the one produced at step top[t][b], or the initial state when top is -1.
// With skip_push, rows whose step produced the returned state (top[t] = t) are left as they
// are (the wide forward kernel writes them).
__global__ void __launch_bounds__(256) k_gather_top(const int32_t* __restrict__ top, const float* __restrict__ cellv,
                                                    const float* __restrict__ init, float* __restrict__ out, int T,
                                                    int B, int H, int skip_push, uint32_t* ctl) {
  const size_t n = (size_t)T * B * H;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    size_t tb = i / H;
    int u = (int)(i - tb * H);
    int b = (int)(tb % B);
    int s = top[tb];
    int t = (int)(tb / B);
    if (skip_push && s == t) continue;
    s = checked_src(s, t, ctl);
    out[i] = (s < 0) ? init[(size_t)b * H + u] : cellv[((size_t)s * B + b) * H + u];
  }
}

// The same for h_top and c_top in one pass (either may be null; skip_h as skip_push for
// h_top), four units per thread: H must be a multiple of 4 and the arrays 16-byte aligned.
__global__ void __launch_bounds__(256) k_gather_top4(const int32_t* __restrict__ top, const float* __restrict__ hcell,
                                                     const float* __restrict__ h0, float* __restrict__ htop,
                                                     const float* __restrict__ ccell, const float* __restrict__ c0,
                                                     float* __restrict__ ctop, int T, int B, int H, int skip_h,
                                                     uint32_t* ctl) {
  const int H4 = H / 4;
  const size_t n = (size_t)T * B * H4;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t tb = i / H4;
    const int u4 = (int)(i - tb * H4);
    const int b = (int)(tb % B), t = (int)(tb / B);
    const int s0 = top[tb];
    const int s = checked_src(s0, t, ctl);
    const size_t src = s < 0 ? (size_t)b * H4 + u4 : ((size_t)s * B + b) * H4 + u4;
    if (htop && !(skip_h && s0 == t)) ((float4*)htop)[i] = s < 0 ? ((const float4*)h0)[src] : ((const float4*)hcell)[src];
    if (ctop) ((float4*)ctop)[i] = s < 0 ? ((const float4*)c0)[src] : ((const float4*)ccell)[src];
  }
}

// W [I][4H] (gate-major columns) -> Wp [I][4H] gate-interleaved, as fp32 or bf16, and its
// transpose WpT [4H][I] in bf16 (each output may be null).
__global__ void __launch_bounds__(256) k_permute_w(const float* __restrict__ W, float* __restrict__ Wp32,
                                                   bf16_t* __restrict__ Wp16, bf16_t* __restrict__ WpT16, int I,
                                                   int H) {
  const size_t n = (size_t)I * 4 * H;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    size_t row = i / (4 * (size_t)H);
    int np = (int)(i - row * 4 * H);
    float v = W[row * 4 * H + perm_to_orig(np, H)];
    if (Wp32) Wp32[i] = v;
    if (Wp16) Wp16[i] = f32_to_bf16_bits(v);
    if (WpT16) WpT16[(size_t)np * I + row] = f32_to_bf16_bits(v);
  }
}

__global__ void __launch_bounds__(256) k_fill_f32(float* __restrict__ p, size_t n, float v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

// Fills `bytes` bytes at p with the 32-bit pattern v (repeated; p and bytes multiples of 2 when
// the pattern's halves are equal, of 4 otherwise): 16-byte stores over the aligned middle.
__global__ void __launch_bounds__(256) k_fill_pattern(unsigned char* __restrict__ p, size_t bytes, uint32_t v) {
  const uintptr_t a0 = (uintptr_t)p;
  size_t head = (size_t)((16 - (a0 & 15)) & 15);
  if (head > bytes) head = bytes;
  const size_t nvec = (bytes - head) / 16;
  const size_t tail0 = head + nvec * 16;
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, nth = (size_t)gridDim.x * blockDim.x;
  uint4* q = (uint4*)(p + head);
  for (size_t i = tid; i < nvec; i += nth) q[i] = uint4{v, v, v, v};
  // edges in 16-bit pieces, taken from the pattern at the piece's address
  for (size_t i = tid * 2; i < head; i += nth * 2)
    *(uint16_t*)(p + i) = (uint16_t)(v >> (8 * ((a0 + i) & 2)));
  for (size_t i = tail0 + tid * 2; i < bytes; i += nth * 2)
    *(uint16_t*)(p + i) = (uint16_t)(v >> (8 * ((a0 + i) & 2)));
}

__global__ void __launch_bounds__(256) k_zero_u32(uint32_t* __restrict__ p, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0u;
}

// bf16 copy of h0 into slot 0 of the bf16 state array (slot s+1 holds the state of step s)
__global__ void __launch_bounds__(256) k_h0_bf16(const float* __restrict__ h0, bf16_t* __restrict__ hx, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    hx[i] = f32_to_bf16_bits(h0[i]);
}

// fp32 -> bf16 (nearest even), eight elements per thread and iteration: 32 bytes read and
// 16 written with vector accesses (in and out 16-byte aligned); the input is read once
__global__ void __launch_bounds__(256) k_to_bf16x8(const float* __restrict__ in, bf16_t* __restrict__ out, size_t n8) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += (size_t)gridDim.x * blockDim.x) {
    const f32x4 lo = __builtin_nontemporal_load((const f32x4*)in + 2 * i);
    const f32x4 hi = __builtin_nontemporal_load((const f32x4*)in + 2 * i + 1);
    const float v[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    ((bf16x8*)out)[i] = pack_bf16x8(v);
  }
}

// Clears the backward's control words: slot counters, group barrier counters, the wait flags
// and the index flag (the op status of the forward stays: the backward reports only its own).
// (keep_errors: a deferred call; the error words stay as earlier calls left them)
__global__ void __launch_bounds__(256) k_zero_ctl_bwd(uint32_t* __restrict__ ctl, int keep_errors) {
  for (int i = threadIdx.x; i < 16; i += blockDim.x) ctl[CTL_XCC_SLOT_B + i] = 0u;
  for (int i = threadIdx.x; i < 16 * MAX_GROUPS; i += blockDim.x) ctl[CTL_BAR_B + i] = 0u;
  if (threadIdx.x == 0) {
    ctl[CTL_ABORT] = 0u;
    if (!keep_errors) {
      ctl[CTL_STATUS] = kStatusOk;
      ctl[CTL_TIMEOUT] = 0u;
      ctl[CTL_BADIDX] = 0u;
    }
  }
}

// Push-row list: rows[k] = t*B + b of the k-th push (op = +1) in increasing row order, and
// *count = the number of pushes. Only push steps have a non-zero gate gradient dA (the
// states other steps write are never read, section 3, Observation 2), so the post-loop
// gradients dW, dU and dx contract over these rows only. One workgroup: tiles of 32 K ops
// go through LDS, each thread counts and writes 32 consecutive ops, offsets from a
// workgroup scan of the counts.
__global__ void __launch_bounds__(1024) k_push_rows(const int8_t* __restrict__ ops, int n, int32_t* __restrict__ rows,
                                                    uint32_t* __restrict__ count) {
  constexpr int TILE = 32768, PER = 32;
  __shared__ __align__(16) int8_t s_ops[TILE];
  __shared__ int s_wsum[16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int base = 0;
  for (int t0 = 0; t0 < n; t0 += TILE) {
    const int len = min(TILE, n - t0);
    // each thread reads its own 32 ops: two 16-byte loads when they are all in range and the
    // array is 16-byte aligned, else bytes through LDS
    uint4 q0, q1;
    const bool vec = ((uintptr_t)ops & 15u) == 0 && tid * PER + PER <= len;
    if (!vec)
      for (int i = 0; i < PER; ++i) s_ops[tid * PER + i] = tid * PER + i < len ? ops[(size_t)t0 + tid * PER + i] : (int8_t)0;
    if (vec) {
      q0 = *(const uint4*)(ops + (size_t)t0 + tid * PER);
      q1 = *(const uint4*)(ops + (size_t)t0 + tid * PER + 16);
    } else {
      q0 = *(const uint4*)&s_ops[tid * PER];
      q1 = *(const uint4*)&s_ops[tid * PER + 16];
    }
    const uint32_t w[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
    uint32_t mask = 0;                               // bit j: op j of this thread is a push
#pragma unroll
    for (int j = 0; j < PER; ++j) mask |= (((w[j >> 2] >> (8 * (j & 3))) & 0xffu) == 1u ? 1u : 0u) << j;
    const int cnt = __popc(mask);
    int incl = cnt;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int v = __shfl_up(incl, d, 64);
      if (lane >= d) incl += v;
    }
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int wbase = 0, total = 0;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int x = s_wsum[v];
      wbase += v < wave ? x : 0;
      total += x;
    }
    int pos = base + wbase + incl - cnt;
    while (mask) {
      const int j = __builtin_ctz(mask);
      mask &= mask - 1;
      rows[pos++] = t0 + tid * PER + j;
    }
    base += total;
    __syncthreads();
  }
  if (tid == 0) *count = (uint32_t)base;
}

// Zeroes the rows of out [n][cols] whose op is not a push (dx is exactly 0 there).
__global__ void __launch_bounds__(256) k_zero_nonpush_rows(const int8_t* __restrict__ ops, float* __restrict__ out,
                                                           size_t n, int cols) {
  const size_t tid = (size_t)blockIdx.x * blockDim.x + threadIdx.x, nth = (size_t)gridDim.x * blockDim.x;
  if ((cols & 3) == 0 && ((uintptr_t)out & 15) == 0) {
    const int cv = cols >> 2;
    const size_t nv = n * cv;
    for (size_t i = tid; i < nv; i += nth)
      if (ops[i / cv] != 1) ((float4*)out)[i] = float4{0.f, 0.f, 0.f, 0.f};
    return;
  }
  for (size_t i = tid; i < n * cols; i += nth)
    if (ops[i / cols] != 1) out[i] = 0.f;
}

// Hprev rows of the push steps: out[k][:] = the state read at the step of row prow[k] =
// t*B + b, for k < *count: h0[b] for t = 0, else the state produced at step top[t-1][b]
// (-1 = h0), from h_cell (fp32).
__global__ void __launch_bounds__(256) k_gather_hprev(const int32_t* __restrict__ top, const float* __restrict__ hcell,
                                                      const float* __restrict__ h0, const int32_t* __restrict__ prow,
                                                      const uint32_t* __restrict__ count, float* __restrict__ out,
                                                      int T, int B, int H, uint32_t* ctl) {
  const size_t n = (size_t)min(*count, (uint32_t)T * (uint32_t)B) * H;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t k = i / H;
    const int u = (int)(i - k * H);
    const int tb = prow[k];
    const int t = tb / B, b = tb - t * B;
    const int s = (t == 0) ? -1 : checked_src(top[tb - B], t - 1, ctl);
    out[i] = (s < 0) ? h0[(size_t)b * H + u] : hcell[((size_t)s * B + b) * H + u];
  }
}

// Gathering transpose to bf16 over the push rows: out[c][k] = bf16(row prow[k], column c)
// for k < *count, and 0 for *count <= k < (*count rounded up to 64), so a GEMM over the
// rounded K adds nothing past the last push; columns beyond are not written. The source row
// r is src + r*ld (fp32 or bf16); with a producer table (gtop != null) row r = t*B + b is
// the state read at step t (Hprev): h0[b] for t = 0, else the state produced at
// top[t-1][b] (-1 = h0), taken from the bf16 state copy (slot s+1 = step s, slot 0 = h0).
// 64x64 tiles through LDS. When rows, columns and both base addresses allow it, every
// global access moves 16 bytes (8 bf16 or 4 fp32 along a source row, 8 consecutive k of an
// output row); otherwise one element per access.
__global__ void __launch_bounds__(256) k_transpose_bf16(const void* __restrict__ src, int src_f32, int ld, int cols,
                                                        const int32_t* __restrict__ prow,
                                                        const uint32_t* __restrict__ count, int ldo,
                                                        const int32_t* __restrict__ gtop, int B,
                                                        bf16_t* __restrict__ out, uint32_t* ctl) {
  __shared__ __align__(16) bf16_t tile[64][72];             // 144-byte rows: 16-byte aligned
  const int rows = (int)min(*count, (uint32_t)ldo);
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  if (r0 >= rows + ((64 - (rows & 63)) & 63)) return;      // past the rounded extent
  const int E = src_f32 ? 4 : 8;                            // elements per 16 bytes of source
  const bool vec = ((uintptr_t)src & 15u) == 0 && ((uintptr_t)out & 15u) == 0 && ld % E == 0 && cols % E == 0 &&
                   ldo % 8 == 0;
  // source row of tile row i (-1: zero row)
  auto src_row = [&](int r) -> long long {
    if (r >= rows) return -1;
    const int pr = prow[r];
    if (!gtop) return pr;
    const int t = pr / B, b = pr - t * B;
    const int s = (t == 0) ? -1 : checked_src(gtop[(size_t)pr - B], t - 1, ctl);
    return (long long)(s + 1) * B + b;
  };
  if (vec) {
    if (src_f32) {
      const int tc = (threadIdx.x & 15) * 4, tr = threadIdx.x >> 4;   // 16 rows per pass
      for (int i = tr; i < 64; i += 16) {
        const long long sr = src_row(r0 + i);
        const int c = c0 + tc;
        uint2 v = uint2{0u, 0u};
        if (sr >= 0 && c < cols) {
          const float4 f = *(const float4*)((const float*)src + (size_t)sr * ld + c);
          v.x = (uint32_t)f32_to_bf16_bits(f.x) | ((uint32_t)f32_to_bf16_bits(f.y) << 16);
          v.y = (uint32_t)f32_to_bf16_bits(f.z) | ((uint32_t)f32_to_bf16_bits(f.w) << 16);
        }
        *(uint2*)&tile[i][tc] = v;
      }
    } else {
      const int tc = (threadIdx.x & 7) * 8, tr = threadIdx.x >> 3;     // 32 rows per pass
      for (int i = tr; i < 64; i += 32) {
        const long long sr = src_row(r0 + i);
        const int c = c0 + tc;
        uint4 v = uint4{0u, 0u, 0u, 0u};
        if (sr >= 0 && c < cols) v = *(const uint4*)((const bf16_t*)src + (size_t)sr * ld + c);
        *(uint4*)&tile[i][tc] = v;
      }
    }
    __syncthreads();
    const int kk = (threadIdx.x & 7) * 8;                   // 8 consecutive k of one column
    for (int ci = threadIdx.x >> 3; ci < 64; ci += 32) {
      const int c = c0 + ci, r = r0 + kk;
      if (c >= cols || r >= ldo) continue;
      uint32_t w[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) w[m] = (uint32_t)tile[kk + 2 * m][ci] | ((uint32_t)tile[kk + 2 * m + 1][ci] << 16);
      *(uint4*)&out[(size_t)c * ldo + r] = uint4{w[0], w[1], w[2], w[3]};
    }
    return;
  }
  const int tc = threadIdx.x & 63, tr = threadIdx.x >> 6;   // 4 rows per pass
  for (int i = tr; i < 64; i += 4) {
    const long long sr = src_row(r0 + i);
    const int c = c0 + tc;
    bf16_t v = 0;
    if (sr >= 0 && c < cols)
      v = src_f32 ? f32_to_bf16_bits(((const float*)src)[(size_t)sr * ld + c]) : ((const bf16_t*)src)[(size_t)sr * ld + c];
    tile[i][tc] = v;
  }
  __syncthreads();
  for (int i = tr; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tc;
    if (c < cols && r < ldo) out[(size_t)c * ldo + r] = tile[tc][i];
  }
}
