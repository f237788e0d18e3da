// Op validation and stack-pointer scan (paper, section 3: the unified update p <- p + op
// with op in {+1 push, -1 pop, 0 hold}). ptr[t][b] is the pointer before step t;
// ptr[T][b] the pointer after the last step, also kept in depth_end[b] for the backward. A pop while only the initial state is on
// the stack (p would become -1) is reported as EUNDERFLOW, an op outside {-1, 0, 1} as
// EOPS; the reported element is the lowest failing batch index, and within it the
// earliest failing step decides the code.
#include "common.h"

__global__ void __launch_bounds__(256) k_init_ctl(uint32_t* ctl) {
  for (int i = threadIdx.x; i < CTL_WORDS; i += blockDim.x) ctl[i] = (i == CTL_STATUS) ? 0x7fffffffu : 0u;
}

// Block of 256 threads = 16 columns x 16 time segments. Two passes over each segment:
// segment sums, a scan of the 16 sums per column in LDS, then the pointer values.
__global__ void __launch_bounds__(256) k_scan(const int8_t* __restrict__ ops, int T, int B, int32_t* __restrict__ ptr,
                                              int32_t* __restrict__ depth_end, uint32_t* ctl) {
  __shared__ int s_sum[16][17];
  __shared__ int s_first_bad[16], s_first_uf[16], s_maxd;
  const int c = threadIdx.x & 15, seg = threadIdx.x >> 4;
  const int b = blockIdx.x * 16 + c;
  const int L = (T + 15) / 16;
  const int t0 = seg * L, t1 = min(T, t0 + L);
  if (threadIdx.x < 16) { s_first_bad[threadIdx.x] = 0x7fffffff; s_first_uf[threadIdx.x] = 0x7fffffff; }
  if (threadIdx.x == 0) s_maxd = 0;
  int sum = 0;
  if (b < B) {
    for (int t = t0; t < t1; ++t) {
      int op = ops[(size_t)t * B + b];
      sum += (op >= -1 && op <= 1) ? op : 0;
    }
  }
  s_sum[c][seg] = sum;
  __syncthreads();
  int off = 0;
  for (int s = 0; s < seg; ++s) off += s_sum[c][s];
  int first_bad = 0x7fffffff, first_uf = 0x7fffffff, maxd = 0;
  if (b < B) {
    if (seg == 0) ptr[b] = 0;
    int p = off, npush = 0;
    for (int t = t0; t < t1; ++t) {
      int op = ops[(size_t)t * B + b];
      if (op < -1 || op > 1) { if (first_bad == 0x7fffffff) first_bad = t; op = 0; }
      npush += op == 1;
      p += op;
      if (p < 0 && first_uf == 0x7fffffff) first_uf = t;
      ptr[(size_t)(t + 1) * B + b] = p;
      maxd = max(maxd, p);
    }
    if (t1 == T && t0 < t1) depth_end[b] = p;      // the pointer after the last step
    if (npush) atomicAdd(&ctl[CTL_NPUSHF], (uint32_t)npush);
    atomicMin(&s_first_bad[c], first_bad);
    atomicMin(&s_first_uf[c], first_uf);
    atomicMax(&s_maxd, maxd);
  }
  __syncthreads();
  if (seg == 0 && b < B) {
    int fb = s_first_bad[c], fu = s_first_uf[c];
    int code = 0;
    if (fb != 0x7fffffff || fu != 0x7fffffff) code = (fu < fb) ? ST_EUNDERFLOW : ST_EOPS;
    if (code) atomicMin((int*)&ctl[CTL_STATUS], b * 8 + code);
  }
  if (threadIdx.x == 0) atomicMax(&ctl[CTL_MAXDEPTH], (uint32_t)s_maxd);
}

// Producer trace from the ops alone (section 3: the unified update p <- p + op on an
// integer stack of step indices): top[t][b] = the step that produced the state at the
// pointer after step t, -1 for the initial state. One thread per batch element keeps its
// stack of cap slots in LDS (slot 0 = the initial state); the ops of CH steps are staged in
// LDS at a time. Ops were validated by k_scan, and cap exceeds the deepest pointer.
__global__ void __launch_bounds__(64) k_trace(const int8_t* __restrict__ ops, int T, int B, int cap,
                                              int32_t* __restrict__ top) {
  constexpr int CH = 64;
  extern __shared__ int s_stk[];                  // [blockDim.x][cap]
  __shared__ int8_t s_ops[CH][64];
  const int R = blockDim.x;
  const int b = blockIdx.x * R + threadIdx.x;
  int* stk = s_stk + threadIdx.x * cap;
  int p = 0, tp = -1;
  stk[0] = -1;
  for (int t0 = 0; t0 < T; t0 += CH) {
    const int n = min(CH, T - t0);
    __syncthreads();
    for (int i = 0; i < n; ++i) s_ops[i][threadIdx.x] = b < B ? ops[(size_t)(t0 + i) * B + b] : (int8_t)0;
    __syncthreads();
    if (b < B) {
      for (int i = 0; i < n; ++i) {
        const int op = s_ops[i][threadIdx.x];
        if (op == 1) {
          ++p;
          if (p < cap) stk[p] = t0 + i;
          tp = t0 + i;
        } else if (op == -1) {
          p = p > 0 ? p - 1 : 0;
          tp = stk[min(p, cap - 1)];
        }
        top[(size_t)(t0 + i) * B + b] = tp;
      }
    }
  }
}

// h_top / c_top materialisation: the state returned at step t (Algorithm 1's return value)
// is the one produced at step top[t][b], or the initial state when top is -1.
// With skip_push, rows whose step produced the returned state (top[t] = t) are left as they
// are (the wide forward kernel writes them).
__global__ void __launch_bounds__(256) k_gather_top(const int32_t* __restrict__ top, const float* __restrict__ cellv,
                                                    const float* __restrict__ init, float* __restrict__ out, int T,
                                                    int B, int H, int skip_push) {
  const size_t n = (size_t)T * B * H;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    size_t tb = i / H;
    int u = (int)(i - tb * H);
    int b = (int)(tb % B);
    int s = top[tb];
    int t = (int)(tb / B);
    if (skip_push && s == t) continue;
    if (s < -1 || s > t) { out[i] = __builtin_nanf(""); continue; }   // not a valid producer
    out[i] = (s < 0) ? init[(size_t)b * H + u] : cellv[((size_t)s * B + b) * H + u];
  }
}

// The same for h_top and c_top in one pass (either may be null; skip_h as skip_push for
// h_top), four units per thread: H must be a multiple of 4 and the arrays 16-byte aligned.
__global__ void __launch_bounds__(256) k_gather_top4(const int32_t* __restrict__ top, const float* __restrict__ hcell,
                                                     const float* __restrict__ h0, float* __restrict__ htop,
                                                     const float* __restrict__ ccell, const float* __restrict__ c0,
                                                     float* __restrict__ ctop, int T, int B, int H, int skip_h) {
  const int H4 = H / 4;
  const size_t n = (size_t)T * B * H4;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t tb = i / H4;
    const int u4 = (int)(i - tb * H4);
    const int b = (int)(tb % B), t = (int)(tb / B);
    const int s = top[tb];
    const bool bad = s < -1 || s > t;             // not a valid producer
    const float nan = __builtin_nanf("");
    const size_t src = (s < 0 || bad) ? (size_t)b * H4 + u4 : ((size_t)s * B + b) * H4 + u4;
    if (htop && !(skip_h && s == t)) {
      const float4 v = bad ? float4{nan, nan, nan, nan} : (s < 0 ? ((const float4*)h0)[src] : ((const float4*)hcell)[src]);
      ((float4*)htop)[i] = v;
    }
    if (ctop) {
      const float4 v = bad ? float4{nan, nan, nan, nan} : (s < 0 ? ((const float4*)c0)[src] : ((const float4*)ccell)[src]);
      ((float4*)ctop)[i] = v;
    }
  }
}

// W [I][4H] (gate-major columns) -> Wp [I][4H] gate-interleaved, as fp32 or bf16.
__global__ void __launch_bounds__(256) k_permute_w(const float* __restrict__ W, float* __restrict__ Wp32,
                                                   bf16_t* __restrict__ Wp16, int I, int H) {
  const size_t n = (size_t)I * 4 * H;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    size_t row = i / (4 * (size_t)H);
    int np = (int)(i - row * 4 * H);
    float v = W[row * 4 * H + perm_to_orig(np, H)];
    if (Wp32) Wp32[i] = v;
    if (Wp16) Wp16[i] = f32_to_bf16_bits(v);
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

// fp32 -> bf16 (nearest even), elementwise
__global__ void __launch_bounds__(256) k_to_bf16(const float* __restrict__ in, bf16_t* __restrict__ out, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    out[i] = f32_to_bf16_bits(in[i]);
}

// Clears the backward's control words: slot counters, group barrier counters, abort flags.
__global__ void __launch_bounds__(256) k_zero_ctl_bwd(uint32_t* __restrict__ ctl) {
  for (int i = threadIdx.x; i < 16; i += blockDim.x) ctl[CTL_XCC_SLOT_B + i] = 0u;
  for (int i = threadIdx.x; i < 16 * MAX_GROUPS; i += blockDim.x) ctl[CTL_BAR_B + i] = 0u;
  if (threadIdx.x < 2) ctl[CTL_ABORT + threadIdx.x] = 0u;
}

// Operand of the input-projection GEMM: out [rows][KA] = [x | nones columns of 1 | 0], in
// fp32 (out32) or bf16 (out16, x rounded as k_to_bf16 does).
__global__ void __launch_bounds__(256) k_augment_x(const float* __restrict__ x, size_t rows, int I, int KA, int nones,
                                                   float* __restrict__ out32, bf16_t* __restrict__ out16) {
  // eight output columns per thread when I and KA are multiples of 8 and x is 16-byte aligned
  if (I % 8 == 0 && KA % 8 == 0 && ((uintptr_t)x & 15u) == 0) {
    const int K8 = KA / 8;
    const size_t n8 = rows * (size_t)K8;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += (size_t)gridDim.x * blockDim.x) {
      const size_t r = i / (size_t)K8;
      const int c = (int)(i - r * (size_t)K8) * 8;
      float v[8];
      if (c < I) {
        const float4 a = *(const float4*)(x + r * (size_t)I + c), b = *(const float4*)(x + r * (size_t)I + c + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = (c + j < I + nones) ? 1.f : 0.f;
      }
      if (out32) {
        *(float4*)(out32 + r * (size_t)KA + c) = float4{v[0], v[1], v[2], v[3]};
        *(float4*)(out32 + r * (size_t)KA + c + 4) = float4{v[4], v[5], v[6], v[7]};
      } else {
        bf16_t q[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) q[j] = f32_to_bf16_bits(v[j]);
        *(uint4*)(out16 + r * (size_t)KA + c) = *(const uint4*)q;
      }
    }
    return;
  }
  const size_t n = rows * (size_t)KA;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t r = i / (size_t)KA;
    const int c = (int)(i - r * (size_t)KA);
    const float v = c < I ? x[r * (size_t)I + c] : (c < I + nones ? 1.f : 0.f);
    if (out32) out32[i] = v;
    else out16[i] = f32_to_bf16_bits(v);
  }
}

// Bias rows under the gate-interleaved Wp: row j < nparts holds the j-th part of b (fp32: b
// itself; bf16: b = p0 + p1 + p2 with p0 = bf16(b), p1 = bf16(b - p0), p2 = bf16(b - p0 - p1),
// each difference exact in fp32), the other rows up to nrows are 0.
__global__ void __launch_bounds__(256) k_bias_rows(const float* __restrict__ b, int H, int nparts, int nrows,
                                                   float* __restrict__ out32, bf16_t* __restrict__ out16) {
  const int H4 = 4 * H;
  const size_t n = (size_t)nrows * H4;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int j = (int)(i / (size_t)H4);
    const int col = (int)(i - (size_t)j * H4);
    float rem = b ? b[perm_to_orig(col, H)] : 0.f;
    float part = 0.f;
    if (out32) {
      part = j == 0 ? rem : 0.f;
      out32[i] = part;
    } else {
      bf16_t bits = 0;
      for (int q = 0; q <= j && q < nparts; ++q) {
        bits = f32_to_bf16_bits(rem);
        const float pv = __uint_as_float((uint32_t)bits << 16);
        if (q < j) rem -= pv;
      }
      out16[i] = j < nparts ? bits : (bf16_t)0;
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
                                                      int T, int B, int H) {
  const size_t n = (size_t)min(*count, (uint32_t)T * (uint32_t)B) * H;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const size_t k = i / H;
    const int u = (int)(i - k * H);
    const int tb = prow[k];
    const int t = tb / B, b = tb - t * B;
    int s = (t == 0) ? -1 : top[tb - B];
    if (s < -1 || s >= t) s = -1;                 // only a valid producer is ever indexed
    out[i] = (s < 0) ? h0[(size_t)b * H + u] : hcell[((size_t)s * B + b) * H + u];
  }
}

// Row gather / scatter over the push rows (k < *count): dst[k] = src[prow[k]] and
// dst[prow[k]] = src[k], rows of `cols` floats (four at a time when cols % 4 == 0).
__global__ void __launch_bounds__(256) k_gather_rows(const float* __restrict__ src, const int32_t* __restrict__ prow,
                                                     const uint32_t* __restrict__ count, size_t max_rows, int cols,
                                                     int scatter, float* __restrict__ dst) {
  const size_t rows = min((size_t)*count, max_rows);
  if (cols % 4 == 0) {
    const int c4 = cols / 4;
    const size_t n = rows * c4;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
      const size_t k = i / c4;
      const int c = (int)(i - k * c4);
      const size_t r = (size_t)prow[k];
      if (scatter) ((float4*)dst)[r * c4 + c] = ((const float4*)src)[i];
      else ((float4*)dst)[i] = ((const float4*)src)[r * c4 + c];
    }
  } else {
    const size_t n = rows * cols;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
      const size_t k = i / cols;
      const int c = (int)(i - k * cols);
      const size_t r = (size_t)prow[k];
      if (scatter) dst[r * cols + c] = src[i];
      else dst[i] = src[r * cols + c];
    }
  }
}

// Gathering transpose to bf16 over the push rows: out[c][k] = bf16(row prow[k], column c)
// for k < *count, and 0 for *count <= k < (*count rounded up to 64), so a GEMM over the
// rounded K adds nothing past the last push; columns beyond are not written. The source row
// r is src + r*ld (fp32 or bf16); with a producer table (gtop != null) row r = t*B + b is
// the state read at step t (Hprev): h0[b] for t = 0, else the state produced at
// top[t-1][b] (-1 = h0), taken from the bf16 state copy (slot s+1 = step s, slot 0 = h0).
// 64x64 tiles through LDS: reads and writes are both along contiguous rows.
__global__ void __launch_bounds__(256) k_transpose_bf16(const void* __restrict__ src, int src_f32, int ld, int cols,
                                                        const int32_t* __restrict__ prow,
                                                        const uint32_t* __restrict__ count, int ldo,
                                                        const int32_t* __restrict__ gtop, int B,
                                                        bf16_t* __restrict__ out) {
  __shared__ bf16_t tile[64][66];
  const int rows = (int)min(*count, (uint32_t)ldo);
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  if (r0 >= rows + ((64 - (rows & 63)) & 63)) return;      // past the rounded extent
  const int tc = threadIdx.x & 63, tr = threadIdx.x >> 6;   // 4 rows per pass
  for (int i = tr; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tc;
    bf16_t v = 0;
    if (r < rows && c < cols) {
      const int pr = prow[r];
      if (gtop) {
        const int t = pr / B, b = pr - t * B;
        int s = (t == 0) ? -1 : gtop[(size_t)pr - B];
        if (s < -1 || s >= t) s = -1;                        // only a valid producer is ever indexed
        v = ((const bf16_t*)src)[((size_t)(s + 1) * B + b) * ld + c];
      } else if (src_f32) {
        v = f32_to_bf16_bits(((const float*)src)[(size_t)pr * ld + c]);
      } else {
        v = ((const bf16_t*)src)[(size_t)pr * ld + c];
      }
    }
    tile[i][tc] = v;
  }
  __syncthreads();
  for (int i = tr; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tc;
    if (c < cols && r < ldo) out[(size_t)c * ldo + r] = tile[tc][i];
  }
}
