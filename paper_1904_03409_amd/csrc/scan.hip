// Op validation and stack-pointer scan (paper, section 3: the unified update p <- p + op
// with op in {+1 push, -1 pop, 0 hold}). ptr[t][b] is the pointer before step t;
// ptr[T][b] the pointer after the last step. A pop while only the initial state is on
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
                                              uint32_t* ctl) {
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
    int p = off;
    for (int t = t0; t < t1; ++t) {
      int op = ops[(size_t)t * B + b];
      if (op < -1 || op > 1) { if (first_bad == 0x7fffffff) first_bad = t; op = 0; }
      p += op;
      if (p < 0 && first_uf == 0x7fffffff) first_uf = t;
      ptr[(size_t)(t + 1) * B + b] = p;
      maxd = max(maxd, p);
    }
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

// h_top / c_top materialisation: the state returned at step t (Algorithm 1's return value)
// is the one produced at step top[t][b], or the initial state when top is -1.
__global__ void __launch_bounds__(256) k_gather_top(const int32_t* __restrict__ top, const float* __restrict__ cellv,
                                                    const float* __restrict__ init, float* __restrict__ out, int T,
                                                    int B, int H) {
  const size_t n = (size_t)T * B * H;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    size_t tb = i / H;
    int u = (int)(i - tb * H);
    int b = (int)(tb % B);
    int s = top[tb];
    int t = (int)(tb / B);
    if (s < -1 || s > t) { out[i] = __builtin_nanf(""); continue; }   // not a valid producer
    out[i] = (s < 0) ? init[(size_t)b * H + u] : cellv[((size_t)s * B + b) * H + u];
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

// Hprev[t][b][:] = the state read at step t: h0[b] for t = 0, else the state produced at step
// top[t-1][b] (-1 = h0). fp32 rows from h_cell, or bf16 rows from the bf16 state copy (slot
// s+1 = step s, slot 0 = h0) in bf16-GEMM mode.
__global__ void __launch_bounds__(256) k_gather_hprev(const int32_t* __restrict__ top, const float* __restrict__ hcell,
                                                      const float* __restrict__ h0, const bf16_t* __restrict__ hx,
                                                      void* __restrict__ out, int T, int B, int H) {
  const size_t n = (size_t)T * B * H;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    size_t tb = i / H;
    int u = (int)(i - tb * H);
    int t = (int)(tb / B), b = (int)(tb - (size_t)t * B);
    int s = (t == 0) ? -1 : top[tb - B];
    if (s < -1 || s >= t) s = -1;                 // only a valid producer is ever indexed
    if (hx) ((bf16_t*)out)[i] = hx[((size_t)(s + 1) * B + b) * H + u];
    else ((float*)out)[i] = (s < 0) ? h0[(size_t)b * H + u] : hcell[((size_t)s * B + b) * H + u];
  }
}

// Tiled transpose to bf16: out[c][r] = bf16(row r, column c) for r < rows, c < cols, where
// row r is src + r*ld (fp32 or bf16). With a producer table (gtop != null) row r = t*B + b is
// the state read at step t (Hprev): h0[b] for t = 0, else the state produced at top[t-1][b]
// (-1 = h0), taken from the bf16 state copy (slot s+1 = step s, slot 0 = h0).
// 64x64 tiles through LDS: reads and writes are both along contiguous rows.
__global__ void __launch_bounds__(256) k_transpose_bf16(const void* __restrict__ src, int src_f32, int ld, int rows,
                                                        int cols, const int32_t* __restrict__ gtop, int B,
                                                        bf16_t* __restrict__ out) {
  __shared__ bf16_t tile[64][66];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tc = threadIdx.x & 63, tr = threadIdx.x >> 6;   // 4 rows per pass
  for (int i = tr; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tc;
    bf16_t v = 0;
    if (r < rows && c < cols) {
      if (gtop) {
        const int t = r / B, b = r - t * B;
        int s = (t == 0) ? -1 : gtop[(size_t)r - B];
        if (s < -1 || s >= t) s = -1;                        // only a valid producer is ever indexed
        v = ((const bf16_t*)src)[((size_t)(s + 1) * B + b) * ld + c];
      } else if (src_f32) {
        v = f32_to_bf16_bits(((const float*)src)[(size_t)r * ld + c]);
      } else {
        v = ((const bf16_t*)src)[(size_t)r * ld + c];
      }
    }
    tile[i][tc] = v;
  }
  __syncthreads();
  for (int i = tr; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tc;
    if (c < cols && r < rows) out[(size_t)c * rows + r] = tile[tc][i];
  }
}
