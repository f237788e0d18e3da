// Tiled MFMA GEMM for the non-recurrent contractions of the StackLSTM step:
//   XW = x Wp + b     (input projection for all T steps at once: the x_t part of the cell's
//                      pre-activation does not depend on the recurrence)
//   dx = dA Wp^T      dW = x^T dA      dU = Hprev^T dA   (Hprev = the state each step read)
// C[M][N] = sum_k A(m, k) B(k, n); A stored MK (A[m*lda+k]) or KM (A[k*lda+m]); B stored KN
// (B[k*ldb+n]) or NK (B[n*ldb+k]). Both operands share one element type: fp32
// (v_mfma_f32_16x16x4f32) or bf16 (v_mfma_f32_16x16x32_bf16), fp32 accumulation; a bf16
// kernel can also read an fp32 A (MK) and round it to bf16 as it loads it.
// 128x128 block tile, four 64x64 wave tiles, K slices of BK; the next slice is fetched
// into registers while the current one is multiplied (two LDS buffers, one barrier per
// slice). Split K writes partials that k_reduce_splits adds in a fixed order.
// The gradient GEMMs run over the push rows only (dA is exactly zero elsewhere): rows of
// A, B and C can be gathered through index tables, and M or K can come from a device-side
// count, so the host launches them without knowing how many rows are pushes.
#include "common.h"
#include "gemm.h"

namespace {

constexpr int BM = 128, BN = 128;
template <int P> struct Cfg;
// fp32: LDS tiles keep the global layout (k-contiguous rows read as 4-wide vectors,
// m/n-contiguous rows read one value per MFMA step); 32-deep K slices.
template <> struct Cfg<0> { using T = float; static constexpr int BK = 32; static constexpr int VE = 4; };
// bf16: LDS tiles are always [m][k] / [n][k] so a lane reads its 8 consecutive k at once;
// m/n-contiguous operands are transposed while being written to LDS. 64-deep K slices.
template <> struct Cfg<1> { using T = bf16_t; static constexpr int BK = 64; static constexpr int VE = 8; };

// LDS geometry of one operand tile (elements): rows x (cols + pad)
template <int P, bool KMAJOR> struct Geo {
  static constexpr int BK = Cfg<P>::BK;
  // fp32 k-major tile stored [k][m]: BK rows of 128 (+4); otherwise [m][k]: 128 rows of BK (+pad)
  static constexpr bool KROWS = (P == 0) && KMAJOR;
  static constexpr int ROWS = KROWS ? BK : 128;
  static constexpr int LD = KROWS ? (128 + 16) : (BK + (P ? 8 : 4));   // pads keep fragment reads conflict-free
  static constexpr int ELEMS = ROWS * LD;
};

// Register staging of one operand tile: NV vectors of VE elements per thread. With F32SRC
// (bf16 kernels only) the stage holds the fp32 values as loaded (f32v) and rounds them to bf16
// (nearest even) when it writes them to LDS, after the slice in between has been multiplied:
// rounding them at load time made every fetch wait for its own loads.
template <int P, bool KMAJOR, bool F32SRC = false> struct Stage {
  using T = typename Cfg<P>::T;
  static constexpr int BK = Cfg<P>::BK, VE = Cfg<P>::VE;
  static constexpr int NV = 128 * BK / VE / 256;
  uint4 v[NV];
  uint4 f32v[F32SRC ? NV : 1][2];
  int prow[NV];   // array row of each of this thread's vectors in the slice loaded next

  // Array row of tile row gr: the gather table's entry, or gr itself. Tiles stored [m/n][k]
  // keep the same rows for every K slice, so they are resolved once; k-major tiles change rows
  // with every slice, and the rows of the next slice are looked up right after the current
  // slice's loads are issued (their latency then overlaps that of the data).
  __device__ __forceinline__ void set_rows(const int32_t* __restrict__ rows, int r0, int rlim) {
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int e = threadIdx.x + 256 * i;
      const int gr = r0 + (KMAJOR ? e / (128 / VE) : e / (BK / VE));
      prow[i] = (rows && gr < rlim) ? rows[gr] : gr;
    }
  }

  // global tile element (r, c): KMAJOR -> row r in [0,BK) of k, col c in [0,128) of m/n;
  // otherwise row r in [0,128) of m/n, col c in [0,BK) of k. The vector path goes through a
  // bounds-checked buffer descriptor: an element past the row or column limit is given an
  // offset beyond the buffer, which reads 0 without a branch or a memory access. It needs
  // the row stride and both limits to be multiples of VE (checked by the host).
  __device__ __forceinline__ void load(const void* __restrict__ vbase, size_t bytes, int ld, int r0, int rlim, int c0,
                                       int clim, bool vec, const int32_t* __restrict__ rows) {
    if constexpr (F32SRC) {
      static_assert(P == 1 && !KMAJOR, "fp32 source: bf16 kernels, k-contiguous rows");
      // two 16-byte loads of four floats per vector; the vector path needs the row stride and
      // both limits to be multiples of 4 (each half lies wholly inside or outside the row)
      const float* fb = (const float*)vbase;
      const rsrc_t rs = make_rsrc(fb, bytes);
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int e = threadIdx.x + 256 * i;
        const int r = e / (BK / VE), c = (e % (BK / VE)) * VE;
        const int gr = r0 + r, gc = c0 + c;
        const int pr = prow[i];
        if (vec) {
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const bool ok = gr < rlim && gc + 4 * hh < clim;
            const uint32_t off = ok ? (uint32_t)(((size_t)pr * ld + gc + 4 * hh) * 4) : 0xffffffffu;
            f32v[i][hh] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
          }
        } else {
          float f[8];
#pragma unroll
          for (int j = 0; j < VE; ++j) f[j] = (gr < rlim && gc + j < clim) ? fb[(size_t)pr * ld + gc + j] : 0.f;
          f32v[i][0] = __builtin_bit_cast(uint4, float4{f[0], f[1], f[2], f[3]});
          f32v[i][1] = __builtin_bit_cast(uint4, float4{f[4], f[5], f[6], f[7]});
        }
      }
      return;
    }
    const T* base = (const T*)vbase;
    if (vec) {
      const rsrc_t rs = make_rsrc(base, bytes);
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const int e = threadIdx.x + 256 * i;
        int r, c;
        if (KMAJOR) { r = e / (128 / VE); c = (e % (128 / VE)) * VE; }
        else        { r = e / (BK / VE);  c = (e % (BK / VE)) * VE; }
        const int gr = r0 + r, gc = c0 + c;
        const bool ok = gr < rlim && gc < clim;
        const int pr = prow[i];
        const uint32_t off = ok ? (uint32_t)(((size_t)pr * ld + gc) * sizeof(T)) : 0xffffffffu;
        v[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
      }
      return;
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int e = threadIdx.x + 256 * i;
      int r, c;
      if (KMAJOR) { r = e / (128 / VE); c = (e % (128 / VE)) * VE; }
      else        { r = e / (BK / VE);  c = (e % (BK / VE)) * VE; }
      const int gr = r0 + r, gc = c0 + c;
      const int pr = prow[i];
      T tmp[VE];
#pragma unroll
      for (int j = 0; j < VE; ++j) tmp[j] = (gr < rlim && gc + j < clim) ? base[(size_t)pr * ld + gc + j] : (T)0;
      v[i] = *(const uint4*)tmp;
    }
  }

  __device__ __forceinline__ void store(T* __restrict__ s) {
    using G = Geo<P, KMAJOR>;
    if constexpr (F32SRC) {
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        const float4 lo = __builtin_bit_cast(float4, f32v[i][0]), hi = __builtin_bit_cast(float4, f32v[i][1]);
        const bf16_t q[8] = {f32_to_bf16_bits(lo.x), f32_to_bf16_bits(lo.y), f32_to_bf16_bits(lo.z),
                             f32_to_bf16_bits(lo.w), f32_to_bf16_bits(hi.x), f32_to_bf16_bits(hi.y),
                             f32_to_bf16_bits(hi.z), f32_to_bf16_bits(hi.w)};
        v[i] = *(const uint4*)q;
      }
    }
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int e = threadIdx.x + 256 * i;
      if (KMAJOR) {
        const int r = e / (128 / VE), c = (e % (128 / VE)) * VE;   // r = k, c = m
        if (G::KROWS) {
          *(uint4*)&s[r * G::LD + c] = v[i];
        } else {                                                    // bf16: transpose to [m][k]
          const bf16_t* h = (const bf16_t*)&v[i];
#pragma unroll
          for (int j = 0; j < VE; ++j) s[(c + j) * G::LD + r] = h[j];
        }
      } else {
        const int r = e / (BK / VE), c = (e % (BK / VE)) * VE;     // r = m, c = k
        *(uint4*)&s[r * G::LD + c] = v[i];
      }
    }
  }
};

}  // namespace

template <int P, int AL, int BL>
__global__ void __launch_bounds__(256, 2) k_gemm(GemmArgs g) {
  using T = typename Cfg<P>::T;
  constexpr int BK = Cfg<P>::BK;
  constexpr bool AKM = (AL == GEMM_KM), BKN = (BL == GEMM_KN);
  constexpr bool AF32 = (AL == GEMM_MK_F32);       // bf16 kernel, fp32 A rounded on load
  using GA = Geo<P, AKM>;
  using GB = Geo<P, BKN>;
  // the two slice buffers of A and B; after the K loop the same bytes hold the output tile
  constexpr int OLD = BN + 4;                       // row stride of the staged output (floats)
  constexpr size_t SLICE_BYTES = (size_t)2 * (GA::ELEMS + GB::ELEMS) * sizeof(T);
  constexpr size_t OUT_BYTES = (size_t)BM * OLD * 4;
  __shared__ __align__(16) unsigned char gsm_s[SLICE_BYTES > OUT_BYTES ? SLICE_BYTES : OUT_BYTES];
  T (*As)[GA::ELEMS] = reinterpret_cast<T (*)[GA::ELEMS]>(gsm_s);
  T (*Bs)[GB::ELEMS] = reinterpret_cast<T (*)[GB::ELEMS]>(gsm_s + (size_t)2 * GA::ELEMS * sizeof(T));
  // Block -> (n tile, m tile, K slice). Workgroups are dealt to the 8 XCDs in turn by their
  // linear id, so ids are renumbered such that each XCD takes a contiguous run of tiles, and
  // that run goes over groups of GM m tiles: for each n tile, the GM m tiles of the group. The
  // A tiles of a group and the B tile in use then stay in that XCD's L2 (one B tile is read
  // once per group rather than once per m tile).
  constexpr int GM = 8;
  const int NTL = (int)gridDim.x, MTL = (int)gridDim.y;
  const int nblk = NTL * MTL * (int)gridDim.z;
  int lid = (int)blockIdx.x + NTL * ((int)blockIdx.y + MTL * (int)blockIdx.z);
  {
    const int full = nblk & ~7;
    if (lid < full) lid = (lid & 7) * (full >> 3) + (lid >> 3);
  }
  int M = g.M, K = g.K, kchunk = g.k_chunk;
  int tn, tm, tz;
  auto grouped = [&](int id, int ntiles_m) {
    const int per = NTL * ntiles_m;
    tz = id / per;
    const int r0 = id - tz * per;
    const int gidx = r0 / (GM * NTL);
    const int gm = min(GM, ntiles_m - gidx * GM);     // m tiles in this group (the last may be short)
    const int r = r0 - gidx * GM * NTL;
    tm = gidx * GM + r % gm;
    tn = r / gm;
  };
  grouped(lid, MTL);
  float* C = g.C;
  int tz_c = -1;                                    // split whose split_stride offsets C (-1: tz)
  if (g.dyn) {
    const int ext = (int)((*g.dyn + (uint32_t)g.dyn_round - 1u) / (uint32_t)g.dyn_round * (uint32_t)g.dyn_round);
    if (g.dyn_axis == 0) {
      // device-side M: the grid covers the static M; the blocks are spread over the tiles in
      // use, each tile's K range cut into s slices (dyn_split, s <= 4) written as partials
      M = min(M, ext);
      if (g.dyn_split) {
        const int active = NTL * ((M + BM - 1) / BM);
        const int sp = gemm_dyn_splits(nblk, active);
        if (active == 0 || lid >= active * sp) return;
        grouped(lid, active / NTL);
        kchunk = ((K + sp - 1) / sp + 63) / 64 * 64;
        C += (size_t)tz * M * g.ldc;                // partial z: rows [0, M) packed
        tz_c = 0;
      }
    } else {
      K = min(K, ext);
      kchunk = ((K + (int)gridDim.z - 1) / (int)gridDim.z + 63) / 64 * 64;
    }
  }
  const int m0 = tm * BM, n0 = tn * BN;
  if (m0 >= M) return;                              // a whole block past a device-side M
  const int kbeg = tz * kchunk;
  const int kend = min(K, kbeg + kchunk);
  C += (size_t)(tz_c < 0 ? tz : tz_c) * g.split_stride;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l16 = lane & 15, lq = lane >> 4;
  const void* A = g.A;
  const T* Bp = (const T*)g.Bm;

  Stage<P, AKM, AF32> sa;
  Stage<P, BKN> sb;
  // buffer extents: the arrays' static sizes (gathered rows index within them)
  const size_t abytes = (AKM ? (size_t)g.K * g.lda : (size_t)g.M * g.lda) * (AF32 ? 4 : sizeof(T));
  const size_t bbytes = (BKN ? (size_t)g.K * g.ldb : (size_t)g.N * g.ldb) * sizeof(T);
  sa.set_rows(g.a_rows, AKM ? kbeg : m0, AKM ? kend : M);
  sb.set_rows(g.b_rows, BKN ? kbeg : n0, BKN ? kend : g.N);
  auto fetch = [&](int k0) {
    if (AKM) sa.load(A, abytes, g.lda, k0, kend, m0, M, g.a_vec, g.a_rows);
    else     sa.load(A, abytes, g.lda, m0, M, k0, kend, g.a_vec, g.a_rows);
    if (BKN) sb.load(Bp, bbytes, g.ldb, k0, kend, n0, g.N, g.b_vec, g.b_rows);
    else     sb.load(Bp, bbytes, g.ldb, n0, g.N, k0, kend, g.b_vec, g.b_rows);
    // k-major tiles: rows of the next slice, looked up behind this slice's loads
    if (AKM) sa.set_rows(g.a_rows, k0 + BK, kend);
    if (BKN) sb.set_rows(g.b_rows, k0 + BK, kend);
  };

  // epilogue operands (bias of this lane's columns, output rows), loaded now: on this GPU loads
  // and stores share one in-order counter, so a load issued among the epilogue's stores would
  // make its use wait for every store before it
  float bias[4][4];

#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int n = n0 + wn * 64 + j * 16 + 4 * lq + r;
      bias[j][r] = (g.bias && n < g.N) ? g.bias[perm_to_orig(n, g.bias_H)] : 0.f;
    }

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  int buf = 0;
  if (kbeg < kend) {
    fetch(kbeg);
    sa.store(As[0]);
    sb.store(Bs[0]);
  }
  __syncthreads();
  for (int k0 = kbeg; k0 < kend; k0 += BK) {
    const bool more = k0 + BK < kend;
    if (more) fetch(k0 + BK);                       // next slice in flight during this one
    const T* as = As[buf];
    const T* bs = Bs[buf];
    if constexpr (P == 0) {
      // one MFMA k-step covers k = 4*kc + lq (A and B use the same k for a lane); the
      // fragments of step kc+1 are read from LDS before the MFMAs of step kc
      auto rd = [&](int kc, float av[4], float bv[4]) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int m = wm * 64 + i * 16 + l16;
          av[i] = AKM ? as[(4 * kc + lq) * GA::LD + m] : as[m * GA::LD + 4 * kc + lq];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = wn * 64 + j * 16 + l16;
          bv[j] = BKN ? bs[(4 * kc + lq) * GB::LD + n] : bs[n * GB::LD + 4 * kc + lq];
        }
      };
      float av[2][4], bv[2][4];
      rd(0, av[0], bv[0]);
#pragma unroll
      for (int kc = 0; kc < BK / 4; ++kc) {
        const int cur = kc & 1;
        if (kc + 1 < BK / 4) rd(kc + 1, av[cur ^ 1], bv[cur ^ 1]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = mfma_f32_16x16x4(bv[cur][j], av[cur][i], acc[i][j]);
      }
    } else {
#pragma unroll
      for (int kc = 0; kc < BK / 32; ++kc) {
        bf16x8 a8[4], b8[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a8[i] = *(const bf16x8*)&as[(wm * 64 + i * 16 + l16) * GA::LD + kc * 32 + 8 * lq];
#pragma unroll
        for (int j = 0; j < 4; ++j) b8[j] = *(const bf16x8*)&bs[(wn * 64 + j * 16 + l16) * GB::LD + kc * 32 + 8 * lq];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = mfma_bf16_16x16x32(b8[j], a8[i], acc[i][j]);
      }
    }
    if (more) {
      sa.store(As[buf ^ 1]);
      sb.store(Bs[buf ^ 1]);
    }
    __syncthreads();
    buf ^= 1;
  }

  // epilogue: the MFMAs ran as C^T = B^T A^T, so a lane holds row l16, columns 4*lq .. 4*lq+3
  // of each 16x16 tile. The tile (bias added) goes through LDS (the slice buffers, free after
  // the loop's last barrier) so that the stores write whole rows: 32 lanes x 16 bytes = one
  // contiguous 512-byte row per half wave, instead of 64-byte pieces of 16 rows (measured: the
  // fp32 input projection wrote 1.39 times its output bytes with those). Non-temporal: the
  // output is streamed out.
  float* os = reinterpret_cast<float*>(gsm_s);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *(f32x4*)&os[(wm * 64 + i * 16 + l16) * OLD + wn * 64 + j * 16 + 4 * lq] =
          f32x4{acc[i][j][0] + bias[j][0], acc[i][j][1] + bias[j][1], acc[i][j][2] + bias[j][2],
                acc[i][j][3] + bias[j][3]};
  __syncthreads();
  const bool cvec = (g.ldc % 4) == 0 && (((uintptr_t)C) & 15u) == 0;
#pragma unroll 4
  for (int it = 0; it < BM * BN / 4 / 256; ++it) {
    const int idx = (int)threadIdx.x + 256 * it, r = idx / (BN / 4), c = (idx % (BN / 4)) * 4;
    const int m = m0 + r, n = n0 + c;
    if (m >= M) continue;
    const f32x4 v = *(const f32x4*)&os[r * OLD + c];
    float* cp = C + (size_t)(g.c_rows ? g.c_rows[m] : m) * g.ldc + n;
    if (cvec && n + 3 < g.N) {
      __builtin_nontemporal_store(v, (f32x4*)cp);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (n + q < g.N) cp[q] = v[q];
    }
  }
}

// out[m][col(n)] = sum_z P[z][m][n] in increasing z (deterministic), col = caller order.
__global__ void __launch_bounds__(256) k_reduce_splits(const float* __restrict__ P, int splits, size_t split_stride,
                                                       int M, int N, int unperm_H, float* __restrict__ out) {
  const size_t n_el = (size_t)M * N;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_el; i += (size_t)gridDim.x * blockDim.x) {
    float s = 0.f;
    for (int z = 0; z < splits; ++z) s += P[(size_t)z * split_stride + i];
    size_t m = i / N;
    int n = (int)(i - m * N);
    int col = unperm_H ? perm_to_orig(n, unperm_H) : n;
    out[m * N + col] = s;
  }
}

// Rows of a device-M GEMM run with dyn_split (N columns, partial z at P + z * nr * N for the
// nr rows in use): dst row rows[k] = the sum over the s K slices of partial row k, in
// increasing z (s as the GEMM computed it from its grid and the device count).
__global__ void __launch_bounds__(256) k_scatter_splits(const float* __restrict__ P, const int32_t* __restrict__ rows,
                                                        const uint32_t* __restrict__ count, size_t max_rows, int N,
                                                        int grid_blocks, int n_tiles, float* __restrict__ dst) {
  const size_t nr = min((size_t)*count, max_rows);
  const int sp = gemm_dyn_splits(grid_blocks, n_tiles * (int)((nr + BM - 1) / BM));
  const size_t n_el = nr * N;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_el; i += (size_t)gridDim.x * blockDim.x) {
    float s = 0.f;
    for (int z = 0; z < sp; ++z) s += P[(size_t)z * n_el + i];
    const size_t k = i / N;
    dst[(size_t)rows[k] * N + (i - k * N)] = s;
  }
}

// Wide-tile bf16 GEMM for A stored MK and B stored NK, both bf16 with 16-byte rows: a
// 256 x 256 block tile, four waves of 128 x 128 (64 MFMA tiles per wave, the accumulators in
// AGPRs), 64-deep K slices double-buffered in LDS, one workgroup per CU. A wave reads 16 B
// fragments per 64 MFMAs: a quarter of the LDS bytes per MFMA of k_gemm's 64 x 64 wave tile,
// whose bf16 form is bound by LDS reads (about 32 B per cycle per wave, eight waves per CU,
// against 128 B per cycle per CU). Split K (gridDim.z) and a device-side K as in k_gemm; no
// row gathers and no device-side M.
static_assert(kGemmWideBN == 256, "one bias column per thread");
__global__ void __launch_bounds__(256, 1) k_gemm_wide(GemmArgs g) {
  constexpr int BMW = kGemmWideBM, BNW = kGemmWideBN, BKW = 64, LDW = BKW + 8;   // LDS row stride: 16-byte pad
  extern __shared__ __align__(16) unsigned char gsm[];
  bf16_t* As = reinterpret_cast<bf16_t*>(gsm);     // [2][BMW][LDW]
  bf16_t* Bs = As + 2 * BMW * LDW;                 // [2][BNW][LDW]
  // block -> (n tile, m tile, K slice): XCD-contiguous runs over groups of GM m tiles, as k_gemm
  constexpr int GM = 4;
  const int NTL = (int)gridDim.x, MTL = (int)gridDim.y;
  const int nblk = NTL * MTL * (int)gridDim.z;
  int lid = (int)blockIdx.x + NTL * ((int)blockIdx.y + MTL * (int)blockIdx.z);
  {
    const int full = nblk & ~7;
    if (lid < full) lid = (lid & 7) * (full >> 3) + (lid >> 3);
  }
  const int per = NTL * MTL;
  const int tz = lid / per;
  const int r0 = lid - tz * per;
  const int gidx = r0 / (GM * NTL);
  const int gm = min(GM, MTL - gidx * GM);
  const int rg = r0 - gidx * GM * NTL;
  const int tm = gidx * GM + rg % gm, tn = rg / gm;
  int K = g.K, kchunk = g.k_chunk;
  if (g.dyn) {                                      // device-side K (the host never passes a device M)
    const int ext = (int)((*g.dyn + (uint32_t)g.dyn_round - 1u) / (uint32_t)g.dyn_round * (uint32_t)g.dyn_round);
    K = min(K, ext);
    kchunk = ((K + (int)gridDim.z - 1) / (int)gridDim.z + 63) / 64 * 64;
  }
  const int M = g.M, N = g.N;
  const int m0 = tm * BMW, n0 = tn * BNW;
  const int kbeg = tz * kchunk, kend = min(K, kbeg + kchunk);
  float* C = g.C + (size_t)tz * g.split_stride;
  const int tid = (int)threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l16 = lane & 15, lq = lane >> 4;
  const rsrc_t ra = make_rsrc(g.A, (size_t)M * g.lda * 2);
  const rsrc_t rb = make_rsrc(g.Bm, (size_t)N * g.ldb * 2);
  // staging of one slice: per operand 256 rows x 64 k, eight 16-byte vectors per thread
  // (vector e = tid + 256 i: row e / 8, k 8 (e % 8)); outside the rows or K: offset beyond the
  // buffer (reads 0, no access)
  uint4 va[8], vb[8];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int e = tid + 256 * i, r = e >> 3, gk = k0 + (e & 7) * 8;
      const bool kin = gk < kend;
      const uint32_t ao = (kin && m0 + r < M) ? (uint32_t)(((size_t)(m0 + r) * g.lda + gk) * 2) : 0xffffffffu;
      const uint32_t bo = (kin && n0 + r < N) ? (uint32_t)(((size_t)(n0 + r) * g.ldb + gk) * 2) : 0xffffffffu;
      va[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(ra, ao, 0, 0));
      vb[i] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rb, bo, 0, 0));
    }
  };
  auto stage = [&](int b) {
    bf16_t* as = As + b * BMW * LDW;
    bf16_t* bs = Bs + b * BNW * LDW;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int e = tid + 256 * i, r = e >> 3, c = (e & 7) * 8;
      *(uint4*)&as[r * LDW + c] = va[i];
      *(uint4*)&bs[r * LDW + c] = vb[i];
    }
  };
  // the block's bias columns, into LDS before the K loop (no registers held through it)
  __shared__ float s_bias[BNW];
  {
    const int n = n0 + tid;
    s_bias[tid] = (g.bias && n < N) ? g.bias[perm_to_orig(n, g.bias_H)] : 0.f;
  }
  f32x4 acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  int buf = 0;
  if (kbeg < kend) {
    fetch(kbeg);
    stage(0);
  }
  __syncthreads();
  for (int k0 = kbeg; k0 < kend; k0 += BKW) {
    const bool more = k0 + BKW < kend;
    if (more) fetch(k0 + BKW);                      // next slice in flight during this one
    const bf16_t* as = As + buf * BMW * LDW;
    const bf16_t* bs = Bs + buf * BNW * LDW;
#pragma unroll
    for (int kc = 0; kc < BKW / 32; ++kc) {
      bf16x8 a8[8], b8[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) a8[i] = *(const bf16x8*)&as[(wm * 128 + i * 16 + l16) * LDW + kc * 32 + 8 * lq];
#pragma unroll
      for (int j = 0; j < 8; ++j) b8[j] = *(const bf16x8*)&bs[(wn * 128 + j * 16 + l16) * LDW + kc * 32 + 8 * lq];
      // C^T = B^T A^T: a lane holds row l16, columns 4*lq .. 4*lq+3 of each 16 x 16 tile
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = mfma_bf16_16x16x32(b8[j], a8[i], acc[i][j]);
    }
    if (more) stage(buf ^ 1);
    __syncthreads();
    buf ^= 1;
  }
  // epilogue through LDS (the K loop's buffers are free now): the block's rows are written
  // out in two halves of 128; the waves of one half put their tiles in LDS, then every wave
  // stores whole rows, 64 lanes x 16 bytes = one contiguous 1 KB row per instruction
  // (non-temporal: the output is streamed out)
  constexpr int OLD = BNW + 4;                     // LDS row stride of the staged output (floats)
  static_assert((size_t)128 * OLD * 4 <= kGemmWideLds, "half the output tile fits the slice buffers");
  float* os = reinterpret_cast<float*>(gsm);
  const bool cvec = (g.ldc % 4) == 0 && (((uintptr_t)C) & 15u) == 0;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (wm == h) {
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          *(f32x4*)&os[(i * 16 + l16) * OLD + wn * 128 + j * 16 + 4 * lq] = acc[i][j];
    }
    __syncthreads();
#pragma unroll 4
    for (int it = 0; it < 32; ++it) {
      const int idx = tid + 256 * it, r = idx >> 6, c = (idx & 63) * 4;
      const int m = m0 + h * 128 + r, n = n0 + c;
      if (m >= M) continue;
      const f32x4 v = *(const f32x4*)&os[r * OLD + c];
      const float4 bv = *(const float4*)&s_bias[c];
      const f32x4 o = f32x4{v[0] + bv.x, v[1] + bv.y, v[2] + bv.z, v[3] + bv.w};
      float* cp = C + (size_t)m * g.ldc + n;
      if (cvec && n + 3 < N) {
        __builtin_nontemporal_store(o, (f32x4*)cp);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (n + q < N) cp[q] = o[q];
      }
    }
    __syncthreads();
  }
}

#define INST(P, A, B) template __global__ void k_gemm<P, A, B>(GemmArgs);
INST(0, GEMM_MK, GEMM_KN)
INST(0, GEMM_MK, GEMM_NK)
INST(0, GEMM_KM, GEMM_KN)
INST(1, GEMM_MK, GEMM_NK)
INST(1, GEMM_MK_F32, GEMM_NK)

// fp32 GEMM for A stored MK and B stored KN (the input projection x Wp + b): the tiles, waves,
// MFMAs and epilogue of k_gemm<0, MK, KN>, but the operand slices (16 deep) go from global
// memory straight into a ring of kRingStages LDS stages by LDS DMA, issued that many slices
// less one ahead (k_gemm stages one slice in registers, one slice ahead, and a second register
// stage does not fit its register budget). A DMA writes one contiguous kilobyte of LDS per wave
// instruction, so the lanes fetch the 16-byte chunks that a swizzled layout puts at their
// slots: A row m holds its chunk c at slot c ^ ((m >> 2) & 3), B row k holds column n at
// n ^ 16 (k & 3), and the fragment reads of a wave then fall in 64 distinct banks. Every
// wave issues four DMAs per slice, also past the last slice (out of range: zeros), so
// "this slice has landed" is always the wait for all but the later slices' DMAs.
// Requires K and N multiples of 4, A and B 16-byte aligned, and A, B under 4 GB.
namespace {
constexpr int kRingK = 16;                                  // K per slice
constexpr int kRingStages = 4;
constexpr int kRingStage = BM * kRingK + kRingK * BN;       // floats per stage: A, then B
__device__ __forceinline__ int ring_a(int m, int k) { return m * kRingK + ((((k >> 2) ^ (m >> 2)) & 3) << 2) + (k & 3); }
__device__ __forceinline__ int ring_b(int k, int n) { return BM * kRingK + k * BN + (n ^ ((k & 3) << 4)); }
}  // namespace

__global__ void __launch_bounds__(256, 2) k_gemm_ring(GemmArgs g) {
  constexpr int OLD = BN + 4;                       // row stride of the staged output (floats)
  constexpr size_t RING_BYTES = (size_t)kRingStages * kRingStage * 4;
  constexpr size_t OUT_BYTES = (size_t)BM * OLD * 4;
  __shared__ __align__(16) float rs_s[(RING_BYTES > OUT_BYTES ? RING_BYTES : OUT_BYTES) / 4];
  // block -> tile: the XCD-contiguous, m-grouped order of k_gemm
  constexpr int GM = 8;
  const int NTL = (int)gridDim.x, MTL = (int)gridDim.y;
  const int nblk = NTL * MTL;
  int lid = (int)blockIdx.x + NTL * (int)blockIdx.y;
  {
    const int full = nblk & ~7;
    if (lid < full) lid = (lid & 7) * (full >> 3) + (lid >> 3);
  }
  const int gidx = lid / (GM * NTL);
  const int gm = min(GM, MTL - gidx * GM);
  const int r = lid - gidx * GM * NTL;
  const int m0 = (gidx * GM + r % gm) * BM, n0 = (r / gm) * BN;
  const int M = g.M, N = g.N, K = g.K;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int l16 = lane & 15, lq = lane >> 4;
  const float* A = (const float*)g.A;
  const float* Bp = (const float*)g.Bm;
  const rsrc_t ra = make_rsrc(A, (size_t)M * g.lda * 4);
  const rsrc_t rb = make_rsrc(Bp, (size_t)K * g.ldb * 4);

  // slice s into stage s % 4: wave w copies A rows [32w, 32w+32) (two DMAs of 16 rows) and B
  // rows [4w, 4w+4) (two DMAs of 2 rows)
  auto issue = [&](int s) {
    float* st = rs_s + (s % kRingStages) * kRingStage;
    const int k0 = s * kRingK;
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int r0 = 32 * wave + 16 * q, rr = r0 + (lane >> 2), c = (lane & 3) ^ ((rr >> 2) & 3);
      const bool ok = m0 + rr < M && k0 + 4 * c < K;
      bdma16(ra, ok ? (uint32_t)(((size_t)(m0 + rr) * g.lda + k0 + 4 * c) * 4) : kOOB, 0u, lds_addr(st + r0 * kRingK));
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int kk0 = 4 * wave + 2 * q, kk = kk0 + (lane >> 5), n = ((lane & 31) * 4) ^ ((kk & 3) << 4);
      const bool ok = k0 + kk < K && n0 + n < N;
      bdma16(rb, ok ? (uint32_t)(((size_t)(k0 + kk) * g.ldb + n0 + n) * 4) : kOOB, 0u,
             lds_addr(st + BM * kRingK + kk0 * BN));
    }
  };

  // epilogue operands, loaded before the DMAs (loads and DMAs share one in-order counter)
  float bias[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int n = n0 + wn * 64 + j * 16 + 4 * lq + q;
      bias[j][q] = (g.bias && n < N) ? g.bias[perm_to_orig(n, g.bias_H)] : 0.f;
    }
  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int ns = (K + kRingK - 1) / kRingK;
#pragma unroll
  for (int s = 0; s < kRingStages - 1; ++s) issue(s);
  for (int s = 0; s < ns; ++s) {
    // this wave's part of slice s has landed (the later slices' DMAs may still be in flight)
    wait_vm<4 * (kRingStages - 2)>();
    // every wave's part has, and every wave is done with the stage slice s-1 used
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    issue(s + kRingStages - 1);
    const float* st = rs_s + (s % kRingStages) * kRingStage;
    // one MFMA k-step covers k = 4*kc + lq; the fragments of step kc+1 are read before the
    // MFMAs of step kc
    float av[2][4], bv[2][4];
    auto rd = [&](int kc, float (&a4)[4], float (&b4)[4]) {
#pragma unroll
      for (int i = 0; i < 4; ++i) a4[i] = st[ring_a(wm * 64 + i * 16 + l16, 4 * kc + lq)];
#pragma unroll
      for (int j = 0; j < 4; ++j) b4[j] = st[ring_b(4 * kc + lq, wn * 64 + j * 16 + l16)];
    };
    rd(0, av[0], bv[0]);
#pragma unroll
    for (int kc = 0; kc < kRingK / 4; ++kc) {
      const int cur = kc & 1;
      if (kc + 1 < kRingK / 4) rd(kc + 1, av[cur ^ 1], bv[cur ^ 1]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma_f32_16x16x4(bv[cur][j], av[cur][i], acc[i][j]);
    }
  }
  wait_vm<0>();                                     // the DMAs past the last slice (zeros)
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");

  // epilogue as k_gemm's: the tile (bias added) through LDS, whole rows stored non-temporally
  float* os = rs_s;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      *(f32x4*)&os[(wm * 64 + i * 16 + l16) * OLD + wn * 64 + j * 16 + 4 * lq] =
          f32x4{acc[i][j][0] + bias[j][0], acc[i][j][1] + bias[j][1], acc[i][j][2] + bias[j][2],
                acc[i][j][3] + bias[j][3]};
  __syncthreads();
  float* C = g.C;
  const bool cvec = (g.ldc % 4) == 0 && (((uintptr_t)C) & 15u) == 0;
#pragma unroll 4
  for (int it = 0; it < BM * BN / 4 / 256; ++it) {
    const int idx = (int)threadIdx.x + 256 * it, rw = idx / (BN / 4), c = (idx % (BN / 4)) * 4;
    const int m = m0 + rw, n = n0 + c;
    if (m >= M) continue;
    const f32x4 v = *(const f32x4*)&os[rw * OLD + c];
    float* cp = C + (size_t)m * g.ldc + n;
    if (cvec && n + 3 < N) {
      __builtin_nontemporal_store(v, (f32x4*)cp);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (n + q < N) cp[q] = v[q];
    }
  }
}
