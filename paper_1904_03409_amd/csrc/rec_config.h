// Compile-time configuration table of the persistent recurrent kernels.
#pragma once
#include <hip/hip_runtime.h>

// K per chunk of the register-resident U slice: 16 (fp32 MFMA, 4 k per lane x 4 steps)
// or 32 (bf16 MFMA, 8 k per lane).
constexpr int rec_kc(int prec) { return prec ? 32 : 16; }
// Padding of a staged row (elements): keeps rows 16-byte aligned and moves consecutive rows
// to other LDS banks for the fragment reads (lane l16 reads row l16).
constexpr int rec_lds_pad(int prec) { return prec ? 8 : 4; }
constexpr int rec_lds_ld(int prec, int ks) { return ks * rec_kc(prec) + rec_lds_pad(prec); }
// Row tiles staged in LDS per pass: as many as fit in about 68 KB, so two workgroups
// can share a CU when the configuration needs it.
constexpr int rec_ntb(int prec, int nt, int ks) {
  int per_tile = 16 * rec_lds_ld(prec, ks) * (prec ? 2 : 4);
  int cap = 69632 / per_tile;
  int ntb = 1;
  while (ntb * 2 <= nt && ntb * 2 <= cap) ntb *= 2;
  return ntb;
}
constexpr size_t rec_lds_bytes(int prec, int ntb, int ks) {
  return (size_t)16 * ntb * rec_lds_ld(prec, ks) * (prec ? 2 : 4);
}
// Fused input projection of the plain bf16 forward: a ring of three buffers of the step's x
// rows (fp32, 1 KB + 16 B per row: I <= 256, i.e. at most 8 chunks of 32, the W slice's
// register capacity).
constexpr size_t rec_fx_lds_bytes(int rows) { return (size_t)3 * rows * 260 * 4; }
constexpr bool rec_fx_built(int prec, int ks) { return prec == 1 && ks <= 16; }
constexpr bool rec_fx_fits(int rows, int kx) { return kx <= 8 && rows > 0; }
// Backward kernel: LDS for the staged dA rows of the direct path (4 waves x 16 rows of the
// wave's K range); the direct path is used when this plus the static LDS fits one CU.
constexpr size_t rec_bwd_lds_bytes(int prec, int ks) { return (size_t)4 * 16 * rec_lds_ld(prec, ks) * (prec ? 2 : 4); }
constexpr size_t rec_bwd_static_lds(int nt) { return (size_t)4 * nt * 16 * 17 * 4 + 16 * 16 * 4 * 4 + 5 * nt * 16 * 4 + 64; }

// Register budget of the kernels for the bf16 K = 32 chunk case (H > 512): 256 registers per
// lane, as for two 256-thread workgroups per CU; the plain forward runs two workgroups of 16
// units per CU, the backward one 512-thread workgroup of 32 units. 1 (the whole register file
// for one 256-thread workgroup) otherwise.
constexpr int rec_occ(int prec, int ks) { return (prec == 1 && ks == 32) ? 2 : 1; }
// Backward instantiations that contain the direct-staging path (LDS DMA of the dA rows with
// hand-counted vmcnt waits): whole 1 KB row segments, at most two per row, one workgroup per
// CU and at most four row tiles per group. The eight-tile variants keep more state per thread
// than the registers hold; their spills would share the counter those waits count, so they
// are built without the path. The build checks that every variant built with it compiles
// without scratch.
constexpr bool rec_bwd_direct_built(int prec, int nt, int ks) {
  return (ks * rec_kc(prec) * (prec ? 2 : 4)) % 1024 == 0 && ks * rec_kc(prec) * (prec ? 2 : 4) / 1024 <= 2 &&
         rec_occ(prec, ks) == 1 && nt <= 4;
}

// Backward instantiations built with the gate-split contraction as well (the planner
// chooses it when the contraction's K columns are exactly H: H = KS * KC; at least two M
// tiles per wave, at most 32 workgroups per group, one workgroup per CU). fp32 only: there a
// push row's dA is 8 KB against 2 KB of partial sums (large fp32 backward 1.68 -> 1.40 ms);
// in bf16 the row is 4 KB, and the extra partial stores made the large backward slower
// (1.26 -> 1.48 ms).
constexpr bool rec_bwd_gs_built(int prec, int nt, int ks) {
  return prec == 0 && ks * rec_kc(prec) >= 128 && ks * rec_kc(prec) <= 512 && nt <= 2 && rec_occ(prec, ks) == 1;
}

#define REC_CASES(X) \
  X(0, 1, 4) X(0, 1, 8) X(0, 1, 16) X(0, 1, 32) \
  X(0, 2, 4) X(0, 2, 8) X(0, 2, 16) X(0, 2, 32) \
  X(0, 4, 4) X(0, 4, 8) X(0, 4, 16) X(0, 4, 32) \
  X(0, 8, 4) X(0, 8, 8) X(0, 8, 16) X(0, 8, 32) \
  X(1, 1, 2) X(1, 1, 4) X(1, 1, 8) X(1, 1, 16) X(1, 1, 32) \
  X(1, 2, 2) X(1, 2, 4) X(1, 2, 8) X(1, 2, 16) X(1, 2, 32) \
  X(1, 4, 2) X(1, 4, 4) X(1, 4, 8) X(1, 4, 16) X(1, 4, 32) \
  X(1, 8, 2) X(1, 8, 4) X(1, 8, 8) X(1, 8, 16) X(1, 8, 32)

// Pipelined forward kernel (two LDS tile buffers, whole 1 KB row segments: K of at least
// 16 chunks, an even number of row tiles per group). Only the variants that compile without
// register spills are built; the others run the plain forward kernel.
constexpr size_t rec_pipe_lds_bytes(int prec, int ks) { return (size_t)2 * 16 * rec_lds_ld(prec, ks) * (prec ? 2 : 4); }
#define REC_PIPE_CASES(X) \
  X(0, 2, 16) X(0, 2, 32) X(0, 4, 16) X(0, 4, 32) X(0, 8, 16) \
  X(1, 2, 16) X(1, 4, 16) X(1, 8, 16)
constexpr bool rec_pipe_built(int prec, int nt, int ks) {
  return prec == 0 ? (ks == 16 || (ks == 32 && nt <= 4)) : ks == 16;
}

// Wide forward (bf16, H > 512): row padding of its staged tiles (elements), then the LDS of
// three 16-row tile buffers of K = 32*KS bf16 columns, the
// per-tile recurrence state (NT tiles x 4 floats x 256 lanes) and three input-projection
// slots (2 float4 x 256 lanes).
constexpr int rec_wide_pad = 8;
constexpr size_t rec_wide_lds_bytes(int ks, int nt) {
  return (size_t)3 * 16 * (ks * 32 + rec_wide_pad) * 2 + (size_t)nt * 4 * 256 * 4 + (size_t)3 * 2 * 256 * 16;
}

hipError_t launch_fwd(const struct RecArgs& a, const struct FxArgs& f, int prec, int NT, int KS, dim3 grid,
                      hipStream_t st, int* occ_out);
hipError_t launch_fwd_pipe(const struct RecArgs& a, int prec, int NT, int KS, dim3 grid, hipStream_t st,
                           int* occ_out);
hipError_t launch_fwd_wide(const struct RecArgs& a, int NT, int KS, dim3 grid, hipStream_t st, int* occ_out);
hipError_t launch_bwd(const struct RecArgs& a, int prec, int NT, int KS, dim3 grid, hipStream_t st, int* occ_out);
