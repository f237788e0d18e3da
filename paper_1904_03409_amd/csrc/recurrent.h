// Launch descriptions of the persistent recurrent kernels (forward and backward).
#pragma once
#include <stddef.h>
#include <stdint.h>

struct RecArgs {
  int T, B, I, H;
  int G, NW, ks_eff, spin_limit;   // batch groups, workgroups per group, K chunks in use, barrier spin limit
  // 1 when a cache line of the exchanged arrays can hold entries of two different steps
  // (rows not 128-byte multiples): then every exchanged value is read with L1-bypassing
  // loads; with aligned rows a line is never read before its only write, plain loads suffice
  int coh_rows;
  int bwd_direct;        // backward stages dA rows with global_load_lds (host checks the LDS fits)
  int poll;              // 1: workgroups exchange rows by polling fill-marked data; 0: group barrier per step
  int bwd_gs;            // backward: gate-split contraction (partial sums exchanged instead of dA rows);
                         // this int fills the padding before the first pointer (layout unchanged)
  const float* xw;       // [T*B][4H] gate-interleaved, bias included (forward; null when fused)
  const int8_t* ops;     // [T][B]
  const float* U;        // [H][4H] caller layout (gate-major columns)
  const float* h0;       // [B][H]
  const float* c0;       // [B][H]
  float* hcell;          // [T][B][H]  state computed at step t (written to slot p+1)
  float* ccell;          // [T][B][H]
  uint16_t* hx;          // [T+1][B][H] bf16 copies: slot 0 = h0, slot t+1 = hcell[t] (bf16-GEMM mode)
  float* stash;          // [T][B][4H] gate activations i, f, g, o, gate-interleaved
  int32_t* top;          // [T][B]     producer step of the state returned at step t (-1 = initial),
                         //            complete before the forward kernel starts (op scan)
  union {
    float* htop;         // forward: [T][B][H] or null: state at the top after step t (wide forward writes it)
    float* gs_part;      // backward with bwd_gs: [2][G][16*NT][NW][H] partial sums of dA U^T by workgroup
  };
  float* ctop;           // [T][B][H] (with htop)
  uint32_t* ctl;         // control block (status, barrier counters)
  // backward
  const float* dh_top;   // [T][B][H]
  const float* dc_top;   // [T][B][H] or null
  void* dA;              // [T][B][4H] fp32 or bf16: gradient w.r.t. the gate pre-activations
  float* dh_acc;         // [T+1][B][H] spilled gradient of the state at each stack depth (backward)
  float* dc_acc;         // [T+1][B][H]
  float* db_part;        // [G][4H] per-group bias gradient (gate-interleaved)
  const int32_t* depth_end;   // [B] stack pointer after the last step (written by k_scan)
  float* dh0;            // [B][H]
  float* dc0;            // [B][H]
  long long* clk;        // optional per-step wall-clock stamps [grid][T][4] (profiling)
};

// Fused input projection of the plain bf16 forward (a second argument of that kernel only).
struct FxArgs {
  int fuse_x;            // 1: the kernel contracts x_t W itself (RecArgs::xw unused)
  int kx;                // K chunks of 32 covering I (at most 8)
  const float* x;        // [T][B][I], 16-byte aligned, I % 4 == 0
  const float* W;        // [I][4H] caller layout
  const float* bias;     // [4H] caller layout
};
