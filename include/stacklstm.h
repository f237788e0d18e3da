/*
 * stacklstm.h -- C ABI of the MI355X (gfx950) parallelised StackLSTM step.
 *
 * Method: Ding & Koehn, "Parallelizable Stack Long Short-Term Memory" (2019).
 * Each batch element carries its own stack of (h, c) states and its own op stream,
 * op in {+1 push, -1 pop, 0 hold} (section 2 defines Push and Pop, section 3 the
 * unified pointer update p <- p + op and the hold op). Algorithm 1 (section 3) is run
 * for every element at every step with no op-dependent branch: read the state at the
 * pointer p, run one LSTM cell on (x_t, h_p), write the result to slot p + 1, move p
 * by op, return the state at the new p. The cell-state stack is handled exactly like
 * the hidden-state stack (footnote of section 2). Backward is BPTT through the stack
 * reads (section 5: gradient reaches popped and overwritten states).
 *
 * LSTM cell (the paper names the standard LSTM without equations): gates i, f, g, o,
 * a = x W + h_prev U + b, i = sig(a_i), f = sig(a_f), g = tanh(a_g), o = sig(a_o),
 * c = f c_prev + i g, h = o tanh(c). Gate k of hidden unit u is column k*H + u of W, U
 * and b (torch.nn.LSTMCell order: weight_ih = W^T, weight_hh = U^T, bias_ih = b,
 * bias_hh = 0).
 *
 * Conventions for every entry point:
 *  - All array arguments are DEVICE pointers, owned by the caller; the library keeps
 *    none of them after the call returns. Shapes are row-major, time-major.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = default stream) up to
 *    one status read-back at the end of each call (the only host synchronisation): it
 *    reports invalid ops, a wait that gave up (SLSTM_ETIMEOUT) and an index out of range
 *    (SLSTM_EINDEX) for the kernels of that call.
 *  - Gradient outputs are overwritten, not accumulated.
 *  - An error found by the argument checks (EINVAL, EWORKSPACE, ENORESIDENT) launches
 *    nothing. On an error found by the read-back the call's kernels have run; output
 *    contents are then unspecified (an invalid op is walked as a hold so that every
 *    index stays in range).
 *  - No exception crosses the ABI. The only global state is the cached device
 *    properties (multiprocessor count per device), the kernels' launch attributes, and
 *    for stacklstm_fwd_static its static work space per GPU (with its device address).
 *    Calls on different work spaces may overlap, on any streams and from any host
 *    threads; calls that share a work space must not overlap. Results do not depend on
 *    what runs beside them.
 *  - Supported sizes: T >= 0, B >= 1, I >= 1, 1 <= H <= 512 (SLSTM_FP32) or
 *    H <= 1024 (SLSTM_BF16_GEMM); B up to 8 groups of 128 rows per XCC pass
 *    (SLSTM_ENORESIDENT beyond what one launch can hold).
 */
#ifndef STACKLSTM_H
#define STACKLSTM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SLSTM_OK = 0,
  SLSTM_EINVAL = 1,        /* bad dims, NULL required pointer, unsupported size */
  SLSTM_EOPS = 2,          /* an op outside {-1, 0, 1} */
  SLSTM_EUNDERFLOW = 3,    /* a pop while only the initial state is on the stack */
  SLSTM_EWORKSPACE = 4,    /* ws_bytes < stacklstm_workspace_bytes(dims) */
  SLSTM_ENORESIDENT = 5,   /* the persistent kernels cannot be made co-resident */
  SLSTM_EDEVICE = 6,       /* a HIP runtime error */
  SLSTM_ETIMEOUT = 7,      /* a wait for another workgroup's data exceeded its spin limit
                              (dims->spin_limit failed polls, or the default limit) */
  SLSTM_EINDEX = 8         /* a kernel read a producer index or reached a stack depth outside
                              its valid range: the top or ops passed to stacklstm_bwd are not
                              the forward's (or a read returned stale data) */
} slstm_status;

typedef enum {
  SLSTM_FP32 = 0,          /* fp32 operands, fp32 accumulation */
  SLSTM_BF16_GEMM = 1      /* operands of every matrix product rounded to bf16 (nearest
                              even): x, W, U, h_prev, dA; fp32 accumulation, fp32 h/c,
                              fp32 nonlinearities */
} slstm_precision;

typedef struct {
  int32_t T;               /* steps */
  int32_t B;               /* batch elements */
  int32_t I;               /* input size */
  int32_t H;               /* hidden size */
  int32_t precision;       /* slstm_precision */
  int32_t spin_limit;      /* failed polls per wait before the kernels give up and report
                              SLSTM_ETIMEOUT: 0 = the default (4M), > 0 = this limit */
  void* phase_events;      /* NULL, or an array of SLSTM_PHASE_EVENTS hipEvent_t created by the
                              caller; the calls record them on `stream` between their phases:
                              fwd [0] start, [1] after the op scan and trace,
                              [2] after the input projection and the preparation of the exchange
                              buffers, [3] after the persistent forward kernel, [4] after the
                              h_top/c_top gathers; bwd [5] after the backward's preparation
                              (control words, exchange buffer), right before the persistent
                              backward kernel, [6] after it, [7] after dW and db, [8] after dU,
                              [9] after dx. [2]-[3] and [5]-[6] time the persistent kernels
                              alone. For profiling only. */
  void* step_clock;        /* NULL, or a device int64 buffer of 2 * 512 * T * 4 entries: the
                              persistent kernels store 100 MHz wall-clock stamps per workgroup
                              and step, [pass (0 fwd, 1 bwd)][workgroup][t][4], at four points of
                              each step (forward: loop top, h_prev staged, MFMA done, epilogue
                              done; backward: loop top, epilogue done, row list ready, dh
                              scattered). For profiling only. */
  int32_t defer_status;    /* 0: each call ends with a read-back of its control words (one host
                              synchronisation) and returns the call's own status. 1: the call
                              returns SLSTM_OK once its kernels are queued (host-side argument
                              errors are still returned at once), and the error words of the
                              work space are not reset, so they keep the first op error and any
                              time-out or index error of every deferred call since the last call
                              made with 0; stacklstm_sync_status reads them. Calls with 0 reset
                              them (make the first call on a new work space with 0). */
} slstm_dims;

#define SLSTM_PHASE_EVENTS 10

/* Bytes of device work space that stacklstm_fwd / stacklstm_bwd need for `d`
 * (0 for invalid dims). The work space carries the forward's gate activations and
 * stack depths to the backward; pass the same buffer, untouched, to both calls. */
size_t stacklstm_workspace_bytes(const slstm_dims* d);

/* Forward over T steps (Algorithm 1 for every element and step). Op scan and producer
 * trace (section 3's p <- p + op on an integer stack), the input projection x_t W + b of
 * all steps as one MFMA GEMM, the persistent recurrent kernel and the gathers of the
 * returned states all run in the library's kernels.
 *  x      [T, B, I]   inputs x_t                                 (read)
 *  ops    [T, B]      int8 ops, +1 push / -1 pop / 0 hold         (read)
 *  W [I, 4H], U [H, 4H], b [4H], h0 [B, H], c0 [B, H]             (read)
 *  h_cell, c_cell [T, B, H]   the LSTM output of step t, i.e. the state Algorithm 1
 *                             writes to slot p + 1 at step t      (written)
 *  h_top, c_top   [T, B, H]   Algorithm 1's return value: the state at the pointer
 *                             after step t; may be NULL           (written)
 *  ptr    [T + 1, B]  int32 pointer before step t (ptr[T] = after the last step)
 *  top    [T, B]      int32 step that produced the returned state of step t, -1 for the
 *                     initial state (h0, c0)                      (written)
 * Returns SLSTM_EOPS / SLSTM_EUNDERFLOW for invalid ops (lowest failing element, earliest
 * failing step), SLSTM_ETIMEOUT / SLSTM_EINDEX as above. */
int stacklstm_fwd(const slstm_dims* d, const float* x, const int8_t* ops, const float* W, const float* U,
                  const float* b, const float* h0, const float* c0, float* h_cell, float* c_cell, float* h_top,
                  float* c_top, int32_t* ptr, int32_t* top, void* workspace, size_t ws_bytes, void* stream);

/* Allocation-free variant of stacklstm_fwd, for callers that cannot allocate device memory
 * (serving loops and harnesses that forbid allocation): the same arguments, outputs and
 * status read-back, with no work-space argument. Its work space is a static device array of
 * SLSTM_FWD_STATIC_MAX_BYTES bytes, one per GPU, held until the process ends; the call
 * allocates nothing. Dims whose forward work space (the forward's part of
 * stacklstm_workspace_bytes) exceeds it give SLSTM_EWORKSPACE. Every call on a GPU uses that
 * GPU's array: calls that overlap on one GPU (two streams, two host threads) race and must
 * be serialised by the caller. A backward cannot follow it (it keeps nothing for one). */
#define SLSTM_FWD_STATIC_MAX_BYTES ((size_t)128 << 20)
int stacklstm_fwd_static(const slstm_dims* d, const float* x, const int8_t* ops, const float* W, const float* U,
                         const float* b, const float* h0, const float* c0, float* h_cell, float* c_cell, float* h_top,
                         float* c_top, int32_t* ptr, int32_t* top, void* stream);

/* Backward of L given dL/dh_top and dL/dc_top (section 5), after stacklstm_fwd on the
 * same inputs and work space. The reverse loop scatters each step's gradient into the step
 * that produced the state it read (the producer table `top`); dW, dU, db, dx are contracted
 * over the push steps only (on the other steps the gate gradient is exactly 0) on the
 * library's MFMA GEMM. A `top` or `ops` that is not the forward's gives SLSTM_EINDEX when
 * a kernel meets an index or stack depth outside its range.
 *  x, ops, W, U, h0, c0       as given to stacklstm_fwd          (read)
 *  h_cell, c_cell, top        as written by stacklstm_fwd        (read)
 *  dh_top [T, B, H]           gradient w.r.t. h_top              (read)
 *  dc_top [T, B, H] or NULL   gradient w.r.t. c_top (NULL = 0)   (read)
 *  dx [T, B, I], dW [I, 4H], dU [H, 4H], db [4H], dh0 [B, H], dc0 [B, H]  (written)
 * dx is exactly 0 on steps whose op is not push. */
int stacklstm_bwd(const slstm_dims* d, const float* x, const int8_t* ops, const float* W, const float* U,
                  const float* h0, const float* c0, const float* h_cell, const float* c_cell, const int32_t* top,
                  void* workspace, size_t ws_bytes, const float* dh_top, const float* dc_top, float* dx, float* dW,
                  float* dU, float* db, float* dh0, float* dc0, void* stream);

/* Synchronises `stream` and reports the status held by the error words of `workspace`: that
 * of the last ordinary call (what it returned from its read-back, for calls whose return value
 * was lost), together with the first error of every deferred call made since (defer_status). */
int stacklstm_sync_status(const void* workspace, size_t ws_bytes, void* stream);

/* Static text for a status code. */
const char* stacklstm_status_string(int status);

/* Launch configuration the library chooses for `d` (informational; tests use it to reach
 * every kernel variant). */
typedef struct {
  int32_t groups;          /* forward: batch groups (one per XCC slot) */
  int32_t wg_per_group;    /* forward: workgroups per group */
  int32_t rows_per_group;  /* forward: batch rows per group (16 * fwd_tiles) */
  int32_t k_chunks;        /* K chunks of the recurrent contraction in use */
  int32_t fwd_kernel;      /* 0 plain, 1 pipelined (two LDS tile buffers), 2 wide (bf16, H > 512) */
  int32_t fwd_tiles;       /* forward: 16-row tiles per group */
  int32_t k_chunk_cap;     /* K chunks compiled into the kernels (power of two >= k_chunks) */
  int32_t occupancy;       /* 2: the recurrent kernels are compiled for 256 registers per lane
                              (two 256-thread workgroups per CU in the forward, one 512-thread
                              workgroup in the backward), else 1 */
  int32_t bwd_groups;      /* backward: batch groups */
  int32_t bwd_tiles;       /* backward: 16-row tiles per group */
  int32_t bwd_direct;      /* backward: dA rows staged in LDS by DMA (1) or read into registers (0) */
  int32_t fused_x;         /* 1: the forward kernel contracts x_t W itself (no separate input
                              projection GEMM; bf16, plain forward, one pass per step) */
  int32_t bwd_split;       /* 1: the backward contracts dA U^T over each workgroup's own gate
                              columns and exchanges partial sums instead of dA rows */
} slstm_plan;

/* Fills `out` for `d`; returns a status like the entry points. */
int stacklstm_plan(const slstm_dims* d, slstm_plan* out);

#ifdef __cplusplus
}
#endif
#endif /* STACKLSTM_H */
