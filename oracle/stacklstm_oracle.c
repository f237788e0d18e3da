/* CPU oracle for the parallelised StackLSTM step -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the CPU-baseline leg of the benchmark call
 * this library; the HIP library never links, includes or calls it, and the two
 * share no code. It is written for checking by eye against the paper
 * (Ding & Koehn, "Parallelizable Stack Long Short-Term Memory", NAACL-SPNLP 2019):
 *
 *   - oracle_run_f64 / oracle_run_f32: the branching StackLSTM of section 2 (Push
 *     and Pop as defined there, hold from section 3), one batch element at a time,
 *     with the cell-state stack handled exactly like the hidden-state stack (the
 *     footnote of section 2), plus its exact gradient by a literal reverse sweep
 *     over the recorded nodes (section 5: popped states keep receiving gradient).
 *   - oracle_alg1_f64: Algorithm 1 of section 3 taken literally (compute every step,
 *     write slot p+1, move p by op, return slot p). It supplies the values written
 *     on non-push steps, which the branching form never computes.
 *
 * Readings where the paper is silent: the LSTM cell is the standard one (gates
 * i, f, g, o in that order along the 4H axis, single bias, no peepholes, no
 * forget-gate offset); slot 0 holds the caller's initial state (h0, c0); a pop with
 * only the initial state on the stack is an error; the returned "top" of step t is
 * the state at the pointer after that step's update.
 *
 * Precision: REAL = double for parity; REAL = float for the timed baseline. The
 * bf16-operand flag rounds both operands of every product in a matrix-product
 * position (x, W, U, h_prev, dA) to bfloat16 with round-to-nearest-even and keeps
 * everything else, including the accumulation, in REAL.
 *
 * Parity pins (tests/test_oracle_*.py): hand-worked index traces, the prefix-sum
 * form of the pointer, three independent derivations of the producer index, an
 * all-push stream against torch.nn.LSTM in float64 (values and autograd
 * gradients), a closed form for W = U = 0 that depends only on stack depth,
 * all-hold streams, central finite differences, torch autograd over a Python list
 * stack, and Observation 2 (branching form == Algorithm 1 on every returned state).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_EINVAL 1
#define ORACLE_EOPS 2
#define ORACLE_EUNDERFLOW 3

/* Round a float to bfloat16 (the top 16 bits of the binary32 pattern) with
 * round-to-nearest, ties to even, and return it widened back to float. */
static float round_bf16(float v) {
  uint32_t u;
  memcpy(&u, &v, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) {            /* inf / nan: truncate, keep nan quiet */
    if (u & 0x007fffffu) u |= 0x00400000u;
    u &= 0xffff0000u;
  } else {
    uint32_t lsb = (u >> 16) & 1u;
    u += 0x7fffu + lsb;
    u &= 0xffff0000u;
  }
  float r;
  memcpy(&r, &u, 4);
  return r;
}

void oracle_round_bf16(const float* in, float* out, long n) {
  for (long k = 0; k < n; ++k) out[k] = round_bf16(in[k]);
}

int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

#define REAL double
#define SFX(n) n##_f64
#define EXPF exp
#define TANHF tanh
#include "oracle_impl.h"
#undef REAL
#undef SFX
#undef EXPF
#undef TANHF

#define REAL float
#define SFX(n) n##_f32
#define EXPF expf
#define TANHF tanhf
#include "oracle_impl.h"
