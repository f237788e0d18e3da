/* Body of the StackLSTM CPU oracle, instantiated twice by stacklstm_oracle.c:
 * REAL = double (parity reference) and REAL = float (timed CPU baseline).
 * Test infrastructure only; see the header comment of stacklstm_oracle.c. */

/* Logistic function, evaluated in the form that does not overflow for large |z|. */
static REAL SFX(sigm)(REAL z) {
  if (z >= 0) return (REAL)1 / ((REAL)1 + EXPF(-z));
  REAL e = EXPF(z);
  return e / ((REAL)1 + e);
}

/* Operand used inside a product: unchanged, or rounded to bfloat16 when the
 * bf16-operand mode is on (only meaningful for the double instantiation). */
static REAL SFX(opnd)(REAL v, int bf16) {
  if (!bf16) return v;
  return (REAL)round_bf16((float)v);
}

/* One LSTM cell (paper, Algorithm 1 "LSTM(x_t, h_prev)"; standard cell with gates
 * i, f, g, o, one bias, no peepholes): a = b + x W + h_prev U,
 * i = sig(a_i), f = sig(a_f), g = tanh(a_g), o = sig(a_o), c = f c_prev + i g,
 * h = o tanh(c). Gate k of unit u sits at column k*H + u of W, U and b.
 * Wq/Uq are the (possibly bf16-rounded) weights. act receives i, f, g, o. */
static void SFX(cell_fwd)(int I, int H, const float* x, const REAL* Wq, const REAL* Uq, const float* bias,
                          const REAL* hp, const REAL* cp, int bf16, REAL* a, REAL* act, REAL* h, REAL* c) {
  const int G = 4 * H;
  for (int n = 0; n < G; ++n) a[n] = (REAL)bias[n];
  for (int i = 0; i < I; ++i) {
    REAL xi = SFX(opnd)((REAL)x[i], bf16);
    const REAL* w = Wq + (size_t)i * G;
    for (int n = 0; n < G; ++n) a[n] += xi * w[n];
  }
  for (int k = 0; k < H; ++k) {
    REAL hk = SFX(opnd)(hp[k], bf16);
    const REAL* u = Uq + (size_t)k * G;
    for (int n = 0; n < G; ++n) a[n] += hk * u[n];
  }
  for (int u = 0; u < H; ++u) {
    REAL ig = SFX(sigm)(a[0 * H + u]);
    REAL fg = SFX(sigm)(a[1 * H + u]);
    REAL gg = TANHF(a[2 * H + u]);
    REAL og = SFX(sigm)(a[3 * H + u]);
    act[0 * H + u] = ig; act[1 * H + u] = fg; act[2 * H + u] = gg; act[3 * H + u] = og;
    c[u] = fg * cp[u] + ig * gg;
    h[u] = og * TANHF(c[u]);
  }
}

/* Per-thread scratch for one batch element. Node k = 0 is the initial state
 * (h0, c0); node t + 1 is the state pushed at step t. */
typedef struct {
  REAL *Hn, *Cn, *dHn, *dCn, *act, *a, *dA, *tmp;
  int *parent, *stk, *opv;
} SFX(scratch);

/* Branching StackLSTM on one batch element (paper, section 2: Push reads the state
 * at the pointer, runs the LSTM, writes it above and moves the pointer up; Pop only
 * moves the pointer down; section 3: hold leaves everything unchanged), followed by
 * its exact reverse-mode gradient (section 5: gradients reach popped states and
 * their precedents). Returns 0, ORACLE_EOPS or ORACLE_EUNDERFLOW. */
static int SFX(element)(int T, int B, int I, int H, int bcol, int j, int nsel,
                        const float* x, const int8_t* ops, const REAL* Wq, const REAL* Uq, const float* bias,
                        const float* h0, const float* c0, const float* dh_top, const float* dc_top, int bf16,
                        REAL* h_top, REAL* c_top, REAL* h_cell, REAL* c_cell, int32_t* ptr, int32_t* top,
                        REAL* dx, REAL* dW, REAL* dU, REAL* db, REAL* dh0, REAL* dc0, SFX(scratch)* s) {
  const int G = 4 * H;
  for (int u = 0; u < H; ++u) { s->Hn[u] = (REAL)h0[(size_t)bcol * H + u]; s->Cn[u] = (REAL)c0[(size_t)bcol * H + u]; }
  int d = 0;              /* number of states above the initial one */
  s->stk[0] = 0;
  ptr[j] = 0;
  for (int t = 0; t < T; ++t) {
    int op = ops[(size_t)t * B + bcol];
    s->opv[t] = op;
    if (op == 1) {
      int par = s->stk[d];
      int node = t + 1;
      REAL* hn = s->Hn + (size_t)node * H;
      REAL* cn = s->Cn + (size_t)node * H;
      SFX(cell_fwd)(I, H, x + ((size_t)t * B + bcol) * I, Wq, Uq, bias, s->Hn + (size_t)par * H, s->Cn + (size_t)par * H,
                    bf16, s->a, s->act + (size_t)t * G, hn, cn);
      s->parent[node] = par;
      s->stk[++d] = node;
      if (h_cell) for (int u = 0; u < H; ++u) {
        h_cell[((size_t)t * nsel + j) * H + u] = hn[u];
        c_cell[((size_t)t * nsel + j) * H + u] = cn[u];
      }
    } else if (op == -1) {
      if (d == 0) return ORACLE_EUNDERFLOW;
      --d;
    } else if (op != 0) {
      return ORACLE_EOPS;
    }
    int tn = s->stk[d];
    top[(size_t)t * nsel + j] = tn - 1;
    ptr[(size_t)(t + 1) * nsel + j] = d;
    for (int u = 0; u < H; ++u) {
      h_top[((size_t)t * nsel + j) * H + u] = s->Hn[(size_t)tn * H + u];
      c_top[((size_t)t * nsel + j) * H + u] = s->Cn[(size_t)tn * H + u];
    }
  }
  if (!dh_top) return 0;

  /* Reverse sweep over the tape. dHn/dCn hold the gradient of the loss with
   * respect to each node's h and c. */
  memset(s->dHn, 0, sizeof(REAL) * (size_t)(T + 1) * H);
  memset(s->dCn, 0, sizeof(REAL) * (size_t)(T + 1) * H);
  for (int t = T - 1; t >= 0; --t) {
    int tn = top[(size_t)t * nsel + j] + 1;        /* node on top after step t */
    for (int u = 0; u < H; ++u) {
      s->dHn[(size_t)tn * H + u] += (REAL)dh_top[((size_t)t * B + bcol) * H + u];
      if (dc_top) s->dCn[(size_t)tn * H + u] += (REAL)dc_top[((size_t)t * B + bcol) * H + u];
    }
    REAL* dxr = dx ? dx + ((size_t)t * nsel + j) * I : NULL;
    if (s->opv[t] != 1) {
      if (dxr) for (int i = 0; i < I; ++i) dxr[i] = 0;
      continue;
    }
    int node = t + 1, par = s->parent[node];
    const REAL* act = s->act + (size_t)t * G;
    const REAL* hp = s->Hn + (size_t)par * H;
    const REAL* cp = s->Cn + (size_t)par * H;
    const REAL* cn = s->Cn + (size_t)node * H;
    for (int u = 0; u < H; ++u) {
      REAL ig = act[u], fg = act[H + u], gg = act[2 * H + u], og = act[3 * H + u];
      REAL tc = TANHF(cn[u]);
      REAL dh = s->dHn[(size_t)node * H + u];
      REAL dc = s->dCn[(size_t)node * H + u] + dh * og * ((REAL)1 - tc * tc);
      s->dA[0 * H + u] = dc * gg * ig * ((REAL)1 - ig);
      s->dA[1 * H + u] = dc * cp[u] * fg * ((REAL)1 - fg);
      s->dA[2 * H + u] = dc * ig * ((REAL)1 - gg * gg);
      s->dA[3 * H + u] = dh * tc * og * ((REAL)1 - og);
      s->dCn[(size_t)par * H + u] += dc * fg;
    }
    /* products with dA: dx = W dA, dh_prev = U dA, dW += x (x) dA, dU += h_prev (x) dA, db += dA */
    for (int n = 0; n < G; ++n) s->tmp[n] = SFX(opnd)(s->dA[n], bf16);
    const float* xr = x + ((size_t)t * B + bcol) * I;
    for (int i = 0; i < I; ++i) {
      const REAL* w = Wq + (size_t)i * G;
      REAL acc = 0;
      for (int n = 0; n < G; ++n) acc += w[n] * s->tmp[n];
      if (dxr) dxr[i] = acc;
      REAL xi = SFX(opnd)((REAL)xr[i], bf16);
      REAL* dwr = dW + (size_t)i * G;
      for (int n = 0; n < G; ++n) dwr[n] += xi * s->tmp[n];
    }
    for (int k = 0; k < H; ++k) {
      const REAL* uu = Uq + (size_t)k * G;
      REAL acc = 0;
      for (int n = 0; n < G; ++n) acc += uu[n] * s->tmp[n];
      s->dHn[(size_t)par * H + k] += acc;
      REAL hk = SFX(opnd)(hp[k], bf16);
      REAL* dur = dU + (size_t)k * G;
      for (int n = 0; n < G; ++n) dur[n] += hk * s->tmp[n];
    }
    for (int n = 0; n < G; ++n) db[n] += s->dA[n];
  }
  for (int u = 0; u < H; ++u) {
    dh0[(size_t)j * H + u] = s->dHn[u];
    dc0[(size_t)j * H + u] = s->dCn[u];
  }
  return 0;
}

int SFX(oracle_run)(int T, int B, int I, int H, const float* x, const int8_t* ops, const float* W, const float* U,
                    const float* bias, const float* h0, const float* c0, const float* dh_top, const float* dc_top,
                    const int32_t* sel, int nsel, int bf16, int nthreads,
                    REAL* h_top, REAL* c_top, REAL* h_cell, REAL* c_cell, int32_t* ptr, int32_t* top,
                    REAL* dx, REAL* dW, REAL* dU, REAL* db, REAL* dh0, REAL* dc0) {
  if (T < 0 || B < 1 || I < 1 || H < 1 || nsel < 0) return ORACLE_EINVAL;
  const int G = 4 * H;
  if (nthreads < 1) nthreads = 1;
  REAL* Wq = (REAL*)malloc(sizeof(REAL) * (size_t)I * G);
  REAL* Uq = (REAL*)malloc(sizeof(REAL) * (size_t)H * G);
  for (size_t k = 0; k < (size_t)I * G; ++k) Wq[k] = SFX(opnd)((REAL)W[k], bf16);
  for (size_t k = 0; k < (size_t)H * G; ++k) Uq[k] = SFX(opnd)((REAL)U[k], bf16);
  size_t wsz = (size_t)I * G + (size_t)H * G + G;
  REAL* part = dh_top ? (REAL*)calloc((size_t)nthreads * wsz, sizeof(REAL)) : NULL;
  int* status = (int*)calloc((size_t)(nsel > 0 ? nsel : 1), sizeof(int));

#pragma omp parallel num_threads(nthreads)
  {
    int tid = 0;
#ifdef _OPENMP
    tid = omp_get_thread_num();
#endif
    SFX(scratch) s;
    s.Hn = (REAL*)malloc(sizeof(REAL) * (size_t)(T + 1) * H);
    s.Cn = (REAL*)malloc(sizeof(REAL) * (size_t)(T + 1) * H);
    s.dHn = (REAL*)malloc(sizeof(REAL) * (size_t)(T + 1) * H);
    s.dCn = (REAL*)malloc(sizeof(REAL) * (size_t)(T + 1) * H);
    s.act = (REAL*)malloc(sizeof(REAL) * ((size_t)T * G + 1));
    s.a = (REAL*)malloc(sizeof(REAL) * G);
    s.dA = (REAL*)malloc(sizeof(REAL) * G);
    s.tmp = (REAL*)malloc(sizeof(REAL) * G);
    s.parent = (int*)malloc(sizeof(int) * (size_t)(T + 1));
    s.stk = (int*)malloc(sizeof(int) * (size_t)(T + 1));
    s.opv = (int*)malloc(sizeof(int) * (size_t)(T + 1));
    REAL* myp = part ? part + (size_t)tid * wsz : NULL;
#pragma omp for schedule(static)
    for (int j = 0; j < nsel; ++j) {
      status[j] = SFX(element)(T, B, I, H, sel[j], j, nsel, x, ops, Wq, Uq, bias, h0, c0, dh_top, dc_top, bf16,
                               h_top, c_top, h_cell, c_cell, ptr, top, dx,
                               myp, myp ? myp + (size_t)I * G : NULL, myp ? myp + (size_t)I * G + (size_t)H * G : NULL,
                               dh0, dc0, &s);
    }
    free(s.Hn); free(s.Cn); free(s.dHn); free(s.dCn); free(s.act); free(s.a); free(s.dA); free(s.tmp);
    free(s.parent); free(s.stk); free(s.opv);
  }
  int rc = 0;
  for (int j = 0; j < nsel && !rc; ++j) rc = status[j];
  if (dh_top) {
    /* reduce the per-thread weight-gradient partials in thread order */
    memset(dW, 0, sizeof(REAL) * (size_t)I * G);
    memset(dU, 0, sizeof(REAL) * (size_t)H * G);
    memset(db, 0, sizeof(REAL) * G);
    for (int th = 0; th < nthreads; ++th) {
      const REAL* p = part + (size_t)th * wsz;
      for (size_t k = 0; k < (size_t)I * G; ++k) dW[k] += p[k];
      for (size_t k = 0; k < (size_t)H * G; ++k) dU[k] += p[(size_t)I * G + k];
      for (int k = 0; k < G; ++k) db[k] += p[(size_t)I * G + (size_t)H * G + k];
    }
  }
  free(Wq); free(Uq); free(part); free(status);
  return rc;
}

/* Algorithm 1 taken literally on one element: a float stack of T + 1 slots, the
 * LSTM is run at every step whatever the op, its result is written to slot p + 1,
 * then p moves by op and the slot at p is returned. An int stack receives the step
 * index the same way, giving the producer of the returned state. Forward only. */
int SFX(oracle_alg1)(int T, int B, int I, int H, const float* x, const int8_t* ops, const float* W, const float* U,
                     const float* bias, const float* h0, const float* c0, const int32_t* sel, int nsel, int bf16,
                     int nthreads, REAL* h_top, REAL* c_top, REAL* h_cell, REAL* c_cell, int32_t* ptr, int32_t* top) {
  if (T < 0 || B < 1 || I < 1 || H < 1 || nsel < 0) return ORACLE_EINVAL;
  const int G = 4 * H;
  if (nthreads < 1) nthreads = 1;
  REAL* Wq = (REAL*)malloc(sizeof(REAL) * (size_t)I * G);
  REAL* Uq = (REAL*)malloc(sizeof(REAL) * (size_t)H * G);
  for (size_t k = 0; k < (size_t)I * G; ++k) Wq[k] = SFX(opnd)((REAL)W[k], bf16);
  for (size_t k = 0; k < (size_t)H * G; ++k) Uq[k] = SFX(opnd)((REAL)U[k], bf16);
  int* status = (int*)calloc((size_t)(nsel > 0 ? nsel : 1), sizeof(int));
#pragma omp parallel num_threads(nthreads)
  {
    REAL* Sh = (REAL*)malloc(sizeof(REAL) * (size_t)(T + 2) * H);
    REAL* Sc = (REAL*)malloc(sizeof(REAL) * (size_t)(T + 2) * H);
    int* Si = (int*)malloc(sizeof(int) * (size_t)(T + 2));
    REAL* a = (REAL*)malloc(sizeof(REAL) * G);
    REAL* act = (REAL*)malloc(sizeof(REAL) * G);
#pragma omp for schedule(static)
    for (int j = 0; j < nsel; ++j) {
      int bcol = sel[j];
      for (int u = 0; u < H; ++u) { Sh[u] = (REAL)h0[(size_t)bcol * H + u]; Sc[u] = (REAL)c0[(size_t)bcol * H + u]; }
      Si[0] = -1;
      int p = 0, rc = 0;
      ptr[j] = 0;
      for (int t = 0; t < T && !rc; ++t) {
        int op = ops[(size_t)t * B + bcol];
        if (op < -1 || op > 1) { rc = ORACLE_EOPS; break; }
        REAL* hn = Sh + (size_t)(p + 1) * H;
        REAL* cn = Sc + (size_t)(p + 1) * H;
        SFX(cell_fwd)(I, H, x + ((size_t)t * B + bcol) * I, Wq, Uq, bias, Sh + (size_t)p * H, Sc + (size_t)p * H, bf16,
                      a, act, hn, cn);
        Si[p + 1] = t;
        for (int u = 0; u < H; ++u) {
          h_cell[((size_t)t * nsel + j) * H + u] = hn[u];
          c_cell[((size_t)t * nsel + j) * H + u] = cn[u];
        }
        p += op;
        if (p < 0) { rc = ORACLE_EUNDERFLOW; break; }
        ptr[(size_t)(t + 1) * nsel + j] = p;
        top[(size_t)t * nsel + j] = Si[p];
        for (int u = 0; u < H; ++u) {
          h_top[((size_t)t * nsel + j) * H + u] = Sh[(size_t)p * H + u];
          c_top[((size_t)t * nsel + j) * H + u] = Sc[(size_t)p * H + u];
        }
      }
      status[j] = rc;
    }
    free(Sh); free(Sc); free(Si); free(a); free(act);
  }
  int rc = 0;
  for (int j = 0; j < nsel && !rc; ++j) rc = status[j];
  free(Wq); free(Uq); free(status);
  return rc;
}
