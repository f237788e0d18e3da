"""Seeded synthetic workloads for the parallelised StackLSTM step.

This module only draws inputs: op streams, activations, weights and the
upstream gradient. It holds none of the method's arithmetic, so the CPU oracle
and the HIP path can both consume its arrays without sharing any computation.

Op encoding (paper, section 3 and the hold paragraph after Algorithm 1):
+1 = push, -1 = pop, 0 = hold, stored as int8 in a time-major [T, B] array.

The paper trains a parser on the Stanford Dependency treebank (section 4.1),
which is not available here; the streams below stand in for its oracle
transition sequences with the same stack-op shape:

* ``tiny``   -- push/pop with p = 0.6 / 0.4 (a pop on an empty stack becomes a
  push), active length uniform in 32..64, padded with hold to T = 64.
* ``parser``, ``large``, ``thru`` -- arc-standard shaped streams: for a sentence
  of n words there are n shifts (push) and n-1 reduces (pop); a shift is forced
  while fewer than two items are on the stack, a reduce is forced once the
  buffer is empty, otherwise reduce with probability 0.5. Padded with hold to
  T = 2 * max n.
* ``deep``   -- bursty runs: push runs of 100..300, pop runs of 100..200
  clamped to the current depth, alternating, truncated at T = 1024.
* ``hybrid`` -- the arc-hybrid parser's two StackLSTMs (paper, section 3 and its
  transition table): per sentence of n words a random arc-hybrid transition
  sequence (n shifts, n-1 left/right arcs, each chosen uniformly among the valid
  ones) drives a stack StackLSTM (shift = push, either arc = pop) and a buffer
  StackLSTM (the n words pushed first, then shift = pop, either arc = hold); both
  run as one doubled batch (rows 0..E-1 the stacks, E..2E-1 the buffers of the E
  sentences) with shared weights, padded with hold to T = 3 * max n - 1.

Every draw comes from one ``numpy.random.default_rng(seed)`` in the fixed order
ops (element by element), x, W, U, b, h0, c0, R (the upstream gradient).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

PUSH, POP, HOLD = 1, -1, 0

FP32 = 0
BF16_GEMM = 1


@dataclass
class Workload:
    name: str
    T: int
    B: int
    I: int
    H: int
    precision: int
    ops: np.ndarray            # int8 [T, B]
    x: np.ndarray              # f32 [T, B, I]
    W: np.ndarray              # f32 [I, 4H]   gate order i, f, g, o along 4H
    U: np.ndarray              # f32 [H, 4H]
    b: np.ndarray              # f32 [4H]
    h0: np.ndarray             # f32 [B, H]
    c0: np.ndarray             # f32 [B, H]
    dh_top: np.ndarray         # f32 [T, B, H]  upstream gradient of the top output
    dc_top: Optional[np.ndarray] = None   # f32 [T, B, H] or None (= 0)
    meta: dict = field(default_factory=dict)

    def op_stats(self) -> dict:
        ops = self.ops.astype(np.int64)
        depth = np.cumsum(ops, axis=0)
        n = ops.size
        return {
            "push": float((ops == PUSH).sum()) / n,
            "pop": float((ops == POP).sum()) / n,
            "hold": float((ops == HOLD).sum()) / n,
            "max_depth": int(depth.max(initial=0)),
            "push_steps": int((ops == PUSH).sum()),
        }


# ----------------------------------------------------------------------------- op streams

def ops_tiny_stream(rng: np.random.Generator, T: int, lo: int, hi: int) -> np.ndarray:
    """push 0.6 / pop 0.4, a pop at depth 0 is drawn as a push, then hold-padded."""
    L = int(rng.integers(lo, hi + 1))
    out = np.zeros(T, dtype=np.int8)
    p = 0
    for t in range(min(L, T)):
        op = PUSH if rng.random() < 0.6 else POP
        if op == POP and p == 0:
            op = PUSH
        out[t] = op
        p += op
    return out


def ops_arc_standard_stream(rng: np.random.Generator, n: int) -> np.ndarray:
    """n shifts and n-1 reduces in an arc-standard order (2n-1 ops, no padding)."""
    out = []
    p = 0
    buf = n
    reduces_left = n - 1
    while buf > 0 or reduces_left > 0:
        if buf > 0 and (p < 2 or reduces_left == 0):
            op = PUSH
        elif buf == 0:
            op = POP
        else:
            op = POP if rng.random() < 0.5 else PUSH
        if op == PUSH:
            buf -= 1
        else:
            reduces_left -= 1
        p += op
        out.append(op)
    return np.asarray(out, dtype=np.int8)


def ops_arc_hybrid_streams(rng: np.random.Generator, n: int) -> tuple:
    """Stack and buffer op streams of one sentence of n words (3n - 1 steps each): the
    buffer first receives the n words (n pushes while the stack holds), then a random
    arc-hybrid transition sequence runs. Valid transitions: shift needs a non-empty
    buffer, left-arc a non-empty stack and a non-empty buffer, right-arc two stack
    items; the sequence ends with an empty buffer and one item on the stack."""
    stack = [HOLD] * n
    buf = [PUSH] * n
    s, b = 0, n
    while b > 0 or s > 1:
        valid = []
        if b > 0:
            valid.append("shift")
        if s >= 1 and b > 0:
            valid.append("left")
        if s >= 2:
            valid.append("right")
        tr = valid[int(rng.integers(len(valid)))]
        if tr == "shift":
            stack.append(PUSH)
            buf.append(POP)
            s, b = s + 1, b - 1
        else:
            stack.append(POP)
            buf.append(HOLD)
            s -= 1
    return np.asarray(stack, dtype=np.int8), np.asarray(buf, dtype=np.int8)


def ops_deep_stream(rng: np.random.Generator, T: int, push_run=(100, 300), pop_run=(100, 200)) -> np.ndarray:
    out = np.zeros(T, dtype=np.int8)
    t = 0
    p = 0
    pushing = True
    while t < T:
        if pushing:
            r = int(rng.integers(push_run[0], push_run[1] + 1))
            r = min(r, T - t)
            out[t:t + r] = PUSH
            p += r
        else:
            r = int(rng.integers(pop_run[0], pop_run[1] + 1))
            r = min(r, p, T - t)
            out[t:t + r] = POP
            p -= r
        t += r
        pushing = not pushing
    return out


def ops_random_valid(rng: np.random.Generator, T: int, B: int, p_push=0.45, p_pop=0.35) -> np.ndarray:
    """Random push/pop/hold streams that never pop an empty stack (test helper)."""
    ops = np.zeros((T, B), dtype=np.int8)
    for b in range(B):
        p = 0
        for t in range(T):
            u = rng.random()
            op = PUSH if u < p_push else (POP if u < p_push + p_pop else HOLD)
            if op == POP and p == 0:
                op = HOLD
            ops[t, b] = op
            p += op
    return ops


# ----------------------------------------------------------------------------- values

def _values(rng, T, B, I, H, wscale, bias_zero, random_state=False, dc_top=False):
    x = rng.standard_normal((T, B, I), dtype=np.float32)
    W = rng.uniform(-wscale, wscale, size=(I, 4 * H)).astype(np.float32)
    U = rng.uniform(-wscale, wscale, size=(H, 4 * H)).astype(np.float32)
    if bias_zero:
        b = np.zeros(4 * H, dtype=np.float32)
    else:
        b = rng.uniform(-wscale, wscale, size=(4 * H,)).astype(np.float32)
    if random_state:
        h0 = rng.uniform(-0.5, 0.5, size=(B, H)).astype(np.float32)
        c0 = rng.uniform(-0.5, 0.5, size=(B, H)).astype(np.float32)
    else:
        h0 = np.zeros((B, H), dtype=np.float32)
        c0 = np.zeros((B, H), dtype=np.float32)
    R = rng.standard_normal((T, B, H), dtype=np.float32)
    Rc = rng.standard_normal((T, B, H), dtype=np.float32) if dc_top else None
    return x, W, U, b, h0, c0, R, Rc


CONFIGS = {
    # name: (B, I, H, precision, seed, op-kind, op-params)
    "tiny": dict(B=8, I=32, H=64, precision=FP32, seed=101, kind="tiny", T=64, lo=32, hi=64, wscale=0.1, bias_zero=True),
    "parser": dict(B=64, I=128, H=256, precision=FP32, seed=102, kind="arc", nlo=10, nhi=60, wscale=0.08, bias_zero=False),
    "large": dict(B=256, I=256, H=512, precision=FP32, seed=103, kind="arc", nlo=20, nhi=120, wscale=0.08, bias_zero=False),
    "deep": dict(B=128, I=256, H=512, precision=FP32, seed=104, kind="deep", T=1024, wscale=0.08, bias_zero=False),
    "thru": dict(B=1024, I=512, H=1024, precision=BF16_GEMM, seed=105, kind="arc", nlo=10, nhi=128, wscale=0.08, bias_zero=False),
    # B counts sentences; the workload has 2B rows (stack StackLSTMs, then buffer StackLSTMs)
    "hybrid": dict(B=128, I=256, H=512, precision=FP32, seed=106, kind="hybrid", nlo=20, nhi=80, wscale=0.08, bias_zero=False),
    # the paper's cell size (hidden dimension 200 for every LSTM, section 4.1) on the
    # arc-hybrid stack + buffer streams of a batch of 64 sentences
    "paper": dict(B=64, I=200, H=200, precision=FP32, seed=107, kind="hybrid", nlo=10, nhi=60, wscale=0.08, bias_zero=False),
}


def layer_params(wl: Workload, L: int) -> tuple:
    """Parameters of L stacked layers for a workload: layer 1 is the workload's own (W, U,
    b, h0, c0); layers 2..L (input size H) are drawn from default_rng(seed + 1000 + l) with
    the workload's recipe (weights and bias U(-0.08, 0.08), zero initial state)."""
    seed = int(wl.meta.get("seed", 0))
    layers = [(wl.W, wl.U, wl.b)]
    h0, c0 = [wl.h0], [wl.c0]
    for l in range(1, L):
        rng = np.random.default_rng(seed + 1000 + l)
        H = wl.H
        layers.append((rng.uniform(-0.08, 0.08, (H, 4 * H)).astype(np.float32),
                       rng.uniform(-0.08, 0.08, (H, 4 * H)).astype(np.float32),
                       rng.uniform(-0.08, 0.08, 4 * H).astype(np.float32)))
        h0.append(np.zeros((wl.B, H), np.float32))
        c0.append(np.zeros((wl.B, H), np.float32))
    return layers, h0, c0


def make(name: str, seed: Optional[int] = None, precision: Optional[int] = None, B: Optional[int] = None,
         T: Optional[int] = None) -> Workload:
    """Build one of the named workloads. ``precision`` overrides the GEMM precision
    (e.g. the large shape in bf16-GEMM mode); ``B`` overrides the batch size (used
    by the batch-size sweep), keeping the rest of the recipe; ``T`` pads the
    arc-standard streams with holds to at least T steps (a fixed length across the
    sweep, so every batch size does the same work per element)."""
    c = dict(CONFIGS[name])
    if B is not None:
        c["B"] = int(B)
    rng = np.random.default_rng(c["seed"] if seed is None else seed)
    Bn, I, H = c["B"], c["I"], c["H"]
    if c["kind"] == "tiny":
        T = max(c["T"], T or 0)
        ops = np.stack([ops_tiny_stream(rng, T, c["lo"], c["hi"]) for _ in range(Bn)], axis=1)
    elif c["kind"] == "arc":
        streams, lengths = [], []
        for _ in range(Bn):
            n = int(rng.integers(c["nlo"], c["nhi"] + 1))
            lengths.append(n)
            streams.append(ops_arc_standard_stream(rng, n))
        T = max(2 * max(lengths), T or 0)
        ops = np.zeros((T, Bn), dtype=np.int8)
        for j, s in enumerate(streams):
            ops[: len(s), j] = s
    elif c["kind"] == "hybrid":
        pairs = [ops_arc_hybrid_streams(rng, int(rng.integers(c["nlo"], c["nhi"] + 1))) for _ in range(Bn)]
        T = max(max(len(st) for st, _ in pairs), T or 0)
        ops = np.zeros((T, 2 * Bn), dtype=np.int8)
        for j, (st, bu) in enumerate(pairs):
            ops[: len(st), j] = st
            ops[: len(bu), Bn + j] = bu
        Bn = 2 * Bn
    elif c["kind"] == "deep":
        T = max(c["T"], T or 0)
        ops = np.stack([ops_deep_stream(rng, T) for _ in range(Bn)], axis=1)
    else:
        raise ValueError(c["kind"])
    x, W, U, b, h0, c0, R, _ = _values(rng, T, Bn, I, H, c["wscale"], c["bias_zero"])
    prec = c["precision"] if precision is None else precision
    return Workload(name=name, T=T, B=Bn, I=I, H=H, precision=prec, ops=np.ascontiguousarray(ops), x=x, W=W, U=U,
                    b=b, h0=h0, c0=c0, dh_top=R, meta={"seed": c["seed"] if seed is None else seed})


def custom(T: int, B: int, I: int, H: int, seed: int, ops: Optional[np.ndarray] = None, wscale: float = 0.1,
           random_state: bool = False, dc_top: bool = False, precision: int = FP32, bias_zero: bool = False,
           name: str = "custom") -> Workload:
    """Small ad-hoc workloads for tests; ``ops`` may be given explicitly ([T, B] int8)."""
    rng = np.random.default_rng(seed)
    if ops is None:
        ops = ops_random_valid(rng, T, B)
    ops = np.ascontiguousarray(np.asarray(ops, dtype=np.int8).reshape(T, B))
    x, W, U, b, h0, c0, R, Rc = _values(rng, T, B, I, H, wscale, bias_zero, random_state, dc_top)
    return Workload(name=name, T=T, B=B, I=I, H=H, precision=precision, ops=ops, x=x, W=W, U=U, b=b, h0=h0, c0=c0,
                    dh_top=R, dc_top=Rc, meta={"seed": seed})
