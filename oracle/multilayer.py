"""Multi-layer StackLSTM oracle -- TEST INFRASTRUCTURE ONLY (tests, the smoke check and
the benchmark's CPU leg may use it; the HIP library never does).

A StackLSTM whose stack element is the state of every layer (the parser the paper builds
on stacks LSTM layers; section 4.1 uses hidden dimension 200 for all of them). Per batch
element, in float64 with torch autograd, written from the definitions of section 2 (and
the hold op of section 3):

  push  read the element at the pointer; layer 1 runs the LSTM cell on (x_t, its state
        there), layer l > 1 on (the new h of layer l-1, its state there); the new states
        of all layers form one element written above the pointer; the pointer moves up;
  pop   the pointer moves down;   hold  nothing changes.

The value returned at step t is the element at the pointer after the update, for every
layer. The loss is sum_t <dh_top[t], h_top_L[t]> (+ <dc_top[t], c_top_L[t]>) on the last
layer L; gradients come from torch autograd over the list stack, so they reach popped
and overwritten states exactly as section 5 describes. The cell is the standard LSTM
(gates i, f, g, o along 4H, one bias, h = o tanh(c)), as in the single-layer oracle.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch


def _cell(x, hp, cp, W, U, b):
    H = hp.shape[-1]
    a = b + x @ W + hp @ U
    i = torch.sigmoid(a[..., 0 * H:1 * H])
    f = torch.sigmoid(a[..., 1 * H:2 * H])
    g = torch.tanh(a[..., 2 * H:3 * H])
    o = torch.sigmoid(a[..., 3 * H:4 * H])
    c = f * cp + i * g
    return o * torch.tanh(c), c


def run(ops: np.ndarray, x: np.ndarray, layers: Sequence[tuple], h0: Sequence[np.ndarray],
        c0: Sequence[np.ndarray], dh_top: np.ndarray, dc_top: Optional[np.ndarray] = None) -> dict:
    """ops [T, B] int8; x [T, B, I]; layers = [(W_l [I_l, 4H], U_l [H, 4H], b_l [4H])], I_1 = I and
    I_l = H after; h0/c0 = per layer [B, H]; dh_top/dc_top [T, B, H] on the last layer.
    Returns h_top/c_top per layer ([T, B, H] each, lists), top [T, B] (producer step of the
    returned element, -1 = initial), and the gradients dx [T, B, I], dW/dU/db/dh0/dc0 per layer."""
    T, B = ops.shape
    L = len(layers)
    d = torch.float64
    xt = torch.tensor(x, dtype=d, requires_grad=True)
    P = [tuple(torch.tensor(p, dtype=d, requires_grad=True) for p in lay) for lay in layers]
    h0t = [torch.tensor(h, dtype=d, requires_grad=True) for h in h0]
    c0t = [torch.tensor(c, dtype=d, requires_grad=True) for c in c0]
    h_top = [[[None] * B for _ in range(T)] for _ in range(L)]
    c_top = [[[None] * B for _ in range(T)] for _ in range(L)]
    top = np.zeros((T, B), np.int32)
    for bb in range(B):
        stack = [(-1, [(h0t[l][bb], c0t[l][bb]) for l in range(L)])]
        for t in range(T):
            op = int(ops[t, bb])
            if op == 1:
                inp = xt[t, bb]
                elem = []
                for l, (W, U, bias) in enumerate(P):
                    hp, cp = stack[-1][1][l]
                    h, c = _cell(inp, hp, cp, W, U, bias)
                    elem.append((h, c))
                    inp = h
                stack.append((t, elem))
            elif op == -1:
                if len(stack) == 1:
                    raise ValueError("pop with only the initial state on the stack")
                stack.pop()
            elif op != 0:
                raise ValueError(f"op {op}")
            top[t, bb] = stack[-1][0]
            for l in range(L):
                h_top[l][t][bb], c_top[l][t][bb] = stack[-1][1][l]
    H_last = [torch.stack([torch.stack(row) for row in h_top[l]]) for l in range(L)]
    C_last = [torch.stack([torch.stack(row) for row in c_top[l]]) for l in range(L)]
    loss = (H_last[-1] * torch.tensor(dh_top, dtype=d)).sum()
    if dc_top is not None:
        loss = loss + (C_last[-1] * torch.tensor(dc_top, dtype=d)).sum()
    loss.backward()
    z = lambda t: np.zeros(tuple(t.shape)) if t.grad is None else t.grad.numpy()
    return {
        "h_top": [h.detach().numpy() for h in H_last], "c_top": [c.detach().numpy() for c in C_last], "top": top,
        "dx": z(xt), "dW": [z(p[0]) for p in P], "dU": [z(p[1]) for p in P], "db": [z(p[2]) for p in P],
        "dh0": [z(h) for h in h0t], "dc0": [z(c) for c in c0t],
    }
