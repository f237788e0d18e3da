"""Independent float64 references built on torch autograd (test-only).

``list_stack_model`` runs the branching StackLSTM over a Python list of tensors,
so its gradient comes from torch's autograd rather than from a hand-written
backward. ``bf16`` rounds both operands of each matrix product (and, in the
backward, the incoming gradient of each product) to bfloat16 through torch's own
dtype conversion.
"""
import numpy as np
import torch


def _rnd(t):
    return t.to(torch.float32).to(torch.bfloat16).to(torch.float64)


class _BF16MM(torch.autograd.Function):
    @staticmethod
    def forward(ctx, a, w):
        ar, wr = _rnd(a), _rnd(w)
        ctx.save_for_backward(ar, wr)
        return ar @ wr

    @staticmethod
    def backward(ctx, g):
        ar, wr = ctx.saved_tensors
        gr = _rnd(g)
        return gr @ wr.t(), ar.t() @ gr


def _mm(a, w, bf16):
    if bf16:
        return _BF16MM.apply(a.reshape(1, -1), w).reshape(-1)
    return a @ w


def list_stack_model(wl, bf16=False, dc_top=None):
    """Returns dict of float64 numpy arrays: h_top, c_top, and gradients of
    L = sum(dh_top * h_top) + sum(dc_top * c_top)."""
    f64 = torch.float64
    T, B, H = wl.T, wl.B, wl.H
    x = torch.tensor(wl.x, dtype=f64, requires_grad=True)
    W = torch.tensor(wl.W, dtype=f64, requires_grad=True)
    U = torch.tensor(wl.U, dtype=f64, requires_grad=True)
    b = torch.tensor(wl.b, dtype=f64, requires_grad=True)
    h0 = torch.tensor(wl.h0, dtype=f64, requires_grad=True)
    c0 = torch.tensor(wl.c0, dtype=f64, requires_grad=True)
    ops = wl.ops
    htop = [[None] * B for _ in range(T)]
    ctop = [[None] * B for _ in range(T)]
    for j in range(B):
        stack = [(h0[j], c0[j])]
        for t in range(T):
            op = int(ops[t, j])
            if op == 1:
                hp, cp = stack[-1]
                a = b + _mm(x[t, j], W, bf16) + _mm(hp, U, bf16)
                i = torch.sigmoid(a[0:H])
                f = torch.sigmoid(a[H:2 * H])
                g = torch.tanh(a[2 * H:3 * H])
                o = torch.sigmoid(a[3 * H:4 * H])
                c = f * cp + i * g
                h = o * torch.tanh(c)
                stack.append((h, c))
            elif op == -1:
                stack.pop()
            htop[t][j], ctop[t][j] = stack[-1]
    Ht = torch.stack([torch.stack(r) for r in htop])
    Ct = torch.stack([torch.stack(r) for r in ctop])
    L = (Ht * torch.tensor(wl.dh_top, dtype=f64)).sum()
    dct = wl.dc_top if dc_top is None else dc_top
    if dct is not None:
        L = L + (Ct * torch.tensor(dct, dtype=f64)).sum()
    L.backward()
    out = dict(h_top=Ht.detach().numpy(), c_top=Ct.detach().numpy())
    for k, v in (("dx", x), ("dW", W), ("dU", U), ("db", b), ("dh0", h0), ("dc0", c0)):
        out[k] = v.grad.numpy().copy()
    return out


def normwise(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.abs(ref).max() if ref.size else 0.0
    num = np.abs(a - ref).max() if ref.size else 0.0
    return num / den if den > 0 else num
