"""Pins of the CPU oracle to things other than itself (paper definitions, closed
forms, textbook LSTM, finite differences, an autograd implementation).

Sections cited are those of the paper: section 2 (Push/Pop definitions and the
cell-state footnote), section 3 (pointer update p <- p + op, Observations 1-2,
Algorithm 1, the hold op), section 5 (gradients flow to popped states).
"""
import os

import numpy as np
import pytest
import torch

from paper_1904_03409_amd import workloads as wk
from tests import trace_ref
from tests.torch_ref import list_stack_model, normwise

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "trace_example.txt")


def _golden():
    rows = {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        k, *v = line.split()
        rows[k] = [int(z) for z in v]
    return rows


def _single(ops, H=3, I=2, seed=0, **kw):
    ops = np.asarray(ops, np.int8).reshape(-1, 1)
    return wk.custom(T=ops.shape[0], B=1, I=I, H=H, seed=seed, ops=ops, **kw)


# ----------------------------------------------------------------------------- index traces

def test_golden_trace(oracle_mod):
    g = _golden()
    r = oracle_mod.run(_single(g["ops"]))
    assert r["ptr"][:, 0].tolist() == g["ptr"]
    assert r["top"][:, 0].tolist() == g["top"]
    src = [-1] + r["top"][:-1, 0].tolist()
    assert src == g["src"]
    # the reference derivations agree with the hand-worked trace too
    assert trace_ref.list_stack(g["ops"]) == (g["top"], g["ptr"])
    assert trace_ref.alg1_int_stack(g["ops"]) == (g["top"], g["ptr"])
    assert trace_ref.parent_pointer(g["ops"]) == (g["top"], g["src"])
    assert trace_ref.closed_form(g["ops"]) == (g["top"], g["ptr"])


@pytest.mark.parametrize("seed", range(6))
def test_trace_invariants_random(oracle_mod, seed):
    rng = np.random.default_rng(seed)
    T, B = 97, 9
    ops = wk.ops_random_valid(rng, T, B, p_push=0.4, p_pop=0.4)
    wl = wk.custom(T=T, B=B, I=2, H=2, seed=seed, ops=ops)
    r = oracle_mod.run(wl, backward=False)
    ptr = np.vstack([np.zeros((1, B), np.int64), np.cumsum(ops.astype(np.int64), axis=0)])
    assert np.array_equal(r["ptr"], ptr) and r["ptr"].min() >= 0        # p <- p + op, never below 0
    for j in range(B):
        col = ops[:, j].tolist()
        top = r["top"][:, j].tolist()
        assert trace_ref.list_stack(col)[0] == top
        assert trace_ref.alg1_int_stack(col)[0] == top
        assert trace_ref.parent_pointer(col)[0] == top
        assert trace_ref.closed_form(col)[0] == top


def test_errors(oracle_mod):
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.run(_single([1, -1, -1, 1]))
    assert e.value.code == 3                                                # pop of the initial state
    wl = _single([1, 2, 0])
    with pytest.raises(oracle_mod.OracleError) as e:
        oracle_mod.run(wl)
    assert e.value.code == 2                                                # op outside {-1, 0, 1}
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.alg1(_single([-1, 1]))


# ----------------------------------------------------------------------------- cell values

def test_all_push_is_textbook_lstm(oracle_mod):
    """A push-only stream is an ordinary LSTM: compare with torch.nn.LSTMCell in float64,
    values and autograd gradients (weight_ih = W^T, weight_hh = U^T, bias_ih = b, bias_hh = 0)."""
    T, B, I, H = 9, 3, 5, 4
    wl = wk.custom(T=T, B=B, I=I, H=H, seed=11, ops=np.ones((T, B), np.int8), wscale=0.5, random_state=True,
                   dc_top=True)
    r = oracle_mod.run(wl)
    f64 = torch.float64
    cell = torch.nn.LSTMCell(I, H, bias=True).to(f64)
    with torch.no_grad():
        cell.weight_ih.copy_(torch.tensor(wl.W.T, dtype=f64))
        cell.weight_hh.copy_(torch.tensor(wl.U.T, dtype=f64))
        cell.bias_ih.copy_(torch.tensor(wl.b, dtype=f64))
        cell.bias_hh.zero_()
    x = torch.tensor(wl.x, dtype=f64, requires_grad=True)
    h = torch.tensor(wl.h0, dtype=f64, requires_grad=True)
    c = torch.tensor(wl.c0, dtype=f64, requires_grad=True)
    h0, c0 = h, c
    hs, cs = [], []
    for t in range(T):
        h, c = cell(x[t], (h, c))
        hs.append(h)
        cs.append(c)
    Hs, Cs = torch.stack(hs), torch.stack(cs)
    L = (Hs * torch.tensor(wl.dh_top, dtype=f64)).sum() + (Cs * torch.tensor(wl.dc_top, dtype=f64)).sum()
    L.backward()
    tol = 1e-12
    assert normwise(r["h_top"], Hs.detach().numpy()) < tol
    assert normwise(r["c_top"], Cs.detach().numpy()) < tol
    assert normwise(r["h_cell"], Hs.detach().numpy()) < tol
    assert normwise(r["dx"], x.grad.numpy()) < tol
    assert normwise(r["dW"], cell.weight_ih.grad.numpy().T) < tol
    assert normwise(r["dU"], cell.weight_hh.grad.numpy().T) < tol
    assert normwise(r["db"], cell.bias_ih.grad.numpy()) < tol
    assert normwise(r["dh0"], h0.grad.numpy()) < tol
    assert normwise(r["dc0"], c0.grad.numpy()) < tol


def test_zero_weights_closed_form(oracle_mod):
    """W = U = 0, h0 = c0 = 0: every push computes the same gates, so the state at
    depth d is c(d) = i g (1 - f^d) / (1 - f), h(d) = o tanh(c(d)). The returned top
    of step t must be the depth-ptr[t+1] state: this pins hold, pop, and a push that
    overwrites a slot freed by an earlier pop, purely numerically."""
    rng = np.random.default_rng(3)
    T, B, H = 60, 4, 3
    ops = wk.ops_random_valid(rng, T, B, p_push=0.45, p_pop=0.35)
    wl = wk.custom(T=T, B=B, I=2, H=H, seed=5, ops=ops)
    wl.W[:] = 0
    wl.U[:] = 0
    wl.b[:] = rng.uniform(-1.5, 1.5, size=4 * H).astype(np.float32)
    r = oracle_mod.run(wl, backward=False)
    bb = wl.b.astype(np.float64)
    sig = lambda z: 1.0 / (1.0 + np.exp(-z))
    i, f, g, o = sig(bb[:H]), sig(bb[H:2 * H]), np.tanh(bb[2 * H:3 * H]), sig(bb[3 * H:])
    depth = r["ptr"][1:]                                              # [T, B]
    cd = i * g * (1.0 - f[None, None, :] ** depth[..., None]) / (1.0 - f)
    hd = o * np.tanh(cd)
    assert np.abs(r["c_top"] - cd).max() < 1e-14
    assert np.abs(r["h_top"] - hd).max() < 1e-14


def test_all_hold_is_identity(oracle_mod):
    T, B = 7, 3
    wl = wk.custom(T=T, B=B, I=4, H=5, seed=2, ops=np.zeros((T, B), np.int8), random_state=True, dc_top=True)
    r = oracle_mod.run(wl)
    assert np.array_equal(r["h_top"], np.broadcast_to(wl.h0.astype(np.float64), (T, B, 5)))
    assert np.array_equal(r["c_top"], np.broadcast_to(wl.c0.astype(np.float64), (T, B, 5)))
    assert np.all(r["top"] == -1) and np.all(r["ptr"] == 0)
    for k in ("dW", "dU", "db", "dx"):
        assert np.all(r[k] == 0), k
    assert np.allclose(r["dh0"], wl.dh_top.astype(np.float64).sum(0), rtol=0, atol=1e-13)
    assert np.allclose(r["dc0"], wl.dc_top.astype(np.float64).sum(0), rtol=0, atol=1e-13)


# ----------------------------------------------------------------------------- gradients

def _loss(oracle_mod, wl):
    r = oracle_mod.run(wl, backward=False)
    L = (r["h_top"] * wl.dh_top.astype(np.float64)).sum()
    if wl.dc_top is not None:
        L += (r["c_top"] * wl.dc_top.astype(np.float64)).sum()
    return L


@pytest.mark.parametrize("seed", [0, 1])
def test_finite_differences(oracle_mod, seed):
    """Central differences in float64 on every input and parameter of a tiny case with
    push, pop and hold. Steps are 2^-12, exact offsets for float32 inputs of this size."""
    ops = np.array([[1, 1], [1, 0], [-1, 1], [0, 1], [1, -1], [-1, 1], [1, 0]], np.int8)
    T, B = ops.shape
    wl = wk.custom(T=T, B=B, I=3, H=2, seed=seed, ops=ops, wscale=0.6, random_state=True, dc_top=True)
    r = oracle_mod.run(wl)
    eps = 2.0 ** -12
    worst = 0.0
    for name, gname in (("W", "dW"), ("U", "dU"), ("b", "db"), ("x", "dx"), ("h0", "dh0"), ("c0", "dc0")):
        arr = getattr(wl, name)
        g = r[gname].reshape(-1)
        fd = np.zeros(arr.size)
        for k in range(arr.size):
            v = arr.reshape(-1)[k]
            arr.reshape(-1)[k] = v + eps
            lp = _loss(oracle_mod, wl)
            arr.reshape(-1)[k] = v - eps
            lm = _loss(oracle_mod, wl)
            arr.reshape(-1)[k] = v
            fd[k] = (lp - lm) / (2 * eps)
        err = normwise(g, fd)
        worst = max(worst, err)
        assert err < 1e-6, (name, err)
    assert worst < 1e-6


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_autograd_list_stack(oracle_mod, seed):
    """Oracle forward and hand-written backward against torch autograd over a Python
    list stack, with random push/pop/hold streams, random h0/c0 and dc_top."""
    rng = np.random.default_rng(100 + seed)
    T, B, I, H = 23, 4, 5, 6
    ops = wk.ops_random_valid(rng, T, B)
    wl = wk.custom(T=T, B=B, I=I, H=H, seed=seed, ops=ops, wscale=0.4, random_state=True, dc_top=True)
    r = oracle_mod.run(wl)
    ref = list_stack_model(wl)
    for k in ("h_top", "c_top", "dx", "dW", "dU", "db", "dh0", "dc0"):
        assert normwise(r[k], ref[k]) < 1e-12, k


def test_dx_zero_off_push(oracle_mod):
    rng = np.random.default_rng(9)
    ops = wk.ops_random_valid(rng, 40, 5)
    wl = wk.custom(T=40, B=5, I=3, H=4, seed=9, ops=ops)
    r = oracle_mod.run(wl)
    mask = ops != 1
    assert np.all(r["dx"][mask] == 0)
    assert np.all(np.abs(r["dx"][~mask]).sum(-1) > 0)


# ----------------------------------------------------------------------------- Observation 2, Algorithm 1

@pytest.mark.parametrize("name", ["tiny", "parser"])
def test_observation2_branching_equals_algorithm1(oracle_mod, name):
    """Algorithm 1 (compute at every step, write slot p+1, move p) returns exactly the
    states the branching form returns (Observation 2): bit-identical, since the cell
    arithmetic is the same code. Its push-step writes are the branching form's states."""
    wl = wk.make(name)
    sel = np.arange(min(wl.B, 16))
    r = oracle_mod.run(wl, sel=sel, backward=False)
    a = oracle_mod.alg1(wl, sel=sel)
    assert np.array_equal(r["h_top"], a["h_top"]) and np.array_equal(r["c_top"], a["c_top"])
    assert np.array_equal(r["top"], a["top"]) and np.array_equal(r["ptr"], a["ptr"])
    push = wl.ops[:, sel] == 1
    assert np.array_equal(r["h_cell"][push], a["h_cell"][push])
    assert np.all(np.isnan(r["h_cell"][~push]))


# ----------------------------------------------------------------------------- bf16 operands, fp32, subsets

def test_round_bf16_matches_torch(oracle_mod):
    rng = np.random.default_rng(0)
    v = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        # exact ties: low 16 bits = 0x8000 with even and odd kept bits
                        np.array([0x3f808000, 0x3f818000, 0xbf808000, 0x00008000, 0x7f7f8000],
                                 np.uint32).view(np.float32),
                        np.array([0.0, -0.0, 1e-40, 3.0e38], np.float32)])
    ours = oracle_mod.round_bf16(v)
    ref = torch.tensor(v).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))


def test_bf16_operand_mode(oracle_mod):
    rng = np.random.default_rng(7)
    T, B, I, H = 17, 3, 6, 5
    ops = wk.ops_random_valid(rng, T, B)
    wl = wk.custom(T=T, B=B, I=I, H=H, seed=7, ops=ops, wscale=0.5, random_state=True, dc_top=True)
    r = oracle_mod.run(wl, bf16=True)
    ref = list_stack_model(wl, bf16=True)
    for k in ("h_top", "c_top", "dx", "dW", "dU", "db", "dh0", "dc0"):
        assert normwise(r[k], ref[k]) < 1e-12, k
    plain = oracle_mod.run(wl)
    assert normwise(r["h_top"], plain["h_top"]) > 1e-5                   # the rounding does act


def test_f32_instantiation_close(oracle_mod):
    wl = wk.make("tiny")
    a = oracle_mod.run(wl)
    b = oracle_mod.run(wl, mode="f32")
    for k in ("h_top", "c_top", "dx", "dW", "dU", "db", "dh0", "dc0"):
        assert normwise(b[k], a[k]) < 1e-5, k
    assert np.array_equal(a["top"], b["top"])


def test_subset_and_additivity(oracle_mod):
    """Batch elements are independent: a subset run equals the matching columns of the
    full run, and the weight gradients add over disjoint subsets."""
    wl = wk.make("tiny")
    full = oracle_mod.run(wl, threads=1)
    s1, s2 = np.array([1, 4, 6]), np.array([0, 2, 3, 5, 7])
    a, b = oracle_mod.run(wl, sel=s1), oracle_mod.run(wl, sel=s2)
    for k in ("h_top", "c_top", "dx"):
        assert np.array_equal(a[k], full[k][:, s1]), k
    assert np.array_equal(a["top"], full["top"][:, s1])
    for k in ("dW", "dU", "db"):
        assert normwise(a[k] + b[k], full[k]) < 1e-13, k
