"""Pins of the multi-layer StackLSTM oracle (oracle/multilayer.py) against things other
than itself: torch.nn.LSTM with two layers on all-push streams, and the C oracle at one
layer."""
import numpy as np
import pytest
import torch

from oracle import multilayer


def _layers(rng, I, H, L, scale=0.3):
    out = []
    for l in range(L):
        Il = I if l == 0 else H
        out.append((rng.uniform(-scale, scale, (Il, 4 * H)), rng.uniform(-scale, scale, (H, 4 * H)),
                    rng.uniform(-scale, scale, 4 * H)))
    return out


def test_all_push_two_layers_equals_torch_lstm():
    """With every op a push the stack is a plain 2-layer LSTM over time: values and every
    gradient match torch.nn.LSTM(num_layers=2) in float64 (weight_ih = W^T, weight_hh =
    U^T, bias_ih = b, bias_hh = 0, gate order i, f, g, o)."""
    rng = np.random.default_rng(0)
    T, B, I, H = 7, 3, 5, 4
    layers = _layers(rng, I, H, 2)
    x = rng.standard_normal((T, B, I))
    h0 = [rng.standard_normal((B, H)) * 0.5 for _ in range(2)]
    c0 = [rng.standard_normal((B, H)) * 0.5 for _ in range(2)]
    R = rng.standard_normal((T, B, H))
    got = multilayer.run(np.ones((T, B), np.int8), x, layers, h0, c0, R)

    lstm = torch.nn.LSTM(I, H, num_layers=2).double()
    with torch.no_grad():
        for l, (W, U, b) in enumerate(layers):
            getattr(lstm, f"weight_ih_l{l}").copy_(torch.tensor(W.T))
            getattr(lstm, f"weight_hh_l{l}").copy_(torch.tensor(U.T))
            getattr(lstm, f"bias_ih_l{l}").copy_(torch.tensor(b))
            getattr(lstm, f"bias_hh_l{l}").zero_()
    xt = torch.tensor(x, requires_grad=True)
    h0t = torch.tensor(np.stack(h0), requires_grad=True)
    c0t = torch.tensor(np.stack(c0), requires_grad=True)
    out, _ = lstm(xt, (h0t, c0t))
    (out * torch.tensor(R)).sum().backward()
    np.testing.assert_allclose(got["h_top"][1], out.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(got["dx"], xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    for l in range(2):
        np.testing.assert_allclose(got["dW"][l], getattr(lstm, f"weight_ih_l{l}").grad.numpy().T, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(got["dU"][l], getattr(lstm, f"weight_hh_l{l}").grad.numpy().T, rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(got["db"][l], getattr(lstm, f"bias_ih_l{l}").grad.numpy(), rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(got["dh0"][l], h0t.grad.numpy()[l], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(got["dc0"][l], c0t.grad.numpy()[l], rtol=1e-10, atol=1e-12)


def test_one_layer_equals_the_c_oracle(oracle_mod):
    """At one layer the multi-layer oracle is the single-layer StackLSTM: the C oracle's
    values, producer trace and gradients on a random push/pop/hold stream."""
    from paper_1904_03409_amd import workloads as wk
    wl = wk.custom(T=40, B=4, I=6, H=5, seed=9, wscale=0.4, random_state=True, dc_top=True)
    ref = oracle_mod.run(wl)
    got = multilayer.run(wl.ops, wl.x.astype(np.float64), [(wl.W, wl.U, wl.b)], [wl.h0], [wl.c0], wl.dh_top, wl.dc_top)
    assert np.array_equal(got["top"], ref["top"])
    np.testing.assert_allclose(got["h_top"][0], ref["h_top"], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(got["c_top"][0], ref["c_top"], rtol=1e-11, atol=1e-12)
    for k in ("dx",):
        np.testing.assert_allclose(got[k], ref[k], rtol=1e-10, atol=1e-11)
    for k in ("dW", "dU", "db", "dh0", "dc0"):
        np.testing.assert_allclose(got[k][0], ref[k], rtol=1e-10, atol=1e-11)


def test_layers_see_their_own_stack_positions():
    """Pop and push move every layer's pointer together: after push, push, pop, push the
    top element of each layer was built on the first push's element (its parent), so it
    equals a fresh 2-step all-push run whose second input is the fourth step's."""
    rng = np.random.default_rng(3)
    T, B, I, H = 4, 1, 3, 4
    layers = _layers(rng, I, H, 2)
    x = rng.standard_normal((T, B, I))
    h0 = [np.zeros((B, H)), np.zeros((B, H))]
    c0 = [np.zeros((B, H)), np.zeros((B, H))]
    ops = np.array([[1], [1], [-1], [1]], np.int8)
    got = multilayer.run(ops, x, layers, h0, c0, np.zeros((T, B, H)))
    x2 = x[[0, 3]]
    ref = multilayer.run(np.ones((2, B), np.int8), x2, layers, h0, c0, np.zeros((2, B, H)))
    for l in range(2):
        np.testing.assert_allclose(got["h_top"][l][3], ref["h_top"][l][1], rtol=1e-13)
        np.testing.assert_allclose(got["h_top"][l][2], ref["h_top"][l][0], rtol=1e-13)
    assert got["top"][:, 0].tolist() == [0, 1, 0, 3]
