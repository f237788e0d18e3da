"""GPU parity of stacked StackLSTM layers (one op stream, the stack element holds every
layer's state) run as chained single-layer calls on the device, against the multi-layer
oracle (oracle/multilayer.py, pinned to torch.nn.LSTM and the C oracle on the CPU)."""
import numpy as np
import pytest

from paper_1904_03409_amd import workloads as wk
from tests.gpu_helpers import need_gpu
from tests.torch_ref import normwise

pytestmark = pytest.mark.gpu

CASES = [
    # (T, B, I, H, layers): the paper's H = 200 (13 workgroups, a partial last one), three layers
    (48, 20, 24, 40, 2),
    (40, 12, 48, 200, 2),
    (36, 9, 16, 32, 3),
]


@pytest.mark.parametrize("case", CASES)
def test_stacked_layers(case):
    need_gpu()
    import torch
    from oracle import multilayer
    from paper_1904_03409_amd.stacklstm import multilayer_runs
    T, B, I, H, L = case
    print(f"[gpu] multilayer T={T} B={B} I={I} H={H} L={L}", flush=True)
    rng = np.random.default_rng(T + B + H)
    ops = wk.ops_random_valid(rng, T, B)
    x = rng.standard_normal((T, B, I)).astype(np.float32)
    layers = []
    for l in range(L):
        Il = I if l == 0 else H
        layers.append(tuple(rng.uniform(-0.3, 0.3, sh).astype(np.float32) for sh in ((Il, 4 * H), (H, 4 * H), (4 * H,))))
    h0 = [(rng.standard_normal((B, H)) * 0.5).astype(np.float32) for _ in range(L)]
    c0 = [(rng.standard_normal((B, H)) * 0.5).astype(np.float32) for _ in range(L)]
    R = rng.standard_normal((T, B, H)).astype(np.float32)
    Rc = rng.standard_normal((T, B, H)).astype(np.float32)
    runs = multilayer_runs(ops, x, layers, h0, c0, R, Rc)
    for r in runs:
        r.forward()
    for r in reversed(runs):
        r.backward()
    torch.cuda.synchronize()
    ref = multilayer.run(ops, x.astype(np.float64), layers, h0, c0, R, Rc)
    tol = 1e-5
    errs = {}
    for l, r in enumerate(runs):
        assert np.array_equal(r.top.cpu().numpy(), ref["top"]), f"layer {l} top trace differs"
        errs[f"h_top{l}"] = normwise(r.h_top.cpu().numpy(), ref["h_top"][l])
        errs[f"c_top{l}"] = normwise(r.c_top.cpu().numpy(), ref["c_top"][l])
        for k in ("dW", "dU", "db", "dh0", "dc0"):
            errs[f"{k}{l}"] = normwise(getattr(r, k).cpu().numpy(), ref[k][l])
    errs["dx"] = normwise(runs[0].dx.cpu().numpy(), ref["dx"])
    print(f"[gpu] errors {errs}", flush=True)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad
