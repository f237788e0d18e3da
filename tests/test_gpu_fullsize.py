"""GPU parity at the full workload sizes, in the launch configuration bench.py times.

The whole batch runs on the GPU; the oracle recomputes a few sampled batch columns
(elements are independent, so every per-element output of those columns is exact
ground truth). Weight gradients sum over all columns, so a second GPU run of the
same launch uses an upstream gradient that is zero outside the sampled columns: its
dW/dU/db must then equal the oracle's sums over those columns alone."""
import numpy as np
import pytest

from paper_1904_03409_amd import workloads as wk
from tests.gpu_helpers import TOL, need_gpu
from tests.torch_ref import normwise

pytestmark = pytest.mark.gpu


def _full(oracle_mod, name, precision, ncols, wl=None):
    need_gpu()
    import torch
    from paper_1904_03409_amd.stacklstm import DeviceRun
    if wl is None:
        wl = wk.make(name, precision=precision)
    print(f"[gpu] full-size {name} T={wl.T} B={wl.B} I={wl.I} H={wl.H} prec={precision}", flush=True)
    sel = np.unique(np.linspace(0, wl.B - 1, ncols).astype(np.int32))
    run = DeviceRun.from_workload(wl, precision=precision)
    run.forward()
    run.backward()
    torch.cuda.synchronize()
    got = run.results()
    bf = precision == 1
    ref = oracle_mod.run(wl, sel=sel, bf16=bf)
    tol = TOL[precision]
    # traces of every column against the prefix sum and the oracle's columns
    ptr = np.vstack([np.zeros((1, wl.B), np.int64), np.cumsum(wl.ops.astype(np.int64), axis=0)])
    assert np.array_equal(got["ptr"], ptr)
    assert np.array_equal(got["top"][:, sel], ref["top"])
    errs = {}
    for k in ("h_top", "c_top", "dx"):
        errs[k] = normwise(got[k][:, sel], ref[k])
    for k in ("dh0", "dc0"):
        errs[k] = normwise(got[k][sel], ref[k])
    push = wl.ops[:, sel] == 1
    errs["h_cell_push"] = normwise(got["h_cell"][:, sel][push], ref["h_cell"][push])
    assert np.all(got["dx"][:, sel][~push] == 0)
    # weight gradients: upstream gradient masked to the sampled columns, same launch
    mask = np.zeros(wl.B, np.float32)
    mask[sel] = 1.0
    run.dh_top.copy_(torch.from_numpy(wl.dh_top * mask[None, :, None]).to(run.dh_top.device))
    if wl.dc_top is not None:
        run.dc_top.copy_(torch.from_numpy(wl.dc_top * mask[None, :, None]).to(run.dc_top.device))
    run.backward()
    torch.cuda.synchronize()
    gw = run.results()
    for k in ("dW", "dU", "db"):
        errs[k] = normwise(gw[k], ref[k])
    print(f"[gpu] {name} prec={precision} errors {errs}", flush=True)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"tolerance {tol} exceeded: {bad}"


@pytest.mark.parametrize("precision", [0, 1])
def test_large(oracle_mod, precision):
    _full(oracle_mod, "large", precision, 4)


def test_deep(oracle_mod):
    _full(oracle_mod, "deep", 0, 3)


def test_thru(oracle_mod):
    _full(oracle_mod, "thru", 1, 2)


def test_hybrid(oracle_mod):
    # 128 sentences: rows 0..127 stack StackLSTMs, 128..255 buffer StackLSTMs (sampled: two of each)
    _full(oracle_mod, "hybrid", 0, 4)


def test_plain_bf16_32_chunks_long(oracle_mod):
    # the plain bf16 forward with 32 K chunks at two workgroups per CU (it polls, and its
    # build spills): H = 1020 keeps the wide forward out (rows not a whole number of 16-byte
    # vectors); 200 steps of random valid ops, three groups of 16*NT rows. Weights of the
    # workloads' scale (0.08): at 0.3 and this width the recurrence amplifies rounding so much
    # that the oracle itself, accumulating in fp32 instead of fp64 over the same bf16 operands,
    # ends 0.36 (normwise) away from its fp64 result at step 200 (0.0007 at 0.08).
    from paper_1904_03409_amd.stacklstm import stacklstm_plan, make_dims
    wl = wk.custom(T=200, B=129, I=64, H=1020, seed=4242, wscale=0.08, random_state=True, dc_top=True, precision=1)
    plan = stacklstm_plan(make_dims(wl.T, wl.B, wl.I, wl.H, 1, 0))
    assert plan["fwd_kernel"] == 0 and plan["k_chunk_cap"] == 32 and plan["occupancy"] == 2, plan
    _full(oracle_mod, "custom H=1020", 1, 3, wl=wl)
