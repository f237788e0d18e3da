"""The allocation-free forward (stacklstm_fwd_static: static per-GPU work space) against the
forward on a caller work space (stacklstm_fwd): two calls in a row, the second on a smaller
problem, in both precisions. The outputs must be identical bit for bit (same kernels, same
arithmetic), which is within the parity bar of the forward itself; dims whose forward work
space exceeds the static array are rejected with SLSTM_EWORKSPACE."""
import numpy as np
import pytest
import torch

from paper_1904_03409_amd import workloads as wk
from tests.gpu_helpers import need_gpu

pytestmark = pytest.mark.gpu

OUTS = ("h_cell", "c_cell", "h_top", "c_top", "ptr", "top")


def _static_forward(run):
    from paper_1904_03409_amd.stacklstm import stacklstm_fwd_static
    out = {k: torch.full_like(getattr(run, k), -7 if k in ("ptr", "top") else float("nan")) for k in OUTS}
    rc = stacklstm_fwd_static(run.dims, run.x, run.ops, run.W, run.U, run.b, run.h0, run.c0, out["h_cell"],
                              out["c_cell"], out["h_top"], out["c_top"], out["ptr"], out["top"], check=False)
    torch.cuda.synchronize()
    return rc, {k: v.cpu().numpy() for k, v in out.items()}


@pytest.mark.parametrize("precision", [0, 1])
def test_static_forward_matches_forward(precision):
    need_gpu()
    from paper_1904_03409_amd.stacklstm import DeviceRun
    for wl in (wk.make("parser", precision=precision), wk.make("tiny", precision=precision)):
        print(f"[gpu] static forward {wl.name} T={wl.T} B={wl.B} I={wl.I} H={wl.H} prec={precision}", flush=True)
        run = DeviceRun.from_workload(wl, precision=precision, want_top=True)
        run.forward()
        torch.cuda.synchronize()
        ref = {k: getattr(run, k).cpu().numpy() for k in OUTS}
        rc, got = _static_forward(run)
        assert rc == 0
        for k in OUTS:
            assert np.array_equal(got[k], ref[k], equal_nan=True), (wl.name, k)


def test_static_forward_rejects_large_dims():
    need_gpu()
    from paper_1904_03409_amd import stacklstm as s
    # the large workload's forward work space (about 0.5 GB) exceeds the static array
    wl = wk.make("large")
    run = s.DeviceRun.from_workload(wl, want_top=True)
    rc, _ = _static_forward(run)
    assert rc == 4
