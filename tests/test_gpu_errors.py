"""Error paths of the C-ABI: every bad input returns its status code, nothing faults."""
import numpy as np
import pytest
import torch

from paper_1904_03409_amd import workloads as wk
from tests.gpu_helpers import need_gpu

pytestmark = pytest.mark.gpu


def _run(wl, **kw):
    from paper_1904_03409_amd.stacklstm import DeviceRun
    r = DeviceRun.from_workload(wl, **kw)
    return r, r.forward(check=False)


def test_bad_op_and_underflow():
    need_gpu()
    ops = np.ones((10, 4), np.int8)
    ops[3, 2] = 5
    r, rc = _run(wk.custom(T=10, B=4, I=3, H=8, seed=0, ops=ops))
    assert rc == 2
    ops = np.ones((10, 4), np.int8)
    ops[0, 1] = -1
    r, rc = _run(wk.custom(T=10, B=4, I=3, H=8, seed=0, ops=ops))
    assert rc == 3
    ops = np.zeros((10, 4), np.int8)
    ops[2, 3] = 1
    ops[3, 3] = -1
    ops[4, 3] = -1                # second pop of element 3 underflows at step 4
    ops[6, 3] = 7                 # a later bad op does not change the code of element 3
    r, rc = _run(wk.custom(T=10, B=4, I=3, H=8, seed=0, ops=ops))
    assert rc == 3


def test_workspace_dims_and_null():
    need_gpu()
    from paper_1904_03409_amd import stacklstm as s
    wl = wk.custom(T=8, B=4, I=3, H=8, seed=0)
    r, rc = _run(wl)
    assert rc == 0
    small = torch.empty(r.workspace.numel() - 256, dtype=torch.uint8, device="cuda")
    rc = s.stacklstm_fwd(r.dims, r.x, r.ops, r.W, r.U, r.b, r.h0, r.c0, r.h_cell, r.c_cell, None, None, r.ptr,
                         r.top, small, check=False)
    assert rc == 4
    bad = s.make_dims(8, 4, 3, 2000)
    assert s.stacklstm_workspace_bytes(bad) == 0
    rc = s.stacklstm_fwd(bad, r.x, r.ops, r.W, r.U, r.b, r.h0, r.c0, r.h_cell, r.c_cell, None, None, r.ptr, r.top,
                         r.workspace, check=False)
    assert rc == 1
    rc = s.stacklstm_fwd(r.dims, None, r.ops, r.W, r.U, r.b, r.h0, r.c0, r.h_cell, r.c_cell, None, None, r.ptr,
                         r.top, r.workspace, check=False)
    assert rc == 1


def test_spin_limit_timeout_reported():
    """A one-poll barrier limit forced from the host: the kernels give up, every
    workgroup leaves its loop, and the call reports SLSTM_ETIMEOUT (also through
    stacklstm_sync_status)."""
    need_gpu()
    from paper_1904_03409_amd import stacklstm as s
    wl = wk.make("parser")
    r, rc = _run(wl, spin_limit=1)
    assert rc == 7
    assert s.stacklstm_sync_status(r.workspace) == 7
    torch.cuda.synchronize()
    # the same buffers run normally afterwards
    r2, rc2 = _run(wl)
    assert rc2 == 0
    assert s.stacklstm_sync_status(r2.workspace) == 0


def test_spin_limit_timeout_reported_polling():
    """The plain bf16 forward exchanges rows by polling fill-marked data: with a one-poll limit
    the first wait that finds a row not yet written gives up (some wait of the deep-stack
    streams always does when the input projection is not fused into the step: its MFMAs
    would sit between the copy and the check), the kernels leave their loops and the call
    reports SLSTM_ETIMEOUT; the same buffers then run normally."""
    need_gpu()
    from paper_1904_03409_amd import stacklstm as s
    deep = wk.make("deep")
    wl = wk.custom(T=deep.T, B=deep.B, I=544, H=deep.H, seed=104, ops=deep.ops, wscale=0.08)
    plan = s.stacklstm_plan(s.make_dims(wl.T, wl.B, wl.I, wl.H, 1, 0))
    assert plan["fwd_kernel"] == 0 and plan["fused_x"] == 0, plan
    r, rc = _run(wl, precision=1, spin_limit=1)
    assert rc == 7
    torch.cuda.synchronize()
    r2, rc2 = _run(wl, precision=1)
    assert rc2 == 0
    assert s.stacklstm_sync_status(r2.workspace) == 0
    r2.backward()
    torch.cuda.synchronize()
    assert s.stacklstm_sync_status(r2.workspace) == 0


def test_empty_T():
    need_gpu()
    wl = wk.custom(T=0, B=3, I=2, H=4, seed=0, ops=np.zeros((0, 3), np.int8))
    from paper_1904_03409_amd.stacklstm import DeviceRun
    r = DeviceRun.from_workload(wl)
    r.forward()
    r.backward()
    torch.cuda.synchronize()
    out = r.results()
    assert np.all(out["ptr"] == 0)
    for k in ("dW", "dU", "db", "dh0", "dc0"):
        assert np.all(out[k] == 0)


@pytest.mark.parametrize("precision", [0, 1])
def test_corrupted_top_reported(precision):
    """A producer table that is not the forward's (indices past their step, below -1) passed
    to stacklstm_bwd: every kernel still finishes (each bad index is replaced by -1 before any
    access), and the call returns SLSTM_EINDEX instead of OK. The same work space then runs a
    normal backward with status OK."""
    need_gpu()
    from paper_1904_03409_amd import stacklstm as s
    wl = wk.make("tiny")
    r, rc = _run(wl, precision=precision)
    assert rc == 0
    torch.cuda.synchronize()
    good = r.top.clone()
    bad = good.clone()
    bad[5:, 1] = 1000                 # past every step
    bad[9, 3] = -7                    # below the initial state's -1
    print(f"[gpu] corrupted top, tiny, precision={precision}", flush=True)
    rc = s.stacklstm_bwd(r.dims, r.x, r.ops, r.W, r.U, r.h0, r.c0, r.h_cell, r.c_cell, bad, r.workspace, r.dh_top,
                         r.dc_top, r.dx, r.dW, r.dU, r.db, r.dh0, r.dc0, check=False)
    assert rc == 8
    assert s.stacklstm_sync_status(r.workspace) == 8
    rc = s.stacklstm_bwd(r.dims, r.x, r.ops, r.W, r.U, r.h0, r.c0, r.h_cell, r.c_cell, good, r.workspace, r.dh_top,
                         r.dc_top, r.dx, r.dW, r.dU, r.db, r.dh0, r.dc0, check=False)
    assert rc == 0
    assert s.stacklstm_sync_status(r.workspace) == 0


def test_deferred_status():
    """Deferred calls return OK without a read-back; they give the same results as ordinary
    calls, keep the first error of any of them for stacklstm_sync_status, and an ordinary call
    resets it."""
    need_gpu()
    from paper_1904_03409_amd.stacklstm import DeviceRun, stacklstm_sync_status
    wl = wk.custom(T=12, B=40, I=8, H=32, seed=3)
    ref = DeviceRun.from_workload(wl)
    assert ref.forward(check=False) == 0 and ref.backward(check=False) == 0
    want = ref.results()
    r = DeviceRun.from_workload(wl)
    assert r.forward(check=False) == 0 and r.backward(check=False) == 0   # resets the error words
    r.dims.defer_status = 1
    for _ in range(2):
        assert r.forward(check=False) == 0 and r.backward(check=False) == 0
    torch.cuda.synchronize()
    assert stacklstm_sync_status(r.workspace) == 0
    got = r.results()
    for k in want:
        assert np.array_equal(want[k], got[k]), k
    # an invalid op in a deferred call, then valid deferred calls: still reported
    bad_ops = wl.ops.copy()
    bad_ops[4, 7] = 5
    rb = DeviceRun.from_workload(wk.custom(T=12, B=40, I=8, H=32, seed=3, ops=bad_ops))
    assert rb.forward(check=False) == 2                                      # ordinary call: its own status
    rb.dims.defer_status = 1
    assert rb.forward(check=False) == 0 and rb.backward(check=False) == 0
    rb.ops.copy_(torch.from_numpy(wl.ops).to(rb.ops.device))
    assert rb.forward(check=False) == 0 and rb.backward(check=False) == 0
    torch.cuda.synchronize()
    assert stacklstm_sync_status(rb.workspace) == 2
    rb.dims.defer_status = 0
    assert rb.forward(check=False) == 0                                      # resets: valid ops now
    assert stacklstm_sync_status(rb.workspace) == 0
