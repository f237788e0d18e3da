"""Shared helpers of the GPU parity tests: run the HIP path through the C-ABI binding,
run the CPU oracle on the same arrays, compare to the stated tolerances."""
import numpy as np
import pytest

from tests.torch_ref import normwise

TOL = {0: 1e-5, 1: 2e-2}      # normwise max|gpu - ref| / max|ref|: fp32, bf16-GEMM


def need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def run_gpu(wl, precision=None, want_top=True, spin_limit=0):
    import torch
    from paper_1904_03409_amd.stacklstm import DeviceRun
    r = DeviceRun.from_workload(wl, precision=precision, want_top=want_top, spin_limit=spin_limit)
    r.forward()
    r.backward()
    torch.cuda.synchronize()
    return r.results(), r


def compare(wl, gpu, ref, precision, sel=None, alg1=None, check_weights=True, tol=None):
    """Element-by-element comparison of the GPU outputs with the oracle's (columns sel)."""
    tol = TOL[precision] if tol is None else tol
    sel = np.arange(wl.B) if sel is None else np.asarray(sel)
    errs = {}
    assert np.array_equal(gpu["ptr"][:, sel], ref["ptr"]), "ptr trace differs"
    assert np.array_equal(gpu["top"][:, sel], ref["top"]), "top trace differs"
    for k in ("h_top", "c_top", "dx", "dh0", "dc0"):
        g = gpu[k][:, sel] if k in ("h_top", "c_top", "dx") else gpu[k][sel]
        errs[k] = normwise(g, ref[k])
    push = wl.ops[:, sel] == 1
    errs["h_cell_push"] = normwise(gpu["h_cell"][:, sel][push], ref["h_cell"][push])
    errs["c_cell_push"] = normwise(gpu["c_cell"][:, sel][push], ref["c_cell"][push])
    if alg1 is not None:
        errs["h_cell_all"] = normwise(gpu["h_cell"][:, sel], alg1["h_cell"])
        errs["c_cell_all"] = normwise(gpu["c_cell"][:, sel], alg1["c_cell"])
    if check_weights:
        for k in ("dW", "dU", "db"):
            errs[k] = normwise(gpu[k], ref[k])
    # dx is exactly zero where the op is not push
    assert np.all(gpu["dx"][:, sel][~push] == 0), "dx not exactly 0 on a non-push step"
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    assert not bad, f"tolerance {tol} exceeded: {bad} (all: {errs})"
    return errs
