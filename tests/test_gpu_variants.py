"""Every kernel variant the planner can choose runs against the oracle.

The planner picks, per call, a forward kernel (plain, pipelined or wide), the row tiles per
group of the forward and the backward, the K-chunk capacity compiled into the kernels, the
occupancy they are built for and whether the backward stages dA rows by DMA. Those choices
depend on H (K chunks), B (co-residency of the groups' workgroups) and the precision. The
test sweeps a grid of (precision, H, B) that crosses every K-chunk bucket, the pipelined and
wide conditions and every row-tile threshold, collects the distinct variants the planner
returns, and runs each once (short T) against the oracle: traces of every column, floats of
sampled columns, and the weight gradients of a second backward whose upstream gradient is
zero outside the sampled columns."""
import numpy as np
import pytest

from paper_1904_03409_amd import workloads as wk
from tests.gpu_helpers import TOL, need_gpu
from tests.torch_ref import normwise

pytestmark = pytest.mark.gpu

GRID_H = {0: [1, 40, 64, 100, 128, 200, 252, 256, 300, 508, 512],
          1: [1, 64, 100, 128, 200, 256, 300, 504, 512, 520, 1020, 1024]}
GRID_B = [1, 17, 64, 100, 128, 129, 200, 256, 257, 300, 384, 400, 512, 513, 600, 700, 768, 769, 900, 1000, 1024]
KEYS = ("fwd_kernel", "fwd_tiles", "k_chunk_cap", "occupancy", "bwd_tiles", "bwd_direct", "fused_x", "bwd_split")


def reachable_variants():
    """{variant: (precision, H, B) of the first grid point that reaches it}."""
    from paper_1904_03409_amd.stacklstm import StackLSTMError, make_dims, stacklstm_plan
    out = {}
    for prec, hs in GRID_H.items():
        for H in hs:
            for B in GRID_B:
                try:
                    plan = stacklstm_plan(make_dims(8, B, 8, H, prec, 0))
                except StackLSTMError:
                    continue
                key = (prec,) + tuple(plan[k] for k in KEYS) + row_class(prec, H, plan)
                out.setdefault(key, (prec, H, B))
    return out


def row_class(prec, H, plan):
    """How the kernels copy state rows for this H: every K chunk in use, rows of whole 1 KB
    segments, rows of whole 128-byte lines (no line shared by two rows)."""
    nbytes = H * (2 if prec else 4)
    return (int(plan["k_chunks"] == plan["k_chunk_cap"]), int(nbytes % 1024 == 0), int(nbytes % 128 == 0))


# shapes run whatever variant they map to: the largest batches at the largest hidden sizes
EXTRA = [(0, 512, 1024), (1, 512, 1024), (1, 1020, 1024), (1, 1024, 1024)]


def _sampled_parity(oracle_mod, wl, precision, ncols=3):
    import torch
    from paper_1904_03409_amd.stacklstm import DeviceRun
    sel = np.unique(np.linspace(0, wl.B - 1, ncols).astype(np.int32))
    run = DeviceRun.from_workload(wl, precision=precision)
    run.forward()
    run.backward()
    torch.cuda.synchronize()
    got = run.results()
    ref = oracle_mod.run(wl, sel=sel, bf16=precision == 1)
    ptr = np.vstack([np.zeros((1, wl.B), np.int64), np.cumsum(wl.ops.astype(np.int64), axis=0)])
    assert np.array_equal(got["ptr"], ptr)
    assert np.array_equal(got["top"][:, sel], ref["top"])
    errs = {k: normwise(got[k][:, sel], ref[k]) for k in ("h_top", "c_top", "dx")}
    errs.update({k: normwise(got[k][sel], ref[k]) for k in ("dh0", "dc0")})
    push = wl.ops[:, sel] == 1
    errs["h_cell_push"] = normwise(got["h_cell"][:, sel][push], ref["h_cell"][push])
    assert np.all(got["dx"][:, sel][~push] == 0)
    mask = np.zeros(wl.B, np.float32)
    mask[sel] = 1.0
    run.dh_top.copy_(torch.from_numpy(wl.dh_top * mask[None, :, None]).to(run.dh_top.device))
    run.dc_top.copy_(torch.from_numpy(wl.dc_top * mask[None, :, None]).to(run.dc_top.device))
    run.backward()
    torch.cuda.synchronize()
    gw = run.results()
    errs.update({k: normwise(gw[k], ref[k]) for k in ("dW", "dU", "db")})
    return errs


def test_every_planner_variant(oracle_mod):
    need_gpu()
    variants = reachable_variants()
    print(f"[gpu] {len(variants)} variants: precision, fwd kernel, fwd tiles, K-chunk cap, occupancy, "
          f"bwd tiles, bwd direct, fused x W, all chunks used, 1 KB rows, 128-byte rows -> first (precision, H, B)", flush=True)
    failures = {}
    cases = sorted(variants.items()) + [(("extra",), s) for s in EXTRA]
    for key, (prec, H, B) in cases:
        T = 10
        wl = wk.custom(T=T, B=B, I=24, H=H, seed=1000 + H + B, wscale=0.3, random_state=True, dc_top=True)
        print(f"[gpu] variant {key} at H={H} B={B} T={T}", flush=True)
        errs = _sampled_parity(oracle_mod, wl, prec)
        bad = {k: v for k, v in errs.items() if not v <= TOL[prec]}
        print(f"[gpu]   max err {max(errs.values()):.2e}" + (f" FAILED {bad}" if bad else ""), flush=True)
        if bad:
            failures[key] = bad
    assert not failures, failures
