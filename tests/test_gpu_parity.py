"""GPU parity: the HIP path (through the C-ABI) against the CPU oracle on the same
seeded inputs. Traces must match bit for bit; floats within the normwise tolerance
(1e-5 fp32, 2e-2 bf16-GEMM against the oracle with bf16-rounded operands)."""
import numpy as np
import pytest

from paper_1904_03409_amd import workloads as wk
from tests.gpu_helpers import compare, need_gpu, run_gpu
from tests.torch_ref import normwise

pytestmark = pytest.mark.gpu


def _check(oracle_mod, wl, precision, sel=None, alg1=True):
    need_gpu()
    print(f"[gpu] {wl.name} T={wl.T} B={wl.B} I={wl.I} H={wl.H} prec={precision}", flush=True)
    gpu, _ = run_gpu(wl, precision=precision)
    bf = precision == 1
    ref = oracle_mod.run(wl, sel=sel, bf16=bf)
    a1 = oracle_mod.alg1(wl, sel=sel, bf16=bf) if alg1 else None
    errs = compare(wl, gpu, ref, precision, sel=sel, alg1=a1, check_weights=sel is None)
    print(f"[gpu] errors {errs}", flush=True)
    return gpu


@pytest.mark.parametrize("precision", [0, 1])
@pytest.mark.parametrize("name", ["tiny", "parser"])
def test_named_configs(oracle_mod, name, precision):
    _check(oracle_mod, wk.make(name), precision)


SHAPES = [
    # (T, B, I, H): odd sizes, ragged batch, the paper's H=200 / I=48 cell, the H=I=1 cell
    (37, 5, 7, 13),
    (50, 17, 48, 200),
    (23, 3, 1, 1),
    (64, 33, 64, 64),
    (41, 130, 32, 96),
]


@pytest.mark.parametrize("precision", [0, 1])
@pytest.mark.parametrize("shape", SHAPES)
def test_odd_shapes(oracle_mod, shape, precision):
    T, B, I, H = shape
    wl = wk.custom(T=T, B=B, I=I, H=H, seed=T * 7 + H, wscale=0.3, random_state=True, dc_top=True)
    _check(oracle_mod, wl, precision)


PIPE_SHAPES = [
    # (T, B, I, H, precision): batches that need two or more 16-row tiles per group, with
    # whole 1 KB state rows, so the forward runs the pipelined kernel
    (20, 1000, 24, 256, 0),
    (16, 1000, 20, 252, 0),   # copied row segments reach past H
    (12, 1000, 16, 512, 1),
]


@pytest.mark.parametrize("shape", PIPE_SHAPES)
def test_pipelined_forward(oracle_mod, shape):
    T, B, I, H, precision = shape
    from paper_1904_03409_amd.stacklstm import make_dims, stacklstm_plan
    need_gpu()
    plan = stacklstm_plan(make_dims(T, B, I, H, precision, 0))
    assert plan["rows_per_group"] >= 32, plan
    wl = wk.custom(T=T, B=B, I=I, H=H, seed=B + H, wscale=0.3, random_state=True, dc_top=True)
    _check(oracle_mod, wl, precision)


def test_arc_hybrid_two_stacks(oracle_mod):
    """The arc-hybrid parser's stack and buffer StackLSTMs of 12 sentences as one doubled
    batch with shared weights (one launch per direction)."""
    rng = np.random.default_rng(11)
    E = 12
    pairs = [wk.ops_arc_hybrid_streams(rng, int(rng.integers(3, 18))) for _ in range(E)]
    T = max(len(s) for s, _ in pairs)
    ops = np.zeros((T, 2 * E), np.int8)
    for j, (st, bu) in enumerate(pairs):
        ops[: len(st), j] = st
        ops[: len(bu), E + j] = bu
    for precision in (0, 1):
        wl = wk.custom(T=T, B=2 * E, I=24, H=48, seed=12, ops=ops, wscale=0.3, random_state=True, dc_top=True)
        _check(oracle_mod, wl, precision)


def _streams(kind, T, B, rng):
    if kind == "all_push":
        return np.ones((T, B), np.int8)
    if kind == "all_hold":
        return np.zeros((T, B), np.int8)
    if kind == "hold_then_push":
        o = np.zeros((T, B), np.int8)
        o[T // 2:] = 1
        return o
    if kind == "alternate":
        o = np.zeros((T, B), np.int8)
        o[0::2] = 1
        o[1::2] = -1
        return o
    if kind == "deep":
        return np.stack([wk.ops_deep_stream(rng, T, (20, 40), (10, 30)) for _ in range(B)], axis=1)
    raise ValueError(kind)


@pytest.mark.parametrize("precision", [0, 1])
@pytest.mark.parametrize("kind", ["all_push", "all_hold", "hold_then_push", "alternate", "deep"])
def test_edge_streams(oracle_mod, kind, precision):
    rng = np.random.default_rng(5)
    T, B = 96, 20
    wl = wk.custom(T=T, B=B, I=24, H=40, seed=3, ops=_streams(kind, T, B, rng), wscale=0.3, random_state=True)
    gpu = _check(oracle_mod, wl, precision)
    if kind == "all_hold":
        assert np.all(gpu["dW"] == 0) and np.all(gpu["dU"] == 0) and np.all(gpu["db"] == 0)


@pytest.mark.parametrize("precision", [0, 1])
def test_deterministic(precision):
    need_gpu()
    wl = wk.make("parser")
    a, _ = run_gpu(wl, precision=precision)
    b, _ = run_gpu(wl, precision=precision)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def _columns(wl, sel):
    """The workload restricted to batch elements sel (every per-element array sliced)."""
    import dataclasses
    sel = np.asarray(sel)
    return dataclasses.replace(
        wl, name=f"{wl.name}[{sel[0]}:{sel[-1] + 1}]", B=len(sel), ops=np.ascontiguousarray(wl.ops[:, sel]),
        x=np.ascontiguousarray(wl.x[:, sel]), h0=np.ascontiguousarray(wl.h0[sel]), c0=np.ascontiguousarray(wl.c0[sel]),
        dh_top=np.ascontiguousarray(wl.dh_top[:, sel]),
        dc_top=None if wl.dc_top is None else np.ascontiguousarray(wl.dc_top[:, sel]))


@pytest.mark.parametrize("precision", [0, 1])
def test_partition_invariance(precision):
    """Batch elements are independent: the same elements run in one batch of 8 groups of 16
    and in batches of 1 and 3 groups (same kernel variants) give bit-identical states, traces
    and initial-state gradients; dx, whose split-K slicing follows the number of push rows in
    the batch, agrees to rounding."""
    need_gpu()
    from paper_1904_03409_amd.stacklstm import stacklstm_plan, make_dims
    wl = wk.custom(T=40, B=128, I=256, H=512, seed=7)
    full, _ = run_gpu(wl, precision=precision)
    for lo, hi in ((0, 16), (48, 96)):
        part = _columns(wl, np.arange(lo, hi))
        pf = stacklstm_plan(make_dims(wl.T, wl.B, wl.I, wl.H, precision, 0))
        pp = stacklstm_plan(make_dims(part.T, part.B, part.I, part.H, precision, 0))
        keys = ("fwd_kernel", "fwd_tiles", "k_chunks", "occupancy", "bwd_tiles", "bwd_direct", "fused_x", "bwd_split")
        assert all(pf[k] == pp[k] for k in keys), (pf, pp)
        print(f"[gpu] partition {lo}:{hi} groups {pp['groups']} of {pf['groups']}", flush=True)
        got, _ = run_gpu(part, precision=precision)
        for k in ("h_cell", "c_cell", "h_top", "c_top", "ptr", "top", "dh0", "dc0"):
            ref = full[k][lo:hi] if k in ("dh0", "dc0") else full[k][:, lo:hi]
            assert np.array_equal(got[k], ref), k
        # dx sums 4H = 2048 products per element, cut into K slices whose number follows the
        # batch's push-row count: two orders of one fp32 sum, held to the fp32 parity bar
        # (measured 1.3e-6 normwise)
        assert normwise(got["dx"], full["dx"][:, lo:hi]) <= 1e-5
        assert np.array_equal(got["dx"] == 0, full["dx"][:, lo:hi] == 0)


WIDE_SHAPES = [
    # (T, B, I, H): bf16 with H > 512 runs the wide forward (32 units per workgroup, groups of
    # 128 rows); units past H (544, 776) and rows past B are masked
    (20, 40, 24, 544),
    (14, 150, 16, 1024),
    (9, 8, 8, 776),
]


@pytest.mark.parametrize("shape", WIDE_SHAPES)
def test_wide_forward(oracle_mod, shape):
    T, B, I, H = shape
    from paper_1904_03409_amd.stacklstm import make_dims, stacklstm_plan
    need_gpu()
    plan = stacklstm_plan(make_dims(T, B, I, H, 1, 0))
    assert plan["rows_per_group"] == 128 and plan["wg_per_group"] == (H + 31) // 32, plan
    wl = wk.custom(T=T, B=B, I=I, H=H, seed=B + H, wscale=0.3, random_state=True, dc_top=True)
    _check(oracle_mod, wl, 1)


@pytest.mark.parametrize("kind", ["all_push", "all_hold", "alternate", "deep"])
def test_wide_forward_streams(oracle_mod, kind):
    rng = np.random.default_rng(9)
    T, B = 48, 24
    wl = wk.custom(T=T, B=B, I=16, H=640, seed=4, ops=_streams(kind, T, B, rng), wscale=0.2, random_state=True)
    _check(oracle_mod, wl, 1)


@pytest.mark.gpu
@pytest.mark.parametrize("threaded", [False, True])
def test_concurrent_calls_on_two_streams(threaded):
    """Two independent problems run fwd + bwd on two HIP streams at once (interleaved from one
    host thread, or from two host threads): the library keeps no state between calls beyond
    the work space, so every output is bit-identical to the same problem run alone."""
    need_gpu()
    import threading
    import torch
    from paper_1904_03409_amd.stacklstm import DeviceRun
    wls = [wk.make("large"), wk.make("large", seed=7)]
    alone = []
    for wl in wls:
        r = DeviceRun.from_workload(wl, precision=0, want_top=True)
        r.forward()
        r.backward()
        torch.cuda.synchronize()
        alone.append(r.results())
    runs = [DeviceRun.from_workload(wl, precision=0, want_top=True) for wl in wls]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    if threaded:
        def work(i):
            with torch.cuda.stream(streams[i]):
                for _ in range(2):
                    runs[i].forward(stream=streams[i])
                    runs[i].backward(stream=streams[i])
        th = [threading.Thread(target=work, args=(i,)) for i in range(2)]
        for x in th:
            x.start()
        for x in th:
            x.join()
    else:
        for _ in range(2):
            for i in range(2):
                with torch.cuda.stream(streams[i]):
                    runs[i].forward(stream=streams[i])
            for i in range(2):
                with torch.cuda.stream(streams[i]):
                    runs[i].backward(stream=streams[i])
    torch.cuda.synchronize()
    for i in range(2):
        got = runs[i].results()
        for k, v in alone[i].items():
            assert np.array_equal(got[k], v), (i, k)


@pytest.mark.gpu
def test_many_streams():
    """Calls on 40 different streams, one after the other on one work space: every call gives
    the same outputs as the first, bit for bit (no per-stream state in the library)."""
    need_gpu()
    import torch
    from paper_1904_03409_amd.stacklstm import DeviceRun
    wl = wk.make("parser")
    r = DeviceRun.from_workload(wl, precision=0, want_top=True)
    r.forward()
    r.backward()
    torch.cuda.synchronize()
    ref = r.results()
    streams = [torch.cuda.Stream() for _ in range(40)]
    for i, s in enumerate(streams):
        with torch.cuda.stream(s):
            r.forward(stream=s)
            r.backward(stream=s)
        s.synchronize()
        got = r.results()
        for k, v in ref.items():
            assert np.array_equal(got[k], v), (i, k)
