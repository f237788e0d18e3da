"""Benchmark of the parallelised StackLSTM step on one MI355X.

One step = the whole hot path over one batch: stacklstm_fwd (op scan, input
projection, persistent recurrent forward, h_top/c_top gathers) followed by
stacklstm_bwd (persistent recurrent backward, dW/db, dU, dx), with every input
already resident in HBM. The workload is the B=256, H=512 batch (I=256, T=240
arc-standard shaped streams, fp32) unless --config says otherwise; a second run of
the same shape in bf16-GEMM mode is reported alongside.

Prints ONE JSON line: the contract fields, a per-phase breakdown timed with HIP
events on the library's stream, the roofline of the dominant kernel and the CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"f32": 157.3, "bf16": 2500.0}           # dense MFMA TFLOP/s (fp32, bf16)


def hip():
    lib = ctypes.CDLL("libamdhip64.so.7")
    lib.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
    lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
    return lib


def timed_run(wl, precision, steps, warmup, torch):
    from paper_1904_03409_amd.stacklstm import DeviceRun, SLSTM_PHASE_EVENTS
    run = DeviceRun.from_workload(wl, precision=precision, want_top=True)
    for _ in range(warmup):
        run.forward()
        run.backward()
    torch.cuda.synchronize()
    lib = hip()
    evs = []
    for _ in range(steps):
        arr = (ctypes.c_void_p * SLSTM_PHASE_EVENTS)()
        for i in range(SLSTM_PHASE_EVENTS):
            h = ctypes.c_void_p()
            assert lib.hipEventCreate(ctypes.byref(h)) == 0
            arr[i] = h
        evs.append(arr)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    # the timed calls defer their status (no host synchronisation inside a call, as in a training
    # loop): the warm-up calls above reset the work space's error words, the timed ones keep
    # every error they raise, and the caller reads them with stacklstm_sync_status afterwards
    run.dims.defer_status = 1
    t0 = time.perf_counter()
    start.record()
    for k in range(steps):
        run.dims.phase_events = ctypes.cast(evs[k], ctypes.c_void_p)
        run.forward()
        run.backward()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    run.dims.phase_events = None
    run.dims.defer_status = 0
    total_ms = start.elapsed_time(stop)
    phase = {}
    f = ctypes.c_float()
    pairs = [(0, 1, "scan"), (1, 2, "xw_gemm+prep"), (2, 3, "rec_fwd"), (3, 4, "top_gather"),
             (5, 6, "rec_bwd"), (6, 7, "dW+db"), (7, 8, "dU"), (8, 9, "dx"), (4, 5, "bwd_prep")]
    for a, b, name in pairs:
        acc = 0.0
        for k in range(steps):
            lib.hipEventElapsedTime(ctypes.byref(f), evs[k][a], evs[k][b])
            acc += f.value
        phase[name] = acc / steps
    per_step = []
    for k in range(steps):
        lib.hipEventElapsedTime(ctypes.byref(f), evs[k][0], evs[k][9])
        per_step.append(f.value)
    phase["_per_step_ms"] = per_step
    for arr in evs:
        for i in range(SLSTM_PHASE_EVENTS):
            lib.hipEventDestroy(arr[i])
    return run, total_ms, wall, phase


def timed_layers(wl, L, precision, steps, warmup, torch):
    """fwd + bwd of L stacked layers on the workload's op streams (chained single-layer
    calls, every step on the GPU), timed with events per step."""
    from paper_1904_03409_amd.stacklstm import multilayer_runs
    from paper_1904_03409_amd.workloads import layer_params
    layers, h0, c0 = layer_params(wl, L)
    runs = multilayer_runs(wl.ops, wl.x, layers, h0, c0, wl.dh_top, None, precision=precision)

    def step():
        for r in runs:
            r.forward()
        for r in reversed(runs):
            r.backward()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in evs:
        a.record()
        step()
        b.record()
    torch.cuda.synchronize()
    per = [a.elapsed_time(b) for a, b in evs]
    del runs
    return per


def flops(wl):
    """Algorithmic flops per phase: every element-step counts (the homogenised method runs
    the cell at every step), 2*4H*H per recurrent contraction and 2*4H*I or 2*4H*H per
    post-loop product."""
    T, B, I, H = wl.T, wl.B, wl.I, wl.H
    rec = 2.0 * T * B * H * 4 * H                 # one recurrent contraction (h_prev U or dA U^T)
    return {"rec_fwd": rec, "rec_bwd": rec, "xw_gemm+prep": 2.0 * T * B * I * 4 * H, "dW+db": 2.0 * T * B * I * 4 * H,
            "dU": 2.0 * T * B * H * 4 * H, "dx": 2.0 * T * B * I * 4 * H}


def executed_flops(wl):
    """Flops of the matrix products on rows that carry work: the gate gradient dA is exactly
    zero on non-push steps, so the backward contraction dA U^T (run on tiles of push rows)
    and the dW, dU, dx products (over the push rows) skip those rows. Padding of the last
    16-row tile of a step is not counted."""
    T, B, I, H = wl.T, wl.B, wl.I, wl.H
    n_push = float((np.asarray(wl.ops) == 1).sum())
    out = flops(wl)
    out["rec_bwd"] = 2.0 * n_push * H * 4 * H
    for k, width in (("dW+db", I), ("dU", H), ("dx", I)):
        out[k] = 2.0 * n_push * width * 4 * H
    return out


def strip_comments(src: str) -> str:
    """C++ source without its comments and with runs of white space collapsed (string
    literals in the library's sources hold no comment markers)."""
    import re
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def kernel_sources_sha1():
    """Hash of the code (comments and layout left out) of every HIP source and header of the
    library: a stored counter reading is valid only for the kernels it was taken from."""
    import glob
    import hashlib
    h = hashlib.sha1()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_1904_03409_amd", "csrc", "*"))):
        if f.endswith((".hip", ".h")):
            h.update(os.path.basename(f).encode())
            with open(f, encoding="utf-8") as fh:
                h.update(strip_comments(fh.read()).encode())
    return h.hexdigest()


def stored_traffic(config, dname, phase):
    """HBM bytes per launch of a phase's kernel from the committed rocprofv3 counter summary
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known size), or None when the
    summary is missing or was taken from other kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("source_sha1") != kernel_sources_sha1():
        return None
    e = t.get("entries", {}).get(f"{config}/{dname}/{phase}")
    return None if e is None else e.get("hbm_bytes_per_launch")


def stored_step_traffic(config, dname):
    """HBM bytes of one whole fwd+bwd step (every kernel) from the committed counter
    summary, or None (see stored_traffic)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if t.get("source_sha1") != kernel_sources_sha1():
        return None
    e = t.get("entries", {}).get(f"{config}/{dname}/step")
    return None if e is None else e.get("hbm_bytes_per_launch")


def host_cpu():
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, os.cpu_count()


def copy_probe(torch, nbytes=256 << 20, reps=3):
    """A plain copy kernel of known size (one elementwise kernel reading nbytes and writing
    nbytes, b = a * 1): its FETCH_SIZE / WRITE_SIZE readings calibrate the counters of the
    other kernels. (A device-to-device memcpy is not used: the runtime splits it into several
    blit dispatches.)"""
    a = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(reps):
        torch.mul(a, 1.0, out=b)
    torch.cuda.synchronize()
    print(f"[bench] copy probe: {reps} x {nbytes} bytes (elementwise b = a * 1)", file=sys.stderr, flush=True)


def normwise(got, ref):
    ref = np.asarray(ref, np.float64)
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    return float(np.abs(np.asarray(got, np.float64) - ref).max() / (scale if scale > 0 else 1.0)) if ref.size else 0.0


def cpu_baseline(wl, gpu_out=None, target_s=12.0):
    """The oracle (float32 instantiation, OpenMP over batch elements, built with -march=native
    on this host) timed on a bounded sample. Its outputs for the sample are then compared with
    the benched GPU run's outputs of the same columns: traces bit for bit, every per-element
    float normwise (weight gradients sum over the whole batch and are not compared here)."""
    import oracle
    oracle.build(force=True, native=True)
    th = oracle.max_threads()
    n0 = min(wl.B, max(th, 8))
    t0 = time.perf_counter()
    oracle.run(wl, sel=np.arange(n0, dtype=np.int32), mode="f32", threads=th, native=True)
    dt0 = time.perf_counter() - t0
    # sample size for about target_s of CPU work (at most the whole batch), then runs of it
    # until about target_s have been spent (small workloads repeat many times); the median
    # run is reported
    n = n0 if dt0 >= target_s / 4 else int(min(wl.B, max(n0, n0 * target_s / max(dt0, 1e-3))))
    times = []
    ref = None
    while True:
        t0 = time.perf_counter()
        ref = oracle.run(wl, sel=np.arange(n, dtype=np.int32), mode="f32", threads=th, native=True)
        times.append(time.perf_counter() - t0)
        if len(times) >= 10000 or sum(times) + float(np.median(times)) > target_s:
            break
    dt = float(np.median(times))
    pushes = int((wl.ops[:, :n] == 1).sum())
    model, ncpu = host_cpu()
    out = {"value": n * wl.T / dt, "unit": "element-steps/s", "cores": th, "kind": "oracle",
           "push_steps_per_s": pushes / dt, "host_cpus": ncpu, "cpu_model": model,
           "sample": f"fwd+bwd of the first {n} of {wl.B} batch elements (all T={wl.T} steps), float32 oracle "
                     f"(gcc -O3 -march=native -fopenmp on this host, {th} threads), median of {len(times)} runs: "
                     f"{dt:.2f} s"}
    if gpu_out is not None:
        sel = slice(0, n)
        errs = {k: normwise(gpu_out[k][:, sel], ref[k]) for k in ("h_top", "c_top", "dx")}
        errs.update({k: normwise(gpu_out[k][sel], ref[k]) for k in ("dh0", "dc0")})
        push = wl.ops[:, sel] == 1
        errs["h_cell_push"] = normwise(gpu_out["h_cell"][:, sel][push], ref["h_cell"][push])
        out["gpu_check"] = {
            "columns": n, "trace_equal": bool(np.array_equal(gpu_out["ptr"][:, sel], ref["ptr"]) and
                                               np.array_equal(gpu_out["top"][:, sel], ref["top"])),
            "max_normwise_err": max(errs.values()), "tolerance": 1e-5,
            "parity": bool(max(errs.values()) <= 1e-5), "errors": {k: float(f"{v:.3g}") for k, v in errs.items()}}
    return out


def amdahl_fit(batches, speedups):
    """Parallel fraction P of Amdahl's law S(b) = 1 / ((1 - P) + P / b): the least-squares
    fit of 1/S - 1 = P (1/b - 1) over the points with b > 1, and P from each point alone."""
    y = np.array([1.0 / s - 1.0 for b, s in zip(batches, speedups) if b > 1])
    z = np.array([1.0 / b - 1.0 for b in batches if b > 1])
    p_fit = float((y * z).sum() / (z * z).sum()) if len(z) else None
    each = {int(b): float((1.0 - 1.0 / s) / (1.0 - 1.0 / b)) for b, s in zip(batches, speedups) if b > 1}
    return p_fit, each


def sweep(args, torch):
    """Batch-scaling sweep (the analogue of the paper's Figure 1 on synthetic streams):
    element-steps/s of the parser-shaped workload (H=256, I=128) at B = 1, 2, 4, .., 1024
    with T fixed, speed-up S(B) = throughput(B) / throughput(1), and the Amdahl parallel
    fraction fitted to it (the paper reports 99.92% at a batch of 64)."""
    from paper_1904_03409_amd import workloads
    prec = 0 if (args.precision or "fp32") == "fp32" else 1
    pts = []
    for B in [1 << k for k in range(11)]:
        wl = workloads.make("parser", B=B, T=120, precision=prec)
        run, total_ms, _, phase = timed_run(wl, prec, args.steps, args.warmup, torch)
        per = phase.pop("_per_step_ms")
        ms = total_ms / args.steps
        pts.append({"B": B, "T": wl.T, "ms_per_step": ms, "step_ms_median": float(np.median(per)),
                    "element_steps_per_s": B * wl.T / (ms / 1e3), "rec_fwd_ms": phase["rec_fwd"],
                    "rec_bwd_ms": phase["rec_bwd"]})
        print(f"[sweep] B={B} {ms:.3f} ms/step", file=sys.stderr, flush=True)
        del run
        torch.cuda.empty_cache()
    base = pts[0]["element_steps_per_s"]
    for p in pts:
        p["speedup"] = p["element_steps_per_s"] / base
    p_fit, each = amdahl_fit([p["B"] for p in pts], [p["speedup"] for p in pts])
    return {"metric": "batch-scaling sweep: fwd+bwd element-steps/s vs batch size, Amdahl fit",
            "unit": "element-steps/s", "dtype": "f32" if prec == 0 else "bf16", "data": "synthetic",
            "config": {"workload": "parser-shaped arc-standard streams, I=128, H=256, T=120 (hold-padded)",
                       "steps": args.steps, "warmup": args.warmup},
            "points": pts, "amdahl": {"P_fit": p_fit, "P_from_each_B": each, "paper_P_at_64": 0.9992}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="large")
    ap.add_argument("--precision", choices=["fp32", "bf16"], default=None)
    ap.add_argument("--no-bf16", action="store_true", help="skip the bf16-GEMM run of the same shape")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extra", action="store_true", help="skip the deep and thru workloads of the default run")
    ap.add_argument("--layers", type=int, default=1,
                    help="stacked StackLSTM layers sharing the op streams (the stack element holds every layer)")
    ap.add_argument("--sweep", action="store_true",
                    help="batch-scaling sweep B = 1..1024 of the parser shape and its Amdahl fit (one JSON line)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 256 MiB device copy (counter calibration for rocprofv3 --pmc runs)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the StackLSTM step is measured on one MI355X "
              "(the batch would shard across GPUs with one all-reduce of dW, dU, db after the backward; that path is not launched)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1904_03409_amd import workloads
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    if args.sweep:
        print(json.dumps(sweep(args, torch)), flush=True)
        return
    if args.layers > 1:
        wl = workloads.make(args.config)
        prec = wl.precision if args.precision is None else (0 if args.precision == "fp32" else 1)
        per = timed_layers(wl, args.layers, prec, args.steps, args.warmup, torch)
        ms = float(np.mean(per))
        T, B, I, H = wl.T, wl.B, wl.I, wl.H
        fl = 3 * 2.0 * T * B * 4 * H * (I + H) + (args.layers - 1) * 3 * 2.0 * T * B * 4 * H * (2 * H)
        dname = "f32" if prec == 0 else "bf16"
        print(json.dumps({
            "metric": "fwd+bwd batch·timesteps/sec, stacked StackLSTM layers", "value": B * T / (ms / 1e3),
            "unit": "element-steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
            "step_ms_median": float(np.median(per)), "step_ms_min": float(np.min(per)), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": dname, "data": "synthetic",
            "config": {"workload": f"{args.config}: {args.layers} stacked layers, B={B} T={T} I={I} H={H}",
                       "layers": args.layers, "global_batch": B, "seq_len": T, "parallelism": "none (1 GPU)"},
            "overall_mfma_frac": fl / (ms / 1e3) / 1e12 / PEAK[dname]}), flush=True)
        return
    wl = workloads.make(args.config)
    prec = wl.precision if args.precision is None else (0 if args.precision == "fp32" else 1)
    dname = "f32" if prec == 0 else "bf16"
    m = measure(wl, prec, args.steps, args.warmup, torch, args.config, keep_outputs=not args.no_cpu)
    ms = m["ms_per_step"]
    fl = flops(wl)
    phase = m["phases_ms"]
    kern = max(fl, key=lambda k: phase.get(k, 0.0))
    achieved = fl[kern] / (phase[kern] / 1e3) / 1e12
    out = {
        "metric": "fwd+bwd batch·timesteps/sec at B=256,H=512; % MFMA peak",
        "value": m["value"], "unit": "element-steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dname,
        "data": "synthetic",
        "config": {"workload": f"{args.config}: StackLSTM fwd+bwd, B={wl.B} T={wl.T} I={wl.I} H={wl.H}, "
                               f"arc-standard op streams, {dname} GEMM operands",
                   "global_batch": wl.B, "seq_len": wl.T, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "mfma", "kernel": kern, "achieved": achieved, "peak": PEAK[dname], "unit": "TFLOP/s",
                     "frac": achieved / PEAK[dname], "traffic": stored_traffic(args.config, dname, kern)},
    }
    out.update({k: v for k, v in m.items() if k not in ("value", "ms_per_step", "out")})
    gpu_out = m.get("out")
    torch.cuda.empty_cache()
    extra = []
    if not args.no_bf16 and prec == 0 and wl.H <= 1024:
        extra.append(("bf16_gemm", wl, 1, args.config))
    if args.config == "large" and not args.no_extra:
        # the other full-size workloads: deep-stack stress (fp32) and throughput (bf16-GEMM)
        extra.append(("deep", workloads.make("deep"), 0, "deep"))
        extra.append(("thru", workloads.make("thru"), 1, "thru"))
    for key, wlx, px, cname in extra:
        mx = measure(wlx, px, args.steps, args.warmup, torch, cname)
        mx.pop("out", None)
        mx["config"] = f"{cname}: B={wlx.B} T={wlx.T} I={wlx.I} H={wlx.H}, {'f32' if px == 0 else 'bf16'} GEMM operands"
        out[key] = mx
        torch.cuda.empty_cache()
    if args.copy_probe:
        copy_probe(torch)
    if not args.no_cpu:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, gpu_out=gpu_out)
    print(json.dumps(out), flush=True)


def measure(wl, prec, steps, warmup, torch, cname, keep_outputs=False):
    """Times `steps` fwd+bwd steps of one workload and checks the run: the status of the last
    calls (stacklstm_sync_status) and the pointer trace of every column against the prefix
    sum of the ops."""
    from paper_1904_03409_amd.stacklstm import stacklstm_sync_status
    dname = "f32" if prec == 0 else "bf16"
    print(f"[bench] {cname} T={wl.T} B={wl.B} I={wl.I} H={wl.H} {dname} steps={steps} warmup={warmup}",
          file=sys.stderr, flush=True)
    run, total_ms, wall, phase = timed_run(wl, prec, steps, warmup, torch)
    status = stacklstm_sync_status(run.workspace)
    per_step = phase.pop("_per_step_ms")
    ms = total_ms / steps
    fl, fx = flops(wl), executed_flops(wl)
    peak = PEAK[dname]
    rec_t = (phase["rec_fwd"] + phase["rec_bwd"]) / 1e3
    got = run.results() if keep_outputs else {"ptr": run.ptr.cpu().numpy()}
    ptr = np.vstack([np.zeros((1, wl.B), np.int64), np.cumsum(wl.ops.astype(np.int64), axis=0)])
    st = wl.op_stats()
    step_bytes = stored_step_traffic(cname, dname)
    m = {"value": wl.B * wl.T / (ms / 1e3), "ms_per_step": ms, "dtype": dname,
         "status": {"code": int(status), "ptr_trace_equal_prefix_sum": bool(np.array_equal(got["ptr"], ptr))},
         "phases_ms": {k: round(v, 4) for k, v in phase.items()},
         "step_ms_median": float(np.median(per_step)), "step_ms_min": float(np.min(per_step)),
         # algorithmic: every element-step's 2*4H*H per recurrent contraction; executed: the
         # backward contraction over push rows only (dA is exactly 0 on the others)
         "recurrent_mfma_frac": (fl["rec_fwd"] + fl["rec_bwd"]) / rec_t / 1e12 / peak,
         "recurrent_mfma_frac_executed": (fx["rec_fwd"] + fx["rec_bwd"]) / rec_t / 1e12 / peak,
         "overall_mfma_frac": sum(fx.values()) / (ms / 1e3) / 1e12 / peak,
         "executed_tflops": {k: round(fx[k] / (phase[k] / 1e3) / 1e12, 2) for k in fx if phase.get(k)},
         "push_steps_per_s": st["push_steps"] / (ms / 1e3), "op_stats": st, "wall_s_timed": wall,
         "hbm_gb_s_whole_run": None if step_bytes is None else step_bytes / (ms / 1e3) / 1e9,
         "out": got if keep_outputs else None}
    if status != 0:
        print(f"[bench] {cname}: status {status} after the timed run", file=sys.stderr, flush=True)
    del run
    return m


if __name__ == "__main__":
    main()
