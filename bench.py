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
    total_ms = start.elapsed_time(stop)
    phase = {}
    f = ctypes.c_float()
    pairs = [(0, 1, "scan+sync"), (1, 2, "xw_gemm+prep"), (2, 3, "rec_fwd"), (3, 4, "top_gather"),
             (5, 6, "rec_bwd"), (6, 7, "dW+db"), (7, 8, "dU"), (8, 9, "dx"), (4, 5, "bwd_prep")]
    for a, b, name in pairs:
        acc = 0.0
        for k in range(steps):
            lib.hipEventElapsedTime(ctypes.byref(f), evs[k][a], evs[k][b])
            acc += f.value
        phase[name] = acc / steps
    for arr in evs:
        for i in range(SLSTM_PHASE_EVENTS):
            lib.hipEventDestroy(arr[i])
    return run, total_ms, wall, phase


def flops(wl):
    T, B, I, H = wl.T, wl.B, wl.I, wl.H
    rec = 2.0 * T * B * H * 4 * H                 # one recurrent contraction (h_prev U or dA U^T)
    return {"rec_fwd": rec, "rec_bwd": rec, "xw_gemm+prep": 2.0 * T * B * I * 4 * H, "dW+db": 2.0 * T * B * I * 4 * H,
            "dU": 2.0 * T * B * H * 4 * H, "dx": 2.0 * T * B * I * 4 * H}


def kernel_sources_sha1():
    """Hash of every HIP source and header of the library: a stored counter reading is
    valid only for the kernels it was taken from."""
    import glob
    import hashlib
    h = hashlib.sha1()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_1904_03409_amd", "csrc", "*"))):
        if f.endswith((".hip", ".h")):
            h.update(os.path.basename(f).encode())
            with open(f, "rb") as fh:
                h.update(fh.read())
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


def cpu_baseline(wl, target_s=12.0):
    """The oracle (float32 instantiation, OpenMP over batch elements) on a bounded sample."""
    import oracle
    th = oracle.max_threads()
    n = min(wl.B, max(th, 8))
    t0 = time.perf_counter()
    oracle.run(wl, sel=np.arange(n, dtype=np.int32), mode="f32", threads=th)
    dt = time.perf_counter() - t0
    if dt < target_s / 4 and n < wl.B:
        n = int(min(wl.B, max(n, n * target_s / max(dt, 1e-3))))
        t0 = time.perf_counter()
        oracle.run(wl, sel=np.arange(n, dtype=np.int32), mode="f32", threads=th)
        dt = time.perf_counter() - t0
    return {"value": n * wl.T / dt, "unit": "element-steps/s", "cores": th, "kind": "oracle",
            "sample": f"fwd+bwd of the first {n} of {wl.B} batch elements (all T={wl.T} steps), float32 oracle, "
                      f"{dt:.1f} s"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="large")
    ap.add_argument("--precision", choices=["fp32", "bf16"], default=None)
    ap.add_argument("--no-bf16", action="store_true", help="skip the bf16-GEMM run of the same shape")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 256 MiB device copy (counter calibration for rocprofv3 --pmc runs)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the StackLSTM step is measured on one MI355X "
              "(batch sharding across GPUs is described in DESIGN.md, not launched)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1904_03409_amd import workloads
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    wl = workloads.make(args.config)
    prec = wl.precision if args.precision is None else (0 if args.precision == "fp32" else 1)
    dname = "f32" if prec == 0 else "bf16"
    print(f"[bench] {args.config} T={wl.T} B={wl.B} I={wl.I} H={wl.H} {dname} steps={args.steps} "
          f"warmup={args.warmup}", file=sys.stderr, flush=True)
    run, total_ms, wall, phase = timed_run(wl, prec, args.steps, args.warmup, torch)
    ms = total_ms / args.steps
    value = wl.B * wl.T / (ms / 1e3)
    fl = flops(wl)
    kern = max(fl, key=lambda k: phase.get(k, 0.0))
    achieved = fl[kern] / (phase[kern] / 1e3) / 1e12
    rec_util = (fl["rec_fwd"] + fl["rec_bwd"]) / ((phase["rec_fwd"] + phase["rec_bwd"]) / 1e3) / 1e12 / PEAK[dname]
    all_util = sum(fl.values()) / (ms / 1e3) / 1e12 / PEAK[dname]
    st = wl.op_stats()
    out = {
        "metric": "fwd+bwd batch·timesteps/sec at B=256,H=512; % MFMA peak",
        "value": value, "unit": "element-steps/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms, "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": dname,
        "data": "synthetic",
        "config": {"workload": f"{args.config}: StackLSTM fwd+bwd, B={wl.B} T={wl.T} I={wl.I} H={wl.H}, "
                               f"arc-standard op streams, {dname} GEMM operands",
                   "global_batch": wl.B, "seq_len": wl.T, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": "mfma", "kernel": kern, "achieved": achieved, "peak": PEAK[dname], "unit": "TFLOP/s",
                     "frac": achieved / PEAK[dname], "traffic": stored_traffic(args.config, dname, kern)},
        "phases_ms": {k: round(v, 4) for k, v in phase.items()},
        "recurrent_mfma_frac": rec_util, "overall_mfma_frac": all_util,
        "push_steps_per_s": st["push_steps"] / (ms / 1e3), "op_stats": st, "wall_s_timed": wall,
    }
    del run
    torch.cuda.empty_cache()
    if not args.no_bf16 and prec == 0 and wl.H <= 1024:
        run2, tot2, _, ph2 = timed_run(wl, 1, args.steps, args.warmup, torch)
        ms2 = tot2 / args.steps
        r2 = (fl["rec_fwd"] + fl["rec_bwd"]) / ((ph2["rec_fwd"] + ph2["rec_bwd"]) / 1e3) / 1e12 / PEAK["bf16"]
        out["bf16_gemm"] = {"value": wl.B * wl.T / (ms2 / 1e3), "ms_per_step": ms2,
                            "recurrent_mfma_frac": r2, "overall_mfma_frac": sum(fl.values()) / (ms2 / 1e3) / 1e12 / PEAK["bf16"],
                            "phases_ms": {k: round(v, 4) for k, v in ph2.items()}}
        del run2
    if args.copy_probe:
        copy_probe(torch)
    if not args.no_cpu:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
