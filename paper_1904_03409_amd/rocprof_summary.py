"""Condenses rocprofv3 CSV output into the short text summaries kept under profiles/.

  python -m paper_1904_03409_amd.rocprof_summary stats DIR
      per-kernel calls / total / average / min / max duration from DIR's *kernel_trace.csv
      (a `rocprofv3 --kernel-trace --output-format csv` run), as a markdown table.

  python -m paper_1904_03409_amd.rocprof_summary traffic --fetch DIR1 --write DIR2 \\
          --copy-bytes N --key CONFIG [--json OUT] [--steps-per-run K]
      HBM bytes per dispatch of every kernel from a FETCH_SIZE run (DIR1) and a WRITE_SIZE
      run (DIR2). Both counters are read in KiB per dispatch and scaled by what they read
      for the plain copy kernel of N bytes in the same run (the elementwise b = a * 1 kernel
      that bench.py --copy-probe launches). With --json, the persistent kernels' entries are
      merged into OUT keyed CONFIG/dtype/phase (dtype from the kernel's precision argument),
      together with the hash of the kernel sources they were taken from (bench.py reports
      them only while that hash still matches). The totals of one whole fwd+bwd step per
      precision (every kernel, K steps per run) are stored as CONFIG/dtype/step.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import json
import os
import sys


def _rows(d, suffix):
    files = glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
    if not files:
        raise SystemExit(f"no *{suffix} under {d}")
    for f in files:
        with open(f, newline="") as fh:
            yield from csv.DictReader(fh)


def stats(d):
    dur = collections.defaultdict(list)
    for r in _rows(d, "kernel_trace.csv"):
        dur[r["Kernel_Name"]].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    tot = sum(sum(v) for v in dur.values())
    lines = ["| Kernel | Calls | Total (us) | Average (us) | Min (us) | Max (us) | % |",
             "|:--|--:|--:|--:|--:|--:|--:|"]
    for k, v in sorted(dur.items(), key=lambda kv: -sum(kv[1])):
        name = k if len(k) <= 70 else k[:67] + "..."
        lines.append(f"| `{name}` | {len(v)} | {sum(v) / 1e3:.1f} | {sum(v) / len(v) / 1e3:.1f} | "
                     f"{min(v) / 1e3:.1f} | {max(v) / 1e3:.1f} | {100.0 * sum(v) / tot:.1f} |")
    return "\n".join(lines)


def _dispatches(d, counter):
    """[(dispatch id, kernel name, counter value summed over the dispatch's instances)] in
    dispatch order."""
    per = collections.defaultdict(float)
    names = {}
    for r in _rows(d, "counter_collection.csv"):
        if r["Counter_Name"] != counter:
            continue
        key = int(r["Dispatch_Id"])
        per[key] += float(r["Counter_Value"])
        names[key] = r["Kernel_Name"]
    return [(k, names[k], per[k]) for k in sorted(per)]


def _per_dispatch(d, counter):
    """Counter value per dispatch, averaged per kernel."""
    out = collections.defaultdict(list)
    for _, name, v in _dispatches(d, counter):
        out[name].append(v)
    return {k: sum(v) / len(v) for k, v in out.items()}


def _step_bytes(d, counter, scale, steps_per_run):
    """Scaled bytes of one fwd+bwd step for the fp32 run and for the bf16 run that bench.py
    starts after it (the bf16 run begins at its first bf16 kernel); the copy probe's kernels
    are left out."""
    seg = {"f32": 0.0, "bf16": 0.0}
    cur = "f32"
    for _, name, v in _dispatches(d, counter):
        if "<1," in name:
            cur = "bf16"
        if "MulFunctor" in name or "FillFunctor" in name:
            continue
        seg[cur] += v * 1024.0 * scale
    return {k: v / steps_per_run for k, v in seg.items()}


PHASE_OF = (("void k_fwd", "rec_fwd"), ("void k_bwd", "rec_bwd"))


def traffic(fetch_dir, write_dir, copy_bytes, key, json_out, steps_per_run):
    fetch = _per_dispatch(fetch_dir, "FETCH_SIZE")
    write = _per_dispatch(write_dir, "WRITE_SIZE")
    probe = "MulFunctor"
    cf = [v for k, v in fetch.items() if probe in k]
    cw = [v for k, v in write.items() if probe in k]
    if not cf or not cw:
        raise SystemExit("no copy probe kernel in the counter runs (run bench.py with --copy-probe)")
    f_scale = copy_bytes / (max(cf) * 1024.0)
    w_scale = copy_bytes / (max(cw) * 1024.0)
    lines = [f"Copy probe (elementwise b = a * 1) of {copy_bytes} bytes: FETCH_SIZE {max(cf):.0f} KiB, WRITE_SIZE {max(cw):.0f} KiB per "
             f"dispatch; scale factors {f_scale:.4f} (fetch), {w_scale:.4f} (write).", "",
             "| Kernel | FETCH_SIZE (KiB) | WRITE_SIZE (KiB) | HBM bytes per launch (scaled) |",
             "|:--|--:|--:|--:|"]
    entries = {}
    for k in sorted(set(fetch) | set(write), key=lambda k: -(fetch.get(k, 0) + write.get(k, 0))):
        fb, wb = fetch.get(k, 0.0), write.get(k, 0.0)
        hbm = fb * 1024.0 * f_scale + wb * 1024.0 * w_scale
        name = k if len(k) <= 70 else k[:67] + "..."
        lines.append(f"| `{name}` | {fb:.0f} | {wb:.0f} | {hbm:.4g} |")
        for prefix, phase in PHASE_OF:
            if k.startswith(prefix):
                dtype = "f32" if k.split("<", 1)[1].startswith("0") else "bf16"
                entries[f"{key}/{dtype}/{phase}"] = {"kernel": k, "fetch_kib": fb, "write_kib": wb,
                                                     "hbm_bytes_per_launch": hbm}
    fs = _step_bytes(fetch_dir, "FETCH_SIZE", f_scale, steps_per_run)
    ws = _step_bytes(write_dir, "WRITE_SIZE", w_scale, steps_per_run)
    lines += ["", f"Whole fwd+bwd step (every kernel, {steps_per_run} steps per run): fp32 "
              f"{(fs['f32'] + ws['f32']) / 1e9:.3f} GB, bf16-GEMM {(fs['bf16'] + ws['bf16']) / 1e9:.3f} GB."]
    for dt in ("f32", "bf16"):
        entries[f"{key}/{dt}/step"] = {"kernel": "all kernels of one fwd+bwd step",
                                       "hbm_bytes_per_launch": fs[dt] + ws[dt]}
    if json_out:
        sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
        from bench import kernel_sources_sha1
        sha = kernel_sources_sha1()
        try:
            with open(json_out) as fh:
                t = json.load(fh)
        except (OSError, ValueError):
            t = {}
        if t.get("source_sha1") != sha:
            t = {"source_sha1": sha, "entries": {}}
        t["entries"].update(entries)
        t["copy_scale"] = {"fetch": f_scale, "write": w_scale}
        with open(json_out, "w") as fh:
            json.dump(t, fh, indent=1, sort_keys=True)
    return "\n".join(lines)


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-bytes", type=int, default=256 << 20)
    t.add_argument("--key", required=True)
    t.add_argument("--json", default=None)
    t.add_argument("--steps-per-run", type=int, default=3, help="warm-up + timed steps of each precision's run")
    a = ap.parse_args()
    if a.cmd == "stats":
        print(stats(a.dir))
    else:
        print(traffic(a.fetch, a.write, a.copy_bytes, a.key, a.json, a.steps_per_run))


if __name__ == "__main__":
    main()
