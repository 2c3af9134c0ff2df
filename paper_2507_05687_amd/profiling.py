"""rocprofv3 driver for the benchmark: kernel timings and HBM byte counters.

    python -m paper_2507_05687_amd.profiling trace    [--raw DIR] [--out DIR]
    python -m paper_2507_05687_amd.profiling counters [--raw DIR] [--out DIR]

`trace` runs ``rocprofv3 --kernel-trace --stats`` over ``bench.py`` and writes
a per-kernel duration table. `counters` takes FETCH_SIZE and WRITE_SIZE (one
counter pass each) over one benchmark step and over a plain 1 GiB device
copy; the copy's readings calibrate the counters (bytes the copy must move /
what the counter reports), and the GEMM kernels' readings, scaled by that
factor, give their HBM bytes per launch. Raw rocprofv3 output stays in
--raw; the text summaries and traffic.json go to --out.
"""
from __future__ import annotations

import argparse
import collections
import glob
import hashlib
import json
import os
import sqlite3
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GEMM_SRC = os.path.join(ROOT, "paper_2507_05687_amd", "csrc", "gemm_bf16.hip")
WORKLOAD = "fwdbwd_bf16"
# library kernel kind -> substring of the kernel symbol
KINDS = {"gemm_logits_lse": "EpiLse", "gemm_recompute_dz": "EpiDz",
         "gemm_grad_hidden": "EpiGradHidden", "gemm_grad_weight": "EpiGradWeight"}
COPY_BYTES = 1 << 30


def _run(cmd: list[str], log: str, limit: int):
    print("+", " ".join(cmd), flush=True)
    with open(log, "w") as f:
        r = subprocess.run(["timeout", "-s", "KILL", str(limit), *cmd], stdout=f,
                           stderr=subprocess.STDOUT, cwd=ROOT)
    if r.returncode != 0:
        sys.exit(f"failed ({r.returncode}): {' '.join(cmd)}; see {log}")


def _db(d: str) -> sqlite3.Connection:
    return sqlite3.connect(glob.glob(os.path.join(d, "*_results.db"))[0])


def _counter(d: str, name: str) -> dict:
    c = _db(d)
    cols = [r[1] for r in c.execute("pragma table_info(counters_collection)")]
    ki, ni, vi = cols.index("kernel_name"), cols.index("counter_name"), cols.index("value")
    out = collections.defaultdict(list)
    for r in c.execute("select * from counters_collection"):
        if r[ni] == name:
            out[r[ki]].append(float(r[vi]))
    return out


def _source_sha() -> str:
    return hashlib.sha256(open(GEMM_SRC, "rb").read()).hexdigest()


def trace(raw: str, out: str, run: bool = True):
    d = os.path.join(raw, "trace")
    cmd = ["rocprofv3", "--kernel-trace", "--stats", "-d", d, "-o", "bench", "--", sys.executable,
           "bench.py", "--steps", "3", "--warmup", "1", "--cpu-sample", "0"]
    if run:
        _run(cmd, os.path.join(raw, "trace.log"), 600)
    rows = _db(d).execute("select name, total_calls, total_duration, average, percentage "
                          "from top_kernels").fetchall()
    lines = [f"# rocprofv3 kernel trace of bench.py, workload {WORKLOAD} (N=131072, H=4096, "
             "V=155136, bf16)",
             "# command: " + " ".join(["rocprofv3", "--kernel-trace", "--stats", "-d", "<raw>",
                                      "-o", "bench", "--", "python", "bench.py", "--steps", "3",
                                      "--warmup", "1", "--cpu-sample", "0"]),
             "# (the warm-up step and the setup scoring call are included: 5 scoring launches)",
             f"# gemm source sha256: {_source_sha()}",
             f"{'calls':>6} {'total_ms':>10} {'avg_ms':>9} {'pct':>6}  kernel"]
    for name, calls, tot, avg, pct in rows:
        if pct < 0.01:
            continue
        # top_kernels reports microseconds
        lines.append(f"{calls:6d} {tot / 1e3:10.3f} {avg / 1e3:9.4f} {pct:6.2f}  {name[:110]}")
    path = os.path.join(out, f"kernels_{WORKLOAD}.txt")
    open(path, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def counters(raw: str, out: str):
    res = {}
    for name in ("FETCH_SIZE", "WRITE_SIZE"):
        d = os.path.join(raw, f"pmc_{name.lower()}")
        _run(["rocprofv3", "--pmc", name, "-d", d, "-o", "bench", "--", sys.executable, "bench.py",
              "--steps", "1", "--warmup", "0", "--cpu-sample", "0"],
             os.path.join(raw, f"pmc_{name.lower()}.log"), 600)
        dc = os.path.join(raw, f"pmc_copy_{name.lower()}")
        _run(["rocprofv3", "--pmc", name, "-d", dc, "-o", "copy", "--", sys.executable, "bench.py",
              "--copy-calibration"], os.path.join(raw, f"pmc_copy_{name.lower()}.log"), 300)
        res[name] = (_counter(d, name), _counter(dc, name))
    copy_f = [v for k, v in res["FETCH_SIZE"][1].items() if "copyBuffer" in k][0]
    copy_w = [v for k, v in res["WRITE_SIZE"][1].items() if "copyBuffer" in k][0]
    kib = COPY_BYTES / 1024
    f_scale = kib / (sum(copy_f) / len(copy_f))
    w_scale = kib / (sum(copy_w) / len(copy_w))
    rec = {"workload": WORKLOAD, "gemm_source_sha256": _source_sha(), "fetch_scale": f_scale,
           "write_scale": w_scale,
           "command": "python -m paper_2507_05687_amd.profiling counters", "kernels": {}}
    lines = [f"# HBM traffic per launch, workload {WORKLOAD}, from rocprofv3 --pmc FETCH_SIZE and "
             "--pmc WRITE_SIZE (one pass each) over `python bench.py --steps 1 --warmup 0 "
             "--cpu-sample 0`",
             "# calibration: `python bench.py --copy-calibration` (1 GiB device copy): "
             f"FETCH_SIZE x{f_scale:.4f}, WRITE_SIZE x{w_scale:.4f} to reach the bytes it moves",
             "# command: python -m paper_2507_05687_amd.profiling counters",
             f"# gemm source sha256: {_source_sha()}",
             f"{'kind':22s} {'launches':>8} {'fetch_GB':>10} {'write_GB':>10} {'total_GB':>10}"]
    for kind, sym in KINDS.items():
        f = [v for k, v in res["FETCH_SIZE"][0].items() if sym in k]
        w = [v for k, v in res["WRITE_SIZE"][0].items() if sym in k]
        if not f or not w:
            continue
        fb = sum(f[0]) / len(f[0]) * 1024 * f_scale
        wb = sum(w[0]) / len(w[0]) * 1024 * w_scale
        rec["kernels"][kind] = {"symbol": sym, "launches": len(f[0]),
                                "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                                "hbm_bytes_per_launch": fb + wb}
        lines.append(f"{kind:22s} {len(f[0]):8d} {fb / 1e9:10.3f} {wb / 1e9:10.3f} "
                     f"{(fb + wb) / 1e9:10.3f}")
    json.dump(rec, open(os.path.join(out, "traffic.json"), "w"), indent=1)
    open(os.path.join(out, f"traffic_{WORKLOAD}.txt"), "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("what", choices=["trace", "counters", "all"])
    ap.add_argument("--raw", default=os.path.join(ROOT, "gpurun_out", "prof"))
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles"))
    ap.add_argument("--summarize-only", action="store_true",
                    help="rewrite the trace summary from an existing --raw directory")
    a = ap.parse_args()
    os.makedirs(a.raw, exist_ok=True)
    os.makedirs(a.out, exist_ok=True)
    os.environ.setdefault("TMPDIR", "/tmp")
    if a.what in ("trace", "all"):
        trace(a.raw, a.out, run=not a.summarize_only)
    if a.what in ("counters", "all"):
        counters(a.raw, a.out)


if __name__ == "__main__":
    main()
