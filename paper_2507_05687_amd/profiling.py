"""rocprofv3 driver for the benchmark: kernel timings and HBM byte counters.

    python -m paper_2507_05687_amd.profiling trace    [--workload W] [--raw DIR] [--out DIR]
    python -m paper_2507_05687_amd.profiling counters [--workload W] [--raw DIR] [--out DIR]
    python -m paper_2507_05687_amd.profiling mfma     [--workload W] [--raw DIR] [--out DIR]

`trace` runs ``rocprofv3 --kernel-trace --stats`` over ``bench.py --workload W``
and writes a per-kernel duration table. `counters` takes FETCH_SIZE and
WRITE_SIZE (one counter pass each) over one benchmark step and over a plain
1 GiB device copy; the copy's readings calibrate the counters (bytes the copy
must move / what the counter reports), and the workload's main kernels'
readings, scaled by that factor, give their HBM bytes per launch. `mfma`
takes GRBM_GUI_ACTIVE, SQ_VALU_MFMA_BUSY_CYCLES and SQ_INSTS_VALU_MFMA_MOPS_BF16
in one pass over one step: per GEMM launch the bf16 MFMA flops executed (512
per MOP), the fraction of SIMD cycles with the MFMA unit busy, the clock, and
the executed flops over the launch's duration in the trace run (no counters)
against the bf16 peak. Raw
rocprofv3 output stays in --raw; the text summaries and traffic_W.json (with
the SHA-256 of the kernels' source and of the host code that sizes their
launches, so that a stale record is never used) go to --out.
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
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join("paper_2507_05687_amd", "csrc")
# library kernel kind -> substring of the kernel symbol
GEMM_KINDS = {"gemm_logits_lse": "EpiLse", "gemm_recompute_dz": "EpiDz",
              "gemm_grad_hidden": "EpiGradHidden", "gemm_grad_weight": "EpiGradWeight"}
# workload -> bench.py arguments, kernels of interest, their source file, description
PROFILED = {
    "fwdbwd_bf16": dict(
        args=[], kinds=GEMM_KINDS, source=os.path.join(CSRC, "gemm_bf16.hip"),
        desc="N=131072, H=4096, V=155136, bf16",
        note="the warm-up step and the setup scoring call are included: 5 scoring launches"),
    "fwd_bf16": dict(
        args=["--workload", "fwd_bf16"], kinds=GEMM_KINDS,
        source=os.path.join(CSRC, "gemm_bf16.hip"),
        desc="log-prob scoring only, N=32768, H=4096, V=155136, bf16",
        note="the warm-up step and the setup scoring call are included: 5 scoring launches"),
    "ragged_bf16": dict(
        args=["--workload", "ragged_bf16"], kinds=GEMM_KINDS,
        source=os.path.join(CSRC, "gemm_bf16.hip"),
        desc="16 prompts x G = 8, lengths U{256..8192} padded to 8192, H=4096, V=155136, bf16",
        note="the warm-up step and the setup scoring call are included: 5 scoring launches"),
    "double_bf16": dict(
        args=["--workload", "double_bf16"], kinds=GEMM_KINDS,
        source=os.path.join(CSRC, "gemm_bf16.hip"),
        desc="policy and reference scoring then loss fwd+bwd, N=262144, H=4096, V=155136, bf16",
        note="the warm-up step and the setup scoring call are included: 9 scoring launches"),
    "sft_bf16": dict(
        args=["--workload", "sft_bf16"], kinds=GEMM_KINDS,
        source=os.path.join(CSRC, "gemm_bf16.hip"),
        desc="one 16384-token sequence, 14336 supervised tokens, H=4096, V=155136, bf16",
        note="the warm-up step is included"),
    "adamw_lmhead": dict(
        args=["--workload", "adamw_lmhead"], kinds={"adamw": "k_adamw"},
        source=os.path.join(CSRC, "aux_kernels.hip"),
        desc="155136 x 4096 fp32 parameters, moments and gradient, bf16 copy",
        note="the warm-up step is included"),
    "rule_reward": dict(
        args=["--workload", "rule_reward"], kinds={"rule_reward": "k_rule_reward"},
        source=os.path.join(CSRC, "reward_kernels.hip"),
        desc="8 prompts x G = 8 generated completions of up to 65,536 bytes, launch check on",
        note="the warm-up step is included"),
}
# the streaming kernels of the loss and scoring calls (HBM-bound; their
# counter bytes are reported with GB/s against the HBM peak)
STREAMING = {"tile_rows": "k_tile_rows", "lse_finalize": "k_lse_finalize",
             "token_objective": "k_token_objective", "loss_final": "k_loss_final",
             "pack_count": "k_pack_count", "pack_scan": "k_pack_scan",
             "pack_scatter": "k_pack_scatter", "sum_splits": "k_sum_splits",
             "sort_init": "k_sort_init", "radix_count": "k_radix_count",
             "radix_scan": "k_radix_scan", "radix_scatter": "k_radix_scatter",
             "onehot_dw": "k_onehot_dw", "zero_masked_rows": "k_zero_masked_rows",
             "group_advantages": "k_group_advantages", "rows_out": "k_rows_out"}
STREAMING_SOURCES = [os.path.join(CSRC, "aux_kernels.hip"), os.path.join(CSRC, "onehot.hip")]
COPY_BYTES = 1 << 30
PEAK_HBM = 8e12     # MI355X HBM3E, bytes/s
PEAK_BF16 = 2.5e15  # MI355X dense bf16 MFMA, flop/s
SIMDS = 256 * 4
XCDS = 8
# the host code that chooses chunk sizes, splits and grids of every launch
HOST_SOURCE = os.path.join(CSRC, "grpo_api.hip")


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


def source_sha(rel: str) -> str:
    return hashlib.sha256(open(os.path.join(ROOT, rel), "rb").read()).hexdigest()


def sources_sha(cfg: dict) -> dict:
    """SHA-256 of the workload's kernel sources and of the host launch code."""
    rels = [cfg["source"], *(STREAMING_SOURCES if cfg["kinds"] is GEMM_KINDS else []), HOST_SOURCE]
    return {rel.replace(os.sep, "/"): source_sha(rel) for rel in rels}


def sha_lines(cfg: dict) -> list[str]:
    return [f"# source sha256 ({os.path.basename(k)}): {v}" for k, v in sources_sha(cfg).items()]


def trace(wl: str, raw: str, out: str, run: bool = True):
    cfg = PROFILED[wl]
    d = os.path.join(raw, f"trace_{wl}")
    bench = ["bench.py", *cfg["args"], "--steps", "3", "--warmup", "1", "--cpu-sample", "0"]
    if run:
        _run(["rocprofv3", "--kernel-trace", "--stats", "-d", d, "-o", "bench", "--",
              sys.executable, *bench], os.path.join(raw, f"trace_{wl}.log"), 600)
    rows = _db(d).execute("select name, total_calls, total_duration, average, percentage "
                          "from top_kernels").fetchall()
    lines = [f"# rocprofv3 kernel trace of bench.py, workload {wl} ({cfg['desc']})",
             "# command: " + " ".join(["rocprofv3", "--kernel-trace", "--stats", "-d", "<raw>",
                                      "-o", "bench", "--", "python", *bench]),
             f"# ({cfg['note']})",
             *sha_lines(cfg),
             f"{'calls':>6} {'total_ms':>10} {'avg_ms':>9} {'pct':>6}  kernel"]
    for name, calls, tot, avg, pct in rows:
        # every kernel, the small streaming ones included; top_kernels reports microseconds
        lines.append(f"{calls:6d} {tot / 1e3:10.3f} {avg / 1e3:9.4f} {pct:6.2f}  {name[:110]}")
    path = os.path.join(out, f"kernels_{wl}.txt")
    open(path, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def counters(wl: str, raw: str, out: str):
    cfg = PROFILED[wl]
    bench = ["bench.py", *cfg["args"], "--steps", "1", "--warmup", "0", "--cpu-sample", "0"]
    res = {}
    for name in ("FETCH_SIZE", "WRITE_SIZE"):
        d = os.path.join(raw, f"pmc_{wl}_{name.lower()}")
        _run(["rocprofv3", "--pmc", name, "-d", d, "-o", "bench", "--", sys.executable, *bench],
             os.path.join(raw, f"pmc_{wl}_{name.lower()}.log"), 600)
        dc = os.path.join(raw, f"pmc_copy_{name.lower()}")
        _run(["rocprofv3", "--pmc", name, "-d", dc, "-o", "copy", "--", sys.executable, "bench.py",
              "--copy-calibration"], os.path.join(raw, f"pmc_copy_{name.lower()}.log"), 300)
        res[name] = (_counter(d, name), _counter(dc, name))
    copy_f = [v for k, v in res["FETCH_SIZE"][1].items() if "copyBuffer" in k][0]
    copy_w = [v for k, v in res["WRITE_SIZE"][1].items() if "copyBuffer" in k][0]
    kib = COPY_BYTES / 1024
    f_scale = kib / (sum(copy_f) / len(copy_f))
    w_scale = kib / (sum(copy_w) / len(copy_w))
    cmd = f"python -m paper_2507_05687_amd.profiling counters --workload {wl}"
    rec = {"workload": wl, "sources_sha256": sources_sha(cfg), "fetch_scale": f_scale, "write_scale": w_scale, "command": cmd, "kernels": {}}
    lines = [f"# HBM traffic per launch, workload {wl}, from rocprofv3 --pmc FETCH_SIZE and "
             f"--pmc WRITE_SIZE (one pass each) over `python {' '.join(bench)}`",
             "# calibration: `python bench.py --copy-calibration` (1 GiB device copy): "
             f"FETCH_SIZE x{f_scale:.4f}, WRITE_SIZE x{w_scale:.4f} to reach the bytes it moves",
             f"# command: {cmd}",
             *sha_lines(cfg),
             f"{'kind':22s} {'launches':>8} {'fetch_GB':>10} {'write_GB':>10} {'total_GB':>10}"]
    for kind, sym in cfg["kinds"].items():
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
    if cfg["kinds"] is GEMM_KINDS:
        # the streaming kernels: bytes per launch, and GB/s over their average
        # duration in the trace run of the same workload (when it is in --raw)
        lines += ["# streaming kernels: counter bytes per launch; GB/s = bytes / average "
                  "duration in the kernel trace; frac = GB/s / 8000",
                  f"{'kind':22s} {'launches':>8} {'fetch_MB':>10} {'write_MB':>10} "
                  f"{'total_MB':>10} {'avg_us':>9} {'GB/s':>8} {'frac':>6}"]
        rec["streaming"] = {}
        for kind, sym in STREAMING.items():
            f = [v for k, v in res["FETCH_SIZE"][0].items() if sym in k]
            w = [v for k, v in res["WRITE_SIZE"][0].items() if sym in k]
            if not f or not w:
                continue
            fv = [x for lst in f for x in lst]
            wv = [x for lst in w for x in lst]
            fb = sum(fv) / len(fv) * 1024 * f_scale
            wb = sum(wv) / len(wv) * 1024 * w_scale
            tms = _trace_avg_ms(raw, wl, sym)
            gbs = (fb + wb) / (tms / 1e3) / 1e9 if tms else None
            rec["streaming"][kind] = {"symbol": sym, "launches": len(fv),
                                      "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
                                      "trace_avg_ms": tms, "gb_per_s": gbs,
                                      "frac_of_hbm_peak": gbs * 1e9 / PEAK_HBM if gbs else None}
            lines.append(f"{kind:22s} {len(fv):8d} {fb / 1e6:10.3f} {wb / 1e6:10.3f} "
                         f"{(fb + wb) / 1e6:10.3f} {tms * 1e3 if tms else float('nan'):9.1f} "
                         f"{gbs if gbs else float('nan'):8.0f} "
                         f"{gbs * 1e9 / PEAK_HBM if gbs else float('nan'):6.3f}")
    json.dump(rec, open(os.path.join(out, f"traffic_{wl}.json"), "w"), indent=1)
    open(os.path.join(out, f"traffic_{wl}.txt"), "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _trace_avg_ms(raw: str, wl: str, sym: str):
    """Average duration (ms) of the kernels matching sym in the trace run, if present."""
    d = os.path.join(raw, f"trace_{wl}")
    if not glob.glob(os.path.join(d, "*_results.db")):
        return None
    n = t = 0.0
    for name, calls, tot in _db(d).execute("select name, total_calls, total_duration "
                                           "from top_kernels"):
        if sym in name:
            n += calls
            t += tot
    return t / n / 1e3 if n else None  # top_kernels reports microseconds


def mfma(wl: str, raw: str, out: str):
    cfg = PROFILED[wl]
    bench = ["bench.py", *cfg["args"], "--steps", "1", "--warmup", "0", "--cpu-sample", "0"]
    names = ["GRBM_GUI_ACTIVE", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16"]
    d = os.path.join(raw, f"pmc_{wl}_mfma")
    _run(["rocprofv3", "--pmc", *names, "-d", d, "-o", "bench", "--", sys.executable, *bench],
         os.path.join(raw, f"pmc_{wl}_mfma.log"), 600)
    c = _db(d)
    cols = [r[1] for r in c.execute("pragma table_info(counters_collection)")]
    ki, ni, vi = cols.index("kernel_name"), cols.index("counter_name"), cols.index("value")
    di, si, ei = cols.index("dispatch_id"), cols.index("start"), cols.index("end")
    per = collections.defaultdict(dict)  # (kernel, dispatch) -> counter -> value
    dur = {}
    for r in c.execute("select * from counters_collection"):
        per[(r[ki], r[di])][r[ni]] = float(r[vi])
        dur[(r[ki], r[di])] = (r[ei] - r[si]) / 1e9
    cmd = f"python -m paper_2507_05687_amd.profiling mfma --workload {wl}"
    rec = {"workload": wl, "sources_sha256": sources_sha(cfg), "command": cmd, "kernels": {}}
    lines = [f"# MFMA counters per launch, workload {wl}, from one rocprofv3 --pmc "
             f"{' '.join(names)} pass over `python {' '.join(bench)}`",
             "# flops = 512 x SQ_INSTS_VALU_MFMA_MOPS_BF16; busy = SQ_VALU_MFMA_BUSY_CYCLES / "
             f"(GRBM_GUI_ACTIVE / {XCDS} x {SIMDS} SIMDs); clock = GRBM_GUI_ACTIVE / {XCDS} / "
             "duration (counters on); frac = flops / trace duration / 2.5 PFLOP/s",
             f"# command: {cmd}",
             *sha_lines(cfg),
             f"{'kind':22s} {'launches':>8} {'TFLOP/launch':>12} {'busy':>6} {'GHz':>5} "
             f"{'trace_ms':>9} {'frac':>6}"]
    for kind, sym in cfg["kinds"].items():
        keys = [k for k in per if sym in k[0]]
        if not keys:
            continue
        avg = {n: sum(per[k].get(n, 0.0) for k in keys) / len(keys) for n in names}
        gui = avg["GRBM_GUI_ACTIVE"] / XCDS
        flops = avg["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
        busy = avg["SQ_VALU_MFMA_BUSY_CYCLES"] / (gui * SIMDS) if gui else None
        ghz = gui / (sum(dur[k] for k in keys) / len(keys)) / 1e9
        tms = _trace_avg_ms(raw, wl, sym)
        frac = flops / (tms / 1e3) / PEAK_BF16 if tms else None
        rec["kernels"][kind] = {"symbol": sym, "launches": len(keys),
                                "mfma_flops_per_launch": flops, "mfma_busy": busy,
                                "clock_ghz_counters_on": ghz, "trace_avg_ms": tms,
                                "executed_frac_of_peak": frac}
        lines.append(f"{kind:22s} {len(keys):8d} {flops / 1e12:12.2f} {busy:6.3f} {ghz:5.2f} "
                     f"{tms if tms else float('nan'):9.3f} "
                     f"{frac if frac else float('nan'):6.3f}")
    json.dump(rec, open(os.path.join(out, f"mfma_{wl}.json"), "w"), indent=1)
    open(os.path.join(out, f"mfma_{wl}.txt"), "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("what", choices=["trace", "counters", "mfma", "all"])
    ap.add_argument("--workload", default="fwdbwd_bf16", choices=sorted(PROFILED))
    ap.add_argument("--raw", default=os.path.join(tempfile.gettempdir(), "grpo_prof_raw"))
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles"))
    ap.add_argument("--summarize-only", action="store_true",
                    help="rewrite the trace summary from an existing --raw directory")
    a = ap.parse_args()
    os.makedirs(a.raw, exist_ok=True)
    os.makedirs(a.out, exist_ok=True)
    os.environ.setdefault("TMPDIR", "/tmp")
    if a.what in ("trace", "all"):
        trace(a.workload, a.raw, a.out, run=not a.summarize_only)
    if a.what in ("counters", "all"):
        counters(a.workload, a.raw, a.out)
    if a.what in ("mfma", "all") and any(k.startswith("gemm") for k in PROFILED[a.workload]["kinds"]):
        mfma(a.workload, a.raw, a.out)


if __name__ == "__main__":
    main()
