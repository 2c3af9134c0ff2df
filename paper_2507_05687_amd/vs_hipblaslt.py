"""The scoring product beside hipBLASLt's plain GEMM of the same shape, on one device.

    python -m paper_2507_05687_amd.vs_hipblaslt [--rounds R] [--step] [--out DIR]
    python -m paper_2507_05687_amd.vs_hipblaslt --kernels-from RAW [--out DIR]

The scoring product (Eq. 1's log-probabilities: z = W h^T with the online
log-sum-exp and the sampled id's logit taken in the epilogue) is timed by the
library's own launch events (summed over the product's vocabulary-chunk
launches); hipBLASLt (through ``torch.matmul``, bf16 in, bf16
z out, no epilogue) by CUDA events around three calls. The two alternate within
each round so that both see the same clock; boxes of one type differ by several
per cent, so only a ratio taken this way compares the kernels. Writes
``vs_hipblaslt_gemms.txt`` (the command, the device, the source hashes and one
row per round) to --out.

With --step, the four products of one loss step at N = 131072 (their launch
times summed per product) are set beside hipBLASLt's plain GEMMs of the same
shapes: z = W h^T for scoring and for the dz recompute, dz W for dL/dh and
dz^T h for dL/dW (dz a random bf16 [N, V] matrix, its transpose stored
contiguous, so that every library call takes plain row-major operands).

Run under ``rocprofv3 --kernel-trace -d RAW``, the trace names the library's
kernels; ``--kernels-from RAW`` then appends each GEMM kernel's name, launch
count and mean duration from that trace to the summary.
"""
from __future__ import annotations

import argparse
import collections
import glob
import hashlib
import os
import sqlite3
import statistics
import sys

import torch

from . import grpo

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SUMMARY = "vs_hipblaslt_gemms.txt"
SOURCES = [os.path.join("paper_2507_05687_amd", "csrc", f) for f in ("gemm_bf16.hip", "grpo_api.hip")]
V, H = 155136, 4096


def _sha(rel: str) -> str:
    return hashlib.sha256(open(os.path.join(ROOT, rel), "rb").read()).hexdigest()


def compare(N: int, rounds: int, reps: int = 3) -> list[tuple[float, float]]:
    g = torch.Generator(device="cuda").manual_seed(0)
    W = (torch.randn(V, H, device="cuda", generator=g) * 0.02).bfloat16()
    h = torch.randn(N, H, device="cuda", generator=g).bfloat16()
    y = torch.randint(0, V, (N,), device="cuda", generator=g)
    z = W @ h.t()
    grpo.logprob_fwd(h, W, y)
    torch.cuda.synchronize()
    rows = []
    for _ in range(rounds):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            z = W @ h.t()
        e1.record()
        torch.cuda.synchronize()
        blas = e0.elapsed_time(e1) / reps
        grpo.profile_reset()
        grpo.profile_enable(True)
        for _ in range(reps):
            grpo.logprob_fwd(h, W, y)
        torch.cuda.synchronize()
        ms = grpo.profile_read()["gemm_logits_lse"][1]  # summed over the product's launches
        grpo.profile_enable(False)
        rows.append((blas, ms / reps))
    del z, W, h, y
    torch.cuda.empty_cache()
    return rows


def compare_step(N: int, rounds: int) -> list[tuple[dict, dict]]:
    g = torch.Generator(device="cuda").manual_seed(1)
    W = (torch.randn(V, H, device="cuda", generator=g) * 0.02).bfloat16()
    h = torch.randn(N, H, device="cuda", generator=g).bfloat16()
    y = torch.randint(0, V, (N,), device="cuda", generator=g)
    B = 64
    cu = torch.arange(B + 1, device="cuda", dtype=torch.int64) * (N // B)
    old = torch.full((N,), -12.0, device="cuda")
    adv = torch.randn(B, device="cuda", generator=g)
    dz = torch.empty(N, V, dtype=torch.bfloat16, device="cuda").normal_(0.0, 1e-3, generator=g)
    dzt = dz.t().contiguous()
    lib = {"scoring": lambda: W @ h.t(), "dz": lambda: W @ h.t(),
           "dh": lambda: dz @ W, "dW": lambda: dzt @ h}
    kinds = {"scoring": "gemm_logits_lse", "dz": "gemm_recompute_dz",
             "dh": "gemm_grad_hidden", "dW": "gemm_grad_weight"}

    def step():
        return grpo.loss_fwd_bwd(h, W, y, None, cu, old, old, adv, 0.2, 0.001,
                                 token_outputs=False)
    out = step()
    for f in lib.values():
        f()
    torch.cuda.synchronize()
    rows = []
    for _ in range(rounds):
        t_lib = {}
        for k, f in lib.items():
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            r = f()
            e1.record()
            torch.cuda.synchronize()
            t_lib[k] = e0.elapsed_time(e1)
            del r
        grpo.profile_reset()
        grpo.profile_enable(True)
        out = step()
        torch.cuda.synchronize()
        p = grpo.profile_read()
        grpo.profile_enable(False)
        rows.append((t_lib, {k: p[kind][1] for k, kind in kinds.items()}))
    del out, dz, dzt, W, h
    torch.cuda.empty_cache()
    return rows


def kernels_from(raw: str) -> list[str]:
    rows = collections.Counter()
    tot = collections.Counter()
    for db in glob.glob(os.path.join(raw, "**", "*_results.db"), recursive=True):
        con = sqlite3.connect(db)
        for name, n, ns in con.execute("select name, count(*), sum(end - start) from kernels "
                                       "group by name"):
            if "Cijk" in name or "k_gemm" in name:
                rows[name] += n
                tot[name] += ns
    lines = ["# GEMM kernels in the trace of the run above: launches, mean ms, name"]
    for name in sorted(rows, key=lambda k: -tot[k]):
        lines.append(f"{rows[name]:5d} {tot[name] / rows[name] / 1e6:9.3f}  {name[:150]}")
    return lines


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--rounds", type=int, default=5)
    ap.add_argument("--sizes", default="32768,131072", help="token counts N")
    ap.add_argument("--step", action="store_true",
                    help="also the four products of a loss step at N = 131072")
    ap.add_argument("--kernels-from", metavar="RAW",
                    help="append the GEMM kernels of a rocprofv3 trace of this run to the summary")
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles"))
    a = ap.parse_args()
    if a.kernels_from:
        lines = kernels_from(a.kernels_from)
        open(os.path.join(a.out, SUMMARY), "a").write("\n".join(lines) + "\n")
        print("\n".join(lines))
        return
    grpo.load()
    prop = torch.cuda.get_device_properties(0)
    cmd = ("rocprofv3 --kernel-trace -d <raw> -o vsb -- python -m paper_2507_05687_amd.vs_hipblaslt "
           + " ".join(sys.argv[1:]) + "; python -m paper_2507_05687_amd.vs_hipblaslt --kernels-from <raw>")
    lines = [f"# GEMM products vs hipBLASLt's plain GEMMs of their shapes (torch.matmul), "
             f"V={V}, H={H}, bf16",
             f"# command: {cmd}",
             f"# device: {prop.gcnArchName}, {prop.multi_processor_count} CUs, "
             f"{prop.total_memory / 2**30:.0f} GiB; torch {torch.__version__}",
             *[f"# source sha256 ({os.path.basename(s)}): {_sha(s)}" for s in SOURCES],
             "# per round: hipBLASLt ms (mean of 3 calls, events), scoring ms (mean of 3 products,"
             " each its launches summed, library events), ratio",
             f"{'N':>7} {'round':>5} {'hipBLASLt_ms':>12} {'scoring_ms':>10} {'ratio':>6}"]
    for N in (int(s) for s in a.sizes.split(",")):
        rows = compare(N, a.rounds)
        for i, (b, s) in enumerate(rows):
            lines.append(f"{N:7d} {i:5d} {b:12.2f} {s:10.2f} {s / b:6.3f}")
        med = statistics.median(s / b for b, s in rows)
        lines.append(f"{N:7d} {'med':>5} {statistics.median(b for b, _ in rows):12.2f} "
                     f"{statistics.median(s for _, s in rows):10.2f} {med:6.3f}")
        print("\n".join(lines[-len(rows) - 1:]), flush=True)
    if a.step:
        N = 131072
        rows = compare_step(N, a.rounds)
        lines.append(f"# loss step at N={N}: per product, hipBLASLt ms (one call of the full shape) /"
                     " library ms (its launches summed) / ratio")
        lines.append(f"{'round':>5} " + " ".join(f"{k:>22}" for k in rows[0][0]))
        for i, (tl, tm) in enumerate(rows):
            lines.append(f"{i:5d} " + " ".join(f"{tl[k]:7.2f} {tm[k]:7.2f} {tm[k] / tl[k]:6.3f}"
                                               for k in tl))
        lines.append(f"{'med':>5} " + " ".join(
            f"{statistics.median(r[0][k] for r in rows):7.2f} "
            f"{statistics.median(r[1][k] for r in rows):7.2f} "
            f"{statistics.median(r[1][k] / r[0][k] for r in rows):6.3f}" for k in rows[0][0]))
        print("\n".join(lines[-len(rows) - 3:]), flush=True)
    os.makedirs(a.out, exist_ok=True)
    open(os.path.join(a.out, SUMMARY), "w").write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
