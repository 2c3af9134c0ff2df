"""Benchmark of the GRPO scoring + loss hot path on one MI355X.

One step = one pass of the whole path over one batch: group advantages
(Eq. 2) from the rewards, then the fused scoring + GRPO loss forward and
backward (Eq. 1 with k3 KL): valid-row packing, LM-head contraction with
online log-sum-exp, the per-token ratio/clip/KL epilogue, the masked
aggregation, and dL/dh, dL/dW through a recomputed, chunked logits
gradient. Inputs are seeded synthetic tensors already resident in HBM.
`--workload sft_bf16` times the supervised stage instead: the same
contractions with the mean cross-entropy over the response tokens.
`--workload adamw_lmhead` times the fused AdamW step of the LM head.
`--workload rule_reward` times the rule-based reward (Eq. 3) of a batch of
completions and the group advantages it feeds.

Prints one JSON line (see the contract in the repository documentation).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "rollout tokens/sec for fused log-prob + GRPO loss fwd+bwd; % bf16 MFMA peak"
METRIC_SFT = "supervised tokens/sec for fused LM-head cross-entropy fwd+bwd (SFT stage); % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA, the published figure (roofline peak)
# the same peak from the unit counts: 256 CUs x 4096 bf16 flop/clock x 2.4 GHz; the
# step's MFMA fractions are taken against this, the larger of the two
PEAK_BF16_UNITS_TFLOPS = 256 * 4096 * 2.4e9 / 1e12
PEAK_HBM_GBS = 8000.0


def host_cpu() -> dict:
    """Model name and online core count of the host that ran the CPU leg."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": os.cpu_count()}


def _to_dev_bf16(bits, torch):
    return torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).cuda()


def _gemm_flops(kind: str, w, n_valid: int, vc_sizes: list[int]) -> float:
    """Contraction flops of all launches of one GEMM kind in one step."""
    H, V = w.hidden, w.vocab
    if kind == "gemm_logits_lse":
        return 2.0 * n_valid * V * H * (2 if w.double_scoring else 1)
    if kind in ("gemm_recompute_dz", "gemm_grad_hidden", "gemm_grad_weight"):
        return 2.0 * n_valid * V * H
    return 0.0


def _profile_record(prefix: str, workload: str):
    """The committed rocprofv3 summary profiles/<prefix>_<workload>.json, if it
    was taken on the current source of its kernels and of the host code that
    sizes their launches; else None."""
    path = os.path.join(ROOT, "profiles", f"{prefix}_{workload}.json")
    if not os.path.exists(path):
        return None
    try:
        import hashlib

        rec = json.load(open(path))
        shas = rec.get("sources_sha256") or {}
        if not shas or rec.get("workload") != workload:
            return None
        for rel, sha in shas.items():
            src = open(os.path.join(ROOT, *rel.split("/")), "rb").read()
            if sha != hashlib.sha256(src).hexdigest():
                return None
        return rec
    except Exception:
        return None


def _traffic_from_profiles(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the counter summary, or None."""
    rec = _profile_record("traffic", workload)
    return rec and rec.get("kernels", {}).get(kernel, {}).get("hbm_bytes_per_launch")


def _mfma_from_profiles(kernel: str, workload: str):
    """(MFMA-busy fraction, executed bf16 flops per launch) of `kernel` from the
    MFMA counter summary, or (None, None)."""
    rec = _profile_record("mfma", workload)
    k = (rec or {}).get("kernels", {}).get(kernel, {})
    return k.get("mfma_busy"), k.get("mfma_flops_per_launch")


def cpu_baseline(w, W_bits, h_bits, batch, adv, old, ref, sample_tokens: int):
    """Time the double-precision oracle on the host cores on a bounded sample
    of the same workload: `sample_tokens` valid rows, scored at full H and V,
    with their loss terms, their dL/dh rows and their contribution to dL/dW
    over the whole vocabulary."""
    import oracle

    oracle.build(force=False)
    rows = np.flatnonzero(batch["mask"])[:sample_tokens]
    hd = oracle.decode(h_bits[rows], "bf16")
    Wd = oracle.decode(W_bits, "bf16")
    y = batch["tokens"][rows]
    B = w.num_seqs
    seq = np.repeat(np.arange(B), np.diff(batch["cu_seqlens"]))[rows]
    counts = np.array([batch["mask"][batch["cu_seqlens"][b]:batch["cu_seqlens"][b + 1]].sum()
                       for b in range(B)])
    t0 = time.perf_counter()
    lse, logp, _ = oracle.score_rows(hd, Wd, y)
    if w.objective == "sft":  # dL/dlogp of the mean cross-entropy over the supervised rows
        g = np.full(len(rows), -1.0 / int(batch["mask"].sum()))
    else:
        c = oracle.seq_weights(counts)
        ell, g, _ = oracle.token_objective(logp, old[rows], ref[rows], adv[seq], c[seq], None,
                                           w.clip_eps, w.beta)
    oracle.grad_hidden_rows(hd, Wd, y, lse, g)
    oracle.grad_weight_rows(hd, Wd, y, lse, g)
    dt = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or os.cpu_count()
    return {"value": len(rows) / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(rows)} valid tokens of {w.name} at H={w.hidden}, V={w.vocab}: "
                      f"scoring, loss terms, dL/dh rows and their dL/dW over all V rows "
                      f"({dt:.1f} s)", **host_cpu()}


def bench_adamw(args):
    """The fused AdamW step on the LM head's V x H fp32 weights, moments and
    gradient (plus the bf16 copy): an HBM-bound pass of 30 bytes per parameter."""
    import torch

    from paper_2507_05687_amd import grpo, workloads

    w = workloads.WORKLOADS["fwdbwd_bf16"]
    n = w.vocab * w.hidden
    gen = torch.Generator(device="cuda").manual_seed(7)
    f32 = dict(dtype=torch.float32, device="cuda")
    weight = torch.randn(n, generator=gen, **f32) * w.weight_sigma
    exp_avg = torch.zeros(n, **f32)
    exp_avg_sq = torch.zeros(n, **f32)
    grad = torch.randn(n, generator=gen, **f32) * 1e-4
    wb = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    lr, b1, b2, eps, wd = 1e-6, 0.9, 0.999, 1e-8, 0.01
    step_no = 0

    def step():
        nonlocal step_no
        step_no += 1
        grpo.adamw_step(weight, exp_avg, exp_avg_sq, grad, step_no, lr, b1, b2, eps, wd,
                        weight_bf16=wb)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    grpo.profile_reset()
    grpo.profile_enable(True)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    grpo.profile_enable(False)
    ms = e0.elapsed_time(e1) / args.steps
    launches, kms = grpo.profile_read()["adamw"]
    bytes_per = 4 * 4 + 3 * 4 + 2  # read w, m, v, g; write w, m, v; write the bf16 copy
    achieved = bytes_per * n / (kms / launches / 1e3) / 1e9
    res = {
        "metric": "parameters/sec for the fused AdamW step of the LM head (fp32 state, bf16 copy)",
        "value": n / (ms / 1e3), "unit": "params/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (seeded torch draws: W N(0,0.02), grad N(0,1e-4))",
        "config": {"workload": "adamw_lmhead", "params": n, "vocab": w.vocab,
                   "hidden": w.hidden, "lr": lr, "betas": [b1, b2], "eps": eps,
                   "weight_decay": wd},
        "roofline": {"kernel": "adamw", "bound": "hbm", "achieved": achieved,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS,
                     "traffic": _traffic_from_profiles("adamw", "adamw_lmhead"),
                     "bytes_per_param": bytes_per,
                     "avg_launch_ms": kms / launches},
    }
    if args.cpu_sample > 0:
        import oracle

        k = 1 << 22
        rng = np.random.default_rng(7)
        a = [rng.standard_normal(k) * s for s in (0.02, 0.0, 0.0, 1e-4)]
        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 10.0:
            oracle.adamw(a[0], np.abs(a[1]), np.abs(a[2]), a[3], 1, lr, b1, b2, eps, wd)
            reps += 1
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": reps * k / dt, "unit": "params/s", "cores": 1,
                               "kind": "oracle",
                               "sample": f"{reps} oracle steps on {k} parameters ({dt:.1f} s)",
                               **host_cpu()}
    else:
        res["cpu_baseline"] = None
    print(json.dumps(res), flush=True)


def bench_rule_reward(args):
    """The rule-based reward (Eq. 3: the @triton.jit rule with the launch
    check, times test_passed) of 8 prompts x G = 8 completions of up to
    16,384 tokens (about 4 bytes each), then the group advantages (Eq. 2)."""
    import torch

    from paper_2507_05687_amd import grpo, workloads

    texts, passed = workloads.make_completions(64, seed=9, mean_len=30000, max_len=65536)
    data, offsets = workloads.pack_completions(texts)
    text_d = torch.from_numpy(data).cuda()
    off_d = torch.from_numpy(offsets).cuda()
    passed_d = torch.from_numpy(passed).cuda()

    def step():
        _, reward = grpo.triton_rule_reward(text_d, off_d, passed_d, require_launch=True)
        grpo.group_advantages(reward, 8)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    grpo.profile_reset()
    grpo.profile_enable(True)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    grpo.profile_enable(False)
    ms = e0.elapsed_time(e1) / args.steps
    launches, kms = grpo.profile_read()["rule_reward"]
    nbytes = int(offsets[-1])
    # every byte is read once by the decorator scan; the launch search reads
    # the completion again for each decorated kernel
    achieved = nbytes / (kms / launches / 1e3) / 1e9
    res = {
        "metric": "completions/sec for the rule-based reward (Eq. 3) and group advantages",
        "value": len(texts) / (ms / 1e3), "unit": "completions/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "u8",
        "data": "synthetic (seeded generated Python/Triton sources, Bernoulli(0.5) test results)",
        "config": {"workload": "rule_reward", "completions": len(texts), "group": 8,
                   "bytes": nbytes, "max_bytes": int(max(len(t) for t in texts)),
                   "require_launch": True},
        "roofline": {"kernel": "rule_reward", "bound": "hbm", "achieved": achieved,
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": achieved / PEAK_HBM_GBS,
                     "traffic": _traffic_from_profiles("rule_reward", "rule_reward"),
                     "bytes_per_launch": nbytes, "avg_launch_ms": kms / launches},
    }
    if args.cpu_sample > 0:
        import oracle

        t0 = time.perf_counter()
        reps = 0
        while time.perf_counter() - t0 < 10.0:
            _, r = oracle.rule_rewards(texts, passed, require_launch=True)
            oracle.advantages(r.astype(np.float64), 8)
            reps += 1
        dt = time.perf_counter() - t0
        res["cpu_baseline"] = {"value": reps * len(texts) / dt, "unit": "completions/s",
                               "cores": 1, "kind": "oracle",
                               "sample": f"{reps} passes of the oracle over the same {len(texts)} "
                                         f"completions ({dt:.1f} s)", **host_cpu()}
    else:
        res["cpu_baseline"] = None
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="fwdbwd_bf16",
                    choices=["fwdbwd_bf16", "fwd_bf16", "ragged_bf16", "double_bf16",
                             "sft_bf16", "adamw_lmhead", "rule_reward"])
    ap.add_argument("--cpu-sample", type=int, default=128,
                    help="valid tokens timed on the CPU oracle (0 skips the CPU baseline)")
    ap.add_argument("--scratch-gb", type=float, default=32.0,
                    help="workspace limit in GB (1e9 bytes): the logits-gradient budget is the "
                         "largest whole GiB that keeps the workspace within it")
    ap.add_argument("--verbose", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library "
              "implements the single-GPU hot path; several GPUs would each take whole prompt "
              "groups and sum dL/dW", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2507_05687_amd import grpo, workloads

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        x = torch.ones(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": x.numel() * 4, "copy_bytes_written": y.numel() * 4,
                          "launches": 3}), flush=True)
        return
    grpo.load()
    if args.workload == "adamw_lmhead":
        return bench_adamw(args)
    if args.workload == "rule_reward":
        return bench_rule_reward(args)
    w = workloads.WORKLOADS[args.workload]
    log = (lambda *a: print(*a, file=sys.stderr, flush=True)) if args.verbose else (lambda *a: None)

    t0 = time.time()
    W_bits = workloads.make_weight(w, "policy")
    h_bits = workloads.make_hidden(w)
    batch = workloads.make_batch(w)
    # the GPU run and the CPU-baseline leg both read these arrays
    inputs_sha256 = workloads.batch_digest(W_bits, h_bits, batch)
    log(f"inputs generated in {time.time() - t0:.1f}s, sha256 {inputs_sha256}")
    W = _to_dev_bf16(W_bits, torch)
    Wref = _to_dev_bf16(workloads.make_weight(w, "reference"), torch) if w.double_scoring else None
    h = _to_dev_bf16(h_bits, torch)
    tokens = torch.from_numpy(batch["tokens"]).cuda()
    mask = torch.from_numpy(batch["mask"]).cuda()
    cu = torch.from_numpy(batch["cu_seqlens"]).cuda()
    rewards = torch.from_numpy(batch["rewards"]).cuda()
    n_valid = int(batch["mask"].sum())
    N, H, V, B = w.num_tokens, w.hidden, w.vocab, w.num_seqs
    sft = w.objective == "sft"
    use_mask = mask if (w.ragged or w.prompt_len) else None

    # old/ref log-probs: the policy's own log-prob plus seeded noise
    if sft:
        old = ref = torch.zeros(N, dtype=torch.float32, device="cuda")
    else:
        base, _ = grpo.logprob_fwd(h, W, tokens, use_mask,
                                   max_valid=n_valid if use_mask is not None else 0)
        old = base + torch.from_numpy(batch["old_noise"]).cuda()
        ref = base + torch.from_numpy(batch["ref_noise"]).cuda()
        del base
    f32 = dict(dtype=torch.float32, device="cuda")
    loss = torch.empty(1, **f32)
    gh = torch.empty(N, H, dtype=torch.bfloat16, device="cuda")
    gw = torch.empty(V, H, **f32)
    adv = torch.empty(B, **f32)
    lse_buf = torch.empty(N, **f32)
    old_buf = torch.empty(N, **f32)
    ref_buf = torch.empty(N, **f32)
    # the valid rows are known on the host (the mask is built there), so the
    # workspace is sized for them; the logits-gradient budget is the largest
    # whole GiB (at most the library default of 48) that keeps it within --scratch-gb
    max_valid = n_valid if use_mask is not None else N
    op_main = grpo.OP_SFT_FWD_BWD if sft else grpo.OP_LOSS_FWD_BWD
    # Double scoring: the reference model is frozen, so its W is tiled once
    # (here, before the timed steps); the policy's W is tiled once per step and
    # read tiled by both calls that use it (its scoring and the loss).
    flag = grpo.WS_TILED_WEIGHT if w.double_scoring else 0

    def ws_need(budget):
        fwd = grpo.workspace_bytes(grpo.OP_LOGPROB_FWD | flag, grpo.BF16, N, H, V, 1, max_valid)
        if args.workload == "fwd_bf16":  # scoring only
            return fwd
        return max(grpo.workspace_bytes(op_main | flag, grpo.BF16, N, H, V, B, max_valid, budget),
                   fwd)
    dz_budget = 48 << 30
    while dz_budget > (1 << 30) and ws_need(dz_budget) > args.scratch_gb * 1e9:
        dz_budget -= 1 << 30
    ws_bytes = ws_need(dz_budget)
    log(f"workspace {ws_bytes / 1e9:.2f} GB (logits-gradient budget {dz_budget >> 30} GiB, "
        f"{max_valid} valid rows)")
    ws = grpo.workspace(ws_bytes)
    lib = grpo.load()
    P = grpo._ptr
    stream = grpo._stream()
    mptr = P(use_mask)
    if w.double_scoring:
        Wref_t = grpo.tile_weight(Wref).buf
        W_t = grpo.tile_weight(W).buf  # rewritten in every step
    else:
        Wref_t = W_t = None

    def step():
        if sft:  # the supervised stage: cross-entropy over the response tokens
            st = lib.sft_ce_fwd_bwd(grpo.BF16, P(h), P(W), None, P(tokens), mptr, N, H, V, P(loss),
                                    None, P(gh), grpo.BF16, P(gw), 0, P(ws), ws.numel(),
                                    max_valid, dz_budget, stream)
            assert st == 0, st
            return
        st = lib.group_advantages(P(rewards), w.prompts, w.group, 1e-6, 1, P(adv), stream)
        assert st == 0, st
        if args.workload == "fwd_bf16":
            st = lib.grpo_logprob_fwd(grpo.BF16, P(h), P(W), None, P(tokens), mptr, N, H, V,
                                      P(old_buf), P(lse_buf), P(ws), ws.numel(), max_valid,
                                      stream)
            assert st == 0, st
            return
        lse_in, o, r = None, old, ref
        if w.double_scoring:  # S8: score under the policy (old) and the reference
            st = lib.grpo_tile_weight(P(W), V, H, P(W_t), W_t.numel(), stream)
            assert st == 0, st
            st = lib.grpo_logprob_fwd(grpo.BF16, P(h), P(W), P(W_t), P(tokens), mptr, N, H, V,
                                      P(old_buf), P(lse_buf), P(ws), ws.numel(), max_valid,
                                      stream)
            assert st == 0, st
            st = lib.grpo_logprob_fwd(grpo.BF16, P(h), P(Wref), P(Wref_t), P(tokens), mptr, N, H,
                                      V, P(ref_buf), None, P(ws), ws.numel(), max_valid, stream)
            assert st == 0, st
            lse_in, o, r = lse_buf, old_buf, ref_buf
        st = lib.grpo_loss_fwd_bwd(grpo.BF16, P(h), P(W), P(W_t), P(tokens), mptr, P(cu), B, N,
                                   H, V, P(o), P(r), P(adv), w.clip_eps, w.beta, 0, P(lse_in),
                                   P(loss),
                                   None, None, None, None, None, P(gh), grpo.BF16, P(gw), 0,
                                   P(ws), ws.numel(), max_valid, dz_budget, stream)
        assert st == 0, st

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    grpo.check_error(ws)
    log(f"warmup done, loss={loss.item():.6g}")

    grpo.profile_reset()
    grpo.profile_enable(True)
    # one event per step boundary, on the stream the library launches on
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    ev[0].record()
    for i in range(args.steps):
        step()
        ev[i + 1].record()
    torch.cuda.synchronize()
    grpo.profile_enable(False)
    total_ms = ev[0].elapsed_time(ev[-1])
    step_ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    prof = grpo.profile_read()
    ms_per_step = total_ms / args.steps
    ms_median = float(np.median(step_ms))
    tokens_per_s = n_valid / (ms_per_step / 1e3)
    log(json.dumps(prof))

    # dominant kernel: the kind with the largest summed time
    kind, (launches, kms) = max(prof.items(), key=lambda kv: kv[1][1])
    flops = _gemm_flops(kind, w, n_valid, []) * args.steps
    achieved = flops / (kms / 1e3) / 1e12 if flops else None
    traffic = _traffic_from_profiles(kind, w.name)
    busy, exe_flops = _mfma_from_profiles(kind, w.name)
    roofline = {"kernel": kind, "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": (achieved / PEAK_BF16_TFLOPS) if achieved else None,
                "traffic": traffic, "launches_per_step": launches / args.steps,
                "avg_launch_ms": kms / launches,
                # rocprofv3 counters of the same kernel (profiles/mfma_<workload>.json):
                # bf16 MFMA flops it executes per launch over this run's launch time, and
                # the fraction of SIMD cycles its MFMA units were busy
                "executed_frac_counters": (exe_flops / (kms / launches / 1e3) /
                                           (PEAK_BF16_TFLOPS * 1e12)) if exe_flops else None,
                "mfma_busy_counters": busy}
    per_tok = {"fwd_bf16": 2, "fwdbwd_bf16": 6, "ragged_bf16": 6, "double_bf16": 8,
               "sft_bf16": 6}[args.workload]
    executed = {"fwd_bf16": 2, "fwdbwd_bf16": 8, "ragged_bf16": 8, "double_bf16": 10,
                "sft_bf16": 8}[args.workload]
    step_s = ms_per_step / 1e3
    alg_frac = per_tok * n_valid * V * H / step_s / (PEAK_BF16_UNITS_TFLOPS * 1e12)
    exe_frac = executed * n_valid * V * H / step_s / (PEAK_BF16_UNITS_TFLOPS * 1e12)

    res = {
        "metric": METRIC_SFT if sft else METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded numpy inputs: h RMS-normalised N(0,1), W N(0,0.02), "
                "uniform token ids" + (", prompt prefix unsupervised)" if sft else
                                       ", Bernoulli rewards)"),
        "config": ({"workload": w.name, "sequences": w.num_seqs, "seq_len": w.seq_len,
                    "prompt_len": w.prompt_len, "valid_tokens": n_valid, "hidden": H,
                    "vocab": V} if sft else
                   {"workload": w.name, "prompts": w.prompts, "group": w.group,
                    "seq_len": w.seq_len, "valid_tokens": n_valid, "hidden": H, "vocab": V,
                    "clip_eps": w.clip_eps, "beta": w.beta}),
        "ms_per_step_median": ms_median,
        "value_median": n_valid / (ms_median / 1e3),
        "step_ms": step_ms,
        "mfma_peak_tflops": PEAK_BF16_UNITS_TFLOPS,
        "workspace_gb": ws_bytes / 1e9,
        "dz_budget_gib": dz_budget >> 30,
        "mfma_frac_algorithmic": alg_frac,
        "mfma_frac_executed": exe_frac,
        "roofline": roofline,
        "kernels_ms_per_step": {k: v[1] / args.steps for k, v in sorted(prof.items())},
        "inputs_sha256": inputs_sha256,
    }
    if args.cpu_sample > 0:
        adv_h = adv.cpu().numpy().astype(np.float64)
        res["cpu_baseline"] = cpu_baseline(w, W_bits, h_bits, batch, adv_h,
                                           old.cpu().numpy().astype(np.float64),
                                           ref.cpu().numpy().astype(np.float64),
                                           args.cpu_sample)
    else:
        res["cpu_baseline"] = None
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
