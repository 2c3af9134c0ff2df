"""Parity of the HIP path (through the C ABI) with the double-precision
oracle, on seeded synthetic inputs. GPU only.

Tolerances: fp32 inputs 1e-5 relative (log-probs, loss, gradients
norm-wise); bf16 inputs 2e-3 relative on log-probs and loss; bf16 gradients
norm-wise within the bound that bf16 rounding of the -g p entries of dz
implies (tests.gpu_util.grad_tolerances: typically 1e-4 or less, larger only
where the softmax is concentrated on few ids), plus 2^-9 for a bf16 dL/dh
output; integer outputs (packing, counts, clip flags away from the clip
boundary) bit-exact.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_05687_amd import grpo, workloads
from tests.gpu_util import (BF16_OUT, dev, grad_tolerances, host64, loss_tolerance_ok, norm_rel,
                            oracle_problem, rel_err, to_dev)

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-3
BF16_GRAD_TOL = None  # the rounding bound of tests.gpu_util.grad_tolerances
F32_TOL = 1e-5


@pytest.fixture(scope="module", autouse=True)
def _setup():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build(force=False)
    grpo.load()
    yield
    grpo.free_workspace()
    torch.cuda.empty_cache()


def _problem(name="tiny_fp32", **kw):
    w = workloads.scaled(workloads.WORKLOADS[name], **kw)
    W = workloads.make_weight(w)
    h = workloads.make_hidden(w)
    b = workloads.make_batch(w)
    adv = oracle.advantages(b["rewards"], w.group).astype(np.float32)
    _, logp, _ = oracle.score_rows(oracle.decode(h, w.dtype), oracle.decode(W, w.dtype),
                                   b["tokens"])
    old = (logp + b["old_noise"]).astype(np.float32)
    ref = (logp + b["ref_noise"]).astype(np.float32)
    return w, W, h, b, adv, old, ref


def _run_loss(w, W, h, b, adv, old, ref, agg=0, **kw):
    return grpo.loss_fwd_bwd(to_dev(h, w.dtype), to_dev(W, w.dtype), dev(b["tokens"]),
                             dev(b["mask"]), dev(b["cu_seqlens"]), dev(old), dev(ref), dev(adv),
                             w.clip_eps, w.beta, agg, check=True, **kw)


def _compare_loss(w, W, h, b, adv, old, ref, out, tol, grad_tol, agg=0):
    o = oracle_problem(h, W, w.dtype, b, adv.astype(np.float64), old.astype(np.float64),
                       ref.astype(np.float64), w.clip_eps, w.beta, agg)
    m = b["mask"].astype(bool)
    torch.cuda.synchronize()
    assert rel_err(host64(out["logp"])[m], o["logp"][m]) <= tol
    assert rel_err(host64(out["lse"])[m], o["lse"][m]) <= tol
    assert np.all(host64(out["logp"])[~m] == 0) and np.all(host64(out["lse"])[~m] == 0)
    # per-row weights of the Eq. 1 sum, for the condition-aware loss check
    counts = np.array([m[b["cu_seqlens"][i]:b["cu_seqlens"][i + 1]].sum()
                       for i in range(w.num_seqs)])
    c = oracle.seq_weights(counts, agg)
    seq = np.repeat(np.arange(w.num_seqs), np.diff(b["cu_seqlens"]))
    abs_sum = float(np.sum(c[seq] * np.abs(o["ell"])))
    assert loss_tolerance_ok(float(out["loss"].item()), o["loss"], abs_sum, tol), \
        (float(out["loss"].item()), o["loss"], abs_sum)
    # token loss and dL/dlogp, absolute scale-aware
    tl = host64(out["token_loss"])
    assert np.max(np.abs(tl - o["ell"])) <= tol * max(1.0, np.max(np.abs(o["ell"])))
    # dL/dlogp jumps at the clip bounds (the clipped branch has zero slope), so a
    # token whose ratio is within rounding of a bound may take either branch: it
    # is compared, like the clip flag, only away from the bounds (the count of
    # such tokens grows with N: about 60 of 4M within 1e-5 of 1.2 at sigma 0.1)
    rho = np.exp(o["logp"] - old)
    band = 1e-3 if w.dtype == "bf16" else 1e-6
    far = (np.abs(rho - (1 - w.clip_eps)) > band) & (np.abs(rho - (1 + w.clip_eps)) > band) & m
    g = host64(out["dlogp"])
    keep = far | ~m
    assert np.max(np.abs(g - o["g"])[keep]) <= tol * np.max(np.abs(o["g"])) + 1e-12
    # clip flags bit-exact away from the clip boundary
    flag = out["clip_flag"].cpu().numpy()
    assert np.array_equal(flag[far], o["clipped"][far])
    assert np.all(flag[~m] == 0)
    dh = host64(out["grad_hidden"])
    dW = host64(out["grad_weight"])
    e_dh, e_dW = norm_rel(dh, o["dh"]), norm_rel(dW, o["dW"])
    if grad_tol is None:  # bf16: the rounding bound of the -g p entries of dz
        tol_dh, tol_dW = grad_tolerances(oracle.decode(h, w.dtype), oracle.decode(W, w.dtype),
                                         np.where(m, o["g"], 0.0), o["dh"], o["dW"])
        if out["grad_hidden"].dtype == torch.bfloat16:
            tol_dh += BF16_OUT
    else:
        tol_dh = tol_dW = grad_tol
    assert e_dh <= tol_dh, (e_dh, tol_dh)
    assert e_dW <= tol_dW, (e_dW, tol_dW)
    assert np.all(dh[~m] == 0)
    return o, dict(dh=e_dh, dW=e_dW)


# ------------------------------------------------------------ advantages
def test_group_advantages_parity():
    g = np.random.default_rng(0)
    G = 8
    r = (g.integers(0, 2, 64 * G) * 0.9 + g.integers(0, 2, 64 * G) * 0.1).astype(np.float32)
    r[:G] = 1.0
    r[G:2 * G] = 0.1  # equal but not exactly representable: must still give 0
    r[2 * G:2 * G + 4] = [0, 0, 1, 1]
    r[2 * G + 4:3 * G] = [0.5, 0.5, 0.5, 0.25]
    for unbiased in (True, False):
        got = grpo.group_advantages(dev(r), G, 1e-6, unbiased).cpu().numpy()
        want = oracle.advantages(r.astype(np.float64), G, 1e-6, unbiased)
        assert np.all(got[want == 0] == 0)
        assert np.max(np.abs(got - want)) <= 1e-6 * max(1.0, np.max(np.abs(want)))
    # G = 4 worked example, one prompt
    got = grpo.group_advantages(dev(np.array([0, 0, 1, 1], np.float32)), 4).cpu().numpy()
    np.testing.assert_allclose(got, [-0.8660239, -0.8660239, 0.8660239, 0.8660239], rtol=1e-6)
    # a large group (several lanes per element)
    r = g.random(3 * 200).astype(np.float32)
    got = grpo.group_advantages(dev(r), 200).cpu().numpy()
    np.testing.assert_allclose(got, oracle.advantages(r.astype(np.float64), 200), rtol=2e-5,
                               atol=2e-6)


# ------------------------------------------------------------ packing
def test_pack_valid_bit_exact():
    g = np.random.default_rng(1)
    T, B = 700, 9
    lens = g.integers(0, T + 1, B)
    lens[3] = 0
    lens[4] = T
    mask = (np.arange(T)[None, :] < lens[:, None]).astype(np.uint8).reshape(-1)
    mask[5 * T + 10] = 0  # a hole inside a rollout
    cu = (np.arange(B + 1) * T).astype(np.int64)
    rows, counts, n = grpo.pack_valid(dev(mask), dev(cu))
    w_rows, w_counts, _ = oracle.pack_valid(mask, cu)
    assert n == len(w_rows)
    assert np.array_equal(rows.cpu().numpy(), w_rows)
    assert np.array_equal(counts.cpu().numpy(), w_counts)


# ------------------------------------------------------------ fp32 config
def test_tiny_fp32_config():
    """2 prompts x G=4 x 16 tokens, H=64, V=1000, fp32 (1e-5)."""
    w, W, h, b, adv, old, ref = _problem("tiny_fp32")
    out = _run_loss(w, W, h, b, adv, old, ref)
    _compare_loss(w, W, h, b, adv, old, ref, out, F32_TOL, F32_TOL)


def test_fp32_at_its_hidden_limit():
    """fp32 with H = 8192 (two LDS rows of H floats, 64 KiB), a ragged mask and
    a vocabulary tail, against the oracle at 1e-5."""
    w, W, h, b, adv, old, ref = _problem("tiny_fp32", hidden=8192, vocab=777, seq_len=12,
                                         ragged=True, min_len=1, seed=24)
    out = _run_loss(w, W, h, b, adv, old, ref)
    _compare_loss(w, W, h, b, adv, old, ref, out, F32_TOL, F32_TOL)


def test_tiny_fp32_pipeline_from_rewards():
    """Rewards -> group_advantages -> loss, all on the device, vs the oracle chain."""
    w, W, h, b, _, old, ref = _problem("tiny_fp32", seed=5)
    adv_dev = grpo.group_advantages(dev(b["rewards"]), w.group)
    out = grpo.loss_fwd_bwd(to_dev(h, "f32"), to_dev(W, "f32"), dev(b["tokens"]), dev(b["mask"]),
                            dev(b["cu_seqlens"]), dev(old), dev(ref), adv_dev, w.clip_eps, w.beta)
    adv_o = oracle.advantages(b["rewards"].astype(np.float64), w.group)
    o = oracle_problem(h, W, "f32", b, adv_o, old.astype(np.float64), ref.astype(np.float64),
                       w.clip_eps, w.beta)
    assert abs(out["loss"].item() - o["loss"]) <= F32_TOL * max(abs(o["loss"]), 1e-3)
    assert norm_rel(host64(out["grad_weight"]), o["dW"]) <= F32_TOL


# ------------------------------------------------------------ bf16, small
SMALL = {
    # several tiles on every axis, ragged token and vocabulary tails
    "ragged_tiles": dict(prompts=3, group=4, seq_len=50, hidden=320, vocab=3000, ragged=True,
                         min_len=1, forced_equal_groups=1),
    # H not a multiple of the 32-wide K step
    "k_tail": dict(prompts=2, group=4, seq_len=40, hidden=200, vocab=1100),
    # several vocabulary chunks in the backward pass
    "multi_chunk": dict(prompts=2, group=4, seq_len=40, hidden=128, vocab=40000),
    # smallest shapes
    "tiny": dict(prompts=1, group=2, seq_len=3, hidden=8, vocab=5),
    # dL/dW of 21 x 16 = 336 tiles: K split in 3 to fill whole rounds of 256 CUs
    "split_rounds": dict(prompts=2, group=4, seq_len=40, hidden=4096, vocab=5376),
    # a wide hidden state: 2048 K steps per scoring tile, 256 gradient tile-columns
    "wide_hidden": dict(prompts=2, group=4, seq_len=32, hidden=65536, vocab=300),
    # dL/dh over 45 token tile-rows: 32 in whole XCD bands, the other 13 shared
    # out as 2 rows to each of 5 XCDs and 1 to each of 3
    "uneven_row_bands": dict(prompts=3, group=4, seq_len=960, hidden=512, vocab=700),
    # 37 token tile-rows: the 5 after the whole bands split by columns over the XCDs
    "few_rows_after_bands": dict(prompts=1, group=8, seq_len=1184, hidden=512, vocab=700),
    # the scoring product launched per 8192 vocabulary rows: a last launch of one row
    "one_row_last_scoring_chunk": dict(prompts=2, group=4, seq_len=40, hidden=64, vocab=8193),
}


@pytest.mark.parametrize("case", list(SMALL))
def test_bf16_loss_parity(case):
    kw = dict(SMALL[case], dtype="bf16", rms_norm_hidden=True, beta=0.01, noise_sigma=0.1,
              seed=11)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    out = _run_loss(w, W, h, b, adv, old, ref)
    _compare_loss(w, W, h, b, adv, old, ref, out, BF16_TOL, BF16_GRAD_TOL)
    # dL/dh in fp32: only the -g p rounding bound
    out = _run_loss(w, W, h, b, adv, old, ref, grad_hidden_dtype=torch.float32)
    _compare_loss(w, W, h, b, adv, old, ref, out, BF16_TOL, BF16_GRAD_TOL)


@pytest.mark.timeout(900)
def test_bf16_backward_at_its_row_limit():
    # 2^22 rows, the most the bf16 backward takes per call: packing and
    # scoring over 16384 token tiles, dz products in column mode, dL/dW with
    # its K (the tokens) split 8 ways, every output against the full oracle
    kw = dict(prompts=2048, group=8, seq_len=256, hidden=32, vocab=512, dtype="bf16",
              rms_norm_hidden=True, beta=0.01, noise_sigma=0.1, seed=21)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    assert w.num_tokens == 1 << 22
    out = _run_loss(w, W, h, b, adv, old, ref)
    _compare_loss(w, W, h, b, adv, old, ref, out, BF16_TOL, BF16_GRAD_TOL)


@pytest.mark.timeout(900)
def test_bf16_vocabulary_of_4m_entries():
    # V = 2^22 with few tokens: 512 vocabulary chunks in the backward pass,
    # 32768 (max, sum-exp) partials per token to merge, a split dL/dW product
    # per chunk; every output against the full oracle
    kw = dict(prompts=2, group=4, seq_len=64, hidden=16, vocab=1 << 22, dtype="bf16",
              rms_norm_hidden=True, beta=0.01, noise_sigma=0.1, seed=22)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    out = _run_loss(w, W, h, b, adv, old, ref)
    _compare_loss(w, W, h, b, adv, old, ref, out, BF16_TOL, BF16_GRAD_TOL)


def test_bf16_token_mean_aggregation():
    kw = dict(SMALL["ragged_tiles"], dtype="bf16", rms_norm_hidden=True, beta=0.01, seed=12)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    out = _run_loss(w, W, h, b, adv, old, ref, agg=1)
    _compare_loss(w, W, h, b, adv, old, ref, out, BF16_TOL, BF16_GRAD_TOL, agg=1)


def test_bf16_f32_grad_hidden_and_accumulate():
    kw = dict(SMALL["k_tail"], dtype="bf16", rms_norm_hidden=True, seed=13)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    base = _run_loss(w, W, h, b, adv, old, ref)
    f32 = _run_loss(w, W, h, b, adv, old, ref, grad_hidden_dtype=torch.float32)
    assert f32["grad_hidden"].dtype == torch.float32
    d = (f32["grad_hidden"].bfloat16() - base["grad_hidden"]).abs().max().item()
    assert d <= 1e-2 * base["grad_hidden"].float().abs().max().item()
    acc = base["grad_weight"].clone()
    again = _run_loss(w, W, h, b, adv, old, ref, grad_weight_out=acc, accumulate_grad_weight=True)
    torch.testing.assert_close(again["grad_weight"], 2 * base["grad_weight"], rtol=1e-6, atol=0)


def test_bf16_logprob_fwd_parity():
    kw = dict(SMALL["ragged_tiles"], dtype="bf16", rms_norm_hidden=True, seed=14)
    w = workloads.scaled(workloads.WORKLOADS["fwd_bf16"], **kw)
    W, h, b = workloads.make_weight(w), workloads.make_hidden(w), workloads.make_batch(w)
    logp, lse = grpo.logprob_fwd(to_dev(h, "bf16"), to_dev(W, "bf16"), dev(b["tokens"]),
                                 dev(b["mask"]), check=True)
    m = b["mask"].astype(bool)
    o_lse, o_logp, _ = oracle.score_rows(oracle.decode(h, "bf16")[m], oracle.decode(W, "bf16"),
                                         b["tokens"][m])
    assert rel_err(host64(logp)[m], o_logp) <= BF16_TOL
    assert rel_err(host64(lse)[m], o_lse) <= BF16_TOL
    assert np.all(host64(logp)[~m] == 0) and np.all(host64(lse)[~m] == 0)


# ------------------------------------------------------------ closed forms on the device
def test_zero_weight_gives_log_vocab():
    N, H, V = 300, 64, 155136
    h = torch.randn(N, H, device="cuda").bfloat16()
    W = torch.zeros(V, H, device="cuda", dtype=torch.bfloat16)
    y = torch.randint(0, V, (N,), device="cuda")
    logp, lse = grpo.logprob_fwd(h, W, y)
    lnV = math.log(V)
    assert torch.all((lse - lnV).abs() <= 2e-6 * lnV)
    assert torch.all((logp + lnV).abs() <= 2e-6 * lnV)


def test_on_policy_and_equal_rewards_closed_forms():
    kw = dict(SMALL["ragged_tiles"], dtype="bf16", rms_norm_hidden=True, seed=15)
    w, W, h, b, adv, _, _ = _problem("fwdbwd_bf16", **kw)
    hd, Wd = to_dev(h, "bf16"), to_dev(W, "bf16")
    logp, _ = grpo.logprob_fwd(hd, Wd, dev(b["tokens"]), dev(b["mask"]))
    # old = ref = own logp: rho = 1, no clipping, kl = 0 -> ell = -A, loss = -(1/B) sum_b A_b
    out = grpo.loss_fwd_bwd(hd, Wd, dev(b["tokens"]), dev(b["mask"]), dev(b["cu_seqlens"]), logp,
                            logp, dev(adv), 0.2, 0.5)
    m = b["mask"].astype(bool)
    seq = np.repeat(np.arange(w.num_seqs), np.diff(b["cu_seqlens"]))
    assert np.all(out["clip_flag"].cpu().numpy() == 0)
    tl = out["token_loss"].cpu().numpy()
    np.testing.assert_allclose(tl[m], -adv[seq[m]], rtol=1e-6, atol=1e-7)
    assert abs(out["loss"].item() + adv[np.diff(b["cu_seqlens"]) > 0].sum() / w.num_seqs) < 1e-5
    # all-equal rewards and beta = 0: loss and gradients exactly zero
    zero = np.zeros_like(adv)
    out = grpo.loss_fwd_bwd(hd, Wd, dev(b["tokens"]), dev(b["mask"]), dev(b["cu_seqlens"]), logp,
                            None, dev(zero), 0.2, 0.0)
    assert out["loss"].item() == 0.0
    assert torch.all(out["grad_hidden"] == 0) and torch.all(out["grad_weight"] == 0)


def test_deterministic_bits():
    kw = dict(SMALL["multi_chunk"], dtype="bf16", rms_norm_hidden=True, seed=16)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    a = _run_loss(w, W, h, b, adv, old, ref)
    c = _run_loss(w, W, h, b, adv, old, ref)
    for k in ("loss", "logp", "lse", "dlogp", "grad_hidden", "grad_weight"):
        assert torch.equal(a[k], c[k]), k


@pytest.mark.parametrize("case", ["ragged_tiles", "multi_chunk", "k_tail"])
def test_tiled_weight_gives_the_same_bits(case):
    # grpo_tile_weight once, then every bf16 entry point given the tiled copy:
    # the same bits as the calls that tile W themselves, with the workspace
    # sized without the copy
    kw = dict(SMALL[case], dtype="bf16", rms_norm_hidden=True, beta=0.01, noise_sigma=0.1,
              seed=17)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    Wd, hd = to_dev(W, "bf16"), to_dev(h, "bf16")
    wt = grpo.tile_weight(Wd)
    grpo.free_workspace()
    a = grpo.logprob_fwd(hd, Wd, dev(b["tokens"]), dev(b["mask"]))
    c = grpo.logprob_fwd(hd, Wd, dev(b["tokens"]), dev(b["mask"]), weight_tiled=wt)
    assert torch.equal(a[0], c[0]) and torch.equal(a[1], c[1])
    a = _run_loss(w, W, h, b, adv, old, ref)
    c = _run_loss(w, W, h, b, adv, old, ref, weight_tiled=wt)
    for k in ("loss", "logp", "lse", "dlogp", "clip_flag", "grad_hidden", "grad_weight"):
        assert torch.equal(a[k], c[k]), k
    # the double-scoring path (lse_in): the gradients read the tiled copy
    lse = a["lse"]
    a = _run_loss(w, W, h, b, adv, old, ref, lse_in=lse)
    c = _run_loss(w, W, h, b, adv, old, ref, lse_in=lse, weight_tiled=wt)
    for k in ("loss", "logp", "grad_hidden", "grad_weight"):
        assert torch.equal(a[k], c[k]), k
    a = grpo.sft_ce_fwd_bwd(hd, Wd, dev(b["tokens"]), dev(b["mask"]))
    c = grpo.sft_ce_fwd_bwd(hd, Wd, dev(b["tokens"]), dev(b["mask"]), weight_tiled=wt)
    for k in ("loss", "logp", "grad_hidden", "grad_weight"):
        assert torch.equal(a[k], c[k]), k
    # a copy of another weight's shape is refused by the binding
    with pytest.raises(ValueError):
        grpo.logprob_fwd(hd, Wd[:-1].contiguous(), dev(b["tokens"]), weight_tiled=wt)


def test_side_stream_and_workspace_per_stream():
    # the binding launches on the caller's current stream, with a workspace of
    # that stream's own; a side stream gives the same bits as the default one
    kw = dict(SMALL["ragged_tiles"], dtype="bf16", rms_norm_hidden=True, seed=18)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    a = _run_loss(w, W, h, b, adv, old, ref)
    ws_default = grpo.workspace(1024)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        c = _run_loss(w, W, h, b, adv, old, ref)
        ws_side = grpo.workspace(1024)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert ws_side.data_ptr() != ws_default.data_ptr()
    assert grpo.workspace(512).data_ptr() == ws_default.data_ptr()
    for k in ("loss", "logp", "lse", "dlogp", "grad_hidden", "grad_weight"):
        assert torch.equal(a[k], c[k]), k


def test_hip_graph_capture_and_replay():
    # the compute entry points only launch kernels (no memset, copy or sync),
    # so a caller can capture them in a HIP graph; every replay, with eager
    # work and synchronisation between replays, must equal the eager result
    kw = dict(SMALL["ragged_tiles"], dtype="bf16", rms_norm_hidden=True, seed=23)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    args = (to_dev(h, w.dtype), to_dev(W, w.dtype), dev(b["tokens"]), dev(b["mask"]),
            dev(b["cu_seqlens"]), dev(old), dev(ref), dev(adv), w.clip_eps, w.beta)
    eager = grpo.loss_fwd_bwd(*args)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        out = grpo.loss_fwd_bwd(*args)
    for i in range(3):
        junk = torch.randn(1 << 20, device="cuda")
        junk.mul_(2.0).add_(1.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in ("loss", "logp", "lse", "token_loss", "dlogp", "clip_flag", "grad_hidden",
                  "grad_weight"):
            assert torch.equal(out[k], eager[k]), (i, k)
    del graph


def test_lse_in_reuse():
    kw = dict(SMALL["ragged_tiles"], dtype="bf16", rms_norm_hidden=True, seed=17)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    hd, Wd = to_dev(h, "bf16"), to_dev(W, "bf16")
    _, lse = grpo.logprob_fwd(hd, Wd, dev(b["tokens"]), dev(b["mask"]))
    a = _run_loss(w, W, h, b, adv, old, ref)
    c = _run_loss(w, W, h, b, adv, old, ref, lse_in=lse)
    torch.testing.assert_close(c["lse"], a["lse"], rtol=0, atol=0)
    torch.testing.assert_close(c["logp"], a["logp"], rtol=1e-5, atol=1e-5)
    torch.testing.assert_close(c["grad_weight"], a["grad_weight"], rtol=1e-2, atol=1e-6)


def test_token_out_of_range_sets_flag():
    w, W, h, b, adv, old, ref = _problem("tiny_fp32", seed=18)
    b["tokens"][7] = w.vocab  # one bad id
    with pytest.raises(grpo.GrpoError) as e:
        _run_loss(w, W, h, b, adv, old, ref)
    assert e.value.status == 9
    # the next call on the same workspace starts clean
    b["tokens"][7] = 0
    _run_loss(w, W, h, b, adv, old, ref)


def test_bf16_token_out_of_range_without_mask_zeroes_its_row():
    # a row whose id is outside [0, V) is dropped by packing even without a
    # mask: its dL/dh row is exactly 0 (as its logp and loss terms) and the
    # call reports the bad id
    kw = dict(SMALL["k_tail"], dtype="bf16", rms_norm_hidden=True, seed=19)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    b["tokens"][5] = w.vocab
    out = grpo.loss_fwd_bwd(to_dev(h, "bf16"), to_dev(W, "bf16"), dev(b["tokens"]), None,
                            dev(b["cu_seqlens"]), dev(old), dev(ref), dev(adv), w.clip_eps,
                            w.beta)
    torch.cuda.synchronize()
    assert torch.all(out["grad_hidden"][5] == 0)
    assert out["logp"][5].item() == 0 and out["token_loss"][5].item() == 0
    assert out["grad_hidden"][4].float().abs().sum().item() > 0
    with pytest.raises(grpo.GrpoError) as e:
        grpo.check_error(grpo.workspace(grpo.workspace_bytes(
            grpo.OP_LOSS_FWD_BWD, grpo.BF16, w.num_tokens, w.hidden, w.vocab, w.num_seqs)))
    assert e.value.status == 9


def test_all_rows_masked():
    """No valid row at all: loss, per-token outputs and both gradients are 0
    (the weight-gradient contraction then has K = 0)."""
    kw = dict(SMALL["ragged_tiles"], dtype="bf16", rms_norm_hidden=True, seed=19)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    b["mask"][:] = 0
    out = _run_loss(w, W, h, b, adv, old, ref)
    assert out["loss"].item() == 0.0
    assert torch.all(out["logp"] == 0) and torch.all(out["dlogp"] == 0)
    assert torch.all(out["grad_hidden"] == 0) and torch.all(out["grad_weight"] == 0)


# ------------------------------------------------------------ SFT cross-entropy
def _sft_problem(**kw):
    w = workloads.scaled(workloads.WORKLOADS["sft_bf16"], **kw)
    return w, workloads.make_weight(w), workloads.make_hidden(w), workloads.make_batch(w)


def _sft_compare(w, W, h, b, out, tol, grad_tol):
    o = oracle.sft_ce(oracle.decode(h, w.dtype), oracle.decode(W, w.dtype), b["tokens"],
                      b["mask"])
    m = b["mask"].astype(bool)
    torch.cuda.synchronize()
    assert abs(out["loss"].item() - o["loss"]) <= tol * max(abs(o["loss"]), 1e-30), \
        (out["loss"].item(), o["loss"])
    lp = host64(out["logp"])
    assert rel_err(lp[m], o["logp"][m]) <= tol
    assert np.all(lp[~m] == 0)
    dh, dW = host64(out["grad_hidden"]), host64(out["grad_weight"])
    if grad_tol is None:  # bf16: the rounding bound of the -g p entries of dz
        tol_dh, tol_dW = grad_tolerances(oracle.decode(h, w.dtype), oracle.decode(W, w.dtype),
                                         np.where(m, o["g"], 0.0), o["dh"], o["dW"])
        if out["grad_hidden"].dtype == torch.bfloat16:
            tol_dh += BF16_OUT
    else:
        tol_dh = tol_dW = grad_tol
    assert norm_rel(dh, o["dh"]) <= tol_dh, (norm_rel(dh, o["dh"]), tol_dh)
    assert norm_rel(dW, o["dW"]) <= tol_dW, (norm_rel(dW, o["dW"]), tol_dW)
    assert np.all(dh[~m] == 0)
    return o


SFT_SMALL = {
    # several tiles on every axis, ragged tails, a masked prompt prefix
    "tiles": dict(prompts=3, group=2, seq_len=90, hidden=320, vocab=3000, prompt_len=17,
                  ragged=True, min_len=20),
    # H not a multiple of 32, several vocabulary chunks
    "chunks": dict(prompts=1, group=2, seq_len=100, hidden=200, vocab=40000, prompt_len=30),
}


@pytest.mark.parametrize("case", list(SFT_SMALL))
def test_sft_bf16_parity(case):
    w, W, h, b = _sft_problem(**SFT_SMALL[case], seed=31)
    out = grpo.sft_ce_fwd_bwd(to_dev(h, "bf16"), to_dev(W, "bf16"), dev(b["tokens"]),
                              dev(b["mask"]), check=True)
    _sft_compare(w, W, h, b, out, BF16_TOL, BF16_GRAD_TOL)


def test_sft_fp32_parity():
    w, W, h, b = _sft_problem(seq_len=64, hidden=64, vocab=1000, prompt_len=9, dtype="f32",
                              rms_norm_hidden=False, seed=32)
    out = grpo.sft_ce_fwd_bwd(to_dev(h, "f32"), to_dev(W, "f32"), dev(b["tokens"]),
                              dev(b["mask"]), check=True)
    _sft_compare(w, W, h, b, out, F32_TOL, F32_TOL)


def test_sft_closed_forms():
    """W = 0 gives loss = ln V exactly up to fp32 and dh = 0; no supervised row
    gives loss 0 and zero gradients."""
    w, W, h, b = _sft_problem(**SFT_SMALL["tiles"], seed=33)
    Wz = torch.zeros(w.vocab, w.hidden, dtype=torch.bfloat16, device="cuda")
    out = grpo.sft_ce_fwd_bwd(to_dev(h, "bf16"), Wz, dev(b["tokens"]), dev(b["mask"]))
    assert out["loss"].item() == pytest.approx(math.log(w.vocab), rel=1e-6)
    assert out["grad_hidden"].abs().max().item() == 0.0
    none = torch.zeros(w.num_tokens, dtype=torch.uint8, device="cuda")
    out = grpo.sft_ce_fwd_bwd(to_dev(h, "bf16"), to_dev(W, "bf16"), dev(b["tokens"]), none)
    assert out["loss"].item() == 0.0
    assert out["grad_hidden"].abs().max().item() == 0.0
    assert out["grad_weight"].abs().max().item() == 0.0


# ------------------------------------------------------------ AdamW step
@pytest.mark.parametrize("n,lr,wd", [(1_000_003, 1e-6, 0.01), (4096, 1e-3, 0.1), (3, 1e-2, 0.0)])
def test_adamw_parity(n, lr, wd):
    """Three fused steps against the float64 oracle; the bf16 copy is the
    round-to-nearest-even of the kernel's own fp32 weight, bit for bit."""
    g = np.random.default_rng(n)
    w = (g.standard_normal(n) * 0.02).astype(np.float32)
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    wt, mt, vt = dev(w), dev(m), dev(v)
    wb = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    b1, b2, eps = 0.9, 0.999, 1e-8
    # the boundary takes fp32 hyper-parameters: the oracle gets the same values
    f = lambda x: float(np.float32(x))  # noqa: E731
    for step in (1, 2, 3):
        gr = (g.standard_normal(n) * 10.0 ** g.uniform(-4, 0)).astype(np.float32)
        w_in, m_in, v_in = host64(wt), host64(mt), host64(vt)
        grpo.adamw_step(wt, mt, vt, dev(gr), step, lr, b1, b2, eps, wd,
                        weight_bf16=wb if step != 2 else None)
        torch.cuda.synchronize()
        ow, om, ov = oracle.adamw(w_in, m_in, v_in, gr, step, f(lr), f(b1), f(b2), f(eps), f(wd))
        kw, km, kv = host64(wt), host64(mt), host64(vt)
        # the first moment is a sum that can cancel: measure against its terms
        scale_m = f(b1) * np.abs(m_in) + (1 - f(b1)) * np.abs(gr.astype(np.float64))
        assert np.all(np.abs(km - om) <= 2e-6 * scale_m + 1e-37)
        np.testing.assert_allclose(kv, ov, rtol=2e-6, atol=1e-37)
        # the new fp32 weight is within about one fp32 spacing of the exact one
        # plus 1e-5 of the step (with lr = 1e-6 the step itself is close to
        # that spacing, so a relative check of the weight is the right scale)
        ulp = np.spacing(np.abs(ow).astype(np.float32)).astype(np.float64)
        assert np.all(np.abs(kw - ow) <= 1.5 * ulp + 1e-5 * np.abs(ow - w_in))
        if step != 2:
            want = workloads.bf16_bits(wt.cpu().numpy())
            got = wb.view(torch.int16).cpu().numpy().view(np.uint16)
            assert np.array_equal(got, want)



# ------------------------------------------------------------ workspace bounds
# ragged rows, several vocabulary tiles, H over two gradient tile-columns
BUDGET_CASE = dict(prompts=3, group=4, seq_len=50, hidden=320, vocab=40000, ragged=True,
                   min_len=1, forced_equal_groups=1)


def test_bf16_max_valid_and_small_budgets():
    # The logits-gradient budget sets the vocabulary chunk width, how many
    # chunks one dL/dh product takes (so the passes over the fp32 dL/dh
    # accumulator) and the dL/dW K splits; max_valid sizes the token-indexed
    # buffers. Each combination against the full oracle; the same arguments
    # give the same bits.
    kw = dict(BUDGET_CASE, dtype="bf16", rms_norm_hidden=True, beta=0.01, noise_sigma=0.1,
              seed=31)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    nv = int(b["mask"].sum())
    for max_valid in (0, nv):
        rows = -(-(w.num_tokens if max_valid == 0 else nv) // 256) * 256
        for cols in (256, 768, 2560, 8192):  # dz columns the budget holds
            budget = 2 * rows * cols
            out = _run_loss(w, W, h, b, adv, old, ref, max_valid=max_valid, dz_budget=budget)
            _compare_loss(w, W, h, b, adv, old, ref, out, BF16_TOL, BF16_GRAD_TOL)
    again = _run_loss(w, W, h, b, adv, old, ref, max_valid=nv, dz_budget=2 * rows * 768)
    first = _run_loss(w, W, h, b, adv, old, ref, max_valid=nv, dz_budget=2 * rows * 768)
    for k in ("loss", "logp", "grad_hidden", "grad_weight"):
        assert torch.equal(again[k].view(torch.uint8), first[k].view(torch.uint8)), k


def test_capacity_error_leaves_outputs_as_for_masked_rows():
    kw = dict(BUDGET_CASE, dtype="bf16", rms_norm_hidden=True, beta=0.01, seed=32)
    w, W, h, b, adv, old, ref = _problem("fwdbwd_bf16", **kw)
    nv = int(b["mask"].sum())
    assert nv > 256  # a max_valid of 200 gives a capacity of 256 rows
    with pytest.raises(grpo.GrpoError) as e:
        _run_loss(w, W, h, b, adv, old, ref, max_valid=200)
    assert e.value.status == 11
    out = grpo.loss_fwd_bwd(to_dev(h, w.dtype), to_dev(W, w.dtype), dev(b["tokens"]),
                            dev(b["mask"]), dev(b["cu_seqlens"]), dev(old), dev(ref), dev(adv),
                            w.clip_eps, w.beta, 0, check=False, max_valid=200)
    torch.cuda.synchronize()
    for k in ("loss", "logp", "lse", "token_loss", "dlogp", "grad_hidden", "grad_weight"):
        assert torch.count_nonzero(out[k]).item() == 0, k
    # the next call on the same workspace starts clean
    _run_loss(w, W, h, b, adv, old, ref, max_valid=nv)
