"""Parity at the benchmark's full sizes (H=4096, V=155136), in the launch
configuration bench.py times. GPU only.

* scoring workload (4 prompts x G=8 x 1024 tokens, N=32768): sampled rows'
  logp and lse against the oracle, a bound on every row.
* fwd+bwd workload (8 prompts x G=8 x 2048 tokens, N=131072): per-token
  outputs (logp, lse, ell, dL/dlogp, dL/dh rows) of a seeded sample of rows
  against the oracle, which scores each sampled row over the whole
  vocabulary; dL/dW through identities that hold at any size.
* reduced N (256 tokens) at full H and V: dL/dW rows against the oracle.
* ragged rollouts with all-equal reward groups, and the two-model
  (policy + reference) scoring sequence, at reduced sizes.
* the SFT cross-entropy workload (one 16384-token sequence, prompt prefix
  unsupervised): sampled rows' logp and dL/dh rows, the loss from the
  per-token log-probs, and the dL/dW identities.
* the ragged workload at full size (1,048,576 padded rows): sampled rows,
  masked rows, the dL/dW identities; the double-scoring workload at full size
  (N = 262144): both scorings and the loss terms of sampled rows.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2507_05687_amd import grpo, workloads
from tests.gpu_util import (BF16_OUT, dev, grad_tolerances, host64, norm_rel, rel_err,
                            rounding_bounds, row_tolerances, to_dev)

pytestmark = pytest.mark.gpu

TOL = 2e-3
# dL/dW and dL/dh: within the bound that bf16 rounding of the -g p entries of
# dz implies (tests.gpu_util), plus 2^-9 for the bf16 dL/dh output; at these
# shapes (V = 155136, logit std 1.3) the bound is about 1e-4


@pytest.fixture(scope="module", autouse=True)
def _setup():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    oracle.build(force=False)
    grpo.load()
    yield
    grpo.free_workspace()
    torch.cuda.empty_cache()


def _seq_weights(batch, B):
    m = batch["mask"]
    cu = batch["cu_seqlens"]
    counts = np.array([m[cu[b]:cu[b + 1]].sum() for b in range(B)])
    return oracle.seq_weights(counts), np.repeat(np.arange(B), np.diff(cu))


def test_fwdbwd_full_size_sampled_rows_and_identities():
    w = workloads.WORKLOADS["fwdbwd_bf16"]
    W_bits = workloads.make_weight(w)
    h_bits = workloads.make_hidden(w)
    b = workloads.make_batch(w)
    N, H, V, B = w.num_tokens, w.hidden, w.vocab, w.num_seqs
    rows = workloads.sample_rows(b["mask"], 24, seed=1)
    Wd = oracle.decode(W_bits, "bf16")
    hs = oracle.decode(h_bits[rows], "bf16")
    o_lse, o_logp, _ = oracle.score_rows(hs, Wd, b["tokens"][rows])
    # old/ref: for sampled rows the oracle's log-prob plus noise; for the
    # others a constant base plus noise (those rows are checked only through
    # identities, so their exact ratio does not matter)
    base = np.full(N, -math.log(V))
    base[rows] = o_logp
    old = (base + b["old_noise"]).astype(np.float32)
    ref = (base + b["ref_noise"]).astype(np.float32)
    adv = oracle.advantages(b["rewards"], w.group).astype(np.float32)

    hd, Wdv = to_dev(h_bits, "bf16"), to_dev(W_bits, "bf16")
    out = grpo.loss_fwd_bwd(hd, Wdv, dev(b["tokens"]), None, dev(b["cu_seqlens"]), dev(old),
                            dev(ref), dev(adv), w.clip_eps, w.beta, check=True)
    torch.cuda.synchronize()

    # per-token outputs of the sampled rows
    c, seq = _seq_weights(b, B)
    o_ell, o_g, _ = oracle.token_objective(o_logp, old[rows], ref[rows], adv[seq[rows]],
                                           c[seq[rows]], None, w.clip_eps, w.beta)
    assert rel_err(host64(out["logp"])[rows], o_logp) <= TOL
    assert rel_err(host64(out["lse"])[rows], o_lse) <= TOL
    tl = host64(out["token_loss"])[rows]
    assert np.max(np.abs(tl - o_ell)) <= TOL * max(1.0, np.max(np.abs(o_ell)))
    g = host64(out["dlogp"])[rows]
    assert np.max(np.abs(g - o_g)) <= TOL * np.max(np.abs(o_g))
    o_dh = oracle.grad_hidden_rows(hs, Wd, b["tokens"][rows], o_lse, o_g)
    dh = host64(out["grad_hidden"][torch.from_numpy(rows).cuda()])
    tols = row_tolerances(rounding_bounds(hs, Wd, o_g, vrows=[])[0], o_dh) + BF16_OUT
    for i in range(len(rows)):
        assert norm_rel(dh[i], o_dh[i]) <= tols[i], (i, norm_rel(dh[i], o_dh[i]), tols[i])
    del Wd

    # the loss is the weighted sum of the per-token terms it also returns
    c_t = torch.from_numpy(c[seq]).cuda()
    want = float((out["token_loss"].double() * c_t).sum())
    scale = float((out["token_loss"].double().abs() * c_t).sum())
    assert abs(out["loss"].item() - want) <= 1e-5 * scale

    _grad_weight_identities(out, hd, Wdv)


def _grad_weight_identities(out, hd, Wdv, dlogp=None):
    """Identities of dL/dW that hold at any size:
    * sum_v dL/dW_v = sum_t h_t g_t (1 - sum_v p_tv) = 0, up to the bf16
      rounding of the -g p entries of dz (the +g of the sampled id is exact):
      |.| <= 2^-9 sum_t |h_t| |g_t|, checked at 2^-8;
    * <dW, W> = <dh, h> = sum_{t,v} dz_tv z_tv (the same dz on both sides),
      up to fp32 accumulation and the bf16 rounding of a bf16 dL/dh: this
      sum nearly cancels (on policy it is close to 0), so it is checked
      against 2^-8 sum |dh| |h| (the rounding bound, doubled) and 1e-4 of
      its own size."""
    gw = out["grad_weight"]
    gt = (out["dlogp"] if dlogp is None else dlogp).double()
    hf = hd.double()
    colsum = gw.double().sum(0)
    bound = 2.0 ** -8 * (hf.abs() * gt.abs()[:, None]).sum(0) + 1e-7
    assert torch.all(colsum.abs() <= bound), float((colsum.abs() / bound).max())
    a = float((gw.double() * Wdv.double()).sum())
    dhf = out["grad_hidden"].double()
    bb = float((dhf * hf).sum())
    scale = float((dhf.abs() * hf.abs()).sum())
    assert abs(a - bb) <= 2.0 ** -8 * scale + 1e-4 * max(abs(a), abs(bb)), (a, bb, scale)
    assert torch.isfinite(gw).all() and torch.isfinite(out["grad_hidden"].float()).all()


def test_fwd_full_size_sampled_rows_and_bounds():
    # log-prob scoring alone (4 prompts x G = 8 x 1024 tokens, N = 32768),
    # through grpo_logprob_fwd without a mask, as bench.py's fwd workload
    w = workloads.WORKLOADS["fwd_bf16"]
    W_bits = workloads.make_weight(w)
    h_bits = workloads.make_hidden(w)
    b = workloads.make_batch(w)
    V = w.vocab
    rows = workloads.sample_rows(b["mask"], 24, seed=2)
    Wd = oracle.decode(W_bits, "bf16")
    hs = oracle.decode(h_bits[rows], "bf16")
    o_lse, o_logp, _ = oracle.score_rows(hs, Wd, b["tokens"][rows])
    del Wd
    hd, Wdv = to_dev(h_bits, "bf16"), to_dev(W_bits, "bf16")
    logp, lse = grpo.logprob_fwd(hd, Wdv, dev(b["tokens"]), None, check=True)
    torch.cuda.synchronize()
    assert rel_err(host64(logp)[rows], o_logp) <= TOL
    assert rel_err(host64(lse)[rows], o_lse) <= TOL
    # every row: a log-probability (< 0 with V = 155136 comparable logits),
    # and Jensen's bound log sum_v e^z_v >= ln V + mean_v z_v = ln V + <h, mean_v W_v>
    lp, ls = host64(logp), host64(lse)
    assert np.all(np.isfinite(lp)) and np.all(np.isfinite(ls)) and np.all(lp < 0)
    zbar = (hd.double() @ Wdv.double().mean(0)).cpu().numpy()
    assert np.all(ls >= math.log(V) + zbar - 1e-3 * np.abs(ls))


def test_reduced_tokens_full_vocab_grad_weight_rows():
    w = workloads.scaled(workloads.WORKLOADS["fwdbwd_bf16"], prompts=1, group=4, seq_len=64,
                         seed=21)
    W_bits = workloads.make_weight(w)
    h_bits = workloads.make_hidden(w)
    b = workloads.make_batch(w)
    Wd, hd64 = oracle.decode(W_bits, "bf16"), oracle.decode(h_bits, "bf16")
    o_lse, o_logp, _ = oracle.score_rows(hd64, Wd, b["tokens"])
    old = (o_logp + b["old_noise"]).astype(np.float32)
    ref = (o_logp + b["ref_noise"]).astype(np.float32)
    adv = oracle.advantages(b["rewards"], w.group).astype(np.float32)
    out = grpo.loss_fwd_bwd(to_dev(h_bits, "bf16"), to_dev(W_bits, "bf16"), dev(b["tokens"]),
                            dev(b["mask"]), dev(b["cu_seqlens"]), dev(old), dev(ref), dev(adv),
                            w.clip_eps, w.beta, check=True)
    c, seq = _seq_weights(b, w.num_seqs)
    o_ell, o_g, _ = oracle.token_objective(o_logp, old, ref, adv[seq], c[seq], None, w.clip_eps,
                                           w.beta)
    assert rel_err(host64(out["logp"]), o_logp) <= TOL
    abs_sum = float(np.sum(c[seq] * np.abs(o_ell)))
    assert abs(out["loss"].item() - float(np.sum(c[seq] * o_ell))) <= TOL * abs_sum
    g = np.random.default_rng(3)
    vrows = np.unique(np.concatenate([b["tokens"][:16], g.integers(0, w.vocab, 32),
                                      [0, w.vocab - 1]]))
    o_dW = oracle.grad_weight_rows(hd64, Wd, b["tokens"], o_lse, o_g, vrows)
    dW = host64(out["grad_weight"][torch.from_numpy(vrows).cuda()])
    m = b["mask"].astype(bool)
    _, dW_b = rounding_bounds(hd64, Wd, np.where(m, o_g, 0.0), vrows=vrows)
    tols = row_tolerances(dW_b, o_dW)
    assert norm_rel(dW, o_dW) <= tols.max(), norm_rel(dW, o_dW)
    for i in range(len(vrows)):
        assert norm_rel(dW[i], o_dW[i]) <= tols[i], (vrows[i], norm_rel(dW[i], o_dW[i]), tols[i])


def test_ragged_equal_groups_zero_gradient():
    """Ragged rollouts; groups whose rewards are all equal get A = 0, so with
    beta = 0 their tokens contribute nothing: dL/dlogp and dL/dh are exactly 0."""
    w = workloads.scaled(workloads.WORKLOADS["ragged_bf16"], prompts=4, group=4, seq_len=300,
                         hidden=256, vocab=5000, min_len=16, forced_equal_groups=2, beta=0.0,
                         seed=31)
    W_bits, h_bits, b = workloads.make_weight(w), workloads.make_hidden(w), workloads.make_batch(w)
    adv_dev = grpo.group_advantages(dev(b["rewards"]), w.group)
    adv = adv_dev.cpu().numpy()
    assert np.all(adv[:2 * w.group] == 0)
    hd64, Wd = oracle.decode(h_bits, "bf16"), oracle.decode(W_bits, "bf16")
    _, o_logp, _ = oracle.score_rows(hd64, Wd, b["tokens"])
    old = (o_logp + b["old_noise"]).astype(np.float32)
    out = grpo.loss_fwd_bwd(to_dev(h_bits, "bf16"), to_dev(W_bits, "bf16"), dev(b["tokens"]),
                            dev(b["mask"]), dev(b["cu_seqlens"]), dev(old), None, adv_dev,
                            w.clip_eps, 0.0, check=True)
    eq_rows = np.arange(b["cu_seqlens"][2 * w.group])
    assert np.all(out["dlogp"].cpu().numpy()[eq_rows] == 0)
    assert torch.all(out["grad_hidden"][:len(eq_rows)] == 0)
    o = oracle.grpo_loss(hd64, Wd, b["tokens"], b["mask"], b["cu_seqlens"], old.astype(np.float64),
                         old.astype(np.float64), adv.astype(np.float64), w.clip_eps, 0.0)
    tol_dh, tol_dW = grad_tolerances(hd64, Wd, np.where(b["mask"].astype(bool), o["g"], 0.0),
                                     o["dh"], o["dW"])
    assert norm_rel(host64(out["grad_weight"]), o["dW"]) <= tol_dW
    assert norm_rel(host64(out["grad_hidden"]), o["dh"]) <= tol_dh + BF16_OUT


def test_double_scoring_sequence():
    """Policy and reference scoring, then the loss on the policy reusing the
    policy's log-sum-exp (the two-model GRPO step), at reduced size."""
    w = workloads.scaled(workloads.WORKLOADS["double_bf16"], prompts=2, group=4, seq_len=64,
                         hidden=512, vocab=6000, seed=41)
    Wp, Wr = workloads.make_weight(w, "policy"), workloads.make_weight(w, "reference")
    h_bits, b = workloads.make_hidden(w), workloads.make_batch(w)
    hd = to_dev(h_bits, "bf16")
    Wpd, Wrd = to_dev(Wp, "bf16"), to_dev(Wr, "bf16")
    y = dev(b["tokens"])
    lp_pol, lse_pol = grpo.logprob_fwd(hd, Wpd, y)
    lp_ref, _ = grpo.logprob_fwd(hd, Wrd, y)
    h64 = oracle.decode(h_bits, "bf16")
    o_lse_p, o_lp_p, _ = oracle.score_rows(h64, oracle.decode(Wp, "bf16"), b["tokens"])
    _, o_lp_r, _ = oracle.score_rows(h64, oracle.decode(Wr, "bf16"), b["tokens"])
    assert rel_err(host64(lp_pol), o_lp_p) <= TOL
    assert rel_err(host64(lp_ref), o_lp_r) <= TOL
    # the loss step takes old = policy log-prob and ref = reference log-prob
    old, ref = o_lp_p.astype(np.float32), o_lp_r.astype(np.float32)
    adv = oracle.advantages(b["rewards"], w.group).astype(np.float32)
    out = grpo.loss_fwd_bwd(hd, Wpd, y, None, dev(b["cu_seqlens"]), dev(old), dev(ref), dev(adv),
                            w.clip_eps, w.beta, lse_in=lse_pol, check=True)
    o = oracle.grpo_loss(h64, oracle.decode(Wp, "bf16"), b["tokens"], None, b["cu_seqlens"],
                         old.astype(np.float64), ref.astype(np.float64), adv.astype(np.float64),
                         w.clip_eps, w.beta)
    assert rel_err(host64(out["logp"]), o["logp"]) <= TOL
    c, seq = _seq_weights(b, w.num_seqs)
    abs_sum = float(np.sum(c[seq] * np.abs(o["ell"])))
    assert abs(out["loss"].item() - o["loss"]) <= TOL * max(abs(o["loss"]), abs_sum)
    tol_dh, tol_dW = grad_tolerances(h64, oracle.decode(Wp, "bf16"), o["g"], o["dh"], o["dW"])
    assert norm_rel(host64(out["grad_weight"]), o["dW"]) <= tol_dW
    assert norm_rel(host64(out["grad_hidden"]), o["dh"]) <= tol_dh + BF16_OUT
    # on policy: rho = exp(logp - old) is 1 up to the difference between the
    # device's and the oracle's log-prob
    rho = np.exp(host64(out["logp"]) - old)
    assert np.max(np.abs(rho - 1)) <= 1e-3


def test_sft_full_size_sampled_rows_and_identities():
    w = workloads.WORKLOADS["sft_bf16"]
    W_bits = workloads.make_weight(w)
    h_bits = workloads.make_hidden(w)
    b = workloads.make_batch(w)
    n_valid = int(b["mask"].sum())
    rows = workloads.sample_rows(b["mask"], 16, seed=2)
    Wd = oracle.decode(W_bits, "bf16")
    hs = oracle.decode(h_bits[rows], "bf16")
    o_lse, o_logp, _ = oracle.score_rows(hs, Wd, b["tokens"][rows])
    hd, Wdv = to_dev(h_bits, "bf16"), to_dev(W_bits, "bf16")
    mask = dev(b["mask"])
    out = grpo.sft_ce_fwd_bwd(hd, Wdv, dev(b["tokens"]), mask, check=True)
    torch.cuda.synchronize()
    assert rel_err(host64(out["logp"])[rows], o_logp) <= TOL
    g_rows = np.full(len(rows), -1.0 / n_valid)
    o_dh = oracle.grad_hidden_rows(hs, Wd, b["tokens"][rows], o_lse, g_rows)
    dh = host64(out["grad_hidden"][torch.from_numpy(rows).cuda()])
    tols = row_tolerances(rounding_bounds(hs, Wd, g_rows, vrows=[])[0], o_dh) + BF16_OUT
    for i in range(len(rows)):
        assert norm_rel(dh[i], o_dh[i]) <= tols[i], (i, norm_rel(dh[i], o_dh[i]), tols[i])
    del Wd
    # masked rows: zero log-prob and gradient
    m = mask.bool()
    assert out["logp"][~m].abs().max().item() == 0.0
    assert out["grad_hidden"][~m].float().abs().max().item() == 0.0
    # the loss is minus the mean of the per-token log-probs it also returns
    want = -float(out["logp"].double().sum()) / n_valid
    assert abs(out["loss"].item() - want) <= 1e-5 * abs(want)
    # dL/dW identities (as for the GRPO loss, with g_t = -1/n on valid rows)
    _grad_weight_identities(out, hd, Wdv, dlogp=-m.double() / n_valid)



@pytest.mark.timeout(600)
def test_ragged_full_size_sampled_rows_and_identities():
    """The ragged workload at full size (16 x 8 rollouts of 256..8192 tokens
    padded to 8192, 1,048,576 rows): the batch's narrow vocabulary chunks take
    the column-split tile mapping and the split-K dL/dW product."""
    w = workloads.WORKLOADS["ragged_bf16"]
    W_bits = workloads.make_weight(w)
    h_bits = workloads.make_hidden(w)
    b = workloads.make_batch(w)
    N, V, B = w.num_tokens, w.vocab, w.num_seqs
    m = b["mask"]
    rows = workloads.sample_rows(m, 16, seed=3)
    Wd = oracle.decode(W_bits, "bf16")
    hs = oracle.decode(h_bits[rows], "bf16")
    o_lse, o_logp, _ = oracle.score_rows(hs, Wd, b["tokens"][rows])
    base = np.full(N, -math.log(V))
    base[rows] = o_logp
    old = (base + b["old_noise"]).astype(np.float32)
    ref = (base + b["ref_noise"]).astype(np.float32)
    adv = oracle.advantages(b["rewards"], w.group).astype(np.float32)
    hd, Wdv = to_dev(h_bits, "bf16"), to_dev(W_bits, "bf16")
    del h_bits
    mask_d = dev(m)
    out = grpo.loss_fwd_bwd(hd, Wdv, dev(b["tokens"]), mask_d, dev(b["cu_seqlens"]), dev(old),
                            dev(ref), dev(adv), w.clip_eps, w.beta, check=True)
    torch.cuda.synchronize()
    c, seq = _seq_weights(b, B)
    o_ell, o_g, _ = oracle.token_objective(o_logp, old[rows], ref[rows], adv[seq[rows]],
                                           c[seq[rows]], None, w.clip_eps, w.beta)
    assert rel_err(host64(out["logp"])[rows], o_logp) <= TOL
    g = host64(out["dlogp"])[rows]
    assert np.max(np.abs(g - o_g)) <= TOL * np.max(np.abs(o_g))
    o_dh = oracle.grad_hidden_rows(hs, Wd, b["tokens"][rows], o_lse, o_g)
    dh = host64(out["grad_hidden"][torch.from_numpy(rows).cuda()])
    tols = row_tolerances(rounding_bounds(hs, Wd, o_g, vrows=[])[0], o_dh) + BF16_OUT
    for i in range(len(rows)):
        if np.linalg.norm(o_dh[i]) > 0:  # rows of all-equal groups have g = 0
            assert norm_rel(dh[i], o_dh[i]) <= tols[i], (i, norm_rel(dh[i], o_dh[i]), tols[i])
    del Wd
    mb = mask_d.bool()
    assert out["logp"][~mb].abs().max().item() == 0.0
    assert out["grad_hidden"][~mb].float().abs().max().item() == 0.0
    # dL/dW identities, as for the fwd+bwd workload (sums over rows in slices)
    gw = out["grad_weight"]
    gt = out["dlogp"].double()
    colsum = gw.double().sum(0)
    bound = torch.zeros_like(colsum)
    bb = scale = 0.0
    for r0 in range(0, N, 1 << 16):
        hc = hd[r0:r0 + (1 << 16)].double()
        dhc = out["grad_hidden"][r0:r0 + (1 << 16)].double()
        bound += (hc.abs() * gt[r0:r0 + (1 << 16)].abs()[:, None]).sum(0)
        bb += float((dhc * hc).sum())
        scale += float((dhc.abs() * hc.abs()).sum())
    bound = 2.0 ** -8 * bound + 1e-7
    assert torch.all(colsum.abs() <= bound), float((colsum.abs() / bound).max())
    a = float((gw.double() * Wdv.double()).sum())
    assert abs(a - bb) <= 2.0 ** -8 * scale + 1e-4 * max(abs(a), abs(bb)), (a, bb, scale)
    assert torch.isfinite(gw).all()


@pytest.mark.timeout(600)
def test_double_scoring_full_size_sampled_rows():
    """The two-model sequence at full size (16 x 8 x 2048 tokens, N = 262144):
    policy and reference scoring, then the loss on the policy reusing its
    log-sum-exp; sampled rows against the oracle and the on-policy ratio. As
    bench.py runs it, each W is tiled once (grpo_tile_weight) and every call
    reads the tiled copy."""
    w = workloads.WORKLOADS["double_bf16"]
    Wp, Wr = workloads.make_weight(w, "policy"), workloads.make_weight(w, "reference")
    h_bits, b = workloads.make_hidden(w), workloads.make_batch(w)
    rows = workloads.sample_rows(b["mask"], 12, seed=4)
    hs = oracle.decode(h_bits[rows], "bf16")
    hd = to_dev(h_bits, "bf16")
    del h_bits
    Wpd, Wrd = to_dev(Wp, "bf16"), to_dev(Wr, "bf16")
    y = dev(b["tokens"])
    wt_pol, wt_ref = grpo.tile_weight(Wpd), grpo.tile_weight(Wrd)
    lp_pol, lse_pol = grpo.logprob_fwd(hd, Wpd, y, weight_tiled=wt_pol)
    lp_ref, _ = grpo.logprob_fwd(hd, Wrd, y, weight_tiled=wt_ref)
    del wt_ref
    Wpo = oracle.decode(Wp, "bf16")
    o_lse_p, o_lp_p, _ = oracle.score_rows(hs, Wpo, b["tokens"][rows])
    _, o_lp_r, _ = oracle.score_rows(hs, oracle.decode(Wr, "bf16"), b["tokens"][rows])
    assert rel_err(host64(lp_pol)[rows], o_lp_p) <= TOL
    assert rel_err(host64(lp_ref)[rows], o_lp_r) <= TOL
    adv = oracle.advantages(b["rewards"], w.group).astype(np.float32)
    out = grpo.loss_fwd_bwd(hd, Wpd, y, None, dev(b["cu_seqlens"]), lp_pol, lp_ref, dev(adv),
                            w.clip_eps, w.beta, lse_in=lse_pol, check=True, weight_tiled=wt_pol)
    torch.cuda.synchronize()
    del wt_pol
    # on policy: old = the policy's own log-prob, so rho = 1 up to the
    # difference between the gathered z_y of the two calls (the reused-lse
    # path takes z_y from a dot product, the scoring call from its GEMM)
    rho = torch.exp(out["logp"].double() - lp_pol.double())
    assert float((rho - 1).abs().max()) <= 1e-3
    c, seq = _seq_weights(b, w.num_seqs)
    o_ell, o_g, _ = oracle.token_objective(o_lp_p, o_lp_p, o_lp_r, adv[seq[rows]],
                                           c[seq[rows]], None, w.clip_eps, w.beta)
    g = host64(out["dlogp"])[rows]
    assert np.max(np.abs(g - o_g)) <= TOL * np.max(np.abs(o_g))
    o_dh = oracle.grad_hidden_rows(hs, Wpo, b["tokens"][rows], o_lse_p, o_g)
    dh = host64(out["grad_hidden"][torch.from_numpy(rows).cuda()])
    tols = row_tolerances(rounding_bounds(hs, Wpo, o_g, vrows=[])[0], o_dh) + BF16_OUT
    for i in range(len(rows)):
        assert norm_rel(dh[i], o_dh[i]) <= tols[i], (i, norm_rel(dh[i], o_dh[i]), tols[i])
    del Wpo
    # dL/dW identities, as for the fwd+bwd workload
    _grad_weight_identities(out, hd, Wpd)
