"""Pins for the CPU oracle: checks against closed forms, invariants, library
routines, brute force and finite differences -- never against the oracle itself.

Each test names the part of AutoTriton Sec. 3.3 it pins (Eq. 1 objective,
Eq. 2 advantage). CPU only.
"""
import math
import os

import numpy as np
import pytest
import scipy.stats
import torch

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([float(x) for x in line.split()])
    return rows


def _rand_problem(seed, B=6, T=5, H=7, V=11, ragged=False, scale=0.5):
    g = np.random.default_rng(seed)
    N = B * T
    h = g.standard_normal((N, H))
    W = g.standard_normal((V, H)) * scale
    y = g.integers(0, V, N)
    cu = np.arange(B + 1) * T
    if ragged:
        lens = g.integers(1, T + 1, B)
        mask = (np.arange(T)[None, :] < lens[:, None]).astype(np.uint8).reshape(N)
    else:
        mask = np.ones(N, np.uint8)
    return h, W, y, mask, cu


# ------------------------------------------------------------------ Eq. 2
def test_advantages_worked_example(oracle_lib):
    """Eq. 2 on rewards {0,0,1,1}; hand-computed values in golden/advantages_worked.txt."""
    for row in _golden_rows("advantages_worked.txt"):
        unbiased, eps = bool(row[0]), row[1]
        r, want = np.array(row[2:6]), np.array(row[6:10])
        got = oracle_lib.advantages(r, 4, std_eps=eps, unbiased=unbiased)
        np.testing.assert_allclose(got, want, rtol=1e-14, atol=0)


def test_advantages_match_scipy_zscore(oracle_lib):
    """Eq. 2 with eps = 0 is the z-score within each group (scipy routine)."""
    g = np.random.default_rng(1)
    for G, ddof in [(4, 1), (8, 1), (8, 0), (16, 1)]:
        r = g.random(G * 5)
        got = oracle_lib.advantages(r, G, std_eps=0.0, unbiased=(ddof == 1))
        want = scipy.stats.zscore(r.reshape(5, G), axis=1, ddof=ddof).reshape(-1)
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


def test_advantages_equal_group_exact_zero(oracle_lib):
    """An all-equal group must give exactly 0, even where the computed mean of
    identical values differs from them by rounding (0.1 summed 7 times)."""
    r = np.concatenate([np.full(7, 0.1), [0.0, 1.0, 0.5, 0.5, 1.0, 0.0, 0.1],
                        np.full(7, 1.0)])
    a = oracle_lib.advantages(r, 7)
    assert np.all(a[:7] == 0.0) and np.all(a[14:] == 0.0)
    assert np.all(a[7:14] != 0.0) or np.count_nonzero(a[7:14]) >= 5
    # the naive formula would not give zero here: mean(0.1 x7) != 0.1 in double
    assert sum([0.1] * 7) / 7 != 0.1


def test_advantages_sum_to_zero_and_unit_scale(oracle_lib):
    g = np.random.default_rng(2)
    r = g.random(8 * 50)
    a = oracle_lib.advantages(r, 8, std_eps=0.0).reshape(50, 8)
    np.testing.assert_allclose(a.sum(axis=1), 0.0, atol=1e-12)
    np.testing.assert_allclose((a * a).sum(axis=1) / 7, 1.0, rtol=1e-12)


# ------------------------------------------------------- |o_i| and packing
def test_pack_valid_brute_force(oracle_lib):
    g = np.random.default_rng(3)
    B, T = 9, 13
    mask = (g.random(B * T) < 0.6).astype(np.uint8)
    mask[2 * T:3 * T] = 0  # an empty rollout
    cu = np.arange(B + 1) * T
    rows, counts, seq = oracle_lib.pack_valid(mask, cu)
    want_rows = [t for t in range(B * T) if mask[t]]
    want_counts = [int(mask[b * T:(b + 1) * T].sum()) for b in range(B)]
    assert rows.tolist() == want_rows
    assert counts.tolist() == want_counts
    assert seq.tolist() == [t // T for t in range(B * T)]


def test_seq_weights_closed_form(oracle_lib):
    counts = np.array([3, 5, 0, 8])
    c = oracle_lib.seq_weights(counts, agg=0)
    np.testing.assert_allclose(c, [1 / 12, 1 / 20, 0.0, 1 / 32], rtol=1e-15)
    c1 = oracle_lib.seq_weights(counts, agg=1)
    np.testing.assert_allclose(c1, [1 / 16, 1 / 16, 0.0, 1 / 16], rtol=1e-15)


# ------------------------------------------------- log-softmax and gather
def test_score_rows_match_torch_log_softmax(oracle_lib):
    h, W, y, _, _ = _rand_problem(4, H=16, V=50, scale=1.0)
    lse, logp, zy = oracle_lib.score_rows(h, W, y)
    z = torch.from_numpy(h) @ torch.from_numpy(W).T
    want = torch.log_softmax(z, dim=1)
    np.testing.assert_allclose(logp, want[torch.arange(len(y)), torch.from_numpy(y)].numpy(),
                               rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(lse, torch.logsumexp(z, 1).numpy(), rtol=1e-13)
    np.testing.assert_allclose(zy, z[torch.arange(len(y)), torch.from_numpy(y)].numpy(),
                               rtol=1e-13, atol=1e-13)


def test_zero_weight_gives_log_vocab(oracle_lib):
    for V, lnV in _golden_rows("logsumexp_closed_forms.txt")[:2]:
        V = int(V)
        h = np.random.default_rng(5).standard_normal((3, 4))
        W = np.zeros((V, 4))
        lse, logp, _ = oracle_lib.score_rows(h, W, np.array([0, V // 2, V - 1]))
        np.testing.assert_allclose(lse, lnV, rtol=1e-15)
        np.testing.assert_allclose(logp, -lnV, rtol=1e-15)


def test_lse_shift_invariance_and_bounds(oracle_lib):
    h, W, y, _, _ = _rand_problem(6, H=9, V=40, scale=2.0)
    lse, logp, _ = oracle_lib.score_rows(h, W, y)
    u = np.random.default_rng(7).standard_normal(9)
    lse2, logp2, _ = oracle_lib.score_rows(h, W + u[None, :], y)
    np.testing.assert_allclose(lse2, lse + h @ u, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(logp2, logp, rtol=1e-10, atol=1e-11)
    zmax = (h @ W.T).max(axis=1)
    assert np.all(lse >= zmax) and np.all(lse <= zmax + math.log(40) + 1e-12)
    assert np.all(logp <= 0)


def test_gather_marker_row(oracle_lib):
    """Setting W[y_t] to a large multiple of h_t makes z_y unique and dominant,
    so logp -> 0 for that token and only that one."""
    h, W, y, _, _ = _rand_problem(8, H=12, V=30, scale=0.1)
    t = 4
    W[y[t]] = 50.0 * h[t] / np.linalg.norm(h[t]) ** 2  # z_y = 50
    _, logp, zy = oracle_lib.score_rows(h, W, y)
    assert abs(zy[t] - 50.0) < 1e-12
    assert -1e-15 < logp[t] <= 0 or abs(logp[t]) < 1e-18


# ------------------------------------------------- Eq. 1 per-token term
def _obj(oracle_lib, logp, old, ref, A, c=1.0, eps=0.2, beta=0.0):
    n = len(logp)
    return oracle_lib.token_objective(np.asarray(logp, float), np.asarray(old, float),
                                      np.asarray(ref, float), np.full(n, A, float),
                                      np.full(n, c, float), None, eps, beta)


def test_ratio_one_and_kl_zero(oracle_lib):
    """old = logp gives rho = 1 (unclipped): ell = -A, g = -c*A; ref = logp gives kl = 0."""
    logp = np.array([-3.0, -0.5, -7.25])
    for A in (0.7, -1.3, 0.0):
        ell, g, clipped = _obj(oracle_lib, logp, logp, logp, A, c=0.25, beta=0.3)
        np.testing.assert_array_equal(ell, -A)
        np.testing.assert_array_equal(g, -0.25 * A)
        assert not clipped.any()


def test_k3_kl_scalar(oracle_lib):
    d, kl, dkl = _golden_rows("logsumexp_closed_forms.txt")[2]
    # logp = old = 0 (rho = 1), A = 0 so only the KL remains; ref - logp = d
    ell, g, _ = _obj(oracle_lib, [0.0], [0.0], [d], 0.0, c=1.0, beta=0.5)
    assert abs(ell[0] - 0.5 * kl) < 1e-15
    assert abs(g[0] - 0.5 * dkl) < 1e-15
    # kl >= 0 everywhere
    g2 = np.random.default_rng(9)
    lp = g2.normal(-5, 2, 1000)
    ref = lp + g2.normal(0, 3, 1000)
    ell, _, _ = _obj(oracle_lib, lp, lp, ref, 0.0, beta=1.0)
    assert np.all(ell >= 0)


def test_clip_branches(oracle_lib):
    """Forced-clip cases, eps = 0.2, beta = 0: the gradient is exactly 0 iff
    (A>0 and rho>1+eps) or (A<0 and rho<1-eps)."""
    lp = 0.0
    hi = math.log(1.5)  # rho = 1.5 when old = logp - ln 1.5
    lo = math.log(0.5)
    cases = [  # (old, A, ell, g)
        (lp - hi, 1.0, -1.2, 0.0),
        (lp - lo, -1.0, 0.8, 0.0),
        (lp - lo, 1.0, -0.5, -0.5),
        (lp - hi, -1.0, 1.5, 1.5),
    ]
    for old, A, ell_w, g_w in cases:
        ell, g, clipped = _obj(oracle_lib, [lp], [old], [lp], A)
        assert abs(ell[0] - ell_w) < 1e-14, (old, A, ell[0])
        assert abs(g[0] - g_w) < 1e-14, (old, A, g[0])
        assert bool(clipped[0]) == (g_w == 0.0)


def test_masked_token_contributes_nothing(oracle_lib):
    ell, g, clipped = oracle_lib.token_objective(
        np.array([-1.0, -2.0]), np.array([-1.5, -1.0]), np.array([-1.0, -3.0]),
        np.array([1.0, 1.0]), np.array([1.0, 1.0]), np.array([1, 0], np.uint8), 0.2, 0.1)
    assert ell[1] == 0.0 and g[1] == 0.0 and clipped[1] == 0


# ------------------------------------------------- whole loss and gradients
def _full(oracle_lib, seed, beta=0.05, eps=0.2, agg=0, ragged=False, equal=False,
          on_policy=False, sigma=0.05, G=3):
    h, W, y, mask, cu = _rand_problem(seed, ragged=ragged)
    B = len(cu) - 1
    g = np.random.default_rng(seed + 100)
    r = g.integers(0, 3, B) * 0.5
    if equal:
        r = np.repeat(g.integers(0, 3, B // G) * 0.5, G)
    adv = oracle_lib.advantages(r, G)
    _, logp, _ = oracle_lib.score_rows(h, W, y)
    if on_policy:
        old, ref = logp.copy(), logp.copy()
    else:
        old = logp + g.normal(0, sigma, len(y))
        ref = logp + g.normal(0, sigma, len(y))
    out = oracle_lib.grpo_loss(h, W, y, mask, cu, old, ref, adv, eps, beta, agg)
    return dict(h=h, W=W, y=y, mask=mask, cu=cu, old=old, ref=ref, adv=adv, beta=beta,
                eps=eps, agg=agg, **out)


def test_equal_rewards_give_zero_loss_and_grads(oracle_lib):
    p = _full(oracle_lib, 10, beta=0.0, equal=True)
    assert np.all(p["adv"] == 0)
    assert p["loss"] == 0.0
    assert np.all(p["dh"] == 0) and np.all(p["dW"] == 0)
    p = _full(oracle_lib, 11, beta=0.5, equal=True, on_policy=True)
    assert p["loss"] == 0.0 and np.all(p["dh"] == 0) and np.all(p["dW"] == 0)


def test_on_policy_loss_is_minus_mean_advantage(oracle_lib):
    p = _full(oracle_lib, 12, beta=0.3, on_policy=True)
    B = len(p["cu"]) - 1
    assert abs(p["loss"] - (-p["adv"].sum() / B)) < 1e-15
    assert abs(p["loss"]) < 1e-14  # advantages sum to zero within each group


def test_token_mean_equals_seq_mean_for_uniform_lengths(oracle_lib):
    a = _full(oracle_lib, 13, agg=0)
    b = _full(oracle_lib, 13, agg=1)
    assert abs(a["loss"] - b["loss"]) < 1e-15
    np.testing.assert_allclose(a["dh"], b["dh"], rtol=1e-13, atol=1e-16)


def test_empty_rollout_counts_in_B(oracle_lib):
    h, W, y, mask, cu = _rand_problem(14)
    mask[cu[1]:cu[2]] = 0
    adv = np.linspace(-1, 1, len(cu) - 1)
    _, logp, _ = oracle_lib.score_rows(h, W, y)
    out = oracle_lib.grpo_loss(h, W, y, mask, cu, logp, logp, adv, 0.2, 0.0)
    B = len(cu) - 1
    want = -sum(adv[b] for b in range(B) if b != 1) / B
    assert abs(out["loss"] - want) < 1e-15
    assert np.all(out["dh"][cu[1]:cu[2]] == 0)


def _torch_loss(p, h, W):
    """Eq. 1 written once more with torch fp64 ops so autograd can differentiate
    it; this pins the oracle's hand-derived gradients, not its loss formula."""
    y = torch.from_numpy(p["y"])
    z = h @ W.T
    logp = torch.log_softmax(z, 1)[torch.arange(len(y)), y]
    old = torch.from_numpy(p["old"])
    ref = torch.from_numpy(p["ref"])
    cu = p["cu"]
    B = len(cu) - 1
    mask = torch.from_numpy(p["mask"].astype(np.float64))
    adv = torch.from_numpy(np.repeat(p["adv"], np.diff(cu)))
    rho = torch.exp(logp - old)
    surr = torch.minimum(rho * adv, torch.clamp(rho, 1 - p["eps"], 1 + p["eps"]) * adv)
    d = ref - logp
    ell = -surr + p["beta"] * (torch.exp(d) - d - 1)
    total = 0.0
    for b in range(B):
        mb = mask[cu[b]:cu[b + 1]]
        if mb.sum() > 0:
            total = total + (ell[cu[b]:cu[b + 1]] * mb).sum() / mb.sum() / B
    return total


@pytest.mark.parametrize("ragged", [False, True])
def test_gradients_match_torch_autograd(oracle_lib, ragged):
    p = _full(oracle_lib, 15 + ragged, beta=0.2, ragged=ragged, sigma=0.3)
    h = torch.from_numpy(p["h"]).requires_grad_(True)
    W = torch.from_numpy(p["W"]).requires_grad_(True)
    L = _torch_loss(p, h, W)
    L.backward()
    assert abs(L.item() - p["loss"]) < 1e-13
    np.testing.assert_allclose(p["dh"], h.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(p["dW"], W.grad.numpy(), rtol=1e-10, atol=1e-14)


def test_gradients_match_weighted_cross_entropy(oracle_lib):
    """On policy with beta = 0 the gradient is that of sum_t w_t * CE(z_t, y_t)
    with w_t = A_b * c_b (torch's cross_entropy routine, fp64)."""
    p = _full(oracle_lib, 17, beta=0.0, on_policy=True)
    cu = p["cu"]
    B = len(cu) - 1
    lens = np.diff(cu)
    w = torch.from_numpy(np.repeat(p["adv"] / (B * lens), lens))
    h = torch.from_numpy(p["h"]).requires_grad_(True)
    W = torch.from_numpy(p["W"]).requires_grad_(True)
    ce = torch.nn.functional.cross_entropy(h @ W.T, torch.from_numpy(p["y"]), reduction="none")
    (w * ce).sum().backward()
    np.testing.assert_allclose(p["dh"], h.grad.numpy(), rtol=1e-10, atol=1e-15)
    np.testing.assert_allclose(p["dW"], W.grad.numpy(), rtol=1e-10, atol=1e-15)


@pytest.mark.parametrize("forced_clip", [False, True])
def test_gradients_match_finite_differences(oracle_lib, forced_clip):
    p = _full(oracle_lib, 18, beta=0.1, sigma=0.05)
    if forced_clip:  # push every ratio well outside [0.8, 1.2]
        g = np.random.default_rng(19)
        p["old"] = p["logp"] + np.where(g.random(len(p["y"])) < 0.5, -0.5, 0.5)

    def loss(h, W):
        return oracle_lib.grpo_loss(h, W, p["y"], p["mask"], p["cu"], p["old"], p["ref"],
                                    p["adv"], p["eps"], p["beta"], want_dh=False,
                                    want_dW=False)["loss"]

    base = oracle_lib.grpo_loss(p["h"], p["W"], p["y"], p["mask"], p["cu"], p["old"],
                                p["ref"], p["adv"], p["eps"], p["beta"])
    rho = np.exp(base["logp"] - p["old"])
    assert np.all(np.abs(rho - 0.8) > 1e-3) and np.all(np.abs(rho - 1.2) > 1e-3)
    if forced_clip:
        assert base["clipped"].sum() > 0
    step = 1e-6
    g = np.random.default_rng(20)
    for _ in range(12):
        i, k = g.integers(0, p["h"].shape[0]), g.integers(0, p["h"].shape[1])
        hp, hm = p["h"].copy(), p["h"].copy()
        hp[i, k] += step
        hm[i, k] -= step
        fd = (loss(hp, p["W"]) - loss(hm, p["W"])) / (2 * step)
        assert abs(fd - base["dh"][i, k]) < 1e-7 + 1e-5 * abs(fd)
        v = g.integers(0, p["W"].shape[0])
        Wp, Wm = p["W"].copy(), p["W"].copy()
        Wp[v, k] += step
        Wm[v, k] -= step
        fd = (loss(p["h"], Wp) - loss(p["h"], Wm)) / (2 * step)
        assert abs(fd - base["dW"][v, k]) < 1e-7 + 1e-5 * abs(fd)


def test_gradient_invariants(oracle_lib):
    """sum_v dW_v = 0 (softmax rows sum to 1); <dW, W> = <dh, h> (both equal
    sum dz*z); dh unchanged by adding one vector to every W row."""
    p = _full(oracle_lib, 21, beta=0.1, ragged=True)
    np.testing.assert_allclose(p["dW"].sum(axis=0), 0.0, atol=1e-14)
    a = float((p["dW"] * p["W"]).sum())
    b = float((p["dh"] * p["h"]).sum())
    assert abs(a - b) < 1e-12 * max(1.0, abs(a))
    assert np.all(p["dh"][p["mask"] == 0] == 0)
    u = np.random.default_rng(22).standard_normal(p["W"].shape[1])
    q = oracle_lib.grpo_loss(p["h"], p["W"] + u, p["y"], p["mask"], p["cu"], p["old"],
                             p["ref"], p["adv"], p["eps"], p["beta"])
    np.testing.assert_allclose(q["dh"], p["dh"], rtol=1e-8, atol=1e-12)


def test_pieces_compose_to_the_whole(oracle_lib):
    """The row-subset entry points (used for full-size spot checks) agree with
    the composed loss on every row."""
    p = _full(oracle_lib, 23, beta=0.1, ragged=True)
    rows, counts, seq = oracle_lib.pack_valid(p["mask"], p["cu"])
    c = oracle_lib.seq_weights(counts)
    lse, logp, _ = oracle_lib.score_rows(p["h"][rows], p["W"], p["y"][rows])
    ell, g, _ = oracle_lib.token_objective(logp, p["old"][rows], p["ref"][rows],
                                           p["adv"][seq[rows]], c[seq[rows]], None,
                                           p["eps"], p["beta"])
    np.testing.assert_array_equal(logp, p["logp"][rows])
    np.testing.assert_array_equal(g, p["g"][rows])
    dh = oracle_lib.grad_hidden_rows(p["h"][rows], p["W"], p["y"][rows], lse, g)
    np.testing.assert_array_equal(dh, p["dh"][rows])
    vr = np.array([0, 3, 10])
    dW = oracle_lib.grad_weight_rows(p["h"][rows], p["W"], p["y"][rows], lse, g, vr)
    np.testing.assert_allclose(dW, p["dW"][vr], rtol=1e-12, atol=1e-15)


# ------------------------------------------------------------ SFT (Sec. 3.2)
@pytest.mark.parametrize("ragged", [False, True])
def test_sft_matches_torch_cross_entropy(oracle_lib, ragged):
    """SFT stage: mean next-token cross-entropy over the supervised rows, and its
    gradients, against torch's fp64 cross_entropy + autograd (a library routine)."""
    h, W, y, mask, _ = _rand_problem(21, ragged=ragged)
    r = oracle_lib.sft_ce(h, W, y, mask)
    ht = torch.from_numpy(h).requires_grad_(True)
    Wt = torch.from_numpy(W).requires_grad_(True)
    keep = torch.from_numpy(mask.astype(bool))
    ce = torch.nn.functional.cross_entropy((ht @ Wt.T)[keep], torch.from_numpy(y)[keep])
    ce.backward()
    assert r["nvalid"] == int(mask.sum())
    assert r["loss"] == pytest.approx(ce.item(), rel=1e-13)
    np.testing.assert_allclose(r["dh"], ht.grad.numpy(), rtol=1e-10, atol=1e-14)
    np.testing.assert_allclose(r["dW"], Wt.grad.numpy(), rtol=1e-10, atol=1e-14)
    assert np.all(r["dh"][mask == 0] == 0.0)


def test_sft_closed_forms(oracle_lib):
    """W = 0: every row is uniform over V, so the loss is exactly ln V and dh = 0;
    no supervised row: loss and gradients 0; a dominant target logit: loss -> 0."""
    h, W, y, mask, _ = _rand_problem(22, V=1000)
    r = oracle_lib.sft_ce(h, np.zeros_like(W), y, mask)
    assert r["loss"] == pytest.approx(math.log(1000), rel=1e-15)
    assert np.all(r["dh"] == 0.0)
    r = oracle_lib.sft_ce(h, W, y, np.zeros_like(mask))
    assert r["loss"] == 0.0 and r["nvalid"] == 0
    assert np.all(r["dh"] == 0.0) and np.all(r["dW"] == 0.0)
    hm = np.zeros_like(h)
    hm[:, 0] = 1.0
    Wm = np.zeros_like(W)
    Wm[y[0], 0] = 60.0  # z = 60 at the target of row 0, 0 elsewhere
    r = oracle_lib.sft_ce(hm[:1], Wm, y[:1])
    assert r["loss"] == pytest.approx(math.log1p((1000 - 1) * math.exp(-60.0)), rel=1e-12)


def test_sft_finite_differences(oracle_lib):
    """Central differences of the SFT loss in h and W (fp64, step 1e-6)."""
    h, W, y, mask, _ = _rand_problem(23, B=3, T=3, H=4, V=6, ragged=True)
    r = oracle_lib.sft_ce(h, W, y, mask)
    eps = 1e-6
    for (i, k) in [(0, 0), (1, 3), (4, 2)]:
        hp, hm = h.copy(), h.copy()
        hp[i, k] += eps
        hm[i, k] -= eps
        fd = (oracle_lib.sft_ce(hp, W, y, mask)["loss"] -
              oracle_lib.sft_ce(hm, W, y, mask)["loss"]) / (2 * eps)
        assert r["dh"][i, k] == pytest.approx(fd, rel=1e-6, abs=1e-9)
    for (v, k) in [(0, 1), (y[0], 2), (5, 3)]:
        Wp, Wn = W.copy(), W.copy()
        Wp[v, k] += eps
        Wn[v, k] -= eps
        fd = (oracle_lib.sft_ce(h, Wp, y, mask)["loss"] -
              oracle_lib.sft_ce(h, Wn, y, mask)["loss"]) / (2 * eps)
        assert r["dW"][v, k] == pytest.approx(fd, rel=1e-6, abs=1e-9)


# ------------------------------------------------ AdamW step (after the gradient)
def test_adamw_matches_torch(oracle_lib):
    """Three steps against torch.optim.AdamW in float64 (a library routine)."""
    g0 = np.random.default_rng(41)
    w0 = g0.standard_normal(1000)
    grads = [g0.standard_normal(1000) * s for s in (1.0, 1e-3, 30.0)]
    p = torch.nn.Parameter(torch.from_numpy(w0.copy()))
    opt = torch.optim.AdamW([p], lr=1e-3, betas=(0.9, 0.95), eps=1e-8, weight_decay=0.1)
    w, m, v = w0.copy(), np.zeros(1000), np.zeros(1000)
    for t, gr in enumerate(grads, start=1):
        p.grad = torch.from_numpy(gr.copy())
        opt.step()
        w, m, v = oracle_lib.adamw(w, m, v, gr, t, 1e-3, 0.9, 0.95, 1e-8, 0.1)
        st = opt.state[p]
        np.testing.assert_allclose(w, p.detach().numpy(), rtol=1e-14, atol=1e-15)
        np.testing.assert_allclose(m, st["exp_avg"].numpy(), rtol=1e-14, atol=1e-300)
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=1e-14, atol=1e-300)


def test_adamw_closed_forms(oracle_lib):
    """Zero gradient from zero moments: pure decay w(1 - lr*wd). First step: the
    bias-corrected moments are g and g^2, so the step is lr*g/(|g| + eps)."""
    w = np.array([1.0, -2.0, 0.5])
    z = np.zeros(3)
    w1, m1, v1 = oracle_lib.adamw(w, z, z, z, 1, 1e-2, 0.9, 0.999, 1e-8, 0.5)
    np.testing.assert_array_equal(w1, w * (1 - 1e-2 * 0.5))
    assert np.all(m1 == 0) and np.all(v1 == 0)
    g = np.array([3.0, -1e-3, 0.25])
    w1, _, _ = oracle_lib.adamw(w, z, z, g, 1, 1e-2, 0.9, 0.999, 1e-8, 0.0)
    np.testing.assert_allclose(w1, w - 1e-2 * g / (np.abs(g) + 1e-8), rtol=1e-14)

