"""Helpers shared by the GPU tests: moving seeded inputs to the device and
comparing with the oracle. No arithmetic of the method lives here."""
from __future__ import annotations

import numpy as np
import torch

import oracle


def to_dev(x: np.ndarray, dtype: str) -> torch.Tensor:
    """numpy input buffer (bf16 bit patterns or fp32) -> device tensor of that dtype."""
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.cuda()


def dev(x: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


def host64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def rel_err(got: np.ndarray, want: np.ndarray) -> float:
    """max_i |got_i - want_i| / |want_i| (elementwise relative)."""
    want = np.asarray(want, np.float64)
    d = np.abs(np.asarray(got, np.float64) - want)
    return float(np.max(d / np.maximum(np.abs(want), 1e-300))) if d.size else 0.0


def norm_rel(got: np.ndarray, want: np.ndarray) -> float:
    """||got - want|| / ||want|| (norm-wise relative; 0 when both are 0)."""
    want = np.asarray(want, np.float64)
    d = np.linalg.norm(np.asarray(got, np.float64) - want)
    n = np.linalg.norm(want)
    return float(d / n) if n > 0 else float(d)


def oracle_problem(h_in, W_in, dtype, batch, adv, old, ref, eps, beta, agg=0):
    """Full oracle loss and gradients for a small problem (all rows)."""
    h = oracle.decode(h_in, dtype)
    W = oracle.decode(W_in, dtype)
    return oracle.grpo_loss(h, W, batch["tokens"], batch["mask"], batch["cu_seqlens"], old, ref,
                            adv, eps, beta, agg)


def loss_tolerance_ok(got: float, want: float, token_loss_abs_sum: float, tol: float) -> bool:
    """|got - want| <= tol * max(|want|, sum_b c_b sum_t |ell_t|): the loss is a
    near-cancelling sum (advantages sum to zero within each group), so its
    error is measured against the size of the terms it sums."""
    return abs(got - want) <= tol * max(abs(want), token_loss_abs_sum)


# ---- gradient tolerances
# The bf16 gradient products multiply dz = -g_t p_{t,v} rounded to bf16 (RNE,
# relative error <= 2^-9 per entry); the sampled id's +g_t is applied in fp32.
# So |dh_t - exact| <= 2^-9 |g_t| sum_v p_{t,v} |W_v| and
# |dW_v - exact| <= 2^-9 sum_t |g_t| p_{t,v} |h_t| elementwise, plus fp32
# accumulation. GRAD_SLACK covers the accumulation and doubles the rounding
# bound; a bf16 output adds its own rounding, 2^-9 relative per element.
GRAD_ROUND = 2.0 ** -9
GRAD_SLACK = 1e-5
BF16_OUT = 2.0 ** -9


def softmax_rows(h: np.ndarray, W: np.ndarray) -> np.ndarray:
    """p_{t,v} = softmax_v(h_t . W_v) in float64, one row per row of h."""
    z = h @ W.T
    z -= z.max(axis=1, keepdims=True)
    p = np.exp(z)
    return p / p.sum(axis=1, keepdims=True)


def rounding_bounds(h: np.ndarray, W: np.ndarray, g: np.ndarray, vrows=None):
    """Norms of the elementwise rounding bounds (without the 2^-9 factor):
    per row t of h, || |g_t| sum_v p_tv |W_v| ||; per vocabulary row v (all, or
    those in vrows), || sum_t |g_t| p_tv |h_t| ||. Rows of h are taken in chunks
    so that p never exceeds about 2^26 entries."""
    aW = np.abs(W)
    cols = np.arange(W.shape[0]) if vrows is None else np.asarray(vrows, dtype=np.int64)
    dh_b = np.empty(h.shape[0])
    dW_acc = np.zeros((len(cols), W.shape[1]))
    step = max(1, (1 << 26) // W.shape[0])
    for a in range(0, h.shape[0], step):
        p = softmax_rows(h[a:a + step], W)
        ag = np.abs(g[a:a + step])[:, None]
        dh_b[a:a + step] = np.linalg.norm(ag * (p @ aW), axis=1)
        dW_acc += p[:, cols].T @ (ag * np.abs(h[a:a + step]))
    return dh_b, np.linalg.norm(dW_acc, axis=1)


def _tol(bound, ref) -> float:
    return 2 * GRAD_ROUND * bound / max(float(np.linalg.norm(ref)), 1e-300) + GRAD_SLACK


def grad_tolerances(h: np.ndarray, W: np.ndarray, g: np.ndarray, dh_ref: np.ndarray,
                    dW_ref: np.ndarray | None = None):
    """Norm-wise relative tolerances (dh, dW) over all rows, from the bf16
    rounding bound above, for the rows h (float64, [n, H]) with dL/dlogp g
    ([n]; 0 for masked rows)."""
    dh_b, dW_b = rounding_bounds(h, W, g)
    tol_dh = _tol(np.linalg.norm(dh_b), dh_ref)
    return tol_dh, (None if dW_ref is None else _tol(np.linalg.norm(dW_b), dW_ref))


def row_tolerances(bounds: np.ndarray, refs: np.ndarray) -> np.ndarray:
    """Per-row norm-wise relative tolerances from rounding_bounds' row bounds."""
    return np.array([_tol(b, r) for b, r in zip(bounds, refs)])
