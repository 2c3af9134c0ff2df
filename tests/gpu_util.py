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
