"""Seeded synthetic inputs for the GRPO scoring + loss hot path.

This module is shared by the tests, the benchmark and the smoke check. It
holds input generation only: random draws, the bf16 round-to-nearest-even
encoding of inputs, and the shapes of the five workloads. None of the
method's arithmetic (log-softmax, ratio, clip, KL, advantages, gradients)
lives here.

Workloads (sizes follow the GRPO stage of AutoTriton, Sec. 3.3 / Eq. 1-2,
with H=4096 and V=155136; the paper trains on TritonBench/KernelBench-style
data, which these seeded synthetic tensors stand in for):

* ``tiny_fp32``     2 prompts x G=4 x 16 tokens, H=64, V=1000, fp32.
* ``fwd_bf16``      4 x 8 x 1024 tokens (N=32768), scoring only.
* ``fwdbwd_bf16``   8 x 8 x 2048 tokens (N=131072), loss fwd+bwd.
* ``ragged_bf16``   16 x 8 rollouts, lengths U{256..8192}, padded to 8192.
* ``double_bf16``   16 x 8 x 2048 tokens (N=262144), policy + reference.
* ``sft_bf16``      the supervised stage before GRPO (Sec. 3.2): one sequence
                    of 16384 tokens per GPU (the paper's maximum length and
                    per-device batch of 1, Sec. 4.1), the first 2048 (the
                    prompt) not supervised.
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor

import numpy as np

_CHUNK = 1 << 22  # elements per independently seeded block


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    prompts: int
    group: int
    seq_len: int  # padded length T per rollout
    hidden: int
    vocab: int
    dtype: str  # "f32" or "bf16"
    clip_eps: float = 0.2
    beta: float = 0.01
    noise_sigma: float = 0.05  # std of old/ref log-prob perturbations
    reward_kind: str = "thirds"  # "thirds": {0,.5,1}; "fmt_exec": .1*Bern+.9*Bern
    ragged: bool = False
    min_len: int = 0
    forced_equal_groups: int = 0  # leading groups given all-equal rewards
    rms_norm_hidden: bool = False
    double_scoring: bool = False
    ref_delta_sigma: float = 0.002  # W_pol = W_ref + N(0, sigma) for double scoring
    weight_sigma: float = 0.02
    seed: int = 0
    fwd_only: bool = False
    objective: str = "grpo"  # "grpo" (Eq. 1) or "sft" (cross-entropy)
    prompt_len: int = 0  # leading tokens of each sequence left out of the mask

    @property
    def num_seqs(self) -> int:
        return self.prompts * self.group

    @property
    def num_tokens(self) -> int:
        return self.num_seqs * self.seq_len


WORKLOADS = {
    "tiny_fp32": Workload("tiny_fp32", 2, 4, 16, 64, 1000, "f32", 0.2, 0.01, 0.05,
                          "thirds", seed=0),
    "fwd_bf16": Workload("fwd_bf16", 4, 8, 1024, 4096, 155136, "bf16",
                         rms_norm_hidden=True, seed=1, fwd_only=True),
    "fwdbwd_bf16": Workload("fwdbwd_bf16", 8, 8, 2048, 4096, 155136, "bf16", 0.2, 0.001,
                            0.1, "fmt_exec", rms_norm_hidden=True, seed=2),
    "ragged_bf16": Workload("ragged_bf16", 16, 8, 8192, 4096, 155136, "bf16", 0.2, 0.001,
                            0.1, "fmt_exec", ragged=True, min_len=256, forced_equal_groups=2,
                            rms_norm_hidden=True, seed=3),
    "double_bf16": Workload("double_bf16", 16, 8, 2048, 4096, 155136, "bf16", 0.2, 0.001,
                            0.1, "fmt_exec", rms_norm_hidden=True, double_scoring=True, seed=4),
    "sft_bf16": Workload("sft_bf16", 1, 1, 16384, 4096, 155136, "bf16", rms_norm_hidden=True,
                         objective="sft", prompt_len=2048, seed=5),
}


def scaled(w: Workload, **kw) -> Workload:
    """A copy of a workload with some fields replaced (e.g. smaller sizes)."""
    return dataclasses.replace(w, **kw)


# ---------------------------------------------------------------- bf16 bits
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even. Finite inputs."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + r) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> the exact fp32 values they encode."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------- draws
def _normal_f32(seed_seq: np.random.SeedSequence, n: int, sigma: float) -> np.ndarray:
    """n N(0, sigma^2) draws in float32; blocks are seeded independently so the
    result does not depend on how many threads fill it."""
    out = np.empty(n, dtype=np.float32)
    nblk = max(1, math.ceil(n / _CHUNK))
    kids = seed_seq.spawn(nblk)

    def fill(i):
        lo, hi = i * _CHUNK, min(n, (i + 1) * _CHUNK)
        g = np.random.Generator(np.random.PCG64(kids[i]))
        g.standard_normal(hi - lo, dtype=np.float32, out=out[lo:hi])
        if sigma != 1.0:
            out[lo:hi] *= np.float32(sigma)

    if nblk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(max_workers=8) as ex:
            list(ex.map(fill, range(nblk)))
    return out


def _rms_normalise_rows(x: np.ndarray) -> np.ndarray:
    """Each row divided by its root mean square (no gain)."""
    out = np.empty_like(x)
    step = 8192
    for lo in range(0, x.shape[0], step):
        blk = x[lo:lo + step].astype(np.float64)
        rms = np.sqrt(np.mean(blk * blk, axis=1, keepdims=True))
        out[lo:lo + step] = (blk / rms).astype(np.float32)
    return out


def _encode(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def make_weight(w: Workload, which: str = "policy") -> np.ndarray:
    """LM-head weight [V, H] (bf16 bits or fp32), rows = vocabulary entries.

    For double scoring, ``"reference"`` is W_ref ~ N(0, sigma^2) and
    ``"policy"`` is W_ref + N(0, ref_delta_sigma^2)."""
    root = np.random.SeedSequence([w.seed, 1])
    base = _normal_f32(root, w.vocab * w.hidden, w.weight_sigma)
    if w.double_scoring and which == "policy":
        base += _normal_f32(np.random.SeedSequence([w.seed, 2]), w.vocab * w.hidden,
                            w.ref_delta_sigma)
    return _encode(base.reshape(w.vocab, w.hidden), w.dtype)


def make_hidden(w: Workload, rows: int | None = None) -> np.ndarray:
    """Final hidden states [N, H] (bf16 bits or fp32)."""
    n = w.num_tokens if rows is None else rows
    x = _normal_f32(np.random.SeedSequence([w.seed, 3]), n * w.hidden, 1.0).reshape(n, w.hidden)
    if w.rms_norm_hidden:
        x = _rms_normalise_rows(x)
    return _encode(x, w.dtype)


def make_batch(w: Workload) -> dict:
    """Everything except the big matrices: sampled ids, mask, sequence offsets,
    rewards and the perturbations that turn a base log-prob into old/ref.

    Returns numpy arrays:
      tokens int64 [N], mask uint8 [N], cu_seqlens int64 [B+1], lengths int64 [B],
      rewards float32 [B], old_noise float32 [N], ref_noise float32 [N].
    """
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, 4])))
    B, T, N = w.num_seqs, w.seq_len, w.num_tokens
    tokens = g.integers(0, w.vocab, size=N, dtype=np.int64)
    if w.ragged:
        lengths = g.integers(w.min_len, T + 1, size=B, dtype=np.int64)
    else:
        lengths = np.full(B, T, dtype=np.int64)
    pos = np.arange(T)[None, :]
    mask = ((pos < lengths[:, None]) & (pos >= w.prompt_len)).astype(np.uint8).reshape(N)
    cu = np.arange(B + 1, dtype=np.int64) * T
    if w.reward_kind == "thirds":
        rewards = g.integers(0, 3, size=B).astype(np.float32) * np.float32(0.5)
    else:
        fmt = g.integers(0, 2, size=B).astype(np.float32)
        ex = g.integers(0, 2, size=B).astype(np.float32)
        rewards = (np.float32(0.1) * fmt + np.float32(0.9) * ex).astype(np.float32)
    for k in range(min(w.forced_equal_groups, w.prompts)):
        rewards[k * w.group:(k + 1) * w.group] = np.float32(1.0 if k % 2 == 0 else 0.0)
    old_noise = (g.standard_normal(N) * w.noise_sigma).astype(np.float32)
    ref_noise = (g.standard_normal(N) * w.noise_sigma).astype(np.float32)
    return dict(tokens=tokens, mask=mask, cu_seqlens=cu, lengths=lengths, rewards=rewards,
                old_noise=old_noise, ref_noise=ref_noise)


def sample_rows(mask: np.ndarray, count: int, seed: int = 0) -> np.ndarray:
    """A seeded, sorted sample of valid row indices (for oracle spot checks)."""
    valid = np.flatnonzero(mask)
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 99])))
    k = min(count, valid.size)
    return np.sort(g.choice(valid, size=k, replace=False)).astype(np.int64)
