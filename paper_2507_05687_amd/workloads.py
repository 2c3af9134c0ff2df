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
import hashlib
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


def input_digest(*arrays: np.ndarray) -> str:
    """SHA-256 over the dtype, shape and bytes of each array, in order: logged
    so that two consumers of a workload's inputs can be shown to read the same
    bytes."""
    d = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        d.update(f"{a.dtype.str}{a.shape}".encode())
        d.update(memoryview(a).cast("B"))
    return d.hexdigest()


def batch_digest(W: np.ndarray, h: np.ndarray, batch: dict) -> str:
    """input_digest of a workload's weight, hidden states and batch arrays."""
    return input_digest(W, h, *(batch[k] for k in sorted(batch)))


def sample_rows(mask: np.ndarray, count: int, seed: int = 0) -> np.ndarray:
    """A seeded, sorted sample of valid row indices (for oracle spot checks)."""
    valid = np.flatnonzero(mask)
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 99])))
    k = min(count, valid.size)
    return np.sort(g.choice(valid, size=k, replace=False)).astype(np.int64)


# ------------------------------------------------------------ completions
# Seeded synthetic completions for the rule-based reward (Sec. 3.3, Eq. 3):
# Python sources assembled from small fragments written for this purpose
# (an elementwise Triton kernel, its launcher, a PyTorch fallback, filler
# statements), with the variations the rule has to tell apart: decorator
# present, commented out, misspelt, with arguments, after other decorators,
# not followed by a function; the kernel launched, launched through a module,
# never launched, or a different name launched. They stand in for the
# paper's rollouts, whose benchmark items are not used.

_HEADER = "import torch\nimport triton\nimport triton.language as tl\n\n"
_KERNEL = (
    "def {name}(x_ptr, y_ptr, out_ptr, n_elements, BLOCK: tl.constexpr):\n"
    "    pid = tl.program_id(axis=0)\n"
    "    offs = pid * BLOCK + tl.arange(0, BLOCK)\n"
    "    mask = offs < n_elements\n"
    "    x = tl.load(x_ptr + offs, mask=mask)\n"
    "    y = tl.load(y_ptr + offs, mask=mask)\n"
    "    tl.store(out_ptr + offs, x {op} y, mask=mask)\n\n")
_LAUNCHER = (
    "def {fn}(x, y):\n"
    "    out = torch.empty_like(x)\n"
    "    n = out.numel()\n"
    "    grid = lambda meta: (triton.cdiv(n, meta['BLOCK']),)\n"
    "    {call}\n"
    "    return out\n\n")
_TORCH = "def {fn}(x, y):\n    return x {op} y\n\n"
_FILLER = [
    "scale = {k} * 0.5\n", "# keep the block size a power of two ({k})\n",
    "values = [i * {k} for i in range(8)]\n", "assert {k} >= 0\n",
    "config = dict(block={k}, warps=4)\n", "total = sum(values) + {k}\n",
]
_VALID_DECOS = ["@triton.jit", "@triton.jit()", "@triton.jit(do_not_specialize=['n_elements'])",
                "@triton.jit(\n    debug=False,\n)", "@triton.autotune(configs=[], key=['n_elements'])\n@triton.jit",
                "@triton.jit\n# the kernel\n", "    @triton.jit"]
_DECOY_DECOS = ["# @triton.jit", "@triton.jitted", "@triton.jit.fn", "@triton.heuristics({})"]
_BROKEN_DECOS = ["@triton.jit x", "@triton.jit(", "y = 1 @triton.jit"]


def _ident(rng, prefix: str) -> str:
    return prefix + "_" + "".join(rng.choice(list("abcdefghijklmnopqrstuvwxyz"), size=5))


def _completion(rng, target_len: int, valid: bool) -> bytes:
    name = _ident(rng, "kernel")
    other = _ident(rng, "helper")
    op = str(rng.choice(["+", "-", "*"]))
    parts = [_HEADER]
    # the kernel, with a decorator variant (or none)
    r = rng.random()
    if r < 0.55:
        deco = str(rng.choice(_VALID_DECOS))
    elif r < 0.75:
        deco = str(rng.choice(_DECOY_DECOS))
    elif r < 0.85 or valid:
        deco = ""
    else:
        deco = str(rng.choice(_BROKEN_DECOS))
    kernel = _KERNEL.format(name=name, op=op)
    if deco.startswith("    "):  # a kernel defined inside a class body
        kernel = "class Ops:\n" + deco + "\n" + "".join("    " + ln + "\n" if ln else "\n"
                                                       for ln in kernel.split("\n"))
    elif deco:
        kernel = deco.rstrip("\n") + "\n" + kernel
    if not valid and rng.random() < 0.05:  # decorator left without a function
        kernel = "@triton.jit\nvalue = 3\n\n" + kernel
    parts.append(kernel)
    # the launcher, with a launch variant (or a PyTorch fallback)
    r = rng.random()
    launches = [f"{name}[grid](x, y, out, n, BLOCK=1024)",
                f"{name} [grid] (x, y, out, n, BLOCK=1024)",
                f"{name}[(triton.cdiv(n, 256), 1)](x, y, out, n, BLOCK=256)"]
    if deco.startswith("    "):
        launches = [f"Ops.{name}[grid](x, y, out, n, BLOCK=1024)"]
    if r < 0.6:
        call = str(rng.choice(launches))
    elif r < 0.7:
        call = f"{other}[grid](x, y, out, n, BLOCK=1024)"
    elif r < 0.8:
        call = f"spec = {name}[grid]"
    elif r < 0.85 and not valid:
        call = f"{name}[grid(x, y, out, n)"
    else:
        call = f"out = x {op} y"
    if rng.random() < 0.3:
        parts.append(_TORCH.format(fn=_ident(rng, "torch_ref"), op=op))
    parts.append(_LAUNCHER.format(fn=_ident(rng, "run"), call=call))
    text = "".join(parts)
    while len(text) < target_len:
        text += str(rng.choice(_FILLER)).format(k=int(rng.integers(0, 1000)))
    if not valid and rng.random() < 0.1:
        text = text.replace("\n", "\r\n")
    if not valid and rng.random() < 0.05:
        text = text[: int(rng.integers(0, len(text) + 1))]  # cut off mid-completion
    data = text.encode("utf-8")
    if not valid and rng.random() < 0.05:
        data += "  # π ≈ 3.14, ü\n".encode("utf-8")
    return data


def make_completions(count: int, seed: int, mean_len: int = 2000, max_len: int = 16384,
                     valid: bool = False, pass_rate: float = 0.5):
    """count seeded synthetic completions (bytes, lengths drawn around
    mean_len, at most max_len bytes) and test_passed flags (u8). With
    valid=True every completion is a syntactically valid Python module (and
    may run a little past max_len)."""
    rng = np.random.default_rng(seed)
    lens = np.minimum(rng.exponential(mean_len, size=count).astype(np.int64) + 200, max_len)
    texts = [_completion(rng, int(n), valid) for n in lens]
    if not valid:
        texts = [t[:max_len] for t in texts]
    passed = (rng.random(count) < pass_rate).astype(np.uint8)
    return texts, passed


def pack_completions(texts):
    """Concatenated bytes (u8) and offsets (int64 [count + 1]) of completions."""
    offsets = np.zeros(len(texts) + 1, dtype=np.int64)
    offsets[1:] = np.cumsum([len(t) for t in texts])
    data = np.frombuffer(b"".join(texts), dtype=np.uint8).copy() if offsets[-1] else np.zeros(
        0, dtype=np.uint8)
    return data, offsets
