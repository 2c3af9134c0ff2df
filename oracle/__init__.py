"""Double-precision CPU oracle for the GRPO scoring + loss hot path.

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the
benchmark's CPU-baseline leg are the only callers. The product path (the
HIP library and its Python binding) never imports this package, and this
package never imports the product path.

The arithmetic lives in ``grpo_oracle.c`` (plain C, double, OpenMP over
independent rows); this module builds it with gcc and marshals numpy
arrays. Inputs are decoded to float64 here: bf16 bit patterns and fp32
values are exactly representable, so the oracle reads the very values the
GPU reads.

What each function follows (AutoTriton, Sec. 3.3):
  advantages        Eq. 2 (statistics over the G rollouts of a prompt)
  pack_valid        the |o_i| token counts of Eq. 1 (valid = mask set)
  seq_weights       the 1/G * 1/|o_i| normalisation of Eq. 1
  score_rows        pi_theta(o_t|q,o_<t): log-softmax of the LM-head logits
  token_objective   the clipped-ratio term minus beta*KL of Eq. 1 (k3 KL)
  grad_hidden_rows  dL/dh, exact chain rule through the log-softmax
  grad_weight_rows  dL/dW, same
  grpo_loss         the whole loss and gradients for small problems
  rule_rewards      Eq. 3: is_Triton (the @triton.jit rule of Sec. 4, plain
                    Python in rule_reward.py) combined with test_passed
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "grpo_oracle.c")
# The test that checks the pins themselves runs them against copies of the
# library with a planted mistake, named by this variable; it is never built
# over. Nothing else sets it.
_OVERRIDE = os.environ.get("GRPO_ORACLE_LIB")
_LIB = _OVERRIDE or os.path.join(_HERE, "libgrpo_oracle.so")
_lib = None

_D = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_I = np.ctypeslib.ndpointer(dtype=np.int64, flags="C_CONTIGUOUS")
_U8 = np.ctypeslib.ndpointer(dtype=np.uint8, flags="C_CONTIGUOUS")
_i64 = ctypes.c_int64
_dbl = ctypes.c_double
_vp = ctypes.c_void_p


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math: sums keep their order)."""
    if _OVERRIDE:
        return _LIB
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                        "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not _OVERRIDE and (not os.path.exists(_LIB) or
                              os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        lib.oracle_group_advantages.argtypes = [_D, _i64, _i64, _dbl, ctypes.c_int, _D]
        lib.oracle_pack_valid.argtypes = [_vp, _I, _i64, _vp, _I, _vp]
        lib.oracle_pack_valid.restype = _i64
        lib.oracle_seq_weights.argtypes = [_I, _i64, ctypes.c_int, _D]
        lib.oracle_score_rows.argtypes = [_D, _D, _I, _i64, _i64, _i64, _D, _D, _vp]
        lib.oracle_token_objective.argtypes = [_D, _D, _D, _D, _D, _vp, _i64, _dbl, _dbl,
                                               _D, _D, _vp]
        lib.oracle_grad_hidden_rows.argtypes = [_D, _D, _I, _D, _D, _i64, _i64, _i64, _D]
        lib.oracle_grad_weight_rows.argtypes = [_D, _D, _I, _D, _D, _i64, _i64, _i64, _vp,
                                                _i64, _D]
        lib.oracle_grpo_loss.argtypes = [_D, _D, _I, _vp, _I, _i64, _i64, _i64, _i64, _D, _D,
                                         _D, _dbl, _dbl, ctypes.c_int, _D, _vp, _vp, _vp, _vp,
                                         _vp, _vp, _vp]
        lib.oracle_grpo_loss.restype = _i64
        lib.oracle_sft_ce.argtypes = [_D, _D, _I, _vp, _i64, _i64, _i64, _D, _vp, _vp, _vp,
                                      _vp, _vp]
        lib.oracle_sft_ce.restype = _i64
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def decode(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of an input buffer: bf16 bit patterns (uint16) or fp32."""
    if dtype == "bf16":
        u = np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    return np.ascontiguousarray(x, dtype=np.float32).astype(np.float64)


def _f64(x):
    return np.ascontiguousarray(x, dtype=np.float64)


def advantages(rewards, group: int, std_eps: float = 1e-6, unbiased: bool = True) -> np.ndarray:
    r = _f64(rewards)
    out = np.empty_like(r)
    _load().oracle_group_advantages(r, r.size // group, group, std_eps, int(unbiased), out)
    return out


def pack_valid(mask, cu_seqlens):
    """(rows of valid tokens in order, |o_b| per rollout, rollout id per row)."""
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int64)
    B = cu.size - 1
    N = int(cu[-1])
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    rows = np.empty(N, dtype=np.int64)
    counts = np.empty(B, dtype=np.int64)
    seq = np.empty(N, dtype=np.int64)
    n = _load().oracle_pack_valid(_ptr(m), cu, B, _ptr(rows), counts, _ptr(seq))
    return rows[:n].copy(), counts, seq


def seq_weights(counts, agg: int = 0) -> np.ndarray:
    c = np.ascontiguousarray(counts, dtype=np.int64)
    out = np.empty(c.size, dtype=np.float64)
    _load().oracle_seq_weights(c, c.size, int(agg), out)
    return out


def score_rows(h, W, y):
    """lse, logp and z_y for tokens with hidden rows h [n,H] (float64) and ids y."""
    h = _f64(h)
    W = _f64(W)
    y = np.ascontiguousarray(y, dtype=np.int64)
    n, H = h.shape
    V = W.shape[0]
    lse = np.empty(n)
    logp = np.empty(n)
    zy = np.empty(n)
    _load().oracle_score_rows(h, W, y, n, H, V, lse, logp, _ptr(zy))
    return lse, logp, zy


def token_objective(logp, old, ref, adv_tok, c_tok, mask, eps: float, beta: float):
    """Per-token ell, g = dL/dlogp and the clipped flag (Eq. 1, k3 KL)."""
    logp = _f64(logp)
    n = logp.size
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    ell = np.empty(n)
    g = np.empty(n)
    clipped = np.empty(n, dtype=np.uint8)
    _load().oracle_token_objective(logp, _f64(old), _f64(ref), _f64(adv_tok), _f64(c_tok),
                                   _ptr(m), n, eps, beta, ell, g, _ptr(clipped))
    return ell, g, clipped


def grad_hidden_rows(h, W, y, lse, g) -> np.ndarray:
    h = _f64(h)
    W = _f64(W)
    n, H = h.shape
    out = np.empty((n, H))
    _load().oracle_grad_hidden_rows(h, W, np.ascontiguousarray(y, dtype=np.int64), _f64(lse),
                                    _f64(g), n, H, W.shape[0], out)
    return out


def grad_weight_rows(h, W, y, lse, g, vrows=None) -> np.ndarray:
    h = _f64(h)
    W = _f64(W)
    n, H = h.shape
    V = W.shape[0]
    vr = None if vrows is None else np.ascontiguousarray(vrows, dtype=np.int64)
    nv = V if vr is None else vr.size
    out = np.empty((nv, H))
    _load().oracle_grad_weight_rows(h, W, np.ascontiguousarray(y, dtype=np.int64), _f64(lse),
                                    _f64(g), n, H, V, _ptr(vr), nv, out)
    return out


def grpo_loss(h, W, tokens, mask, cu_seqlens, old, ref, adv_seq, eps: float, beta: float,
              agg: int = 0, want_dh: bool = True, want_dW: bool = True) -> dict:
    """Whole loss + gradients (h [N,H], W [V,H] float64; per-row old/ref; adv per rollout)."""
    h = _f64(h)
    W = _f64(W)
    N, H = h.shape
    V = W.shape[0]
    cu = np.ascontiguousarray(cu_seqlens, dtype=np.int64)
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    out = dict(lse=np.empty(N), logp=np.empty(N), ell=np.empty(N), g=np.empty(N),
               clipped=np.empty(N, dtype=np.uint8))
    dh = np.empty((N, H)) if want_dh else None
    dW = np.empty((V, H)) if want_dW else None
    loss = np.zeros(1)
    nvalid = _load().oracle_grpo_loss(
        h, W, np.ascontiguousarray(tokens, dtype=np.int64), _ptr(m), cu, cu.size - 1, N, H, V,
        _f64(old), _f64(ref), _f64(adv_seq), eps, beta, int(agg), loss, _ptr(out["lse"]),
        _ptr(out["logp"]), _ptr(out["ell"]), _ptr(out["g"]), _ptr(out["clipped"]), _ptr(dh),
        _ptr(dW))
    out.update(loss=float(loss[0]), dh=dh, dW=dW, nvalid=int(nvalid))
    return out


def sft_ce(h, W, tokens, mask=None, want_dh: bool = True, want_dW: bool = True) -> dict:
    """SFT cross-entropy (mean of -logp over valid rows) and its gradients."""
    h = _f64(h)
    W = _f64(W)
    N, H = h.shape
    V = W.shape[0]
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    out = dict(lse=np.empty(N), logp=np.empty(N), g=np.empty(N))
    dh = np.empty((N, H)) if want_dh else None
    dW = np.empty((V, H)) if want_dW else None
    loss = np.zeros(1)
    n = _load().oracle_sft_ce(h, W, np.ascontiguousarray(tokens, dtype=np.int64), _ptr(m), N, H,
                              V, loss, _ptr(out["lse"]), _ptr(out["logp"]), _ptr(out["g"]),
                              _ptr(dh), _ptr(dW))
    out.update(loss=float(loss[0]), dh=dh, dW=dW, nvalid=int(n))
    return out


def adamw(w, m, v, g, step: int, lr: float, beta1: float, beta2: float, eps: float,
          weight_decay: float):
    """One AdamW step (Adam with decoupled weight decay, Loshchilov & Hutter), written
    out in float64 the way the algorithm states it: moments, bias corrections,
    decay of the previous weight, then the normalised step. Returns (w, m, v)."""
    w, m, v, g = (np.asarray(x, np.float64) for x in (w, m, v, g))
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    m_hat = m / (1.0 - beta1 ** step)
    v_hat = v / (1.0 - beta2 ** step)
    w = w - lr * weight_decay * w - lr * m_hat / (np.sqrt(v_hat) + eps)
    return w, m, v


from .rule_reward import is_triton, rule_rewards  # noqa: E402,F401
