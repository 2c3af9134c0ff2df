"""Python binding of libgrpo (include/grpo.h): argument marshalling only.

Tensors supply device pointers and the current HIP stream; every step of
the computation runs in the library's HIP kernels. There is no CPU or
PyTorch fallback: if libgrpo.so is missing or the device is not gfx950 the
calls raise.
"""
from __future__ import annotations

import ctypes
import functools
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgrpo.so")

F32, BF16 = 0, 1
AGG_SEQ_MEAN, AGG_TOKEN_MEAN = 0, 1
OP_LOGPROB_FWD, OP_LOSS_FWD_BWD, OP_SFT_FWD_BWD = 0, 1, 2
WS_TILED_WEIGHT = 0x100  # OR-ed into an op: the call is given a tiled weight

STATUS = {0: "GRPO_OK", 1: "GRPO_ERR_NULL", 2: "GRPO_ERR_SHAPE", 3: "GRPO_ERR_DTYPE",
          4: "GRPO_ERR_PARAM", 5: "GRPO_ERR_ALIGN", 6: "GRPO_ERR_WORKSPACE",
          7: "GRPO_ERR_DEVICE", 8: "GRPO_ERR_HIP", 9: "GRPO_ERR_TOKEN_RANGE",
          10: "GRPO_ERR_SEQLENS", 11: "GRPO_ERR_CAPACITY"}

# Every symbol include/grpo.h declares, with its ctypes signature.
_vp, _i64, _i32, _f32, _sz = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float,
                              ctypes.c_size_t)
SIGNATURES = {
    "group_advantages": (_i32, [_vp, _i64, _i32, _f32, _i32, _vp, _vp]),
    "grpo_pack_valid": (_i32, [_vp, _vp, _i64, _i64, _vp, _vp, _vp, _vp, _sz, _vp]),
    "grpo_pack_valid_static": (_i32, [_vp, _vp, _i64, _i64, _vp, _vp, _vp, _vp, _vp]),
    "grpo_logprob_fwd": (_i32, [_i32, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp,
                                _sz, _i64, _vp]),
    "grpo_loss_fwd_bwd": (_i32, [_i32, _vp, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, _vp,
                                 _vp, _vp, _f32, _f32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                 _vp, _i32, _vp, _i32, _vp, _sz, _i64, _sz, _vp]),
    "sft_ce_fwd_bwd": (_i32, [_i32, _vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _vp, _vp, _vp,
                              _i32, _vp, _i32, _vp, _sz, _i64, _sz, _vp]),
    "adamw_step": (_i32, [_vp, _vp, _vp, _vp, _vp, _i64, _f32, _f32, _f32, _f32, _f32, _i64,
                          _vp]),
    "triton_rule_reward": (_i32, [_vp, _i64, _vp, _i64, _vp, _i32, _i32, _f32, _f32, _vp, _vp,
                               _vp]),
    "grpo_workspace_bytes": (_sz, [_i32, _i32, _i64, _i64, _i64, _i64, _i64, _sz]),
    "grpo_weight_tiled_bytes": (_sz, [_i64, _i64]),
    "grpo_tile_weight": (_i32, [_vp, _i64, _i64, _vp, _sz, _vp]),
    "grpo_check_error": (_i32, [_vp, _vp]),
    "grpo_status_string": (ctypes.c_char_p, [_i32]),
    "grpo_profile_enable": (None, [_i32]),
    "grpo_profile_reset": (None, []),
    "grpo_profile_num_kinds": (_i32, []),
    "grpo_profile_kind_name": (ctypes.c_char_p, [_i32]),
    "grpo_profile_query": (_i32, [_i32, ctypes.POINTER(_i64), ctypes.POINTER(ctypes.c_double)]),
}

_lib = None


class GrpoError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} ({status_string(status)})")


def load(path: str = LIB_PATH):
    """Load libgrpo.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() or "
                               "python -m paper_2507_05687_amd.build")
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def status_string(st: int) -> str:
    return load().grpo_status_string(st).decode()


def _check(st: int, where: str):
    if st != 0:
        raise GrpoError(st, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _need(t, name, dtype=None, device=None):
    if t is None:
        raise ValueError(f"{name} is required")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{name} is on {t.device}, the call's other tensors on "
                         f"cuda:{torch.cuda.current_device()}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    return t


def _extent(t, name, *shape):
    """Raises ValueError unless t (if given) has exactly the given shape; the C ABI
    receives bare pointers and cannot check extents itself."""
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _matrices(hidden, weight):
    """(N, H, V) of hidden [N, H] and weight [V, H]."""
    if hidden.dim() != 2 or weight.dim() != 2:
        raise ValueError("hidden and weight must be 2-D ([N, H] and [V, H])")
    N, H = hidden.shape
    V = weight.shape[0]
    _extent(weight, "weight", V, H)
    return N, H, V


def _on_tensor_device(fn):
    """Runs an entry point with its first device tensor's GPU current, so that
    the library launches on that GPU's current stream."""
    @functools.wraps(fn)
    def wrapped(*args, **kw):
        t = next((a for a in (*args, *kw.values()) if isinstance(a, torch.Tensor) and a.is_cuda),
                 None)
        if t is None:
            return fn(*args, **kw)
        with torch.cuda.device(t.device):
            return fn(*args, **kw)
    return wrapped


# ------------------------------------------------------------ workspace
# One buffer per (device, stream): calls on different streams may overlap and
# must not share scratch; calls on one stream run in order.
_ws_cache: dict = {}


def workspace_bytes(op: int, dt: int, N: int, H: int, V: int, num_seqs: int = 1,
                    max_valid: int = 0, dz_budget: int = 0) -> int:
    return int(load().grpo_workspace_bytes(op, dt, N, H, V, num_seqs, max_valid, dz_budget))


def workspace(nbytes: int, device=None) -> torch.Tensor:
    """A 256-byte-aligned device byte buffer of at least nbytes, cached per
    device and current stream (allocated on, and used only by, that stream, so
    that torch's allocator reuses a replaced buffer only after the work queued
    on it)."""
    device = torch.device(device if device is not None else torch.cuda.current_device())
    key = (device.index, torch.cuda.current_stream(device).cuda_stream)
    buf = _ws_cache.get(key)
    if buf is None or buf.numel() < nbytes + 256:
        _ws_cache.pop(key, None)
        buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        _ws_cache[key] = buf
    off = (-buf.data_ptr()) % 256
    return buf[off:off + nbytes]


def free_workspace():
    _ws_cache.clear()


class TiledWeight:
    """A bf16 head weight [V, H] in the library's tiled operand layout
    (grpo_tile_weight), for calls that share one W: pass it as weight_tiled
    together with the same weight. It is only valid while W is unchanged."""

    def __init__(self, buf: torch.Tensor, V: int, H: int):
        self.buf, self.V, self.H = buf, V, H  # buf: 256-byte-aligned uint8 view


@_on_tensor_device
def tile_weight(weight: torch.Tensor) -> TiledWeight:
    """grpo_tile_weight: W [V, H] bf16 -> a TiledWeight on W's device and stream."""
    _need(weight, "weight", torch.bfloat16)
    if weight.dim() != 2:
        raise ValueError("weight must be 2-D [V, H]")
    V, H = weight.shape
    nbytes = int(load().grpo_weight_tiled_bytes(V, H))
    if nbytes == 0:
        raise ValueError(f"weight shape {(V, H)} is outside the library's limits")
    raw = torch.empty(nbytes + 256, dtype=torch.uint8, device=weight.device)
    off = (-raw.data_ptr()) % 256
    buf = raw[off:off + nbytes]
    st = load().grpo_tile_weight(_ptr(weight), V, H, _ptr(buf), nbytes, _stream())
    _check(st, "grpo_tile_weight")
    return TiledWeight(buf, V, H)


def _tiled(weight_tiled, weight) -> tuple:
    """(pointer, op flag) for an optional TiledWeight matching weight."""
    if weight_tiled is None:
        return None, 0
    if not isinstance(weight_tiled, TiledWeight):
        raise TypeError("weight_tiled must come from tile_weight()")
    if (weight_tiled.V, weight_tiled.H) != tuple(weight.shape) or weight.dtype != torch.bfloat16:
        raise ValueError(f"weight_tiled is for a bf16 [{weight_tiled.V}, {weight_tiled.H}] "
                         f"weight, the call's weight is {weight.dtype} {tuple(weight.shape)}")
    if weight_tiled.buf.device != weight.device:
        raise ValueError("weight_tiled is on another device than weight")
    return _ptr(weight_tiled.buf), WS_TILED_WEIGHT


# ------------------------------------------------------------ entry points
@_on_tensor_device
def group_advantages(rewards: torch.Tensor, group_size: int, std_eps: float = 1e-6,
                     unbiased: bool = True, out: torch.Tensor | None = None) -> torch.Tensor:
    """Eq. 2: per-prompt group-normalised advantages (rewards [P*G] fp32, prompt-major)."""
    _need(rewards, "rewards", torch.float32)
    n = rewards.numel()
    if n % group_size:
        raise ValueError("rewards length must be a multiple of group_size")
    out = torch.empty_like(rewards) if out is None else _need(out, "out", torch.float32)
    if out.numel() != n:
        raise ValueError(f"out has {out.numel()} elements, rewards {n}")
    st = load().group_advantages(_ptr(rewards), n // group_size, group_size, std_eps,
                                 int(unbiased), _ptr(out), _stream())
    _check(st, "group_advantages")
    return out


@_on_tensor_device
def pack_valid(mask: torch.Tensor | None, cu_seqlens: torch.Tensor):
    """(rows int32 [num_valid], counts int32 [B], num_valid int) of the valid rows."""
    _need(cu_seqlens, "cu_seqlens", torch.int64)
    B = cu_seqlens.numel() - 1
    N = int(cu_seqlens[-1].item()) if mask is None else mask.numel()
    dev = cu_seqlens.device
    rows = torch.empty(N, dtype=torch.int32, device=dev)
    counts = torch.empty(B, dtype=torch.int32, device=dev)
    nv = torch.empty(1, dtype=torch.int32, device=dev)
    ws = workspace(workspace_bytes(OP_LOGPROB_FWD, F32, N, 1, 1, B), dev)
    m = None if mask is None else _need(mask, "mask").view(torch.uint8)
    if B < 1:
        raise ValueError("cu_seqlens needs at least two entries")
    st = load().grpo_pack_valid(_ptr(m), _ptr(cu_seqlens), B, N, _ptr(rows), _ptr(counts),
                                _ptr(nv), _ptr(ws), ws.numel(), _stream())
    _check(st, "grpo_pack_valid")
    n = int(nv.item())
    return rows[:n], counts, n


@_on_tensor_device
def logprob_fwd(hidden: torch.Tensor, weight: torch.Tensor, tokens: torch.Tensor,
                mask: torch.Tensor | None = None, check: bool = False, max_valid: int = 0,
                weight_tiled: TiledWeight | None = None):
    """Per-token log-prob and log-sum-exp over the vocabulary: (logp, lse), fp32 [N].
    max_valid: the most valid rows the mask has (0: N), which sizes the workspace;
    weight_tiled: tile_weight(weight), to skip tiling W in this call."""
    _need(hidden, "hidden")
    _need(weight, "weight", hidden.dtype)
    _need(tokens, "tokens", torch.int64)
    N, H, V = _matrices(hidden, weight)
    _extent(tokens.view(-1), "tokens", N)
    if mask is not None and mask.numel() != N:
        raise ValueError(f"mask has {mask.numel()} elements, expected {N}")
    dt = _dt(hidden)
    logp = torch.empty(N, dtype=torch.float32, device=hidden.device)
    lse = torch.empty(N, dtype=torch.float32, device=hidden.device)
    wt, flag = _tiled(weight_tiled, weight)
    ws = workspace(workspace_bytes(OP_LOGPROB_FWD | flag, dt, N, H, V, 1, max_valid),
                   hidden.device)
    m = None if mask is None else _need(mask, "mask").view(torch.uint8)
    st = load().grpo_logprob_fwd(dt, _ptr(hidden), _ptr(weight), wt, _ptr(tokens), _ptr(m), N,
                                 H, V, _ptr(logp), _ptr(lse), _ptr(ws), ws.numel(), max_valid,
                                 _stream())
    _check(st, "grpo_logprob_fwd")
    if check:
        check_error(ws)
    return logp, lse


@_on_tensor_device
def loss_fwd_bwd(hidden, weight, tokens, mask, cu_seqlens, old_logp, ref_logp, adv,
                 clip_eps: float = 0.2, beta: float = 0.0, agg: int = AGG_SEQ_MEAN,
                 lse_in=None, grad_hidden: bool = True, grad_weight: bool = True,
                 grad_hidden_dtype=None, grad_weight_out: torch.Tensor | None = None,
                 accumulate_grad_weight: bool = False, token_outputs: bool = True,
                 check: bool = False, max_valid: int = 0, dz_budget: int = 0,
                 weight_tiled: TiledWeight | None = None) -> dict:
    """GRPO loss (Eq. 1, k3 KL) and its gradients. Returns a dict of tensors:
    loss [1], logp/lse/token_loss/dlogp [N], clip_flag uint8 [N],
    grad_hidden [N,H], grad_weight [V,H] fp32 (as requested). max_valid (0: N)
    and dz_budget (bytes, 0: default) size the workspace (see grpo.h);
    weight_tiled: tile_weight(weight), to skip tiling W in this call."""
    _need(hidden, "hidden")
    _need(weight, "weight", hidden.dtype)
    _need(tokens, "tokens", torch.int64)
    _need(cu_seqlens, "cu_seqlens", torch.int64)
    _need(old_logp, "old_logp", torch.float32)
    _need(adv, "adv", torch.float32)
    if ref_logp is not None:
        _need(ref_logp, "ref_logp", torch.float32)
    if lse_in is not None:
        _need(lse_in, "lse_in", torch.float32)
    N, H, V = _matrices(hidden, weight)
    B = cu_seqlens.numel() - 1
    if B < 1:
        raise ValueError("cu_seqlens needs at least two entries")
    for t, name in ((tokens, "tokens"), (old_logp, "old_logp"), (ref_logp, "ref_logp"),
                    (lse_in, "lse_in"), (mask, "mask")):
        if t is not None and t.numel() != N:
            raise ValueError(f"{name} has {t.numel()} elements, expected N = {N}")
    if adv.numel() != B:
        raise ValueError(f"adv has {adv.numel()} elements, expected one per rollout ({B})")
    dt = _dt(hidden)
    dev = hidden.device
    f32 = dict(dtype=torch.float32, device=dev)
    out = {"loss": torch.empty(1, **f32)}
    if token_outputs:
        out.update(logp=torch.empty(N, **f32), lse=torch.empty(N, **f32),
                   token_loss=torch.empty(N, **f32), dlogp=torch.empty(N, **f32),
                   clip_flag=torch.empty(N, dtype=torch.uint8, device=dev))
    gh_dt = hidden.dtype if grad_hidden_dtype is None else grad_hidden_dtype
    if grad_hidden:
        out["grad_hidden"] = torch.empty(N, H, dtype=gh_dt, device=dev)
    if grad_weight:
        if grad_weight_out is not None:
            out["grad_weight"] = _extent(_need(grad_weight_out, "grad_weight_out",
                                               torch.float32), "grad_weight_out", V, H)
        else:
            out["grad_weight"] = torch.empty(V, H, **f32)
    wt, flag = _tiled(weight_tiled, weight)
    ws = workspace(workspace_bytes(OP_LOSS_FWD_BWD | flag, dt, N, H, V, B, max_valid, dz_budget),
                   dev)
    m = None if mask is None else _need(mask, "mask").view(torch.uint8)
    g = out.get
    st = load().grpo_loss_fwd_bwd(
        dt, _ptr(hidden), _ptr(weight), wt, _ptr(tokens), _ptr(m), _ptr(cu_seqlens), B, N, H, V,
        _ptr(old_logp), _ptr(ref_logp), _ptr(adv), clip_eps, beta, agg, _ptr(lse_in),
        _ptr(out["loss"]), _ptr(g("logp")), _ptr(g("lse")), _ptr(g("token_loss")),
        _ptr(g("dlogp")), _ptr(g("clip_flag")), _ptr(g("grad_hidden")),
        _dt(out["grad_hidden"]) if grad_hidden else F32, _ptr(g("grad_weight")),
        int(accumulate_grad_weight), _ptr(ws), ws.numel(), max_valid, dz_budget, _stream())
    _check(st, "grpo_loss_fwd_bwd")
    if check:
        check_error(ws)
    return out


@_on_tensor_device
def sft_ce_fwd_bwd(hidden, weight, tokens, mask=None, grad_hidden: bool = True,
                   grad_weight: bool = True, grad_hidden_dtype=None,
                   grad_weight_out: torch.Tensor | None = None,
                   accumulate_grad_weight: bool = False, logp_out: bool = True,
                   check: bool = False, max_valid: int = 0, dz_budget: int = 0,
                   weight_tiled: TiledWeight | None = None) -> dict:
    """SFT next-token cross-entropy (mean over supervised tokens) and its gradients.
    Returns loss [1], logp [N] (if logp_out), grad_hidden [N,H], grad_weight [V,H] fp32;
    weight_tiled: tile_weight(weight), to skip tiling W in this call."""
    _need(hidden, "hidden")
    _need(weight, "weight", hidden.dtype)
    _need(tokens, "tokens", torch.int64)
    N, H, V = _matrices(hidden, weight)
    for t, name in ((tokens, "tokens"), (mask, "mask")):
        if t is not None and t.numel() != N:
            raise ValueError(f"{name} has {t.numel()} elements, expected N = {N}")
    dt = _dt(hidden)
    dev = hidden.device
    f32 = dict(dtype=torch.float32, device=dev)
    out = {"loss": torch.empty(1, **f32)}
    if logp_out:
        out["logp"] = torch.empty(N, **f32)
    gh_dt = hidden.dtype if grad_hidden_dtype is None else grad_hidden_dtype
    if grad_hidden:
        out["grad_hidden"] = torch.empty(N, H, dtype=gh_dt, device=dev)
    if grad_weight:
        if grad_weight_out is not None:
            out["grad_weight"] = _extent(_need(grad_weight_out, "grad_weight_out",
                                               torch.float32), "grad_weight_out", V, H)
        else:
            out["grad_weight"] = torch.empty(V, H, **f32)
    wt, flag = _tiled(weight_tiled, weight)
    ws = workspace(workspace_bytes(OP_SFT_FWD_BWD | flag, dt, N, H, V, 1, max_valid, dz_budget),
                   dev)
    m = None if mask is None else _need(mask, "mask").view(torch.uint8)
    g = out.get
    st = load().sft_ce_fwd_bwd(
        dt, _ptr(hidden), _ptr(weight), wt, _ptr(tokens), _ptr(m), N, H, V, _ptr(out["loss"]),
        _ptr(g("logp")), _ptr(g("grad_hidden")),
        _dt(out["grad_hidden"]) if grad_hidden else F32, _ptr(g("grad_weight")),
        int(accumulate_grad_weight), _ptr(ws), ws.numel(), max_valid, dz_budget, _stream())
    _check(st, "sft_ce_fwd_bwd")
    if check:
        check_error(ws)
    return out


@_on_tensor_device
def adamw_step(weight, exp_avg, exp_avg_sq, grad, step: int, lr: float = 1e-6,
               beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
               weight_decay: float = 0.01, weight_bf16: torch.Tensor | None = None):
    """In-place fused AdamW step on fp32 weight/moments; optionally writes a bf16 copy."""
    for t, name in ((weight, "weight"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq"),
                    (grad, "grad")):
        _need(t, name, torch.float32)
    n = weight.numel()
    if any(t.numel() != n for t in (exp_avg, exp_avg_sq, grad)):
        raise ValueError("weight, exp_avg, exp_avg_sq and grad must have the same size")
    if weight_bf16 is not None:
        _need(weight_bf16, "weight_bf16", torch.bfloat16)
        if weight_bf16.numel() != n:
            raise ValueError("weight_bf16 must have the size of weight")
    st = load().adamw_step(_ptr(weight), _ptr(exp_avg), _ptr(exp_avg_sq), _ptr(grad),
                           _ptr(weight_bf16), n, lr, beta1, beta2, eps, weight_decay, int(step),
                           _stream())
    _check(st, "adamw_step")


@_on_tensor_device
def triton_rule_reward(text, offsets, test_passed, require_launch: bool = False,
                       weighted: bool = False, rule_weight: float = 0.0,
                       exec_weight: float = 0.0):
    """(is_triton u8, reward f32) per completion: Eq. 3's product of the
    @triton.jit rule and test_passed, or the weighted sum. text: u8 device
    bytes of the concatenated completions; offsets: int64 [B + 1]."""
    _need(text, "text", torch.uint8)
    _need(offsets, "offsets", torch.int64)
    _need(test_passed, "test_passed", torch.uint8)
    b = offsets.numel() - 1
    if b < 0 or test_passed.numel() != b:
        raise ValueError("offsets must have one entry more than test_passed")
    flags = torch.empty(b, dtype=torch.uint8, device=text.device)
    reward = torch.empty(b, dtype=torch.float32, device=text.device)
    nbytes = text.numel()
    if nbytes == 0:  # every completion is empty: any valid pointer will do
        text = torch.zeros(1, dtype=torch.uint8, device=offsets.device)
    st = load().triton_rule_reward(_ptr(text), nbytes, _ptr(offsets), b, _ptr(test_passed),
                                   int(require_launch), int(weighted), rule_weight, exec_weight,
                                   _ptr(flags), _ptr(reward), _stream())
    _check(st, "triton_rule_reward")
    return flags, reward


@_on_tensor_device
def check_error(ws: torch.Tensor):
    st = load().grpo_check_error(_ptr(ws), _stream())
    _check(st, "device")


# ------------------------------------------------------------ timing
def profile_enable(on: bool = True):
    load().grpo_profile_enable(int(on))


def profile_reset():
    load().grpo_profile_reset()


def profile_read() -> dict:
    """{kernel kind: (launches, total_ms)} for every kind launched since the last reset."""
    lib = load()
    res = {}
    for k in range(lib.grpo_profile_num_kinds()):
        n = ctypes.c_int64(0)
        ms = ctypes.c_double(0.0)
        _check(lib.grpo_profile_query(k, ctypes.byref(n), ctypes.byref(ms)), "profile")
        if n.value:
            res[lib.grpo_profile_kind_name(k).decode()] = (n.value, ms.value)
    return res
