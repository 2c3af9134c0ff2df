"""C-ABI checks that need no GPU: libgrpo.so loads, exports every function
include/grpo.h declares, and rejects bad arguments on the host before any
launch (these paths return before touching the device)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "grpo.h")


@pytest.fixture(scope="module")
def lib():
    from paper_2507_05687_amd import grpo

    if not os.path.exists(grpo.LIB_PATH):
        pytest.skip("libgrpo.so not built")
    return grpo.load()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][\w\s\*]*?\b([a-z_][a-z0-9_]*)\s*\(", text,
                       flags=re.M)
    return sorted(set(n for n in names if n not in ("defined",)))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in ("group_advantages", "grpo_logprob_fwd", "grpo_loss_fwd_bwd",
                     "sft_ce_fwd_bwd", "adamw_step", "triton_rule_reward", "grpo_pack_valid",
                     "grpo_workspace_bytes", "grpo_tile_weight", "grpo_weight_tiled_bytes",
                     "grpo_check_error", "grpo_status_string"):
        assert required in names


def test_every_declared_symbol_is_exported(lib):
    from paper_2507_05687_amd import grpo

    names = _declared_functions()
    assert set(names) == set(grpo.SIGNATURES), "binding and header disagree"
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for st in range(12):
        s = lib.grpo_status_string(st)
        assert s and s != b"unknown status"
    assert lib.grpo_status_string(99) == b"unknown status"


def test_workspace_bytes(lib):
    def ws(op, dt, N, H, V, B, max_valid=0, dz_budget=0):
        return lib.grpo_workspace_bytes(op, dt, N, H, V, B, max_valid, dz_budget)
    assert ws(0, 1, 100, 64, 1000, 1) > 0
    assert ws(1, 1, 100, 64, 1000, 4) > ws(0, 1, 100, 64, 1000, 4)
    assert ws(1, 1, 1000, 64, 1000, 4) > ws(1, 1, 100, 64, 1000, 4)
    assert ws(0, 1, 0, 64, 1000, 1) == 0       # N < 1
    assert ws(0, 1, 10, 60, 1000, 1) == 0      # bf16 needs H % 8 == 0
    assert ws(0, 0, 10, 60, 1000, 1) > 0       # fp32 does not
    assert ws(0, 7, 10, 64, 1000, 1) == 0      # unknown dtype
    assert ws(9, 1, 10, 64, 1000, 1) == 0      # unknown op
    # SFT uses the loss layout with one sequence
    assert ws(2, 1, 100, 64, 1000, 1) == ws(1, 1, 100, 64, 1000, 1)
    assert ws(2, 1, 100, 60, 1000, 1) == 0
    # full-size loss workspace stays well inside one MI355X's 288 GB
    assert ws(1, 1, 131072, 4096, 155136, 64) < 32 << 30
    # the bf16 backward takes at most 2^22 rows per call (the scoring alone more)
    assert ws(1, 1, 1 << 22, 64, 1000, 1) > 0 and ws(2, 1, 1 << 22, 64, 1000, 1) > 0
    assert ws(1, 1, (1 << 22) + 1, 64, 1000, 1) == 0
    assert ws(2, 1, (1 << 22) + 1, 64, 1000, 1) == 0
    assert ws(0, 1, (1 << 22) + 1, 64, 1000, 1) > 0
    assert ws(1, 0, (1 << 22) + 1, 64, 1000, 1) > 0
    # max_valid caps the token-indexed buffers; beyond N (or negative) it is an error
    full = ws(1, 1, 131072, 4096, 155136, 64)
    assert ws(1, 1, 131072, 4096, 155136, 64, 131072) == full
    # (at a fixed logits-gradient budget: fewer rows otherwise get wider chunks)
    assert (ws(1, 1, 131072, 4096, 155136, 64, 65536, 4 << 30) <
            ws(1, 1, 131072, 4096, 155136, 64, 0, 4 << 30) - (1 << 30))
    assert ws(1, 1, 131072, 4096, 155136, 64, 131073) == 0
    assert ws(1, 1, 131072, 4096, 155136, 64, -1) == 0
    assert ws(0, 1, 1000, 64, 1000, 1, 100) < ws(0, 1, 1000, 64, 1000, 1)
    # a smaller logits-gradient budget gives a smaller workspace
    assert ws(1, 1, 131072, 4096, 155136, 64, 0, 4 << 30) < full - (2 << 30)
    assert ws(2, 1, 131072, 4096, 155136, 1, 0, 4 << 30) < ws(2, 1, 131072, 4096, 155136, 1)


NULL = None
P = ctypes.c_void_p(0x1000)  # a non-NULL, 256-byte-aligned dummy (never dereferenced)


def _loss(lib, **kw):
    a = dict(dt=1, hidden=P, weight=P, wt=NULL, tokens=P, mask=NULL, cu=P, B=2, N=8, H=64, V=100,
             old=P, ref=P, adv=P, eps=0.2, beta=0.01, agg=0, lse_in=NULL, loss=P, logp=NULL,
             lse=NULL, tl=NULL, dlogp=NULL, clip=NULL, gh=NULL, gh_dt=1, gw=NULL, acc=0,
             ws=NULL, ws_bytes=0, max_valid=0, dz_budget=0, stream=NULL)
    a.update(kw)
    return lib.grpo_loss_fwd_bwd(*a.values())


def test_loss_argument_errors(lib):
    assert _loss(lib, hidden=NULL) == 1
    assert _loss(lib, loss=NULL) == 1
    assert _loss(lib, beta=0.1, ref=NULL) == 1
    assert _loss(lib, N=0) == 2
    assert _loss(lib, N=(1 << 22) + 1) == 2
    assert _loss(lib, H=60) == 2
    assert _loss(lib, B=0) == 2
    assert _loss(lib, B=9) == 2
    assert _loss(lib, dt=5) == 3
    assert _loss(lib, gh=P, gh_dt=7) == 3
    assert _loss(lib, dt=0, gh=P, gh_dt=1) == 3
    assert _loss(lib, eps=0.0) == 4
    assert _loss(lib, eps=1.0) == 4
    assert _loss(lib, beta=-1.0) == 4
    assert _loss(lib, beta=float("nan")) == 4
    assert _loss(lib, agg=3) == 4
    assert _loss(lib, hidden=ctypes.c_void_p(0x1008)) == 5
    for k in ("ref", "lse_in", "logp", "lse", "tl", "dlogp", "gw"):
        assert _loss(lib, **{k: ctypes.c_void_p(0x1002)}) == 5, k
    assert _loss(lib) == 6                          # no workspace
    assert _loss(lib, ws=ctypes.c_void_p(0x1010), ws_bytes=1 << 40) == 6  # misaligned
    assert _loss(lib, ws=P, ws_bytes=16) == 6       # too small
    assert _loss(lib, max_valid=-1) == 2
    assert _loss(lib, max_valid=9) == 2             # more than N


def test_other_entry_point_errors(lib):
    adv = lib.group_advantages
    assert adv(NULL, 2, 4, 1e-6, 1, P, NULL) == 1
    assert adv(P, 2, 1, 1e-6, 1, P, NULL) == 2
    assert adv(P, 0, 4, 1e-6, 1, P, NULL) == 2
    assert adv(P, 2, 4, -1.0, 1, P, NULL) == 4
    # one wave per prompt: the grid's thread count must stay below 2^32
    assert adv(P, 4 * ((1 << 24) - 1) + 1, 2, 1e-6, 1, P, NULL) == 2
    fwd = lib.grpo_logprob_fwd
    assert fwd(1, NULL, P, NULL, P, NULL, 8, 64, 100, P, P, P, 1 << 30, 0, NULL) == 1
    assert fwd(1, P, P, NULL, P, NULL, 8, 12, 100, P, P, P, 1 << 30, 0, NULL) == 2
    assert fwd(1, P, P, NULL, P, NULL, 8, 64, 0, P, P, P, 1 << 30, 0, NULL) == 2
    assert fwd(2, P, P, NULL, P, NULL, 8, 64, 100, P, P, P, 1 << 30, 0, NULL) == 3
    assert fwd(1, P, P, NULL, P, NULL, 8, 64, 100, P, P, P, 8, 0, NULL) == 6
    # bf16 scoring grid beyond 32 bits; fp32 H beyond its LDS rows
    assert fwd(1, P, P, NULL, P, NULL, 1 << 22, 8, (1 << 31) - 512, P, P, P, 1 << 30, 0, NULL) == 2
    assert fwd(0, P, P, NULL, P, NULL, 8, 8200, 100, P, P, P, 1 << 30, 0, NULL) == 2
    assert fwd(1, P, P, NULL, P, NULL, 8, 64, 100, P, P, P, 1 << 30, 9, NULL) == 2
    pk = lib.grpo_pack_valid
    assert pk(NULL, NULL, 2, 8, P, P, P, P, 1 << 30, NULL) == 1
    assert pk(NULL, P, 0, 8, P, P, P, P, 1 << 30, NULL) == 2
    assert pk(NULL, P, 2, 8, P, P, P, NULL, 0, NULL) == 6
    assert lib.grpo_check_error(NULL, NULL) == 1


def test_tiled_weight_host_checks(lib):
    tb = lib.grpo_weight_tiled_bytes
    # 256-row x 32-column bf16 blocks, ceil(H/32) + 1 blocks per tile-row
    assert tb(100, 64) == 2 * 256 * (2 + 1) * 32
    assert tb(155136, 4096) == 2 * 155136 * (128 + 1) * 32
    assert tb(257, 8) == 2 * 512 * 2 * 32
    assert tb(0, 64) == 0 and tb(100, 60) == 0 and tb(100, 1 << 20) == 0
    # a workspace for a call given the tiled weight holds no copy of it
    flag = 0x100
    for op, B in ((0, 1), (1, 4), (2, 1)):
        full = lib.grpo_workspace_bytes(op, 1, 1000, 4096, 155136, B, 0, 0)
        lean = lib.grpo_workspace_bytes(op | flag, 1, 1000, 4096, 155136, B, 0, 0)
        assert full - lean == tb(155136, 4096), op
    assert lib.grpo_workspace_bytes(0 | flag, 0, 1000, 64, 1000, 1, 0, 0) == 0  # bf16 only
    tile = lib.grpo_tile_weight
    big = 1 << 40
    assert tile(NULL, 100, 64, P, big, NULL) == 1
    assert tile(P, 100, 64, NULL, big, NULL) == 1
    assert tile(P, 100, 60, P, big, NULL) == 2
    assert tile(P, 0, 64, P, big, NULL) == 2
    assert tile(P, 100, 64, P, tb(100, 64) - 1, NULL) == 2    # out too small
    assert tile(ctypes.c_void_p(0x1008), 100, 64, P, big, NULL) == 5
    assert tile(P, 100, 64, ctypes.c_void_p(0x1010), big, NULL) == 5
    # the compute calls: bf16 only, 256-byte aligned; the lean workspace needs it
    fwd = lib.grpo_logprob_fwd
    assert fwd(0, P, P, P, P, NULL, 8, 64, 100, P, P, P, 1 << 30, 0, NULL) == 3
    assert fwd(1, P, P, ctypes.c_void_p(0x1010), P, NULL, 8, 64, 100, P, P, P, 1 << 30, 0,
               NULL) == 5
    lean = lib.grpo_workspace_bytes(0 | flag, 1, 8, 64, 100, 1, 0, 0)
    assert fwd(1, P, P, NULL, P, NULL, 8, 64, 100, P, P, P, lean, 0, NULL) == 6
    assert _loss(lib, dt=0, wt=P) == 3
    assert _loss(lib, wt=ctypes.c_void_p(0x1040)) == 5
    lean = lib.grpo_workspace_bytes(1 | flag, 1, 8, 64, 100, 2, 0, 0)
    assert _loss(lib, ws=P, ws_bytes=lean) == 6
    assert _sft(lib, dt=0, wt=P) == 3
    lean = lib.grpo_workspace_bytes(2 | flag, 1, 8, 64, 100, 1, 0, 0)
    assert _sft(lib, ws=P, ws_bytes=lean) == 6


def _sft(lib, **kw):
    a = dict(dt=1, hidden=P, weight=P, wt=NULL, tokens=P, mask=NULL, N=8, H=64, V=100, loss=P,
             logp=NULL, gh=NULL, gh_dt=1, gw=NULL, acc=0, ws=NULL, ws_bytes=0, max_valid=0,
             dz_budget=0, stream=NULL)
    a.update(kw)
    return lib.sft_ce_fwd_bwd(*a.values())


def test_sft_argument_errors(lib):
    assert _sft(lib, hidden=NULL) == 1
    assert _sft(lib, tokens=NULL) == 1
    assert _sft(lib, loss=NULL) == 1
    assert _sft(lib, N=0) == 2
    assert _sft(lib, N=(1 << 22) + 1) == 2
    assert _sft(lib, H=60) == 2
    assert _sft(lib, dt=4) == 3
    assert _sft(lib, gh=P, gh_dt=7) == 3
    assert _sft(lib, dt=0, gh=P, gh_dt=1) == 3
    assert _sft(lib, weight=ctypes.c_void_p(0x1008)) == 5
    assert _sft(lib, logp=ctypes.c_void_p(0x1002)) == 5
    assert _sft(lib) == 6                           # no workspace
    assert _sft(lib, ws=P, ws_bytes=16) == 6        # too small
    assert _sft(lib, max_valid=9) == 2


def test_adamw_argument_errors(lib):
    f = lib.adamw_step
    a = [P, P, P, P, NULL, 10, 1e-3, 0.9, 0.999, 1e-8, 0.01, 1, NULL]

    def call(i, x):
        b = list(a)
        b[i] = x
        return f(*b)

    assert call(0, NULL) == 1
    assert call(3, NULL) == 1
    assert call(5, 0) == 2                # n
    assert call(11, 0) == 2               # step
    assert call(6, -1.0) == 4             # lr
    assert call(7, 1.0) == 4              # beta1
    assert call(8, -0.1) == 4             # beta2
    assert call(9, 0.0) == 4              # eps
    assert call(10, float("inf")) == 4    # weight decay
    assert call(1, ctypes.c_void_p(0x1004)) == 5
    assert call(4, ctypes.c_void_p(0x1002)) == 5


def test_rule_reward_argument_errors(lib):
    f = lib.triton_rule_reward
    a = [P, 64, P, 4, P, 0, 0, 0.0, 0.0, P, P, NULL]

    def call(i, x):
        b = list(a)
        b[i] = x
        return f(*b)

    assert call(3, -1) == 2                  # count
    assert call(3, 1 << 31) == 2
    assert call(1, -1) == 2                  # text_bytes
    assert call(0, NULL) == 1
    assert call(2, NULL) == 1
    assert call(4, NULL) == 1
    assert call(9, NULL) == 1
    assert call(10, NULL) == 1
    assert call(5, 2) == 4                   # require_launch
    assert call(6, -1) == 4                  # weighted
    assert call(7, float("nan")) == 4
    assert call(8, float("inf")) == 4
    assert call(0, ctypes.c_void_p(0x1008)) == 5   # text not 16-byte aligned
    assert call(2, ctypes.c_void_p(0x1004)) == 5
    assert call(3, 0) == 0                   # nothing to do: no launch, no device needed
    assert f(NULL, 0, NULL, 0, NULL, 0, 0, 0.0, 0.0, NULL, NULL, NULL) == 0


def test_profile_interface_without_launches(lib):
    n = lib.grpo_profile_num_kinds()
    assert n >= 8
    names = [lib.grpo_profile_kind_name(k).decode() for k in range(n)]
    assert "gemm_logits_lse" in names and "gemm_grad_weight" in names
    lib.grpo_profile_reset()
    c = ctypes.c_int64(-1)
    t = ctypes.c_double(-1)
    assert lib.grpo_profile_query(0, ctypes.byref(c), ctypes.byref(t)) == 0
    assert c.value == 0 and t.value == 0.0
    assert lib.grpo_profile_query(n, ctypes.byref(c), ctypes.byref(t)) == 4


def test_binding_rejects_host_tensors():
    # argument marshalling checks run before any library call
    import torch

    from paper_2507_05687_amd import grpo

    x = torch.zeros(8)
    with pytest.raises(ValueError, match="device tensor"):
        grpo.group_advantages(x, 4)
    bf = torch.zeros(4, 8, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="device tensor"):
        grpo.logprob_fwd(bf, bf, torch.zeros(4, dtype=torch.int64))


def test_static_pack_limits_without_a_device(lib):
    f = lib.grpo_pack_valid_static
    assert f(NULL, NULL, 4, 100, P, P, P, NULL, NULL) == 1
    assert f(NULL, P, 4, 100, NULL, P, P, NULL, NULL) == 1
    assert f(NULL, P, 0, 100, P, P, P, NULL, NULL) == 2
    assert f(NULL, P, 101, 100, P, P, P, NULL, NULL) == 2
    # more rollouts than the static scratch holds
    assert f(NULL, P, (1 << 20) + 1, 1 << 21, P, P, P, NULL, NULL) == 6


def test_binding_fails_loudly_without_the_library(monkeypatch):
    # no fallback: a missing libgrpo.so is an error, not a silent CPU path
    from paper_2507_05687_amd import grpo

    monkeypatch.setattr(grpo, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        grpo.load("/nonexistent/libgrpo.so")
