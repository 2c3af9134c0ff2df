"""The allocation-free packing entry point (grpo_pack_valid_static) against
grpo_pack_valid, through the C ABI: bit-exact rows, counts and valid count on
two calls in a row (the second smaller, so that it runs on the scratch the
first one left behind), and its error output. GPU only."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2507_05687_amd import grpo

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _setup():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    grpo.load()
    yield
    grpo.free_workspace()


def _batch(B, T, seed, ragged=True):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, T + 1, B) if ragged else np.full(B, T)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    N = int(cu[-1])
    mask = (rng.random(N) < 0.7).astype(np.uint8)
    return cu, mask


def _static(cu_d, mask_d, N, B):
    lib = grpo.load()
    rows = torch.full((N,), -7, dtype=torch.int32, device="cuda")
    counts = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    nv = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    err = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    st = lib.grpo_pack_valid_static(grpo._ptr(mask_d), grpo._ptr(cu_d), B, N, grpo._ptr(rows),
                                    grpo._ptr(counts), grpo._ptr(nv), grpo._ptr(err),
                                    grpo._stream())
    assert st == 0, grpo.status_string(st)
    torch.cuda.synchronize()
    return rows, counts, int(nv.item()), int(err.item())


def test_static_pack_matches_workspace_pack_twice():
    for B, T, seed in [(300, 200, 1), (9, 50, 2)]:  # the second call is smaller
        cu, mask = _batch(B, T, seed)
        N = int(cu[-1])
        cu_d, mask_d = torch.from_numpy(cu).cuda(), torch.from_numpy(mask).cuda()
        want_rows, want_counts, want_n = grpo.pack_valid(mask_d, cu_d)
        rows, counts, n, err = _static(cu_d, mask_d, N, B)
        assert err == 0
        assert n == want_n == int(mask.sum())
        assert torch.equal(rows[:n], want_rows)
        assert torch.equal(counts, want_counts)
        assert np.array_equal(rows[:n].cpu().numpy(), np.flatnonzero(mask))


def test_static_pack_without_mask_and_bad_seqlens():
    cu = np.array([0, 5, 3, 12], dtype=np.int64)  # not monotone
    cu_d = torch.from_numpy(cu).cuda()
    rows, counts, n, err = _static(cu_d, None, 12, 3)
    assert err == 10  # GRPO_ERR_SEQLENS
    # a well-formed call on the same scratch starts clean
    cu = np.array([0, 5, 9, 12], dtype=np.int64)
    cu_d = torch.from_numpy(cu).cuda()
    rows, counts, n, err = _static(cu_d, None, 12, 3)
    assert err == 0 and n == 12
    assert counts.cpu().tolist() == [5, 4, 3]
    assert rows.cpu().tolist() == list(range(12))


def test_static_pack_rejects_more_rollouts_than_its_scratch():
    lib = grpo.load()
    P = ctypes.c_void_p(0x1000)
    assert lib.grpo_pack_valid_static(None, P, (1 << 20) + 1, 1 << 21, P, P, P, None, None) == 6
