"""GPU parity of the rule-based reward (Sec. 3.3, Eq. 3) against the oracle:
flags and rewards bit-exact on seeded synthetic completions, hand-written
cases and edge cases, through the C-ABI."""
import numpy as np
import pytest
import torch

import oracle
from paper_2507_05687_amd import grpo, workloads

from test_rule_reward_pins import CASES

pytestmark = pytest.mark.gpu


def _run(texts, passed, **kw):
    data, offsets = workloads.pack_completions(texts)
    flags, reward = grpo.triton_rule_reward(torch.from_numpy(data).cuda(),
                                            torch.from_numpy(offsets).cuda(),
                                            torch.from_numpy(np.asarray(passed, np.uint8)).cuda(),
                                            **kw)
    torch.cuda.synchronize()
    return flags.cpu().numpy(), reward.cpu().numpy()


def _check(texts, passed, **kw):
    for launch in (False, True):
        got_f, got_r = _run(texts, passed, require_launch=launch, **kw)
        want_f, want_r = oracle.rule_rewards(texts, passed, require_launch=launch, **kw)
        bad = np.flatnonzero(got_f != want_f)
        assert bad.size == 0, (launch, bad[:5], texts[bad[0]][:400])
        assert np.array_equal(got_r.view(np.uint32), want_r.view(np.uint32)), launch


@pytest.mark.parametrize("seed", [0, 1])
def test_generated_completions(seed):
    texts, passed = workloads.make_completions(300, seed=seed, mean_len=1500)
    _check(texts, passed)
    _check(texts, passed, weighted=True, rule_weight=0.1, exec_weight=0.9)


def test_hand_written_cases():
    texts = [c[0].encode() for c in CASES]
    passed = np.ones(len(texts), np.uint8)
    f0, _ = _run(texts, passed)
    f1, _ = _run(texts, passed, require_launch=True)
    assert np.array_equal(f0, np.array([c[1] for c in CASES], np.uint8))
    assert np.array_equal(f1, np.array([c[2] for c in CASES], np.uint8))


def test_full_size_batch():
    # 8 prompts x G = 8 completions of up to 16,384 tokens (about 4 bytes each)
    texts, passed = workloads.make_completions(64, seed=7, mean_len=30000, max_len=65536)
    assert max(len(t) for t in texts) > 60000
    _check(texts, passed)


def test_edges():
    kernel = b"@triton.jit\ndef k(x):\n    pass\n"
    long_filler = b"x = 1\n" * 200000  # 1.2 MB
    texts = [
        b"", b"@", b"@triton.jit", kernel, kernel + b"k[(1,)](0)\n",
        b"k[(1,)](0)\n" + long_filler + kernel,           # launch far before the kernel
        kernel + long_filler + b"k[" + b"[" * 5000,         # unclosed brackets to the end
        kernel.replace(b"\n", b"\r\n") + "# é ü\n".encode() + b"\x00\xff k [g]\t(1)",
        b"@triton.jit\n" * 300 + b"def k(x):\n    pass\nk[1](2)\n",  # decorators stacked
    ]
    # more decorated functions than the per-completion list holds
    many = b"".join(b"@triton.jit\ndef k%d(x):\n    pass\n" % i for i in range(100))
    texts += [many, many + b"k99[1](0)\n", many + b"k100[1](0)\n"]
    # long bracket runs: nested, balanced and not, over lines
    texts += [kernel + b"k[" + b"[]" * 3000 + b"](0)",
              kernel + b"k[" + b"x]" * 50 + b"[" * 40 + b"]" * 41 + b"(1)",
              kernel + b"k [" + b"[[]]\n" * 1000 + b"]\t(1)",
              b"@triton.jit(" + b"(" * 100 + b")" * 101 + b"\ndef q(x):\n  pass\nq[0](1)"]
    passed = np.array([1, 0] * 8, np.uint8)
    _check(texts, passed)
    # no completions; only empty ones
    f, r = _run([], [])
    assert f.size == 0 and r.size == 0
    f, r = _run([b"", b""], [1, 1])
    assert np.array_equal(f, [0, 0]) and np.array_equal(r, [0.0, 0.0])


def test_deep_decorator_stacks():
    # repetition loops of decorators (each resolved up to the next one of the
    # same function), with the lines where that shortcut must not apply: text
    # after the decorator, a parenthesis inside its comment, arguments over
    # several lines, other decorators in between, no function at the end
    n = 1500
    kernel = b"def k(x):\n    pass\nk[1](0)\n"
    stacks = [
        b"@triton.jit\n" * n + kernel,
        b"@triton.jit\n" * n,
        b"@triton.jit\n" * n + b"x = 1\n" + kernel,
        b"@triton.jit\n" * (n // 2) + b"@triton.jit x\n" + b"@triton.jit\n" * (n // 2) + kernel,
        b"@triton.jit x\n" * n + kernel,
        b"@triton.jit  # f(x)\n" * n + kernel,
        b"@triton.jit  # f(x\n" * n + kernel,
        b"@triton.jit(\n  a=(1, 2),\n)\n" * (n // 3) + kernel,
        (b"@triton.jit\n@triton.autotune(configs=[])\n" * (n // 2)) + kernel,
        b"\t@triton.jit()\n\n# c\n" * (n // 2) + kernel,
        b"@triton.jit\n" * n + b"def 9k(x):\n",
    ]
    _check(stacks, np.array([1, 0] * 5 + [1], np.uint8))


def test_repeated_definitions():
    # more decorated functions than the name list holds: one definition
    # repeated (searched once), a few alternating, and distinct names with the
    # only launch at the end or of an earlier name
    one = b"@triton.jit\ndef add(x):\n    pass\n"
    alt = b"".join(b"@triton.jit\ndef f%d(x):\n    pass\n" % (i % 3) for i in range(300))
    distinct = b"".join(b"@triton.jit\ndef g%d(x):\n    pass\n" % i for i in range(150))
    texts = [one * 400, one * 400 + b"add[(1,)](0)\n", one * 200 + b"adder[1](0)\n" + one * 200,
             alt, alt + b"f2[g](1)\n", alt + b"f3[g](1)\n",
             distinct + b"g149[1](0)\n", distinct + b"g0[1](0)\n", distinct + b"g150[1](0)\n"]
    _check(texts, np.ones(len(texts), np.uint8))


def test_decreasing_offsets_count_as_empty():
    data = np.frombuffer(b"@triton.jit\ndef k(x):\n    pass\n", np.uint8).copy()
    offsets = np.array([0, len(data), 5], np.int64)
    flags, reward = grpo.triton_rule_reward(torch.from_numpy(data).cuda(),
                                            torch.from_numpy(offsets).cuda(),
                                            torch.ones(2, dtype=torch.uint8, device="cuda"))
    assert flags.cpu().tolist() == [1, 0]
    assert reward.cpu().tolist() == [1.0, 0.0]


def test_many_small_completions():
    texts, passed = workloads.make_completions(4096, seed=3, mean_len=300, max_len=2000)
    _check(texts, passed)


def test_reward_feeds_group_advantages():
    # Eq. 3 rewards of G = 8 rollouts per prompt into Eq. 2
    texts, passed = workloads.make_completions(64, seed=5, mean_len=800)
    data, offsets = workloads.pack_completions(texts)
    _, reward = grpo.triton_rule_reward(torch.from_numpy(data).cuda(),
                                        torch.from_numpy(offsets).cuda(),
                                        torch.from_numpy(passed).cuda())
    adv = grpo.group_advantages(reward, 8).cpu().numpy()
    _, want_r = oracle.rule_rewards(texts, passed)
    want = oracle.advantages(want_r.astype(np.float64), 8)
    assert np.max(np.abs(adv - want)) <= 1e-5 * max(1.0, np.max(np.abs(want)))


def test_offsets_outside_the_text_are_empty_completions():
    # pairs reaching before the text or past text_bytes count as empty
    # completions (no byte outside the buffer is read), as decreasing ones do
    good = b"@triton.jit\ndef k(x):\n    pass\nk[(1,)](x)\n"
    data, offsets = workloads.pack_completions([good, good])
    n = len(data)
    bad = np.array([0, len(good), -16, n + 64, 3, 1 << 40], dtype=np.int64)
    offs = np.concatenate([offsets, bad])
    # completions: good, good, [n, 0) decreasing, [0, len) good again,
    # [len, -16) and [-16, n+64) and [n+64, 3) and [3, 2^40) outside the text
    passed = np.ones(len(offs) - 1, np.uint8)
    flags, reward = grpo.triton_rule_reward(torch.from_numpy(data).cuda(),
                                            torch.from_numpy(offs).cuda(),
                                            torch.from_numpy(passed).cuda(), require_launch=True,
                                            weighted=True, rule_weight=0.25, exec_weight=0.5)
    torch.cuda.synchronize()
    f = flags.cpu().numpy()
    assert list(f) == [1, 1, 0, 1, 0, 0, 0, 0]
    assert np.allclose(reward.cpu().numpy(), np.where(f == 1, 0.75, 0.5))


# ---- adversarial completions: the check's cost per completion is bounded

KERNEL_K = b"@triton.jit\ndef k(x):pass\n"


def _distinct_names(count, launch=None):
    """count decorated functions with distinct names (28 bytes each), then
    optionally a launch line."""
    text = b"".join(b"@triton.jit\ndef n%04d(x):pass\n" % i for i in range(count))
    return text + (launch or b"")


def _unclosed(count, tail=b""):
    """a decorated k, then count unclosed launch candidates k[ (2 bytes each)"""
    return KERNEL_K + b"k[" * count + tail


def _timed_flags(texts, require_launch):
    data, offsets = workloads.pack_completions(texts)
    d, o = torch.from_numpy(data).cuda(), torch.from_numpy(offsets).cuda()
    p = torch.ones(len(texts), dtype=torch.uint8, device="cuda")
    grpo.triton_rule_reward(d, o, p, require_launch=require_launch)  # warm-up
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    f, _ = grpo.triton_rule_reward(d, o, p, require_launch=require_launch)
    e1.record()
    torch.cuda.synchronize()
    return f.cpu().numpy(), e0.elapsed_time(e1)


def test_many_distinct_names_parity():
    # parity with the oracle at full size: 2,200 names per completion (61.6 KB)
    texts = [_distinct_names(2200),
             _distinct_names(2200, b"n2199[(1,)](0)\n"),
             _distinct_names(2200, b"n2200[(1,)](0)\n"),   # not a decorated name
             _distinct_names(2200, b"n0000 [g]\t(1)\n"),
             _distinct_names(2200, b"xn0001[g](1)\n"),      # preceded by an identifier byte
             _distinct_names(3000)]
    _check(texts, np.ones(len(texts), np.uint8))


def test_many_distinct_names_batch_time():
    texts = [_distinct_names(2200)] * 64
    f, ms = _timed_flags(texts, require_launch=True)
    print(f"64 completions x 2,200 distinct names, no launch: {ms:.2f} ms")
    assert not f.any()
    assert ms < 10.0


def test_unclosed_candidates_parity():
    # the oracle's bracket matching is quadratic here: parity at 4,000 candidates
    texts = [_unclosed(4000), _unclosed(4000, b"](0)"), _unclosed(4000, b"]"),
             _unclosed(4000, b"]" * 3999 + b" (1)"), _unclosed(4000, b"]" * 4000 + b"(1)"),
             _unclosed(4000, b"\n" + b"]" * 2000 + b"(1)")]
    _check(texts, np.ones(len(texts), np.uint8))


def test_unclosed_candidates_batch_time():
    # 32,000 unclosed k[ per completion (64 KB); the answer follows from the
    # construction: no "[" is ever closed, so there is no launch; closing the
    # last one with "](" makes a launch of k
    texts = [_unclosed(32000)] * 63 + [_unclosed(32000, b"](0)")]
    f, ms = _timed_flags(texts, require_launch=True)
    print(f"64 completions x 32,000 unclosed k[: {ms:.2f} ms")
    assert not f[:63].any() and f[63] == 1
    assert ms < 10.0
    f0, _ = _timed_flags(texts, require_launch=False)
    assert f0.all()


def test_bracket_soup():
    # random runs of launch-like tokens over decorated k and j: every bracket
    # match of the index against the oracle's scan
    rng = np.random.default_rng(11)
    alphabet = [b"k", b"j", b"q", b"[", b"]", b"(", b")", b" ", b"\n", b"[", b"]", b"x"]
    texts = []
    for i in range(64):
        n = int(rng.integers(200, 3000))
        body = b"".join(alphabet[c] for c in rng.integers(0, len(alphabet), n))
        head = b"@triton.jit\ndef k(x):pass\n@triton.jit\ndef j(y):pass\n"
        texts.append(head + body if i % 2 else body + b"\n" + head)
    _check(texts, np.ones(len(texts), np.uint8))


# ---- completions longer than the LDS copy (96 KiB): the same bounded passes
# over the caller's text, with a coarser bracket index

def test_long_generated_completions():
    # generated sources of 100-400 KB, the last one ending the text (its
    # length not a multiple of 16), against the oracle
    texts, passed = workloads.make_completions(16, seed=5, mean_len=250_000, max_len=400_000)
    keep = [i for i, t in enumerate(texts) if len(t) > 96 * 1024]
    texts = [texts[i] + b"x" * (131 if i % 3 == 0 else 0) for i in keep]
    passed = passed[keep]
    assert len(texts) >= 8 and len(b"".join(texts)) % 16 != 0
    _check(texts, passed)


def test_long_adversarial_completions():
    # 9,000 distinct decorated names (270 KB): more than the long path's name
    # table takes, so the names are taken in rounds by hash class (8,000 too);
    # 128,000 unclosed k[ (256 KB)
    texts = [_distinct_names(8000), _distinct_names(8000, b"n7999[(1,)](0)\n"),
             _distinct_names(9000, b"n8999[(1,)](0)\n"), _distinct_names(9000),
             _distinct_names(8000, b"n8000[(1,)](0)\n")]
    _check(texts, np.ones(len(texts), np.uint8))
    big = [_unclosed(128000)] * 15 + [_unclosed(128000, b"](0)")]
    f, ms = _timed_flags(big, require_launch=True)
    print(f"16 completions x 128,000 unclosed k[ (256 KB): {ms:.2f} ms")
    assert not f[:15].any() and f[15] == 1
    assert ms < 100.0
    f, ms = _timed_flags([_distinct_names(8000)] * 16, require_launch=True)
    print(f"16 completions x 8,000 distinct names (240 KB), no launch: {ms:.2f} ms")
    assert not f.any()
    assert ms < 100.0


def test_long_bracket_soup():
    # a 200 KB soup of launch-like tokens around decorated k and j: parity at
    # the coarser index granularity (one index chunk spans several 32-byte parts)
    rng = np.random.default_rng(12)
    alphabet = [b"k", b"j", b"q", b"[", b"]", b"(", b")", b" ", b"\n", b"[", b"]", b"x"]
    head = b"@triton.jit\ndef k(x):pass\n@triton.jit\ndef j(y):pass\n"
    texts = []
    for i in range(4):
        body = b"".join(alphabet[c] for c in rng.integers(0, len(alphabet), 200_000 + 977 * i))
        texts.append(head + body if i % 2 else body + b"\n" + head)
    _check(texts, np.ones(len(texts), np.uint8))
