"""Pins for the rule-based reward oracle (Sec. 3.3, Eq. 3; the @triton.jit
check and the never-launched kernel of Sec. 4).

The paper prints no worked example, so the oracle is pinned by hand-written
completions whose flags follow from the stated rule, and by Python's own
parser (the ast module, a library routine independent of the oracle's byte
scanning) on syntactically valid generated completions, where the lexical
rule and the syntax tree must agree.
"""
import ast

import numpy as np
import pytest

from oracle import rule_reward as rr
from paper_2507_05687_amd import workloads

KERNEL = "def add(x_ptr, n):\n    tl.store(x_ptr, n)\n"
LAUNCH = "def run(x):\n    add[(1,)](x, 4)\n"

# (completion, is_Triton without the launch requirement, with it)
CASES = [
    ("", False, False),
    ("@triton.jit\n" + KERNEL + LAUNCH, True, True),
    ("@triton.jit\n" + KERNEL, True, False),                      # never launched
    ("# @triton.jit\n" + KERNEL + LAUNCH, False, False),          # commented out
    ("@triton.jitted\n" + KERNEL + LAUNCH, False, False),         # another attribute
    ("@triton.jit.fn\n" + KERNEL + LAUNCH, False, False),
    ("x = 1 @triton.jit\n" + KERNEL + LAUNCH, False, False),      # not at line start
    ("   \t@triton.jit\n" + KERNEL + LAUNCH, True, True),         # indented
    ("@triton.jit()\n" + KERNEL + LAUNCH, True, True),
    ("@triton.jit(\n  debug=(1, 2),\n)  # args\n" + KERNEL + LAUNCH, True, True),
    ("@triton.jit(\n" + KERNEL + LAUNCH, False, False),           # unclosed arguments
    ("@triton.jit x\n" + KERNEL + LAUNCH, False, False),          # text after it
    ("@triton.autotune(configs=[\n  1])\n@triton.jit\n" + KERNEL + LAUNCH, True, True),
    ("@triton.jit\n@triton.heuristics({'a': (1)})\n\n# c\n" + KERNEL + LAUNCH, True, True),
    ("@triton.jit\nvalue = 3\n" + KERNEL + LAUNCH, False, False),  # no function follows
    ("@triton.jit\n", False, False),
    ("@triton.jit", False, False),
    ("@triton.jit\ndef 9add(x):\n    pass\n", False, False),       # not a name
    ("@triton.jit\ndef\tadd (x):\n    pass\nadd  [g] (x)\n", True, True),
    ("@triton.jit\n" + KERNEL + "def run(x):\n    spec = add[(1,)]\n", True, False),  # no call
    ("@triton.jit\n" + KERNEL + "def run(x):\n    add2[(1,)](x)\n", True, False),     # other name
    ("@triton.jit\n" + KERNEL + "def run(x):\n    madd[(1,)](x)\n", True, False),     # suffix match
    ("@triton.jit\n" + KERNEL + "def run(x):\n    ops.add[(1,)](x)\n", True, True),   # via module
    ("@triton.jit\n" + KERNEL + "def run(x):\n    add[(f(x[0]), [2])](x)\n", True, True),
    ("@triton.jit\n" + KERNEL + "def run(x):\n    add[(1,)(x)\n", True, False),       # unclosed
    ("@triton.jit\r\n" + KERNEL.replace("\n", "\r\n") + LAUNCH.replace("\n", "\r\n"), True, True),
    ("def helper():\n    pass\n@triton.jit\n" + KERNEL + LAUNCH, True, True),
    ("@triton.jit\n" + KERNEL + "@triton.jit\ndef mul(x):\n    pass\nmul[(2,)](x)\n", True, True),
]


@pytest.mark.parametrize("i", range(len(CASES)))
def test_hand_written_cases(i):
    text, deco, launch = CASES[i]
    t = text.encode()
    assert rr.is_triton(t, require_launch=False) == deco, text
    assert rr.is_triton(t, require_launch=True) == launch, text


def _ast_flags(src: str):
    """(some function is decorated with triton.jit, some such function is
    called as name[...](...)) from the syntax tree."""
    tree = ast.parse(src)
    names = set()
    for node in ast.walk(tree):
        if isinstance(node, ast.FunctionDef):
            for d in node.decorator_list:
                f = d.func if isinstance(d, ast.Call) else d
                if (isinstance(f, ast.Attribute) and f.attr == "jit" and
                        isinstance(f.value, ast.Name) and f.value.id == "triton"):
                    names.add(node.name)
    launched = False
    for node in ast.walk(tree):
        if isinstance(node, ast.Call) and isinstance(node.func, ast.Subscript):
            v = node.func.value
            n = v.id if isinstance(v, ast.Name) else v.attr if isinstance(v, ast.Attribute) else None
            launched |= n in names
    return bool(names), launched


def test_agrees_with_the_syntax_tree():
    texts, _ = workloads.make_completions(400, seed=11, mean_len=600, valid=True)
    seen = set()
    for t in texts:
        want = _ast_flags(t.decode())
        got = (rr.is_triton(t, False), rr.is_triton(t, True))
        assert got == want, t.decode()
        seen.add(got)
    # the generated set covers every outcome
    assert seen == {(False, False), (True, False), (True, True)}


def test_reward_forms():
    texts = [c[0].encode() for c in CASES]
    passed = np.array([i % 3 != 0 for i in range(len(texts))], dtype=np.uint8)
    flags, r = rr.rule_rewards(texts, passed)
    deco = np.array([c[1] for c in CASES])
    assert np.array_equal(flags, deco.astype(np.uint8))
    # Eq. 3: 1 exactly when both checks pass
    assert np.array_equal(r, (deco & (passed != 0)).astype(np.float32))
    flags2, r2 = rr.rule_rewards(texts, passed, require_launch=True, weighted=True, rule_weight=0.1,
                                 exec_weight=0.9)
    launch = np.array([c[2] for c in CASES])
    assert np.array_equal(flags2, launch.astype(np.uint8))
    want = np.where(launch, np.float32(0.1), np.float32(0)) + np.where(passed != 0, np.float32(0.9),
                                                                        np.float32(0))
    assert r2.dtype == np.float32 and np.array_equal(r2, want.astype(np.float32))
