"""Rule-based reward of AutoTriton's RL stage, written out in plain Python.

TEST INFRASTRUCTURE ONLY (like the rest of this package): the tests, the
smoke check and the benchmark's CPU-baseline leg are the only callers.

Sec. 3.3, Eq. 3: the reward of a completion is 1 when it is Triton code
(is_Triton, a rule-based check) and passes its tests (test_passed, decided by
an execution harness outside this library), else 0. Sec. 4 names the rule
that is checked (the @triton.jit decorator) and a way it is gamed: a
decorated kernel that is never launched. Sec. 4 also reports training with
the rule-based reward *alongside* the execution reward, hence the weighted
form rule_weight * is_Triton + exec_weight * test_passed offered next to Eq. 3.

The check is lexical, over the bytes of the completion (no parsing of
strings or comments beyond what is stated here):

* blank: space, tab or carriage return; identifier byte: [A-Za-z0-9_].
* A decorator is "@triton.jit" whose line holds only blanks before it and
  that is not followed by an identifier byte or ".". Arguments in
  parentheses may follow (balanced "(" / ")", possibly over several lines);
  the rest of that line must be blank or a "#" comment.
* The decorated function: the following lines are skipped while they are
  blank, "#" comments or other decorators (a line starting with "@", its
  parentheses balanced over lines as above); the next line must start,
  after blanks, with "def", one or more blanks, a name (an identifier byte
  run not starting with a digit), optional blanks and "(".
* A launch of a name: the name, not preceded by an identifier byte,
  followed by optional blanks, "[", a bracket-balanced run up to the
  matching "]" (possibly over lines), optional blanks and "(" -- Triton's
  kernel[grid](...) call.

is_Triton is true when some decorator has a decorated function and, when
launches are required, that function's name is launched somewhere in the
completion.
"""
from __future__ import annotations

import numpy as np

_BLANK = b" \t\r"
_IDENT = set(b"abcdefghijklmnopqrstuvwxyzABCDEFGHIJKLMNOPQRSTUVWXYZ0123456789_")
_DECO = b"@triton.jit"


def _is_ident(c: int) -> bool:
    return c in _IDENT


def _skip_blanks(t: bytes, i: int) -> int:
    while i < len(t) and t[i] in _BLANK:
        i += 1
    return i


def _line_end(t: bytes, i: int) -> int:
    """Index of the newline ending the line that holds i (or len(t))."""
    j = t.find(b"\n", i)
    return len(t) if j < 0 else j


def _match_close(t: bytes, i: int, open_b: int, close_b: int) -> int:
    """t[i] is an opening bracket: index just past its matching closing
    bracket (nesting counts only this bracket pair), or -1 if unclosed."""
    depth = 0
    for j in range(i, len(t)):
        if t[j] == open_b:
            depth += 1
        elif t[j] == close_b:
            depth -= 1
            if depth == 0:
                return j + 1
    return -1


def _finish_line(t: bytes, i: int) -> int:
    """From i, skip a parenthesised run if one starts the rest of the line
    (after blanks), then require blanks or a comment up to the newline.
    Returns the start of the next line, or -1 if the line has other text."""
    i = _skip_blanks(t, i)
    if i < len(t) and t[i] == ord("("):
        i = _match_close(t, i, ord("("), ord(")"))
        if i < 0:
            return -1
        i = _skip_blanks(t, i)
    if i < len(t) and t[i] not in b"\n#":
        return -1
    return _line_end(t, i) + 1


def decorator_positions(t: bytes) -> list[int]:
    """Positions of the @triton.jit decorators of the completion."""
    out = []
    p = t.find(_DECO)
    while p >= 0:
        ls = t.rfind(b"\n", 0, p) + 1
        if all(c in _BLANK for c in t[ls:p]):
            q = p + len(_DECO)
            if q >= len(t) or not (_is_ident(t[q]) or t[q] == ord(".")):
                out.append(p)
        p = t.find(_DECO, p + 1)
    return out


def decorated_name(t: bytes, p: int) -> bytes | None:
    """Name of the function decorated by the decorator at p, or None."""
    i = _finish_line(t, p + len(_DECO))
    while 0 <= i < len(t) + 1:
        if i >= len(t):
            return None
        j = _skip_blanks(t, i)
        if j >= len(t):
            return None
        c = t[j]
        if c == ord("\n") or c == ord("#"):  # blank or comment line
            i = _line_end(t, j) + 1
            continue
        if c == ord("@"):  # another decorator
            k = j + 1
            while k < len(t) and t[k] not in b"(\n":
                k += 1
            i = _finish_line(t, k) if k < len(t) and t[k] == ord("(") else _line_end(t, k) + 1
            continue
        if t[j:j + 3] != b"def" or j + 3 >= len(t) or t[j + 3] not in _BLANK:
            return None
        k = _skip_blanks(t, j + 3)
        s = k
        if k >= len(t) or not _is_ident(t[k]) or t[k] in b"0123456789":
            return None
        while k < len(t) and _is_ident(t[k]):
            k += 1
        name = t[s:k]
        k = _skip_blanks(t, k)
        return name if k < len(t) and t[k] == ord("(") else None
    return None


def is_launched(t: bytes, name: bytes) -> bool:
    """True if t holds name[...](: a Triton launch of that kernel."""
    r = t.find(name)
    while r >= 0:
        if r == 0 or not _is_ident(t[r - 1]):
            s = _skip_blanks(t, r + len(name))
            if s < len(t) and t[s] == ord("["):
                e = _match_close(t, s, ord("["), ord("]"))
                if e >= 0:
                    e = _skip_blanks(t, e)
                    if e < len(t) and t[e] == ord("("):
                        return True
        r = t.find(name, r + 1)
    return False


def is_triton(t: bytes, require_launch: bool = False) -> bool:
    for p in decorator_positions(t):
        name = decorated_name(t, p)
        if name is None:
            continue
        if not require_launch or is_launched(t, name):
            return True
    return False


def rule_rewards(texts, test_passed, require_launch: bool = False, weighted: bool = False,
                 rule_weight: float = 0.0, exec_weight: float = 0.0):
    """(is_Triton flags u8, rewards f32) for a batch of completions: Eq. 3's
    product of the two checks, or rule_weight * is_Triton + exec_weight * test_passed
    in fp32."""
    flags = np.array([is_triton(bytes(t), require_launch) for t in texts], dtype=np.uint8)
    passed = np.asarray(test_passed).astype(bool)
    if weighted:
        r = (np.float32(rule_weight) * flags.astype(np.float32) +
             np.float32(exec_weight) * passed.astype(np.float32)).astype(np.float32)
    else:
        r = ((flags != 0) & passed).astype(np.float32)
    return flags, r
