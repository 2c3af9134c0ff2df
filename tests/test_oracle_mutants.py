"""The oracle's pins catch plausible mistakes. Each mutant is a copy of the
oracle with one planted error -- a flipped sign, a dropped term, a wrong index,
a transposed operand, a wrong normalisation -- built and run on the CPU; the
pin suite must fail on every one of them, and pass on an unaltered copy built
the same way. (Mistakes are planted in the oracle only; the HIP path is not
involved.)"""
import importlib.util
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_C = os.path.join(ROOT, "oracle", "grpo_oracle.c")
PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")

# (name, text of the oracle, its mutated form); each text occurs once
C_MUTANTS = [
    ("unaltered", "", ""),
    # Eq. 2
    ("adv_no_mean", "a[i] = (r[i] - mean) / (sd + std_eps);", "a[i] = r[i] / (sd + std_eps);"),
    ("adv_std_swapped", "(double)(unbiased ? group - 1 : group)",
     "(double)(unbiased ? group : group - 1)"),
    ("adv_no_equal_test", "if (lo == hi) {", "if (0) {"),
    # packing and the Eq. 1 weights
    ("pack_ignores_mask", "      if (mask == NULL || mask[t]) {\n        if (rows) rows[n] = t;",
     "      if (1) {\n        if (rows) rows[n] = t;"),
    ("weight_no_B", "c[b] = 1.0 / ((double)num_seqs * (double)counts[b]);",
     "c[b] = 1.0 / (double)counts[b];"),
    ("empty_rollout_not_counted", "c[b] = 1.0 / ((double)num_seqs * (double)counts[b]);",
     "c[b] = 1.0 / ((double)(num_seqs - 1) * (double)counts[b]);"),
    # scoring
    ("lse_no_shift", "  return m + log(s);", "  return log(s);"),
    ("gather_off_by_one", "logp[i] = z[y[i]] - l;", "logp[i] = z[y[i] > 0 ? y[i] - 1 : 1] - l;"),
    ("logits_transposed", "const double* w = W + v * H;\n    double s = 0.0;",
     "const double* w = W + v;\n    double s = 0.0;"),
    # the per-token term of Eq. 1
    ("kl_sign", "double d = ref_logp[i] - logp[i];", "double d = logp[i] - ref_logp[i];"),
    ("kl_no_minus_one", "double kl = ed - d - 1.0;", "double kl = ed - d;"),
    ("max_not_min", "double pg = -(u < cl ? u : cl);", "double pg = -(u > cl ? u : cl);"),
    ("clip_upper_only",
     "double rc = rho < 1.0 - eps ? 1.0 - eps : (rho > 1.0 + eps ? 1.0 + eps : rho);",
     "double rc = rho > 1.0 + eps ? 1.0 + eps : rho;"),
    ("clipped_branch_has_slope", "double dpg = unclipped ? -adv[i] * rho : 0.0;",
     "double dpg = -adv[i] * rho;"),
    ("kl_grad_sign", "g[i] = c[i] * (dpg + beta * (1.0 - ed));",
     "g[i] = c[i] * (dpg + beta * (ed - 1.0));"),
    ("g_no_weight", "g[i] = c[i] * (dpg + beta * (1.0 - ed));",
     "g[i] = (dpg + beta * (1.0 - ed));"),
    # gradients
    ("dh_no_indicator",
     "double dz = g[i] * ((v == y[i] ? 1.0 : 0.0) - exp(z[v] - lse[i]));",
     "double dz = g[i] * (0.0 - exp(z[v] - lse[i]));"),
    ("dw_wrong_operand", "for (int64_t k = 0; k < H; ++k) out[k] += dz * hi[k];",
     "for (int64_t k = 0; k < H; ++k) out[k] += dz * w[k];"),
    ("dw_prob_sign", "double dz = g[i] * ((v == y[i] ? 1.0 : 0.0) - exp(z - lse[i]));",
     "double dz = g[i] * ((v == y[i] ? 1.0 : 0.0) + exp(z - lse[i]));"),
    # SFT
    ("sft_no_mean", "g[t] = -1.0 / (double)n;", "g[t] = -1.0;"),
    ("sft_loss_sign", "*loss = n > 0 ? -s / (double)n : 0.0;", "*loss = n > 0 ? s / (double)n : 0.0;"),
]


@pytest.mark.parametrize("name,old,new", C_MUTANTS, ids=[m[0] for m in C_MUTANTS])
def test_pins_catch_c_mutant(tmp_path, name, old, new):
    src = open(ORACLE_C).read()
    if old:
        assert src.count(old) == 1, f"{name}: mutation site not unique"
        src = src.replace(old, new)
    c = tmp_path / "oracle_mutant.c"
    c.write_text(src)
    lib = tmp_path / "liboracle_mutant.so"
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-o", str(lib),
                    str(c), "-lm"], check=True)
    env = dict(os.environ, GRPO_ORACLE_LIB=str(lib), OMP_NUM_THREADS="4")
    r = subprocess.run([sys.executable, "-m", "pytest", PINS, "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu"], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    if name == "unaltered":
        assert r.returncode == 0, r.stdout[-3000:]
    else:
        # 1 = some test failed (not a collection or usage error)
        assert r.returncode == 1, f"{name} survived the pins:\n{r.stdout[-3000:]}"


# the rule-based reward oracle (Python): the same checks as its pins
R_MUTANTS = [
    ("deco_anywhere_on_line", "        if all(c in _BLANK for c in t[ls:p]):",
     "        if True:"),
    ("cr_not_blank", "_BLANK = b\" \\t\\r\"", "_BLANK = b\" \\t\""),
    ("launch_needs_no_call", "                    if e < len(t) and t[e] == ord(\"(\"):",
     "                    if True:"),
    ("launch_suffix_match", "        if r == 0 or not _is_ident(t[r - 1]):", "        if True:"),
    ("no_bracket_nesting", "        if t[j] == open_b:\n            depth += 1",
     "        if t[j] == open_b:\n            depth = 1"),
    ("comment_lines_not_skipped", "        if c == ord(\"\\n\") or c == ord(\"#\"):  # blank or comment line",
     "        if c == ord(\"\\n\"):  # blank or comment line"),
]


def _load_rule_mutant(tmp_path, old, new):
    path = os.path.join(ROOT, "oracle", "rule_reward.py")
    src = open(path).read()
    assert src.count(old) == 1, old
    f = tmp_path / "rule_reward_mutant.py"
    f.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("rule_reward_mutant", f)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _rule_pins_pass(rr) -> bool:
    from paper_2507_05687_amd import workloads
    from test_rule_reward_pins import CASES, _ast_flags

    for text, deco, launch in CASES:
        t = text.encode()
        if rr.is_triton(t, False) != deco or rr.is_triton(t, True) != launch:
            return False
    texts, _ = workloads.make_completions(200, seed=11, mean_len=600, valid=True)
    return all((rr.is_triton(t, False), rr.is_triton(t, True)) == _ast_flags(t.decode())
               for t in texts)


@pytest.mark.parametrize("name,old,new", R_MUTANTS, ids=[m[0] for m in R_MUTANTS])
def test_pins_catch_rule_mutant(tmp_path, name, old, new):
    import oracle

    assert _rule_pins_pass(oracle.rule_reward)
    assert not _rule_pins_pass(_load_rule_mutant(tmp_path, old, new)), f"{name} survived"
