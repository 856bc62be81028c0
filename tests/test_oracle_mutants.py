"""Mutation check of the oracle's pins (CPU only).

Each mutant plants one plausible mistake in a copy of the oracle -- a dropped
term, a wrong sign or bound, a swapped operand, an off-by-one -- builds the
copy in a temporary directory and runs the oracle's pin tests against it in a
child process.  Every mutant must turn at least one pin red; the unaltered
copy must leave them green.  The repository's own oracle is never modified.

Passages the mutated lines follow: Sec. 3.2 Eqs. 4-6 and the closing
advantage sentence (tiers, tournament, reward, advantage); Sec. 3.1 Eqs. 1-2
(gate); Sec. 3.3 (discount) and Sec. 4.1 (aggregation weight); Sec. 3.1 Eq. 3
per token (log-softmax, ratio, clip, surrogate, KL, gradient); Sec. 4
(training statistics).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PIN_FILES = [os.path.join(HERE, f) for f in (
    "test_oracle_rank.py", "test_oracle_gate_discount.py", "test_oracle_grpo.py",
    "test_oracle_lmhead.py", "test_oracle_vocab_shard.py", "test_oracle_rollout_stats.py",
    "test_oracle_properties.py")]

C = "leap_oracle.c"
PY = "__init__.py"

# (name, file, [(original text, replacement), ...]); each original must occur
# exactly once in the file.
MUTANTS = [
    # Sec. 3.2: tiers, tournament, reward, advantage
    ("tier equals the pass turn", C, [("return M - m + 1;", "return m;")]),
    ("a tie counts as a win", C, [("if (c > 0) worse += 1;", "if (c >= 0) worse += 1;")]),
    ("reward divided by G", C, [("(double)(worse - better) / (double)(G - 1);",
                                 "(double)(worse - better) / (double)G;")]),
    ("biased standard deviation", C, [("var /= (double)(G - 1);", "var /= (double)G;")]),
    ("eps added after the division", C, [("(reward[base + i] - mean) / (sd + eps);",
                                          "(reward[base + i] - mean) / sd + eps;")]),
    ("LEX: more tokens preferred", C, [("if (na < nb) return 1;\n        if (na > nb) return -1;",
                                        "if (na > nb) return 1;\n        if (na < nb) return -1;")]),
    ("LEX: speedup ignored", C, [("if (sa > sb) return 1;\n        if (sa < sb) return -1;\n", "")]),
    # Sec. 3.1, Eqs. 1-2: gate
    ("gate lower bound exclusive", C, [("(tau_min <= nf && nf <= tau_max)",
                                        "(tau_min < nf && nf <= tau_max)")]),
    ("gate counts passes", C, [("if (first_turn_pass[g * (int64_t)G + i] == 0) nf += 1;",
                                "if (first_turn_pass[g * (int64_t)G + i] != 0) nf += 1;")]),
    # Sec. 3.3 and Sec. 4.1: discount and weight
    ("discount exponent T - t", C, [("pow(beta, (double)(T - t - 1))", "pow(beta, (double)(T - t))")]),
    ("negative advantages discounted", C, [("beta = (a >= 0.0) ? gamma : 1.0;", "beta = gamma;")]),
    ("sequence weight without |M_i|", C, [("w_tok[k] = 1.0 / (denom * (double)n_gen_tokens[i]);",
                                           "w_tok[k] = 1.0 / denom;")]),
    ("token-mean weight of 1", C, [("w_tok[k] = 1.0 / denom;\n        else", "w_tok[k] = 1.0;\n        else")]),
    # Sec. 3.1, Eq. 3 per token
    ("log-sum-exp without the log", C, [("lse = m + log(s);", "lse = m + s;")]),
    ("log-sum-exp without the max", C, [("lse = m + log(s);", "lse = log(s);")]),
    ("temperature dropped from the logits", C, [("z_scratch[v] = inv_temp * x[v];",
                                                 "z_scratch[v] = x[v];")]),
    ("ratio inverted", C, [("rho = exp(logp - old_lp);", "rho = exp(old_lp - logp);")]),
    ("clip bounds swapped", C, [
        ("if (clipped < 1.0 - eps_lo) clipped = 1.0 - eps_lo;",
         "if (clipped < 1.0 - eps_hi) clipped = 1.0 - eps_hi;"),
        ("if (clipped > 1.0 + eps_hi) clipped = 1.0 + eps_hi;",
         "if (clipped > 1.0 + eps_lo) clipped = 1.0 + eps_lo;")]),
    ("activity bounds swapped", C, [
        ("active = (ahat > 0.0 && rho <= 1.0 + eps_hi) || (ahat < 0.0 && rho >= 1.0 - eps_lo);",
         "active = (ahat > 0.0 && rho <= 1.0 + eps_lo) || (ahat < 0.0 && rho >= 1.0 - eps_hi);")]),
    ("clip and activity bounds both swapped", C, [
        ("if (clipped < 1.0 - eps_lo) clipped = 1.0 - eps_lo;",
         "if (clipped < 1.0 - eps_hi) clipped = 1.0 - eps_hi;"),
        ("if (clipped > 1.0 + eps_hi) clipped = 1.0 + eps_hi;",
         "if (clipped > 1.0 + eps_lo) clipped = 1.0 + eps_lo;"),
        ("active = (ahat > 0.0 && rho <= 1.0 + eps_hi) || (ahat < 0.0 && rho >= 1.0 - eps_lo);",
         "active = (ahat > 0.0 && rho <= 1.0 + eps_lo) || (ahat < 0.0 && rho >= 1.0 - eps_hi);")]),
    ("max instead of min", C, [("surr = fmin(rho * ahat, clipped * ahat);",
                                "surr = fmax(rho * ahat, clipped * ahat);")]),
    ("clip activity ignored", C, [
        ("active = (ahat > 0.0 && rho <= 1.0 + eps_hi) || (ahat < 0.0 && rho >= 1.0 - eps_lo);",
         "active = 1;")]),
    ("k3 sign", C, [("kl = exp(d) - d - 1.0;", "kl = exp(d) + d - 1.0;")]),
    ("k3 gradient sign", C, [("dkl = 1.0 - exp(d);", "dkl = exp(d) - 1.0;")]),
    ("k2 without the half", C, [("kl = 0.5 * (logp - ref_lp) * (logp - ref_lp);",
                                 "kl = (logp - ref_lp) * (logp - ref_lp);")]),
    ("k1 sign", C, [("kl = logp - ref_lp;\n        dkl = 1.0;", "kl = ref_lp - logp;\n        dkl = 1.0;")]),
    ("KL gradient dropped", C, [("dl = (active ? -ahat * rho : 0.0) + kl_coef * dkl;",
                                 "dl = (active ? -ahat * rho : 0.0);")]),
    ("no temperature in the gradient", C, [("g = w * dl * inv_temp;", "g = w * dl;")]),
    ("weight dropped from the gradient", C, [("g = w * dl * inv_temp;", "g = dl * inv_temp;")]),
    ("one-hot sign", C, [("dlog_row[v] = g * ((v == y ? 1.0 : 0.0) - p);",
                          "dlog_row[v] = g * (p - (v == y ? 1.0 : 0.0));")]),
    ("bf16 decode shift", C, [("uint32_t u = (uint32_t)b << 16;", "uint32_t u = (uint32_t)b << 15;")]),
    ("masked rows evaluated", C, [("if (w == 0.0) return 0;", "")]),
    ("loss total unweighted", C, [("total += w[k] * tok_loss[j];\n    }\n    *loss_total = total;\n    return bad;\n}\n\n/* The same pass on bf16",
                                   "total += tok_loss[j];\n    }\n    *loss_total = total;\n    return bad;\n}\n\n/* The same pass on bf16")]),
    ("forward log-prob without temperature", C, [
        ("for (v = 0; v < V; ++v) zs[v] = inv_temp * bf16_to_double(row[v]);\n            logp[k]",
         "for (v = 0; v < V; ++v) zs[v] = bf16_to_double(row[v]);\n            logp[k]")]),
    ("entropy sign", C, [("if (p > 0.0) h -= p * logp;", "if (p > 0.0) h += p * logp;")]),
    ("entropy of unnormalised logits", C, [("const double logp = zs[v] - lse;",
                                            "const double logp = zs[v] - m_unused;")]),
    # Sec. 4: training statistics
    ("debugging test uses m != 0", C, [("if (activated && m != 1) {", "if (activated && m != 0) {")]),
    ("recovery only on the second turn", C, [("if (m >= 2) ++n_recovered;", "if (m == 2) ++n_recovered;")]),
    ("recovery counts final failures", C, [("if (m >= 2) ++n_recovered;", "if (m == 0) ++n_recovered;")]),
    ("debugging group without a trajectory", C, [("if (n_multi > 0) {", "if (1) {")]),
    ("pass-rate bucket rounded up", C, [("int64_t b = n_pass * (int64_t)n_buckets / G;",
                                         "int64_t b = (n_pass * (int64_t)n_buckets + G - 1) / G;")]),
    ("outcome classes swapped", C, [("const int o = (m == 1) ? 0 : (m >= 2 ? 1 : 2);",
                                     "const int o = (m == 1) ? 1 : (m >= 2 ? 0 : 2);")]),
    ("turns taken from pass_turn", C, [("counters[7] += T;", "counters[7] += m;")]),
    ("zero advantages counted", C, [("if (a == 0.0 || a != a) continue;", "if (a != a) continue;")]),
    # fused LM head and vocabulary shard (numpy side of the oracle)
    ("LM head: dW scaled", PY, [("dW = dZ.T @ Hm", "dW = 2.0 * (dZ.T @ Hm)")]),
    ("LM head: temperature factor in dH", PY, [
        ("dH += dZ[:, v0:v0 + v_block] @ Wm[v0:v0 + v_block]",
         "dH += inv_temp * (dZ[:, v0:v0 + v_block] @ Wm[v0:v0 + v_block])")]),
    ("LM head: rows reordered", PY, [("Z[:, v0:v0 + v_block] = Hs @ Wm[v0:v0 + v_block].T",
                                      "Z[:, v0:v0 + v_block] = Hs[::-1] @ Wm[v0:v0 + v_block].T")]),
    ("LM head: dW rows reversed", PY, [("dW = dZ.T @ Hm", "dW = (dZ.T @ Hm)[::-1]")]),
    ("shard: max without the scale", PY, [("m2[k] = c * mx", "m2[k] = mx")]),
    ("shard: owns one column too many", PY, [("owned = ((yl >= 0) & (yl < V))",
                                              "owned = ((yl >= 0) & (yl <= V))")]),
    ("shard: token logit off by one", PY, [("zy[k] = x[k, yl[k]]", "zy[k] = x[k, yl[k] - 1]")]),
    ("pass-rate window: strict ignored", PY, [("a = (q > lo) if lo_strict else (q >= lo)",
                                               "a = (q >= lo) if lo_strict else (q >= lo)")]),
    ("statistics: per-group recovery over activated groups", PY, [
        ('ratio(out["recovered_groups"], out["debugging_groups"])',
         'ratio(out["recovered_groups"], out["activated_groups"])')]),
]

# The one identifier the entropy mutant introduces.
_EXTRA_DECL = {"entropy of unnormalised logits": ("double lse, h = 0.0;",
                                                  "double lse, h = 0.0, m_unused = 0.0;")}


def _make_copy(dest: str, name: str | None, file: str | None, edits) -> None:
    pkg = os.path.join(dest, "oracle")
    os.makedirs(pkg)
    for f in (C, PY):
        text = open(os.path.join(ROOT, "oracle", f)).read()
        if f == file:
            for a, b in edits:
                assert text.count(a) == 1, f"mutant {name!r}: {a!r} occurs {text.count(a)} times"
                text = text.replace(a, b)
            if name in _EXTRA_DECL:
                a, b = _EXTRA_DECL[name]
                assert text.count(a) == 1
                text = text.replace(a, b)
        open(os.path.join(pkg, f), "w").write(text)
    oracle.build(src=os.path.join(pkg, C), out=os.path.join(pkg, "liboracle.so"))


def _run_pins(dest: str) -> subprocess.CompletedProcess:
    """The pin tests in a child whose ``import oracle`` finds the copy in
    ``dest`` (the working directory; pytest appends the repository root to
    the module path instead of prepending it)."""
    env = dict(os.environ, PYTHONPATH=dest, OMP_NUM_THREADS="1")
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           "--import-mode=append", "-m", "not gpu", *PIN_FILES],
                          cwd=dest, env=env, capture_output=True, text=True, timeout=600)


@pytest.fixture(scope="module")
def outcomes(tmp_path_factory):
    cases = [("control", None, [])] + [(n, f, e) for n, f, e in MUTANTS]
    dirs = {}
    for i, (name, file, edits) in enumerate(cases):
        d = str(tmp_path_factory.mktemp(f"mutant{i:02d}"))
        _make_copy(d, name, file, edits)
        dirs[name] = d

    def one(name):
        r = _run_pins(dirs[name])
        return name, r.returncode, (r.stdout + r.stderr)[-3000:]

    with ThreadPoolExecutor(max_workers=6) as ex:
        res = {n: (rc, out) for n, rc, out in ex.map(one, [c[0] for c in cases])}
    for d in dirs.values():
        shutil.rmtree(d, ignore_errors=True)
    return res


def test_unaltered_copy_passes_every_pin(outcomes):
    rc, out = outcomes["control"]
    assert rc == 0, out


@pytest.mark.parametrize("name", [m[0] for m in MUTANTS])
def test_mutant_fails_a_pin(outcomes, name):
    rc, out = outcomes[name]
    # exit status 1: tests ran and at least one failed (not a collection or
    # usage error, which would be 2 or more)
    assert rc == 1, f"mutant {name!r} survived the pins (exit {rc}):\n{out}"
