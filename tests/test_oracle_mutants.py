"""Plant plausible mistakes in the oracle (on the CPU) and require the pins to catch each one.

Every mutant is a one-spot edit of ``oracle/oracle.c`` -- a dropped term, a
wrong sign or index, a non-strict comparison, a transposed operand -- built
into a temporary library.  All of ``tests/oracle_checks.py`` runs against it,
and at least one check must fail.  This is what makes the pins evidence that
the oracle computes what the paper defines rather than a restatement of it.
"""
import os
import subprocess

import pytest

from oracle import oracle as O
from tests import oracle_checks as C

SRC = os.path.join(os.path.dirname(O.__file__), "oracle.c")

MUTANTS = [
    ("lse drops the max shift", "*log_s_out = log(s);", "*log_s_out = log(s) + m;"),
    ("sum drops the last term", "for (int64_t v = 0; v < vocab; ++v) s += exp(",
     "for (int64_t v = 0; v < vocab - 1; ++v) s += exp("),
    ("max ignores the first element", "for (int64_t v = 0; v < vocab; ++v) {\n        double x = load_logit(row, dtype, v);",
     "for (int64_t v = 1; v < vocab; ++v) {\n        double x = load_logit(row, dtype, v);"),
    ("logp sign flipped", "lp = (load_logit(row, dtype, y) - m) - log_s;", "lp = log_s - (load_logit(row, dtype, y) - m);"),
    ("gather takes the next token", "lp = (load_logit(row, dtype, y) - m) - log_s;",
     "lp = (load_logit(row, dtype, (y + 1) % vocab) - m) - log_s;"),
    ("rows strided by vocab instead of ld", "const void *row = base + i * ld * es;",
     "const void *row = base + i * vocab * es;"),
    ("bf16 decoded with the wrong shift", "uint32_t u = (uint32_t)b << 16;", "uint32_t u = (uint32_t)b << 15;"),
    ("non-finite row accepted", "if (isnan(x) || x == INFINITY) return 0;", "if (isnan(x)) return 0;"),
    ("token id bound off by one", "if (y < 0 || (int64_t)y >= vocab) {\n            flags |= OR_TOKEN_OOB;\n            lp = NAN;\n        } else {\n            lp = (load_logit(row",
     "if (y < 0 || (int64_t)y > vocab) {\n            flags |= OR_TOKEN_OOB;\n            lp = NAN;\n        } else {\n            lp = (load_logit(row"),
    ("kl sign flipped", "kl[i] = logp_s[i] - logp_t[i];", "kl[i] = logp_t[i] - logp_s[i];"),
    ("exact kl weights by the teacher", "double ps = exp(lps);", "double ps = exp(lpt);"),
    ("turn mean divides by n+1", "out[k] = s / (double)(b - a);", "out[k] = s / (double)(b - a + 1);"),
    ("turn mean skips the first token", "for (int64_t i = a; i < b; ++i) s += logp_t[i];",
     "for (int64_t i = a + 1; i < b; ++i) s += logp_t[i];"),
    ("stop test not strict", "if (s < 0 && c < lambda[r]) s = (int32_t)u;", "if (s < 0 && c <= lambda[r]) s = (int32_t)u;"),
    ("stop reports the unit after the trigger", "if (s < 0 && c < lambda[r]) s = (int32_t)u;",
     "if (s < 0 && c < lambda[r]) s = (int32_t)(u + 1 < n ? u + 1 : u);"),
    ("prefix K0 ignored", "int64_t k0 = start ? start[r] : 0;", "int64_t k0 = 0;"),
    ("prefix summed but not tested", "if (u < k0) { cum[first + u] = 0.0; continue; }",
     "if (u < k0) { c += values[first + u]; cum[first + u] = 0.0; continue; }"),
    ("retained drops the trigger unit", "int64_t end = (s >= 0) ? (int64_t)s + 1 : n;", "int64_t end = (s >= 0) ? (int64_t)s : n;"),
    ("correct gate not strict", "(values[g] > alpha[r]);", "(values[g] >= alpha[r]);"),
    ("mask ignored", "int ok = (mask == NULL || mask[g] != 0) &&", "int ok = 1 &&"),
    ("argmin ties to the last index", "values[first + u] < values[first + best]", "values[first + u] <= values[first + best]"),
    ("k* is an argmax", "values[first + u] < values[first + best]", "values[first + u] > values[first + best]"),
    ("record length ignored", "int64_t len = record_len ? record_len[r] : n;", "int64_t len = n;"),
    ("K0 not clamped at zero", "k0[r] = best > 0 ? best : 0;", "k0[r] = best;"),
    ("K0 one past k*", "k0[r] = best > 0 ? best : 0;", "k0[r] = best + 1;"),
    ("lm_head read transposed", "const uint16_t *wrow = w + k * vocab;\n                for (int64_t v = 0; v < vocab; ++v) z[v] += h * bf16_bits_to_double(wrow[v]);",
     "for (int64_t v = 0; v < vocab; ++v) z[v] += h * bf16_bits_to_double(w[v * d + k]);"),
    ("gradient sign flipped", "double c = -scale * r[i];", "double c = scale * r[i];"),
    ("gradient drops the sampled-token term", "g[v] = c * (((int64_t)y == v ? 1.0 : 0.0) - p);",
     "g[v] = c * (-p);"),
    ("gradient ignores the mask", "        if (!mask[i]) {\n            for (int64_t v = 0; v < vocab; ++v) g[v] = 0.0;",
     "        if (0) {\n            for (int64_t v = 0; v < vocab; ++v) g[v] = 0.0;"),
    ("gradient probability without the normaliser", "double p = exp((load_logit(row, dtype, v) - m) - log_s);",
     "double p = exp(load_logit(row, dtype, v) - m);"),
    ("projection skips a hidden unit", "for (int64_t k = 0; k < d; ++k) {\n                double h",
     "for (int64_t k = 1; k < d; ++k) {\n                double h"),
]


@pytest.fixture(scope="module")
def source():
    with open(SRC) as f:
        return f.read()


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(name, old, new, source, tmp_path):
    assert source.count(old) >= 1, f"mutation site for '{name}' not found in oracle.c"
    mutated = source.replace(old, new, 1)
    c_path = tmp_path / "oracle_mutant.c"
    so_path = tmp_path / "liboracle_mutant.so"
    c_path.write_text(mutated)
    subprocess.run(["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
                    "-o", str(so_path), str(c_path), "-lm"], check=True)
    prev = O.use_library(str(so_path))
    failed = []
    try:
        for check in C.ALL_CHECKS:
            try:
                check()
            except (AssertionError, ValueError, IndexError):
                failed.append(check.__name__)
    finally:
        O.use_library(None)
        O._lib = prev
    assert failed, f"no pin catches the mutant '{name}'"
