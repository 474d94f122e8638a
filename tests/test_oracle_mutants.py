"""Mutation tests of the oracle's pins.  Each mutant is a copy of oracle.c with
one plausible mistake planted (an index off by one, a dropped term, a wrong
sign or tie rule, a transposed operand, a wrong rounding or saturation rule).
It is compiled into a temporary library, and the pin suite (test_oracle_pins.py)
is run against it in a subprocess: every mutant must make at least one pin
fail.  The planted mistakes live only in those temporary copies.
"""
import os
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)
from oracle import build as oracle_build  # noqa: E402

SRC = os.path.join(ROOT, "oracle", "oracle.c")

# (name, original text, mutated text): every occurrence is replaced
MUTANTS = [
    ("ring slot off by one", "return s + (int)((p - s) % r);", "return s + (int)((p - s + 1) % r);"),
    ("n_topk counts one candidate too many", "int64_t n = L - (int64_t)s - (int64_t)r;",
     "int64_t n = L - (int64_t)s - (int64_t)r + 1;"),
    ("window rows shifted by one position", "int64_t i = L - w + ii; /* absolute",
     "int64_t i = L - w + ii + 1; /* absolute"),
    ("softmax scale dropped in the window scores",
     "        z[j] = sm_scale * acc;\n        if (z[j] > m) m = z[j];\n      }\n      double Z",
     "        z[j] = acc;\n        if (z[j] > m) m = z[j];\n      }\n      double Z"),
    ("normaliser over the whole row in NORM_CAND", "int64_t lo = (norm == NORM_CAND) ? c0 : 0;",
     "int64_t lo = 0;"),
    ("last visible candidate dropped from the column sum",
     "for (int64_t j = c0; j <= jc_hi; ++j) A[j] +=", "for (int64_t j = c0; j < jc_hi; ++j) A[j] +="),
    ("one head of the group left out", "  for (int h = 0; h < G; ++h) {\n    for (int ii = w - we;",
     "  for (int h = 0; h < G - 1 + (G == 1); ++h) {\n    for (int ii = w - we;"),
    ("query operand transposed (window and head)", "const double* qi = q + ((size_t)h * w + ii) * D;",
     "const double* qi = q + ((size_t)ii * G + h) * D;"),
    ("pool radius one too wide", "int half = kp / 2;", "int half = kp / 2 + 1;"),
    ("avg pool divisor kp - 1", "P[j] = (pool == POOL_MAX) ? acc : acc / (double)kp;",
     "P[j] = (pool == POOL_MAX) ? acc : acc / (double)(kp - 1 + (kp == 1));"),
    ("pool window leaks outside the candidates", "if (t < c0 || t >= c1) continue;",
     "if (t < 0 || t >= L) continue;"),
    ("ties go to the higher index", "return (x->t < y->t) ? -1 : (x->t > y->t); /* equal scores",
     "return (x->t > y->t) ? -1 : (x->t < y->t); /* equal scores"),
    ("smallest pooled scores kept",
     "if (x->p > y->p) return -1; /* larger pooled score first */\n  if (x->p < y->p) return 1;",
     "if (x->p < y->p) return -1; /* larger pooled score first */\n  if (x->p > y->p) return 1;"),
    ("ring rows stored linearly", "int row = oracle_slot_of(t, s, r);", "int row = (int)(t - lo + s);"),
    ("kept rows read one token early", "x + (size_t)sel[m] * width", "x + (size_t)(sel[m] - (sel[m] > 0)) * width"),
    ("decode misses the new token", "int n1 = (int)((p + 1) < (int64_t)(s + r) ? (p + 1) : (int64_t)(s + r));",
     "int n1 = (int)((p) < (int64_t)(s + r) ? (p) : (int64_t)(s + r));"),
    ("decode reads ring rows not filled yet",
     "int n1 = (int)((p + 1) < (int64_t)(s + r) ? (p + 1) : (int64_t)(s + r));", "int n1 = s + r;"),
    ("softmax scale dropped in decode",
     "      z[j] = sm_scale * acc;\n      if (z[j] > m) m = z[j];\n    }\n    double Z = 0.0;\n    double* oh",
     "      z[j] = acc;\n      if (z[j] > m) m = z[j];\n    }\n    double Z = 0.0;\n    double* oh"),
    ("decode value dims transposed in pairs", "oh[d] += e * cv[(size_t)j * cv_width + d];",
     "oh[d] += e * cv[(size_t)j * cv_width + (d ^ 1)];"),
    ("prefill row does not see its own key",
     "for (int64_t j = 0; j <= i; ++j) {", "for (int64_t j = 0; j < i + (i == 0); ++j) {"),
    ("prefill row sees the next key too",
     "for (int64_t j = 0; j <= i; ++j) {", "for (int64_t j = 0; j <= i + (i + 1 < L); ++j) {"),
    ("softmax scale dropped in prefill attention",
     "        z[j] = sm_scale * acc;\n        if (z[j] > m) m = z[j];\n      }\n      double Z = 0.0;\n      double* oi",
     "        z[j] = acc;\n        if (z[j] > m) m = z[j];\n      }\n      double Z = 0.0;\n      double* oi"),
    ("prefill value dims transposed in pairs", "oi[d] += e * v[(size_t)j * dv + d];",
     "oi[d] += e * v[(size_t)j * dv + (d ^ 1)];"),
    ("prefill query rows read position-major", "const double* qi = q + ((size_t)h * L + i) * dk;",
     "const double* qi = q + ((size_t)i * G + h) * dk;"),
    ("prefill normaliser without the row max", "lse[(size_t)h * n + (i - i0)] = m + log(Z);",
     "lse[(size_t)h * n + (i - i0)] = log(Z);"),
    ("prefill rows of a range written one row late", "double* oi = out + ((size_t)h * n + (i - i0)) * dv;",
     "double* oi = out + ((size_t)h * n + (i - i0 + (i0 > 0 && i + 1 < i1))) * dv;"),
    ("fp8 data scale from the largest positive value, not magnitude", "double a = fabs(x[i]);\n    if (a > amax)",
     "double a = x[i];\n    if (a > amax)"),
    ("fp8 data scale for the wrong top code", "return af / 448.0f;", "return af / 240.0f;"),
    ("e4m3 ties to odd", "(d == bestd && (c & 1) == 0)", "(d == bestd && (c & 1) == 1)"),
    ("e4m3 overflow to NaN instead of saturating", "if (a >= 448.0) return sign | 0x7E;",
     "if (a >= 464.0) return sign | 0x7F;"),
    ("e4m3 subnormal scale", "ldexp((double)m, -9)", "ldexp((double)m, -10)"),
    ("quantiser multiplies by the scale", "float qv = xf / scale;", "float qv = xf * scale;"),
]


def _run(tmp, i, name, old, new):
    text = open(SRC).read()
    assert old in text, f"mutant '{name}': the oracle no longer contains the text it mutates"
    src = os.path.join(tmp, f"mutant{i}.c")
    lib = os.path.join(tmp, f"libmutant{i}.so")
    open(src, "w").write(text.replace(old, new))
    oracle_build.build(src=src, out=lib)
    env = dict(os.environ, SNAP_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(HERE, "test_oracle_pins.py"), "-x", "-q",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    caught = [l for l in r.stdout.splitlines() if l.startswith("FAILED") or l.startswith("ERROR")]
    return name, r.returncode, caught[:1]


def test_every_mutant_fails_a_pin():
    with tempfile.TemporaryDirectory() as tmp:
        with ThreadPoolExecutor(max(1, min(8, os.cpu_count() or 1))) as ex:
            results = list(ex.map(lambda a: _run(tmp, *a), [(i, *m) for i, m in enumerate(MUTANTS)]))
    survivors = [name for name, rc, _ in results if rc == 0]
    for name, rc, caught in results:
        print(f"  {name:52s} {'caught by ' + caught[0][7:] if caught else 'SURVIVED'}")
    assert not survivors, f"mutants no pin catches: {survivors}"
