"""Plant plausible mistakes in copies of the oracle and require the pins to catch each.

Every mutant is built from the oracle's C source with one textual change, on
the CPU, and the pin tests are run against it in a child process. A mutant
that passes every pin would mean a mistake of that kind in the oracle could go
unnoticed.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "rb_oracle.c")

# (name, original text, mutated text); each original must occur exactly once.
MUTANTS = [
    ("distance drops the square", "s += diff * diff;", "s += diff;"),
    ("tie goes to the higher index", "(d1 == d2 && i1 < i2)", "(d1 == d2 && i1 > i2)"),
    ("label matrix read transposed", "sq += (double)qual[(size_t)n * M + m];",
     "sq += (double)qual[(size_t)m * N + n];"),
    ("mean divides by k+1", "q_hat[(size_t)b * M + m] = sq / k;",
     "q_hat[(size_t)b * M + m] = sq / (k + 1);"),
    ("input and output price swapped",
     "C[i] = plen * in->cin[i] + l_hat_r[m] * in->cout[i];",
     "C[i] = plen * in->cout[i] + l_hat_r[m] * in->cin[i];"),
    ("prefill drained at the decode rate",
     "T[i] = (p[i] + plen) / in->P[i] + (a[i] + l_hat_r[m]) / in->D[i];",
     "T[i] = (p[i] + plen) / in->D[i] + (a[i] + l_hat_r[m]) / in->P[i];"),
    ("own prompt left out of the latency",
     "T[i] = (p[i] + plen) / in->P[i]", "T[i] = (p[i]) / in->P[i]"),
    ("latency and cost weights swapped",
     "S[i] = w[0] * q_hat_r[m] + w[2] * (1.0 - cost_ratio) + w[1] * (1.0 - lat_ratio);",
     "S[i] = w[0] * q_hat_r[m] + w[1] * (1.0 - cost_ratio) + w[2] * (1.0 - lat_ratio);"),
    ("argmax tie goes to the last index", "if (S[i] > S[best])", "if (S[i] >= S[best])"),
    ("decode grows by the wrong model's length", "a[best] += lr[model[best]];",
     "a[best] += lr[0];"),
    ("prompt not added to the queued prefill", "p[best] += (double)plen[r];", "(void)0;"),
    ("normalised by the minimum", "if (i == 0 || C[i] > cmax)", "if (i == 0 || C[i] < cmax)"),
    ("drain does not clamp at zero", "p[i] = fmax(0.0, p[i] - P[i] * dt);",
     "p[i] = p[i] - P[i] * dt;"),
]


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, orig, mut):
    src = open(SRC).read()
    assert src.count(orig) == 1, name
    msrc = tmp_path / "mutant.c"
    msrc.write_text(src.replace(orig, mut))
    lib = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread", "-o", str(lib),
                           str(msrc), "-lm"])
    env = dict(os.environ, RB_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"pins did not catch mutant '{name}':\n{r.stdout[-2000:]}"
