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
    ("label matrix read transposed", "sq += wj * (double)qual[(size_t)n * M + m];",
     "sq += wj * (double)qual[(size_t)m * N + n];"),
    ("mean divides by one more", "q_hat[(size_t)b * M + m] = sq / sw;",
     "q_hat[(size_t)b * M + m] = sq / (sw + 1);"),
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
    ("argmax tie goes to the last index", "S[i] > S[best]))", "S[i] >= S[best]))"),
    ("decode grows by the wrong model's length", "a[best] += lr[model[best]];",
     "a[best] += lr[0];"),
    ("prompt not added to the queued prefill", "p[best] += (double)plen[r];", "(void)0;"),
    ("normalised by the minimum", "if (!seen || C[i] > cmax)", "if (!seen || C[i] < cmax)"),
    ("drain does not clamp at zero", "p[i] = fmax(0.0, p[i] - P[i] * dt);",
     "p[i] = p[i] - P[i] * dt;"),
    ("LPT runs shortest first", "return u->key > v->key ? -1 : 1;",
     "return u->key < v->key ? -1 : 1;"),
    ("LPT ties go to the higher index", "return u->r < v->r ? -1 : (u->r > v->r);",
     "return u->r > v->r ? -1 : (u->r < v->r);"),
    ("LPT key is the first model's length",
     "key = fmax(key, l_hat[(size_t)r * M + m]);", "(void)0;"),
    ("LPT order not applied", "if (lpt)\n        oracle_lpt_order", "if (0)\n        oracle_lpt_order"),
    ("weight from the squared distance", "return 1.0 / (sqrt(fmax(d, 0.0)) + 1e-6);",
     "return 1.0 / (fmax(d, 0.0) + 1e-6);"),
    ("negative distance not clamped", "sqrt(fmax(d, 0.0))", "sqrt(fabs(d))"),
    ("weights not normalised", "sw += wj;", "sw += 1.0;"),
    ("budget admits strictly below only", "ok = c <= (double)*budget_r;",
     "ok = c < (double)*budget_r;"),
    ("budget admission in fp32 rounding",
     "double c = plen * in->cin[i] + l_hat_r[in->model[i]] * in->cout[i];",
     "double c = fmaf((float)plen, (float)in->cin[i],\n"
     "                            (float)l_hat_r[in->model[i]] * (float)in->cout[i]);"),
    ("budget compared with the output cost only",
     "double c = plen * in->cin[i] + l_hat_r[in->model[i]] * in->cout[i];",
     "double c = l_hat_r[in->model[i]] * in->cout[i];"),
    ("mask ignored", "int ok = mask ? mask[i] != 0 : 1;", "int ok = 1;"),
    ("maxima over every instance",
     "        if (cand && !cand[i])\n            continue;\n        if (!seen || C[i] > cmax)",
     "        if (!seen || C[i] > cmax)"),
    ("no candidate falls back to instance 0", "assign[r] = best;",
     "assign[r] = best < 0 ? 0 : best;"),
]


@pytest.mark.parametrize("name,orig,mut", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, orig, mut):
    src = open(SRC).read()
    assert src.count(orig) == 1, name
    msrc = tmp_path / "mutant.c"
    msrc.write_text(src.replace(orig, mut))
    lib = tmp_path / "libmutant.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
                           "-ffp-contract=off", "-o", str(lib), str(msrc), "-lm"])
    env = dict(os.environ, RB_ORACLE_LIB=str(lib))
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"pins did not catch mutant '{name}':\n{r.stdout[-2000:]}"
