"""Mutation check of the oracle's pins (CPU only).

Each case plants one plausible mistake in a copy of ``oracle/cyfa_oracle.c`` --
a flipped sign, a transposed operand, a wrong index, a dropped factor or term
-- builds the copy into a temporary library, and runs the pin suite
(``tests/test_oracle_pins.py``) against it.  The pins must reject every mutant,
and must accept an unmodified copy built the same way (which shows that the
pins really ran against the copy).
"""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "cyfa_oracle.c")
PINS = os.path.join(ROOT, "tests", "test_oracle_pins.py")

# (name, text in the source, replacement): each text occurs exactly once
MUTANTS = [
    ("rotation_direction", "U[a * m + b] = -s;\n        U[b * m + a] = s;",
     "U[a * m + b] = s;\n        U[b * m + a] = -s;"),
    ("basis_cos_sin_swapped", "phi[r * m + 2 * j - 1] = ac * cos(ang);",
     "phi[r * m + 2 * j - 1] = ac * sin(ang);"),
    ("basis_dc_weight", "const double dc = 1.0 / sqrt((double)m);",
     "const double dc = 1.0 / (double)m;"),
    ("shift_transposed", "const double prs = P[(size_t)r * m + s];",
     "const double prs = P[(size_t)s * m + r];"),
    ("decay_dropped", "S[i] = alpha * tmp[i];", "S[i] = tmp[i];"),
    ("write_strength_dropped", "S[c] += beta * (double)x[c];", "S[c] += (double)x[c];"),
    ("write_into_last_slot", "S[c] += beta * (double)x[c];",
     "S[(size_t)(m - 1) * d + c] += beta * (double)x[c];"),
    ("logit_R_transposed", "if (R) {\n                for (int r = 0; r < m; ++r) acc += R[(size_t)i * m + r] * y[r];",
     "if (R) {\n                for (int r = 0; r < m; ++r) acc += R[(size_t)r * m + i] * y[r];"),
    ("readout_R_not_transposed", "for (int i = 0; i < m; ++i) acc += R[(size_t)i * m + r] * w[i];",
     "for (int i = 0; i < m; ++i) acc += R[(size_t)r * m + i] * w[i];"),
    ("logit_scale_dropped", "zl[i] = scale * acc;", "zl[i] = acc;"),
    ("softmax_not_normalised", "for (int i = 0; i < m; ++i) w[i] /= den;", "(void)den;"),
    ("clock_doubled", "*lam += dlt;", "*lam += 2.0 * dlt;"),
    ("absolute_map_sign", "cyfa_oracle_rotation(m, -lam, U);\n    for (int i = 0; i < m; ++i)\n        for (int c = 0; c < d; ++c) {\n            double acc = 0.0;\n            for (int r = 0; r < m; ++r) acc += phi",
     "cyfa_oracle_rotation(m, lam, U);\n    for (int i = 0; i < m; ++i)\n        for (int c = 0; c < d; ++c) {\n            double acc = 0.0;\n            for (int r = 0; r < m; ++r) acc += phi"),
    ("query_from_key", "qt[c] = (double)q[(size_t)t * sq + c];", "qt[c] = (double)k[(size_t)t * sq + c];"),
]


def _build(src_text: str, path: str):
    c = path + ".c"
    with open(c, "w") as f:
        f.write(src_text)
    r = subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=gnu11", "-o", path, c, "-lm"],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def _run_pins(lib: str) -> subprocess.CompletedProcess:
    env = dict(os.environ, CYFA_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    return subprocess.run([sys.executable, "-m", "pytest", PINS, "-x", "-q", "-p", "no:cacheprovider"],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)


def _source() -> str:
    with open(SRC) as f:
        return f.read()


def test_unmodified_copy_passes(tmp_path):
    lib = str(tmp_path / "liboracle_copy.so")
    _build(_source(), lib)
    r = _run_pins(lib)
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_reject_mutant(tmp_path, name, old, new):
    src = _source()
    assert src.count(old) == 1, f"{name}: the mutated text must occur exactly once"
    lib = str(tmp_path / f"liboracle_{name}.so")
    _build(src.replace(old, new), lib)
    r = _run_pins(lib)
    assert r.returncode != 0, f"{name}: every pin passed with the mutant planted"
