"""The oracle's pins must catch plausible mistakes (CPU only).

Each case plants one mistake in a private copy of oracle.c (a transposed tap,
a swapped gate, a wrong plane index, a dropped or altered term of the
back-propagation), rebuilds it, and runs the pin suite against it; the suite
must fail.  Nothing here touches the real oracle or the GPU path.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = [
    # recurrent convolution taps transposed
    ("whd[(((size_t)gn * O + j) * K + ka) * K + kb]",
     "whd[(((size_t)gn * O + j) * K + kb) * K + ka]"),
    # input convolution taps transposed
    ("acc += xv[c] * wxd[(((size_t)gn * C + c) * K + ka) * K + kb]",
     "acc += xv[c] * wxd[(((size_t)gn * C + c) * K + kb) * K + ka]"),
    # input and forget gate swapped in the cell update
    ("const double c = gg * gi + (cprev ? cprev[o] * gf : 0.0);",
     "const double c = gg * gf + (cprev ? cprev[o] * gi : 0.0);"),
    # previous plane of a negative sweep taken on the wrong side
    ("const int sp = (dir_sign(d) > 0) ? s - 1 : s + 1;     /* previous plane */",
     "const int sp = s - 1;"),
    # transposed convolution of the recurrent gradient with the wrong sign
    ("const int pp = p - (ka - r), qq = q - (kb - r);",
     "const int pp = p + (ka - r), qq = q + (kb - r);"),
    # forget-gate gradient against c_t instead of c_{t-1}
    ("dA[v * G + 1 * O + j] = gcv * cprev * gf * (1.0 - gf);",
     "dA[v * G + 1 * O + j] = gcv * c * gf * (1.0 - gf);"),
    # tanh derivative dropped a square
    ("double gcv = gh * go * (1.0 - tc * tc);", "double gcv = gh * go * (1.0 - tc);"),
    # cell carry uses this plane's forget gate instead of the next plane's
    ("if (t + 1 < T) gcv += gc[vn * O + j] * gdir[vn * G + 1 * O + j];",
     "if (t + 1 < T) gcv += gc[vn * O + j] * gdir[v * G + 1 * O + j];"),
    # input-gradient transposed convolution with the wrong sign
    ("const int p = pp - (ka - r), q = qq - (kb - r);",
     "const int p = pp + (ka - r), q = qq + (kb - r);"),
    # Eq. (13) keeps only the last direction instead of the sum
    ("hn[i] += hdir[i];", "hn[i] = hdir[i];"),
    # FC weight read transposed
    ("acc += w[(size_t)o * Cin + i] * x[(size_t)m * Cin + i];",
     "acc += w[(size_t)i * Cout + o] * x[(size_t)m * Cin + i];"),
    # cross-entropy gradient not divided by the voxel count
    ("const double g = (p[(size_t)m * Kc + k] - (labels[m] == k ? 1.0 : 0.0)) / (double)M;",
     "const double g = (p[(size_t)m * Kc + k] - (labels[m] == k ? 1.0 : 0.0));"),
]


@pytest.mark.parametrize("idx", range(len(MUTANTS)))
def test_pins_catch_planted_mistake(idx, tmp_path):
    src, bad = MUTANTS[idx]
    for sub in ("oracle", "synth", "tests"):
        shutil.copytree(os.path.join(ROOT, sub), tmp_path / sub,
                        ignore=shutil.ignore_patterns("*.so", "__pycache__", "golden"))
    shutil.copytree(os.path.join(ROOT, "tests", "golden"), tmp_path / "tests" / "golden")
    shutil.copy(os.path.join(ROOT, "pytest.ini"), tmp_path / "pytest.ini")
    path = tmp_path / "oracle" / "oracle.c"
    text = path.read_text()
    assert text.count(src) >= 1, src
    path.write_text(text.replace(src, bad, 1))
    env = dict(os.environ, PYTHONPATH=str(tmp_path), OMP_NUM_THREADS="1")
    res = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                          "tests/test_oracle_pins.py"], cwd=tmp_path, env=env,
                         capture_output=True, text=True, timeout=600)
    assert res.returncode != 0, "mutant survived: %s -> %s\n%s" % (src, bad, res.stdout[-2000:])
