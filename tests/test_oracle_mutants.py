"""Mutation check of the oracle's pins (CPU only).

Each case plants one plausible mistake in a copy of the oracle's C source
(in a temporary directory; the repository's oracle is untouched), then runs
the pin tests of tests/test_oracle.py against the copy in a subprocess and
requires that at least one pin fails.  Planted: a shifted bitmask bit, a
reversed k index, wrong fp16 and bf16 exponent biases, a swapped dequant
scale, floor instead of round-to-nearest-even, an off-by-one value index, a
perturbed int8 sum, a shifted row offset, a dropped k term, and in the
activation quantiser truncation instead of round-to-nearest-even and a
divisor of 128 instead of 127."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

MUTANTS = [
    ("bitmask bit", "bitmask[n * words + k / 32] |= (uint32_t)1u << (k % 32);",
     "bitmask[n * words + k / 32] |= (uint32_t)1u << ((k + 1) % 32);"),
    ("reversed k", "s += Xd[m * K + k] * Dn[k];", "s += Xd[m * K + k] * Dn[K - 1 - k];"),
    ("fp16 bias", "v = ldexp((double)(1024 + f), e - 25);", "v = ldexp((double)(1024 + f), e - 24);"),
    ("dequant scale", "volatile float y = t * sw;", "volatile float y = t * sx;"),
    ("rounding", "double r = rint(a / q) * q;", "double r = floor(a / q) * q;"),
    ("value index", "out[k] = elem_to_f64(values, c, dtype);", "out[k] = elem_to_f64(values, c + 1, dtype);"),
    ("int8 sum", "s += (int64_t)Xq[m * K + k] * (int64_t)values[c];",
     "s += (int64_t)Xq[m * K + k] * (int64_t)values[c] + (k == 5 ? 1 : 0);"),
    ("row offset", "row_offsets[n] = (int32_t)c;", "row_offsets[n] = (int32_t)(c + (n == 1));"),
    ("bf16 bias", "v = ldexp((double)(128 + f), e - 134);", "v = ldexp((double)(128 + f), e - 133);"),
    ("dropped k", "for (int64_t k = 0; k < K; ++k) s += Xd", "for (int64_t k = 1; k < K; ++k) s += Xd"),
    ("quantiser rounding", "float q = nearbyintf(r);", "float q = truncf(r);"),
    ("quantiser scale", "volatile float scale = amax / 127.0f;", "volatile float scale = amax / 128.0f;"),
]


@pytest.mark.slow
@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_planted_mistake(tmp_path, name, old, new):
    src = open(os.path.join(ROOT, "oracle", "spl_oracle.c")).read()
    assert src.count(old) >= 1, f"mutation site for '{name}' not found: update this test"
    pkg = tmp_path / "oracle"
    pkg.mkdir()
    shutil.copy(os.path.join(ROOT, "oracle", "__init__.py"), pkg / "__init__.py")
    (pkg / "spl_oracle.c").write_text(src.replace(old, new))
    env = dict(os.environ, PYTHONPATH=f"{tmp_path}{os.pathsep}{ROOT}")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle.py")],
                       cwd=tmp_path, env=env, capture_output=True, text=True, timeout=600)
    assert "liboracle.so" in "".join(os.listdir(pkg)), "the mutated oracle was not the one built"
    assert r.returncode == 1, f"'{name}' was not caught (pytest exit {r.returncode}):\n{r.stdout[-2000:]}"
