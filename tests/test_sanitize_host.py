"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

* The oracle (oracle/spl_oracle.c), built with gcc and the sanitizers, runs
  tests/sanitize/oracle_driver.c: every routine on small ragged shapes,
  with round trips and sparse-vs-dense cross-checks.
* The library's host code (every csrc/*.hip translation unit, sanitizers on
  the host side only; device code is built as usual but never run) runs
  tests/sanitize/host_checks.cpp: every entry point with arguments its host
  checks must reject before any HIP call, and every size function at its
  limits.  No GPU is touched.

Any sanitizer report aborts the program (-fno-sanitize-recover=all)."""
import concurrent.futures as cf
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
HOST_SAN = [a for f in SAN for a in ("-Xarch_host", f)]         # host side only: no GPU sanitizer
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, cwd, timeout=600):
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True, timeout=timeout, env=ENV)
    assert r.returncode == 0, f"{' '.join(cmd[:3])} ... failed ({r.returncode}):\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r.stdout


@pytest.mark.timeout(600)
def test_oracle_under_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-std=c11", "-g", "-O1", "-fopenmp", "-ffp-contract=off", *SAN,
          os.path.join(ROOT, "oracle", "spl_oracle.c"), os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"),
          "-o", exe, "-lm"], str(tmp_path))
    out = _run([exe], str(tmp_path))
    assert out.startswith("ok "), out


@pytest.mark.timeout(900)
def test_library_host_checks_under_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2405_03594_amd", "csrc")]
    common = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", *HOST_SAN, *inc,
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    sources = sorted(glob.glob(os.path.join(ROOT, "paper_2405_03594_amd", "csrc", "*.hip")))
    sources.append(os.path.join(ROOT, "tests", "sanitize", "host_checks.cpp"))

    def compile_one(src):
        obj = str(tmp_path / (os.path.basename(src) + ".o"))
        _run([HIPCC, *common, "-c", src, "-o", obj], str(tmp_path))
        return obj

    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        objs = list(ex.map(compile_one, sources))
    exe = str(tmp_path / "host_checks")
    _run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, *objs, "-o", exe], str(tmp_path))
    out = _run([exe], str(tmp_path), timeout=300)
    assert out.startswith("ok "), out
