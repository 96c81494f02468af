"""Properties of the generated gfx950 code that the sources rely on (no GPU).

The weight gradient's direct-to-LDS requests are issued from inline assembly
that sets M0 (the request's LDS base) and declares it clobbered; the compiler
treats M0 as reserved, so the kernel is correct only while no other
instruction in it reads M0.  The requests are opaque precisely so that the
compiler does not wait for all of them before each LDS transpose read, which
is checked too (a performance property, but one that a compiler change could
silently undo)."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2405_03594_amd import build as B

SRC = os.path.join(B.CSRC, "k_prefill.hip")


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    if not os.path.exists(B.HIPCC) and not shutil.which("hipcc"):
        pytest.skip("hipcc is not available")
    out = tmp_path_factory.mktemp("asm") / "k_prefill.s"
    flags = [f for f in B.CFLAGS if f != "-fPIC"]
    r = subprocess.run([B.HIPCC, *flags, "-S", "--cuda-device-only", SRC, "-o", str(out)], capture_output=True,
                       text=True)
    assert r.returncode == 0, r.stderr
    return out.read_text()


def _kernels(asm, pattern):
    bodies = {}
    for m in re.finditer(r"^(_Z\w*" + pattern + r"\w*):", asm, re.M):
        i = m.start()
        bodies[m.group(1)] = asm[i:asm.index(".Lfunc_end", i)]
    assert bodies, pattern
    return bodies


def test_transposed_core_reads_m0_only_for_its_requests(asm):
    for name, body in _kernels(asm, "k_dense_prefill_dma_tr").items():
        lines = [l.strip() for l in body.split("\n") if l.strip() and not l.strip().startswith(";")]
        for i, l in enumerate(lines):
            if re.search(r"\bm0\b", l):
                assert l.startswith("s_mov_b32 m0,"), (name, l)
                assert lines[i + 1] == "s_nop 0" and lines[i + 2].startswith("global_load_lds_dwordx4"), (name, l)


def test_transposed_reads_do_not_wait_for_every_request(asm):
    for name, body in _kernels(asm, "k_dense_prefill_dma_tr").items():
        lines = [l.strip() for l in body.split("\n") if l.strip() and not l.strip().startswith(";")]
        # between a request and the next LDS transpose read, no wait for all vector-memory operations
        last_request = None
        for i, l in enumerate(lines):
            if l.startswith("global_load_lds_dwordx4"):
                last_request = i
            elif l.startswith("ds_read_b64_tr_b16") and last_request is not None:
                between = lines[last_request:i]
                assert not any(re.match(r"s_waitcnt vmcnt\(0\)", x) for x in between), name
                last_request = None
