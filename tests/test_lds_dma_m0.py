"""The LDS-direct operand loads set M0 in inline assembly and leave it changed, which is
correct only while the kernels that issue them use M0 for nothing else.  Compile those
sources for gfx950 to assembly (code built here) and check, in every function that issues
a global_load_lds, that M0 is written only by the load sequence (M0 write, one wait state,
the load) and read by nothing else."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2606_09377_amd", "csrc")
INCLUDE = os.path.join(os.path.dirname(CSRC), "..", "include")


def _hipcc():
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    pytest.skip("hipcc not found")


def _functions(asm):
    """(name, body lines) of every kernel in an assembly listing."""
    out, name, body = [], None, []
    for line in asm.splitlines():
        m = re.match(r"^(_Z\S+):", line)
        if m:
            name, body = m.group(1), []
            continue
        if name is not None:
            if line.strip().startswith("s_endpgm"):
                out.append((name, body))
                name = None
            else:
                body.append(line.strip())
    return out


@pytest.mark.parametrize("src", ["gemm.hip", "conv.hip"])
def test_m0_only_feeds_the_lds_loads(src):
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        subprocess.run([_hipcc(), "-O3", "-std=c++17", "--offload-arch=gfx950", "--offload-device-only", "-S",
                        "-I", INCLUDE, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-x", "hip", os.path.join(CSRC, src), "-o", out],
                       check=True, capture_output=True)
        asm = open(out).read()
    checked = 0
    for name, body in _functions(asm):
        code = [l for l in body if l and not l.startswith((";", "."))]
        if not any(l.startswith("global_load_lds") for l in code):
            continue
        checked += 1
        for i, l in enumerate(code):
            if "m0" not in l.split(";")[0]:
                continue
            assert re.match(r"s_mov_b32 m0, s\d+$", l), f"{name}: other use of M0: {l}"
            assert code[i + 1] == "s_nop 0" and code[i + 2].startswith("global_load_lds_dwordx4"), \
                f"{name}: M0 write not followed by the wait state and the load"
    assert checked >= 4, f"{src}: expected kernels with LDS-direct loads, found {checked}"
