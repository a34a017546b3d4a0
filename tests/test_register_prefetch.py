"""The kernels that prefetch MFMA operands into registers (the small-tile GEMM's ring of K
tiles, the stem's stream of block-pair chunks) rely on the compiler waiting for the tile
about to be multiplied only.  Register copies between prefetch sets, or a prefetch under a
condition, make it wait for every load in flight instead (vmcnt(0) before the multiply),
which silently turns the prefetch off.  Compile the sources for gfx950 to assembly (code
built here) and check the waits inside those kernels' main loops."""
import functools
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


@functools.lru_cache(maxsize=None)
def _asm(src):
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "k.s")
        subprocess.run([_hipcc(), "-O3", "-std=c++17", "--offload-arch=gfx950", "--offload-device-only", "-S",
                        "-I", INCLUDE, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-x", "hip", os.path.join(CSRC, src), "-o", out],
                       check=True, capture_output=True)
        return open(out).read()


def _kernels(asm, prefix):
    """{name: lines} of the kernels whose mangled name starts with prefix."""
    out = {}
    for m in re.finditer(r"^(" + re.escape(prefix) + r"[^\s:]*):", asm, re.M):
        end = asm.find(".Lfunc_end", m.end())
        if end > 0:   # a function body, not another label of that name
            out[m.group(1)] = [l.strip() for l in asm[m.end():end].splitlines()]
    return out


def _mfma_loop(lines):
    """Lines of the loop whose own blocks hold the MFMAs (the innermost one), gathered from the
    compiler's block comments (a block inside a loop names that loop's header block)."""
    blocks, cur = [], None
    for l in lines:
        m = re.match(r"^\.L(BB\w+):", l) or re.match(r"^; (%bb\.\d+):", l)
        if m:
            cur = {"name": m.group(1), "lines": [], "loop": None}
            blocks.append(cur)
        if cur is None:
            continue
        cur["lines"].append(l)
        h = re.search(r"in Loop: Header=(BB\w+)", l)
        if h and cur["loop"] is None:
            cur["loop"] = h.group(1)
        if "Loop Header" in l and cur["loop"] is None:
            cur["loop"] = cur["name"]
    loops = {}
    for bl in blocks:
        if bl["loop"]:
            loops.setdefault(bl["loop"], []).extend(bl["lines"])
    with_mfma = [body for body in loops.values() if any(x.startswith("v_mfma") for x in body)]
    return min(with_mfma, key=len) if with_mfma else None


def _vmcnt(body):
    return [int(m.group(1)) for x in body for m in [re.search(r"vmcnt\((\d+)\)", x)] if x.startswith("s_waitcnt") and m]


def test_small_gemm_multiplies_with_three_tiles_in_flight():
    ks = _kernels(_asm("gemm.hip"), "_ZN3vcr12k_gemm_small")
    assert len(ks) >= 4
    for name, lines in ks.items():
        body = _mfma_loop(lines)
        assert body is not None, name
        assert sum(x.startswith("v_mfma") for x in body) == 64, name   # four K tiles per round
        waits = _vmcnt(body)
        # each multiply waits for its own tile only: three tiles of 8 loads stay in flight
        assert waits and min(waits) >= 24, (name, waits)


def test_small_gemm_fits_three_waves_per_simd():
    asm = _asm("gemm.hip")
    for m in re.finditer(r"\.name:\s+(_ZN3vcr12k_gemm_small\S+)", asm):
        meta = asm[m.start():m.start() + 4000]
        vg = int(re.search(r"\.vgpr_count:\s+(\d+)", meta).group(1))
        assert vg <= 168, (m.group(1), vg)


def test_stem_step_loop_keeps_the_next_step_in_flight():
    ks = _kernels(_asm("conv.hip"), "_ZN3vcr6k_stem")
    assert len(ks) >= 3
    for name, lines in ks.items():
        body = _mfma_loop(lines)
        assert body is not None, name
        waits = _vmcnt(body)
        # no wait for every load in flight inside the step loop: the step being multiplied
        # is waited for while the next one's 8 loads (or part of them) stay outstanding
        assert waits and 0 not in waits, (name, waits)
        assert max(waits) >= 8, (name, waits)
