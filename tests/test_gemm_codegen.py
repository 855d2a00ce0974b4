"""Code generation of the grouped GEMMs (CPU only: hipcc cross-compiles gfx950 device assembly).

Some tile configurations use all 256 architectural registers of a wave and spill a few values
to scratch.  Those accesses must stay outside the K loops: inside, a scratch load is a vector
memory load like the slice copies, and waiting for it (vmcnt counts in issue order) would also
wait for every copy in flight.  For every kernel with MFMAs this test finds its innermost loops
that contain MFMAs (a backward branch to an earlier label) and checks that no scratch access sits
inside one."""
import os
import re
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_18631_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

pytestmark = pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")


def _device_asm(src, out):
    from paper_2607_18631_amd import build
    cmd = [HIPCC, *build.FLAGS, "-I", CSRC, "-x", "hip", "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", out]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    with open(out) as f:
        return f.read()


def _mfma_loops(lines):
    """(first, last) line spans of the innermost loops that contain an MFMA."""
    labels = {}
    for i, l in enumerate(lines):
        m = re.match(r"(\.LBB\d+_\d+):", l)
        if m:
            labels[m.group(1)] = i
    loops = []
    for i, l in enumerate(lines):
        m = re.search(r"s_(?:cbranch_\w+|branch)\s+(\.LBB\d+_\d+)", l)
        if m and m.group(1) in labels and labels[m.group(1)] < i:
            loops.append((labels[m.group(1)], i))
    has_mfma = [(a, b) for a, b in loops if any("v_mfma" in lines[k] for k in range(a, b))]
    return [(a, b) for a, b in has_mfma
            if not any((c, d) != (a, b) and a <= c and d <= b for c, d in has_mfma)]


@pytest.fixture(scope="module")
def device_asm(tmp_path_factory):
    d = tmp_path_factory.mktemp("asm")
    srcs = ["gemm.hip", "gemm_bwd.hip"]
    with ThreadPoolExecutor(len(srcs)) as ex:
        texts = list(ex.map(lambda s: _device_asm(s, str(d / (s + ".s"))), srcs))
    return dict(zip(srcs, texts))


@pytest.mark.parametrize("src", ["gemm.hip", "gemm_bwd.hip"])
def test_no_scratch_in_mfma_loops(device_asm, src):
    funcs = re.split(r"\n(?=_Z\S+:)", device_asm[src])
    checked = 0
    for f in funcs:
        if "v_mfma" not in f:
            continue
        name = f.split(":", 1)[0]
        lines = f.split("\n")
        loops = _mfma_loops(lines)
        assert loops, f"no MFMA loop found in {name}"
        inside = [lines[i].strip() for a, b in loops for i in range(a, b + 1) if "scratch_" in lines[i]]
        assert not inside, f"{name}: scratch accesses inside an MFMA loop: {inside[:4]}"
        checked += 1
    assert checked >= 8, f"only {checked} MFMA kernels found in {src}"
    print(f"[codegen] {src}: {checked} MFMA kernels, no scratch access inside their K loops")


def test_loop_finder_sees_scratch_in_a_loop():
    """The loop finder on a hand-written listing: a scratch reload inside the MFMA loop is found,
    one in the prologue or in an outer loop's tile code is not."""
    asm = """_Zk:
\tscratch_load_dword v1, off, off
.LBB0_1:
\tscratch_load_dword v2, off, off offset:4
.LBB0_2:
\tv_mfma_f32_32x32x16_bf16 a[0:15], v[0:3], v[4:7], a[0:15]
\tscratch_load_dword v3, off, off offset:8
\ts_cbranch_scc1 .LBB0_2
\tglobal_store_dword v0, v1, s[0:1]
\ts_cbranch_vccnz .LBB0_1
\ts_endpgm""".split("\n")
    loops = _mfma_loops(asm)
    assert loops == [(4, 7)]
    inside = [asm[i] for a, b in loops for i in range(a, b + 1) if "scratch_" in asm[i]]
    assert inside == ["\tscratch_load_dword v3, off, off offset:8"]
