"""Assembly-level invariants of the GEMM kernels (CPU only: cross-compiles
csrc/gemm.hip for gfx950 and reads the generated assembly).

The activation fragments and the weight chunks are loaded by inline assembly
that the compiler does not track (its own waits would stall on younger loads),
which is only correct if the compiler never reads or moves those registers
while the loads are in flight. These tests make that a checked property of
every build instead of an assumption:
  * a register written by an inline-assembly global_load_dwordx4 is, until an
    s_waitcnt vmcnt(0), only read as an MFMA source (never copied, spilled,
    or reused);
  * no gemm kernel uses scratch memory;
  * the MFMA loop blocks contain no AGPR/VGPR copies (the accumulators stay in
    place).
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    out = str(tmp_path_factory.mktemp("asm") / "gemm.s")
    cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"),
           "--cuda-device-only", "-S", os.path.join(ROOT, "paper_2512_16229_amd", "csrc", "gemm.hip"),
           "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read()


def _kernels(s):
    for name in re.findall(r"^(_Z[\w.]+gemm_kernel[\w.]+):", s, re.M):
        i = s.index(name + ":")
        j = s.index(".Lfunc_end", i)
        yield name, s[i:j].split("\n")


def _regs(tok):
    m = re.match(r"v\[(\d+):(\d+)\]", tok)
    if m:
        return set(range(int(m.group(1)), int(m.group(2)) + 1))
    m = re.match(r"v(\d+)$", tok)
    return {int(m.group(1))} if m else set()


def test_kernels_found(asm):
    names = [n for n, _ in _kernels(asm)]
    assert len(names) >= 6, names


def test_inflight_activation_registers_untouched(asm):
    for name, body in _kernels(asm):
        inflight, bad = set(), []
        for line in body:
            t = line.strip()
            if not t or t.startswith((";", ".")):
                continue
            if t.startswith("global_load_dwordx4"):
                inflight |= _regs(t.split()[1].rstrip(","))
                continue
            if re.match(r"s_waitcnt vmcnt\(0\)", t):
                inflight = set()
                continue
            ops = [o.strip() for o in t.split(None, 1)[1].split(",")] if " " in t else []
            regs = set()
            for o in ops:
                if o:
                    regs |= _regs(o.split()[0])
            if not regs & inflight:
                continue
            if t.startswith("v_mfma") and not (_regs(ops[0]) & inflight):
                continue
            bad.append(t)
        assert not bad, f"{name}: in-flight registers touched: {bad[:5]}"


def test_no_scratch(asm):
    for name, body in _kernels(asm):
        text = "\n".join(body)
        assert "scratch_" not in text, f"{name} spills to scratch"


def test_mfma_loops_keep_accumulators_in_place(asm):
    for name, body in _kernels(asm):
        block, blocks = [], []
        for line in body:
            if re.match(r"^(\.LBB\w+|; %bb\.\d+):", line):
                blocks.append(block)
                block = []
            block.append(line.strip())
        blocks.append(block)
        for b in blocks:
            if sum(1 for t in b if t.startswith("v_mfma")) >= 32:
                copies = [t for t in b if t.startswith(("v_accvgpr_read", "v_accvgpr_write",
                                                        "v_accvgpr_mov"))]
                assert not copies, f"{name}: {len(copies)} accumulator copies in an MFMA loop"
