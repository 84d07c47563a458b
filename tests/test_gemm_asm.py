"""Assembly-level invariants of the kernels that issue untracked loads (CPU
only: cross-compiles csrc/gemm.hip and csrc/attention.hip for gfx950 and reads
the generated assembly).

The GEMM's activation fragments and weight copies and the attention kernel's
K / V tiles are loaded by inline assembly that the compiler does not track (its
own waits would stall on younger loads), which is only correct if the compiler
never reads, moves or reuses those registers while the loads are in flight.
These tests make that a checked property of every build instead of an
assumption:
  * vector memory operations complete in issue order, so after
    `s_waitcnt vmcnt(N)` all but the N most recent ones have landed; walking
    each kernel in program order with that rule, no instruction other than
    the load itself touches a register whose load may still be in flight;
  * no gemm or attention kernel uses scratch memory;
  * the MFMA loop blocks of the GEMM contain no AGPR/VGPR copies (the
    accumulators stay in place).
The walk follows the text in order, which matches the control flow of these
kernels: their loads are issued on every path (clamped indices instead of
branches), so no conditional block holds a load.
"""
import importlib.util
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
MEM = re.compile(r"^(global|buffer|flat|scratch)_(load|store|atomic)")


def _build_module():
    # the library's own compile flags (build.py loaded by path: importing the
    # package would load the library)
    spec = importlib.util.spec_from_file_location(
        "lopa_build", os.path.join(ROOT, "paper_2512_16229_amd", "build.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    return b


def _compile(tmp_path_factory, src):
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not available")
    b = _build_module()
    out = str(tmp_path_factory.mktemp("asm") / (src + ".s"))
    flags = [f for f in b.FLAGS if f != "-fPIC"] + b.EXTRA_FLAGS.get(src + ".hip", [])
    cmd = [HIPCC, *flags, "--cuda-device-only", "-S",
           os.path.join(ROOT, "paper_2512_16229_amd", "csrc", src + ".hip"), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read()


@pytest.fixture(scope="module")
def asm(tmp_path_factory):
    return _compile(tmp_path_factory, "gemm")


@pytest.fixture(scope="module")
def attn_asm(tmp_path_factory):
    return _compile(tmp_path_factory, "attention")


def _kernels(s, kind="gemm_kernel"):
    for name in re.findall(r"^(_Z[\w.]+" + kind + r"[\w.]+):", s, re.M):
        i = s.index(name + ":")
        j = s.index(".Lfunc_end", i)
        yield name, s[i:j].split("\n")


def _regs(tok):
    m = re.match(r"([va])\[(\d+):(\d+)\]", tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"([va])(\d+)$", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def _inflight_violations(body):
    """Instructions that touch a register while a load into it may be in flight."""
    fifo, bad = [], []
    for line in body:
        t = line.strip()
        if not t or t.startswith((";", ".")) or t.endswith(":"):
            continue
        if t.startswith("s_waitcnt"):
            m = re.search(r"vmcnt\((\d+)\)", t)
            if m:
                del fifo[:max(0, len(fifo) - int(m.group(1)))]
            continue
        op = t.split()[0]
        ops = [o.strip() for o in t.split(None, 1)[1].split(",")] if " " in t else []
        used = set()
        for o in ops:
            if o:
                used |= _regs(o.split()[0])
        inflight = set().union(*fifo) if fifo else set()
        if used & inflight:
            bad.append(t)
        if MEM.match(op):
            dest = set()
            if "_load" in op and "_lds" not in op and ops:
                dest = _regs(ops[0].split()[0])
            fifo.append(dest)
    return bad


def test_kernels_found(asm, attn_asm):
    assert len(list(_kernels(asm))) >= 6
    assert len(list(_kernels(attn_asm, "attn_kernel"))) >= 8


def test_inflight_registers_untouched(asm, attn_asm):
    for s, kind in ((asm, "gemm_kernel"), (attn_asm, "attn_kernel")):
        for name, body in _kernels(s, kind):
            bad = _inflight_violations(body)
            assert not bad, f"{name}: in-flight registers touched: {bad[:5]}"


def test_no_scratch(asm, attn_asm):
    for s, kind in ((asm, "gemm_kernel"), (attn_asm, "attn_kernel")):
        for name, body in _kernels(s, kind):
            assert "scratch_" not in "\n".join(body), f"{name} spills to scratch"


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


def test_attention_inline_asm_is_memory_only(attn_asm):
    """The attention kernels' MFMAs are compiler builtins, so the compiler
    inserts the wait states before their results are read; that holds only
    for instructions it sees. Its inline assembly is therefore limited to the
    asynchronous copies and explicit waits (no vector arithmetic that could
    read an MFMA result too early)."""
    allowed = re.compile(r"^(s_mov_b32 m0,|global_load_lds_dwordx4|s_waitcnt)")
    for kind in ("attn_kernel", "attn_prefix_kernel", "attn_block_kernel"):
        for name, body in _kernels(attn_asm, kind):
            inside = False
            for line in body:
                t = line.strip()
                if t.startswith(";;#ASMSTART"):
                    inside = True
                elif t.startswith(";;#ASMEND"):
                    inside = False
                elif inside and t and not t.startswith(";"):
                    assert allowed.match(t), f"{name}: inline asm {t!r}"
