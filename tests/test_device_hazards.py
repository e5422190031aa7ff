"""Wait states the compiler cannot insert: scan the gfx950 assembly of the
library for two ISA hazards around the direct global->LDS copies, which are
written as inline assembly (the compiler inserts no wait states inside or in
front of assembly it cannot see into).

  * A vector instruction (v_readfirstlane and the like) writes a scalar
    register, and a vector-memory instruction reads it as its base fewer than
    five wait states later: the load may use the register's previous value.
  * s_mov to M0 directly followed by a copy to LDS, which reads M0: one wait
    state is required.

A kernel of this repository once loaded from a stale scalar base this way and
faulted; the scanner is checked on snippets first, then run on the real build.
"""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _sregs(tok):
    out = set()
    for m in re.finditer(r"s\[(\d+):(\d+)\]|\bs(\d+)\b", tok):
        if m.group(1):
            out |= set(range(int(m.group(1)), int(m.group(2)) + 1))
        else:
            out.add(int(m.group(3)))
    return out


def scan(asm: str):
    """Findings as (line, text, reason)."""
    found = []
    recent = []      # (line, scalar registers written by a vector instruction, wait states since)
    m0_since = None  # wait states since the last write of M0
    for i, raw in enumerate(asm.split("\n"), 1):
        s = raw.strip()
        if re.match(r"^_Z\w+:", s):
            recent, m0_since = [], None
        if not s or s[0] in ";.":
            continue
        op = s.split()[0]
        states = int(s.split()[1]) + 1 if op == "s_nop" else 1
        is_vmem = op.startswith(("global_", "buffer_", "scratch_"))
        if is_vmem:
            args = s[len(op):]
            tail = args.split(",", 2)[-1] if "," in args else ""
            for (j, regs, w) in recent:
                if regs & _sregs(tail):
                    found.append((i, s, f"reads scalar registers a vector instruction wrote {w} wait states before"))
            if "global_load_lds" in op and m0_since == 0:
                found.append((i, s, "reads M0 right after its write"))
        # advance the wait-state counters past this instruction
        recent = [(j, r, w + states) for (j, r, w) in recent if w + states < 5]
        if m0_since is not None:
            m0_since += states
        if op.startswith("v_") and "," in s:
            dst = s[len(op):].split(",")[0]
            r = _sregs(dst) if re.search(r"\bs\[|\bs\d", dst) else set()
            if r:
                recent.append((i, r, 0))
        if op.startswith("s_") and "," in s and s[len(op):].split(",")[0].strip() == "m0":
            m0_since = 0
    return found


def test_scanner_finds_the_hazards_it_looks_for():
    bad = "\n".join([
        "_Zk:",
        "\tv_readfirstlane_b32 s3, v90",
        "\tv_readfirstlane_b32 s2, v91",
        "\tglobal_load_dwordx4 v[70:73], v204, s[2:3]",
        "\ts_mov_b32 m0, s11",
        "\tglobal_load_lds_dwordx4 v[2:3], off",
    ])
    reasons = [r for _, _, r in scan(bad)]
    assert len(reasons) == 3 and sum("M0" in r for r in reasons) == 1
    good = "\n".join([
        "_Zk:",
        "\tv_readfirstlane_b32 s3, v90",
        "\tv_readfirstlane_b32 s2, v91",
        "\ts_nop 4",
        "\tglobal_load_dwordx4 v[70:73], v204, s[2:3]",
        "\ts_add_u32 s4, s22, 0x400",  # scalar-unit writes need no wait states
        "\tglobal_load_dwordx4 v[74:77], v204, s[4:5]",
        "\ts_mov_b32 m0, s11",
        "\ts_nop 0",
        "\tglobal_load_lds_dwordx4 v[2:3], off",
    ])
    assert scan(good) == []


def test_library_assembly_has_no_scalar_base_or_m0_hazards():
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    import importlib.util
    spec = importlib.util.spec_from_file_location("ts3_build", os.path.join(ROOT, "paper_2602_04940_amd", "build.py"))
    build = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(build)
    flags = [f for f in build.HIP_FLAGS if f not in ("-shared", "-fPIC")]
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "dev.s")
        r = subprocess.run([hipcc, *flags, "--cuda-device-only", "-S", "-o", out, build.SRC],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        with open(out) as f:
            asm = f.read()
    assert asm.count("global_load_lds") > 0  # the copies are there to be checked
    found = scan(asm)
    assert not found, "\n".join(f"line {i}: {s} ({why})" for i, s, why in found[:20])
