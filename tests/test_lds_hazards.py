"""The streamed-weight halo kernel reads its MFMA operands from LDS with
inline-assembly `ds_read_b128` whose destination registers are only safe to
use after the wave's own `s_waitcnt lgkmcnt` that covers them (the kernel
waits for them itself, a step later).  Register allocation decides whether
that holds: an allocator copying a still-loading register (for instance into
an accumulation register to relieve pressure) would move stale data without
any error.  This test compiles the kernel source to gfx950 assembly on the
CPU and scans every kernel in it, instruction by instruction, for a use of a
`ds_read` destination before the `lgkmcnt` wait that covers it."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2003_01538_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _regs(tok):
    m = re.match(r"^([va])\[(\d+):(\d+)\]$", tok)
    if m:
        return {(m.group(1), i) for i in range(int(m.group(2)), int(m.group(3)) + 1)}
    m = re.match(r"^([va])(\d+)$", tok)
    return {(m.group(1), int(m.group(2)))} if m else set()


def lds_hazards(lines):
    """(line, text) of every instruction that reads or writes a register an
    LDS read still in flight will write.  LDS operations complete in order
    for lgkmcnt; a straight-line scan (branch targets are not assumed to
    have waited) is conservative for the kernels' unrolled steps."""
    pending, found = [], []
    for ln, raw in lines:
        line = raw.split(";")[0].strip()
        if not line or line.endswith(":") or line.startswith("."):
            continue
        op = line.split()[0]
        ops = [t.strip().split()[0] for t in line[len(op):].split(",") if t.strip()]
        if op == "s_waitcnt":
            m = re.search(r"lgkmcnt\((\d+)\)", line)
            if m:
                n = int(m.group(1))
                pending = pending[len(pending) - n:] if 0 < n < len(pending) else ([] if n == 0 else pending)
            continue
        srcs, dsts = set(), set()
        if op.startswith("ds_read"):
            dsts = _regs(ops[0]) if ops else set()
            for o in ops[1:]:
                srcs |= _regs(o)
        elif op.startswith("ds_") or "store" in op:
            for o in ops:
                srcs |= _regs(o)
        else:
            if ops:
                dsts = _regs(ops[0])
            for o in ops[1:]:
                srcs |= _regs(o)
        live = set().union(*pending) if pending else set()
        if (srcs | (set() if op.startswith("ds_read") else dsts)) & live:
            found.append((ln, raw.strip()))
        if op.startswith("ds_"):
            pending.append(dsts if op.startswith("ds_read") else set())
    return found


def _functions(asm):
    funcs, cur = {}, None
    for i, l in enumerate(asm.splitlines()):
        m = re.match(r"^(_Z\S+):", l)
        if m:
            cur = m.group(1)
            funcs[cur] = []
        elif cur and l.strip().startswith(".size"):
            cur = None
        elif cur:
            funcs[cur].append((i + 1, l))
    return funcs


def test_scanner_flags_an_early_use():
    asm = ["\tds_read_b128 v[8:11], v2", "\tds_read_b128 v[12:15], v2 offset:16", "\tv_accvgpr_write_b32 a5, v10",
           "\ts_waitcnt lgkmcnt(1)", "\tv_mov_b32 v20, v9", "\tv_mov_b32 v21, v13", "\ts_waitcnt lgkmcnt(0)",
           "\tv_mov_b32 v22, v13"]
    found = lds_hazards(list(enumerate(asm, 1)))
    assert [ln for ln, _ in found] == [3, 6]


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc not installed")
def test_streamed_weight_halo_kernel_uses_lds_reads_only_after_their_wait():
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, "conv_hs.s")
        cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
               "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-x", "hip",
               "--cuda-device-only", "-S", os.path.join(CSRC, "conv_hs.hip"), "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        funcs = _functions(open(out).read())
    kernels = {f: lines for f, lines in funcs.items() if "k_conv_hs" in f}
    assert kernels
    for f, lines in kernels.items():
        found = lds_hazards(lines)
        assert not found, f"{f}: {len(found)} uses before the wait, first {found[:3]}"
