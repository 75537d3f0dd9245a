"""The streamed-weight halo kernel reads its MFMA operands from LDS with
inline-assembly `ds_read_b128` whose destination registers are only safe to
use after the wave's own `s_waitcnt lgkmcnt` that covers them (the kernel
waits for them itself, a step later).  Register allocation decides whether
that holds: an allocator copying a still-loading register (for instance into
an accumulation register to relieve pressure) would move stale data without
any error.  This test compiles the kernel source to gfx950 assembly on the
CPU and scans every kernel in it, along its control flow (basic blocks,
branches, loops), for a use of a `ds_read` destination before the `lgkmcnt`
wait that covers it on some path."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2003_01538_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
LGKM_MAX = 15  # lgkmcnt field width on gfx9: the wave stalls rather than exceed it


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


def _step(state, line):
    """One instruction on a pending-read state (a list of register sets, the
    oldest first): returns (new state, whether the instruction touches a
    register that an earlier LDS read may still be writing)."""
    line = line.split(";")[0].strip()
    if not line or line.endswith(":") or line.startswith("."):
        return state, False
    op = line.split()[0]
    ops = [t.strip().split()[0] for t in line[len(op):].split(",") if t.strip()]
    if op == "s_waitcnt":
        m = re.search(r"lgkmcnt\((\d+)\)", line)
        if m:
            n = int(m.group(1))
            state = state[len(state) - n:] if 0 < n < len(state) else ([] if n == 0 else state)
        return state, False
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
    live = set().union(*state) if state else set()
    bad = bool((srcs | (set() if op.startswith("ds_read") else dsts)) & live)
    if op.startswith("ds_"):
        # the counter holds at most 15 outstanding operations: an older one
        # has completed
        state = (state + [dsts if op.startswith("ds_read") else set()])[-LGKM_MAX:]
    return state, bad


def _merge(x, y):
    """Union of two pending states, aligned on the newest read (lgkmcnt(n)
    keeps the n newest on every path)."""
    n = max(len(x), len(y))
    x = [set()] * (n - len(x)) + list(x)
    y = [set()] * (n - len(y)) + list(y)
    return [a | b for a, b in zip(x, y)]


def lds_hazards_cfg(lines):
    """The same check along the control flow: basic blocks from labels and
    branches, the pending reads that may reach a block merged over its
    predecessors until nothing changes, then every instruction checked
    against what may be pending before it."""
    blocks, labels, cur = [], {}, None
    for ln, raw in lines:
        t = raw.split(";")[0].strip()
        m = re.match(r"^(\.LBB\S+):", t)
        if m or cur is None:
            cur = dict(label=m.group(1) if m else None, body=[], succ=[], falls=True)
            blocks.append(cur)
            if m:
                labels[m.group(1)] = len(blocks) - 1
                continue
        if not t or t.startswith("."):
            continue
        cur["body"].append((ln, raw))
        op = t.split()[0]
        if op.startswith("s_branch") or op.startswith("s_cbranch") or op == "s_endpgm" or op == "s_setpc_b64":
            tgt = t.split()[1] if op.startswith("s_branch") or op.startswith("s_cbranch") else None
            cur["succ"] = [tgt] if tgt else []
            cur["falls"] = op.startswith("s_cbranch")
            cur = dict(label=None, body=[], succ=[], falls=True)
            blocks.append(cur)
    succ = []
    for i, b in enumerate(blocks):
        s_ = [labels[t] for t in b["succ"] if t in labels]
        if b["falls"] and i + 1 < len(blocks):
            s_.append(i + 1)
        succ.append(s_)
    inn = [None] * len(blocks)
    inn[0] = []
    work = [0]
    while work:
        i = work.pop()
        st = inn[i]
        for _, raw in blocks[i]["body"]:
            st, _ = _step(st, raw)
        for j in succ[i]:
            new = st if inn[j] is None else _merge(inn[j], st)
            if inn[j] is None or new != inn[j]:
                inn[j] = new
                work.append(j)
    found = []
    for i, b in enumerate(blocks):
        st = inn[i] if inn[i] is not None else []
        for ln, raw in b["body"]:
            st, bad = _step(st, raw)
            if bad:
                found.append((ln, raw.strip()))
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


def test_flow_scan_follows_a_loop():
    # reads issued at the loop head and waited for in the body: a copy on the
    # exit path, after the body's wait, is safe; one on the way into the body,
    # before the wait, is not
    asm = [".LBB0_1:", "\tds_read_b128 v[8:11], v2", "\ts_cbranch_scc1 .LBB0_3", "\tv_mov_b32 v30, v9",
           ".LBB0_2:", "\ts_waitcnt lgkmcnt(0)", "\tv_mov_b32 v20, v9", "\ts_cbranch_scc0 .LBB0_1",
           ".LBB0_3:", "\ts_waitcnt lgkmcnt(0)", "\tv_mov_b32 v21, v10", "\ts_endpgm"]
    found = lds_hazards_cfg(list(enumerate(asm, 1)))
    assert [ln for ln, _ in found] == [4]
    # a read left in flight around the back edge reaches the head again
    asm2 = [".LBB1_1:", "\tv_mov_b32 v40, v9", "\tds_read_b128 v[8:11], v2", "\ts_cbranch_scc0 .LBB1_1",
            "\ts_waitcnt lgkmcnt(0)", "\ts_endpgm"]
    assert [ln for ln, _ in lds_hazards_cfg(list(enumerate(asm2, 1)))] == [2]


def test_scanner_flags_an_early_use():
    asm = ["\tds_read_b128 v[8:11], v2", "\tds_read_b128 v[12:15], v2 offset:16", "\tv_accvgpr_write_b32 a5, v10",
           "\ts_waitcnt lgkmcnt(1)", "\tv_mov_b32 v20, v9", "\tv_mov_b32 v21, v13", "\ts_waitcnt lgkmcnt(0)",
           "\tv_mov_b32 v22, v13"]
    found = lds_hazards(list(enumerate(asm, 1)))
    assert [ln for ln, _ in found] == [3, 6]


def _compile_functions(src):
    with tempfile.TemporaryDirectory() as d:
        out = os.path.join(d, src + ".s")
        cmd = [HIPCC, "-O3", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
               "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-x", "hip",
               "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", out]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr[-2000:]
        return _functions(open(out).read())


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="hipcc not installed")
def test_streamed_weight_halo_kernel_uses_lds_reads_only_after_their_wait():
    funcs = _compile_functions("conv_hs.hip")
    kernels = {f: lines for f, lines in funcs.items() if "k_conv_hs" in f}
    assert kernels
    for f, lines in kernels.items():
        found = lds_hazards_cfg(lines)
        assert not found, f"{f}: {len(found)} uses before the wait, first {found[:3]}"
