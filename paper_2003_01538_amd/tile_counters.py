"""rocprofv3 evidence for the conv tile table: every candidate tile of every
layer shape whose kernel family has more than one tile, per batch bucket,
timed by the kernel trace and measured by the matrix-core counters.

The committed table (csrc/tile_table.inc) is written by make_tile_table.py
from HIP-event timings inside the library's tuner.  This tool re-runs each
(layer shape, bucket, candidate) as a standalone launch (fs_bench_conv: the
layer's shape, Z models per launch, the library's K-split rule, no
projection shortcut) so that a profiler run can attribute every dispatch:

  run        launch every case in a fixed order (run it under rocprofv3)
  summarize  map the dispatches of a kernel trace and of a counter run back
             to the cases and write a markdown summary

Usage (repository root, on an MI355X, export TMPDIR=/tmp; OUT is any scratch
directory):
  rocprofv3 --kernel-trace --output-format csv -d OUT/trace -o tc -- \
      python3 -m paper_2003_01538_amd.tile_counters run
  rocprofv3 --pmc SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE --output-format csv \
      -d OUT/pmc -o tc -- python3 -m paper_2003_01538_amd.tile_counters run
  python3 -m paper_2003_01538_amd.tile_counters summarize --trace OUT/trace/tc_kernel_trace.csv \
      --pmc OUT/pmc/tc_counter_collection.csv --out profiles/conv_tile_counters.md
"""
from __future__ import annotations

import argparse
import csv
import os
import re
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
TABLE = os.path.join(HERE, "csrc", "tile_table.inc")

PEAK_TFLOPS = 2500.0   # dense bf16 MFMA peak of the MI355X
SIMDS = 1024           # 256 CUs x 4 SIMDs: SQ_VALU_MFMA_BUSY_CYCLES is summed over them
XCDS = 8               # GRBM_GUI_ACTIVE is summed over the XCDs
WARMUP = 3             # fs_bench_conv's untimed launches before the timed ones
ITERS = 5

# workload, buckets (batch sizes), models per launch
PLAN = [("resnet18x3_bf16_b32", (1, 8, 32, 64), 3),
        ("resnet50x5_bf16_b256", (32, 256), 5)]


def conv_shapes(models, in_h, in_w):
    """Distinct conv layer shapes of a network launched by the implicit GEMM
    family: (H, W, Cin, Cout, k, stride, pad, relu, residual, proj, layers).
    A 1x1 conv read only as a residual is the projection shortcut of the
    conv that reads it (computed inside that conv's launch), so it is not
    listed on its own, and proj=True marks its consumer."""
    import workloads as wl
    layers = models[0]
    shapes = wl.layer_shapes(layers, in_h, in_w)
    proj_of = {}
    for i, L in enumerate(layers):
        if L["op"] == "conv" and L.get("res", -1) >= 0:
            r = L["res"]
            R = layers[r]
            if R["op"] == "conv" and R["k"] == 1 and not R["relu"]:
                readers = [j for j, M in enumerate(layers) if M.get("src") == r or M.get("res") == r]
                if readers == [i]:
                    proj_of[r] = i
    out = {}
    for i, L in enumerate(layers):
        if L["op"] != "conv" or i in proj_of:
            continue
        H, W, C = (in_h, in_w, 3) if L["src"] < 0 else shapes[L["src"]]
        key = (H, W, L["cin"], L["cout"], L["k"], L["stride"], L["pad"], int(L["relu"]),
               int(L.get("res", -1) >= 0), int(i in proj_of.values()))
        out.setdefault(key, []).append(i)
    return [k + (tuple(v),) for k, v in out.items()]


def patch_px(shape, B, bm):
    """Patch pixels the halo kernels need for tiles of bm consecutive output
    pixels (the band of padded rows from above a tile's first pixel through
    its last pixel's bottom-right tap), as the library computes it."""
    H, W = shape[0], shape[1]
    HW, PW, HP, M = H * W, W + 2, H + 2, B * H * W
    need = 0
    for m0 in range(0, M, bm):
        m1 = min(M, m0 + bm) - 1
        R0 = (m0 // HW) * HP + (m0 % HW) // W
        b1, y1, x1 = m1 // HW, (m1 % HW) // W, (m1 % HW) % W
        need = max(need, (b1 * HP + y1 - R0) * PW + x1 + 2 * PW + 2 + 1)
    return need


def family_tiles(fsb, shape, B):
    """Names of the candidate tiles for a layer shape at batch B: those of
    the layer's kernel family (the library's shape rule), or [] when the
    family has a single tile (the stem with its pool, the resident-weight
    halo kernel)."""
    H, W, Cin, Cout, k, s, p = shape[:7]
    names = [fsb.fs_conv_tile_name(fsb.FS_BF16, t) for t in range(fsb.fs_conv_num_tiles(fsb.FS_BF16))]
    if Cin == 3:
        return []   # the space-to-depth stem (fused with its max pool)
    if k == 3 and s == 1 and p == 1 and Cin == 64 and W == 56:
        return []   # resident-weight halo kernel
    if k == 3 and s == 1 and p == 1 and Cin % 128 == 0 and Cout % 128 == 0 and not shape[9]:
        out = []    # streamed-weight halo family: 128-pixel tiles (weights through LDS), 160 and 96 (in registers)
        for n in names:
            if "hs_" in n and patch_px(shape, B, 128) <= 8 * 48:
                out.append(n)
            elif "hr_160" in n and patch_px(shape, B, 160) <= 8 * 40:
                out.append(n)
            elif "hr_96" in n and patch_px(shape, B, 96) <= 8 * 40:
                out.append(n)
        return out
    return [n for n in names if "dma" in n]


def cases():
    import workloads as wl
    from paper_2003_01538_amd import flexserve as fsb
    out = []
    for wname, buckets, Z in PLAN:
        w = wl.workload(wname)
        for shape in conv_shapes(w["models"], *w["out_hw"]):
            if shape[9]:
                continue  # carries a projection shortcut, which fs_bench_conv does not take
            for B in buckets:
                for tn in family_tiles(fsb, shape, B):
                    out.append(dict(workload=wname, B=B, Z=Z, shape=shape, tile=tn))
    return out


def run():
    sys.path.insert(0, ROOT)
    from paper_2003_01538_amd import flexserve as fsb
    fsb.load(fsb.LIB_PATH)
    names = {fsb.fs_conv_tile_name(fsb.FS_BF16, t): t for t in range(fsb.fs_conv_num_tiles(fsb.FS_BF16))}
    n = 0
    for c in cases():
        H, W, Cin, Cout, k, s, p, relu, res = c["shape"][:9]
        ms, used = fsb.fs_bench_conv(c["B"], H, W, Cin, Cout, k, s, p, relu, res, fsb.FS_BF16, names[c["tile"]],
                                     c["Z"], ITERS)
        n += 1
        print(f"{c['workload']} B={c['B']} {H}x{W}x{Cin}->{Cout} k{k}s{s} {c['tile']}: {ms * 1e3:.1f} us", flush=True)
    print(f"{n} cases", flush=True)


def table_choice(entries, B, Z, shape):
    H, W, Cin, Cout, k, s, p = shape[:7]
    for e in entries:
        if (e["bucket"], e["z"], e["h"], e["w"], e["cin"], e["cout"], e["kh"], e["stride"], e["pad"]) == \
                (B, Z, H, W, Cin, Cout, k, s, p) and (e["proj_cin"] > 0) == bool(shape[9]):
            return e["tile"]
    return None


def read_table(path=TABLE):
    keys = ("bucket", "prec", "kh", "kw", "stride", "pad", "cin", "cout", "h", "w", "z", "proj_cin", "proj_stride")
    out = []
    for line in open(path):
        m = re.match(r"\s*\{([\d, ]+), \"(\S+)\"\}", line)
        if m:
            vals = [int(v) for v in m.group(1).split(",")]
            out.append(dict(zip(keys, vals), tile=m.group(2)))
    return out


def conv_dispatches(rows):
    """Conv kernel dispatches in dispatch order, each with the split-K
    completion that follows it folded in: [(kernel name, [rows])]."""
    rows = sorted(rows, key=lambda r: int(r["Dispatch_Id"]))
    out = []
    for r in rows:
        name = r["Kernel_Name"]
        if "k_conv_splitk_reduce" in name:
            if out:
                out[-1][1].append(r)
        elif "k_conv" in name or "k_stem_pool" in name:
            out.append((name, [r]))
    return out


def per_dispatch(path):
    """Counter CSV -> {dispatch id: {counter: summed value}} and the rows."""
    agg, meta = {}, {}
    for r in csv.DictReader(open(path)):
        d = int(r["Dispatch_Id"])
        agg.setdefault(d, {})
        agg[d][r["Counter_Name"]] = agg[d].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        meta[d] = r
    rows = [dict(meta[d], Dispatch_Id=str(d)) for d in sorted(meta)]
    return agg, rows


def assign(cs, disp):
    """Split the dispatch list over the cases: WARMUP + ITERS each, in order;
    returns per case the timed dispatches."""
    per = WARMUP + ITERS
    if len(disp) != per * len(cs):
        raise SystemExit(f"{len(disp)} conv dispatches for {len(cs)} cases x {per}")
    out = []
    for i, c in enumerate(cs):
        ds = disp[i * per:(i + 1) * per]
        kern = "k_conv_hr" if "hr_" in c["tile"] else "k_conv_hs" if "hs_" in c["tile"] else "k_conv_dma"
        if any(kern not in name for name, _ in ds):
            raise SystemExit(f"case {i} ({c['tile']}): unexpected kernel {ds[0][0]}")
        out.append(ds[WARMUP:])
    return out


def summarize(trace_csv, pmc_csv, out_path, cmdline):
    sys.path.insert(0, ROOT)
    cs = cases()
    tr = assign(cs, conv_dispatches(list(csv.DictReader(open(trace_csv)))))
    agg, prow = per_dispatch(pmc_csv)
    pm = assign(cs, conv_dispatches(prow))
    table = read_table()
    dur = lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    L = ["# Conv tile candidates under rocprofv3: kernel-trace time and matrix-core counters", "",
         "Commands (repository root on an MI355X, `export TMPDIR=/tmp`):", "", "```"] + cmdline + ["```", "",
         "Every candidate tile of every conv layer shape whose kernel family has several (the implicit GEMM; "
         "the streamed-weight halo family of the 3x3/1 layers with Cin >= 128; the stem and the "
         "resident-weight halo kernel have one tile and are not listed), per batch size, launched alone by "
         "`fs_bench_conv` "
         f"({WARMUP} untimed + {ITERS} timed launches, Z models per launch, the library's K-split rule; a layer "
         "that carries a projection shortcut is left out: the other layers of its stage have its "
         "shape without the shortcut).  `us`: kernel-trace "
         "duration per launch (conv plus its split-K completion), mean of the timed launches.  `TF/s` and "
         "`frac`: algorithmic FLOP (2 M N K Z) over that time, against the 2.5 PFLOP/s dense bf16 peak.  "
         f"`MFMA busy`: `SQ_VALU_MFMA_BUSY_CYCLES` / (`GRBM_GUI_ACTIVE` / {XCDS} x {SIMDS} SIMDs) of the conv "
         "dispatch (the counter run serialises dispatches, so this is per launch).  `table`: the tile the "
         "committed table picks for this layer and bucket (`*`), chosen from HIP-event timings inside the "
         "library on the whole network, where a later candidate had to win by 3 %.", ""]
    groups = {}
    for c, tdisp, pdisp in zip(cs, tr, pm):
        groups.setdefault((c["workload"], c["B"], c["Z"], c["shape"]), []).append((c, tdisp, pdisp))
    agree = total = 0
    for (wname, B, Z, shape), items in groups.items():
        H, W, Cin, Cout, k, s, p, relu, res, proj, lays = shape
        Ho, Wo = (H + 2 * p - k) // s + 1, (W + 2 * p - k) // s + 1
        fl = 2.0 * B * Ho * Wo * Cout * k * k * Cin * Z
        chosen = table_choice(table, B, Z, shape)
        rows = []
        for c, t, pp in items:
            us = sum(sum(dur(r) for r in rs) for _, rs in t) / len(t)
            busy = []
            for _, rs in pp:
                d = int(rs[0]["Dispatch_Id"])
                a = agg[d]
                busy.append(a["SQ_VALU_MFMA_BUSY_CYCLES"] / (a["GRBM_GUI_ACTIVE"] / XCDS * SIMDS))
            rows.append((us, c["tile"], fl / us / 1e6, sum(busy) / len(busy)))
        best = min(rows)[1]
        if chosen is not None:
            total += 1
            cu = next((r[0] for r in rows if r[1] == chosen), None)
            agree += int(cu is not None and cu <= 1.05 * min(rows)[0])
        L += [f"### {wname}, B = {B}: {H}x{W}x{Cin} -> {Cout}, {k}x{k}/{s}"
              f"{' +res' if res else ''} (layers {', '.join(str(x) for x in lays)}; M {B * Ho * Wo} x N {Cout} x "
              f"K {k * k * Cin}, Z {Z})", "",
              "| tile | us | TF/s | frac | MFMA busy | table |", "|---|---|---|---|---|---|"]
        for us, tn, tf, bz in sorted(rows):
            L.append(f"| {tn}{' (fastest)' if tn == best else ''} | {us:.1f} | {tf:.0f} | {tf / PEAK_TFLOPS:.3f} | "
                     f"{bz:.3f} | {'*' if tn == chosen else ''} |")
        L.append("")
    L.append(f"Table choices within 5 % of the fastest standalone candidate: {agree} of {total}.")
    with open(out_path, "w") as f:
        f.write("\n".join(L) + "\n")
    print(f"{len(groups)} layer shapes x buckets; table within 5 %: {agree}/{total} -> {out_path}")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("mode", choices=("run", "summarize", "list"))
    ap.add_argument("--trace")
    ap.add_argument("--pmc")
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "conv_tile_counters.md"))
    args = ap.parse_args()
    sys.path.insert(0, ROOT)
    if args.mode == "run":
        run()
    elif args.mode == "list":
        cs = cases()
        print(len(cs), "cases")
    else:
        def run_cmd(path, what, tail):
            d, f = os.path.split(path)
            return f"rocprofv3 {what} --output-format csv -d {d} -o {f.split(tail)[0]} -- " \
                   "python3 -m paper_2003_01538_amd.tile_counters run"
        cmd = [run_cmd(args.trace, "--kernel-trace", "_kernel_trace"),
               run_cmd(args.pmc, "--pmc SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE", "_counter_collection"),
               f"python3 -m paper_2003_01538_amd.tile_counters summarize --trace {args.trace} --pmc {args.pmc} "
               f"--out {os.path.relpath(args.out, ROOT) if os.path.isabs(args.out) else args.out}"]
        summarize(args.trace, args.pmc, args.out, cmd)


if __name__ == "__main__":
    main()
