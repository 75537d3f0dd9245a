"""Regenerate the committed conv tile table (csrc/tile_table.inc) on an MI355X.

For every benchmark workload and every batch bucket it serves, the ensemble
is built with FS_TUNE=3, so the first pass of each bucket times every
candidate tile of every conv layer's kernel family (HIP events, two launches
after a warm-up) and keeps the fastest, where the committed table's tile,
timed first, is replaced only by a candidate that wins by 3 % (as is any
earlier candidate by a later one): re-timing does not swap near-equal tiles
on noise.
The choices become the table the library uses by default (no timing on a
server's first request of a batch size); the candidate timings are written
as a summary, the evidence for each choice.

Usage (repository root, on an MI355X):
  python -m paper_2003_01538_amd.make_tile_table [--summary profiles/conv_tile_choices.md]
Rebuild the library afterwards (python -m paper_2003_01538_amd.build).
"""
from __future__ import annotations

import argparse
import os
import re
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
TABLE = os.path.join(HERE, "csrc", "tile_table.inc")

# workload, ensemble max_batch, batch buckets timed
PLAN = [
    ("tiny2_fp32_b4", 4, (1, 2, 4)),
    ("resnet18x3_bf16_b32", 64, (1, 2, 4, 8, 16, 32, 64)),
    ("hetero_r18_r50_vgg11_bf16_b32", 32, (1, 2, 4, 8, 16, 32)),
    ("resnet50x5_bf16_b256", 256, (1, 2, 4, 8, 16, 32, 64, 128, 256)),
]
KEYS = ("bucket", "prec", "kh", "kw", "stride", "pad", "cin", "cout", "h", "w", "z", "proj_cin", "proj_stride")
CAND = re.compile(r"bucket (\d+) group (\d+) layer (\d+) M (\d+) N (\d+) K (\d+) Z (\d+) split (\d+) tile (\S+) us ([\d.]+)")


def parse_log(log):
    """The tuning log of one ensemble -> (its table entries, one per timed
    layer, as dicts over KEYS plus "tile"; the evidence rows).  A row covers
    the layers of one bucket that share the whole table key (stride,
    shortcut and all, not only the GEMM shape: a stride-2 3x3 layer and a
    stride-1 one can have equal M, N and K but different kernel families),
    with the chosen tile's time and the best other candidate's."""
    cands, choice, choices = {}, {}, []
    for line in log.splitlines():
        m = CAND.match(line)
        if m:
            bk, gi, li = int(m.group(1)), int(m.group(2)), int(m.group(3))
            cands.setdefault((bk, gi, li), []).append((m.group(9), float(m.group(10)), m.groups()[3:8]))
        elif line.startswith("choice "):
            f = line.split()
            kv = dict(zip(f[1::2], f[2::2]))
            c = {k: int(kv[k]) for k in KEYS}
            c["tile"] = kv["tile"]
            choices.append(c)
            choice[(c["bucket"], int(kv["group"]), int(kv["layer"]))] = c
    groups = {}  # repeated layers of a network are alike
    for (bk, gi, li), cs in sorted(cands.items()):
        if len(cs) < 2:
            continue  # a kernel family with one tile: nothing was chosen
        c = choice[(bk, gi, li)]
        pick = [x for x in cs if x[0] == c["tile"]][0]
        alt = min((x for x in cs if x[0] != pick[0]), key=lambda x: x[1])
        key = tuple(c[k] for k in KEYS) + tuple(cs[0][2])
        if key in groups:
            groups[key][1].append(li)
        else:
            groups[key] = (gi, [li], c, cs[0][2], pick, alt)
    rows = []
    for gi, lis, c, (M, N, K, Z, sp), pick, alt in groups.values():
        conv = f"{c['kh']}x{c['kw']}/{c['stride']}"
        if c["proj_cin"]:
            conv += f" + 1x1/{c['proj_stride']} shortcut"
        rows.append(f"| {c['bucket']} | {gi} | {','.join(map(str, lis))} | {conv} | {M} x {N} x {K} ({Z}, {sp}) | "
                    f"{pick[0].replace('bf16', '')} | {pick[1]:.1f} | {alt[0].replace('bf16', '')} | {alt[1]:.1f} |")
    return choices, rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--summary", default=os.path.join(ROOT, "profiles", "conv_tile_choices.md"))
    ap.add_argument("--table", default=TABLE)
    args = ap.parse_args()
    os.environ["FS_TUNE"] = "3"
    sys.path.insert(0, ROOT)
    import workloads as wl
    from paper_2003_01538_amd import flexserve as fsb

    entries, seen = [], set()
    summary = ["# Conv tile choices per batch bucket (MI355X, HIP-event timing of every candidate)", "",
               "Command: `python -m paper_2003_01538_amd.make_tile_table` (repository root, on an MI355X).", "",
               "Per bucket and distinct layer (conv form, shortcut and GEMM shape; alike layers of a network "
               "listed together; layers whose kernel family has a single tile omitted): the chosen tile and "
               "its time per launch, then the "
               "next-best candidate (a later candidate must win by 3 % to be chosen; the table's previous "
               "tile is timed first).", ""]
    for wname, max_batch, buckets in PLAN:
        w = wl.workload(wname)
        with fsb.Ensemble(w["models"], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, w["precision"],
                          max_batch=max_batch) as ens:
            for b in buckets:
                ens.infer(list(wl.images_uniform(w["image_seed"], b, *w["in_hw"])), want_logits=False)
                print(f"{wname}: bucket {b} timed", flush=True)
            log = fsb.fs_tuning_log(ens.handle)
        choices, rows = parse_log(log)
        summary += [f"## {wname} (max_batch {max_batch})", "",
                    "| bucket | group | layers | conv | M x N x K (Z, split) | chosen | us | next best | us |",
                    "|---|---|---|---|---|---|---|---|---|"]
        summary += rows
        summary.append("")
        for c in choices:
            key = tuple(c[k] for k in KEYS)
            if key not in seen:
                seen.add(key)
                entries.append(c)
    with open(args.table, "w") as f:
        f.write("// Conv tile per layer shape and batch bucket, chosen by timing every\n"
                "// candidate of the layer's kernel family on an MI355X (written by\n"
                "// paper_2003_01538_amd/make_tile_table.py; do not edit by hand).\n"
                "// bucket, precision, kh, kw, stride, pad, Cin, Cout, H, W, Z, projection Cin, projection stride, tile\n")
        for c in entries:
            f.write("    {" + ", ".join(str(c[k]) for k in KEYS) + f', "{c["tile"]}"' + "},\n")
    with open(args.summary, "w") as f:
        f.write("\n".join(summary) + "\n")
    print(f"{len(entries)} table entries -> {args.table}; evidence -> {args.summary}")


if __name__ == "__main__":
    main()
