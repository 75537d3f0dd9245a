"""Regenerate the committed conv tile table (csrc/tile_table.inc) on an MI355X.

For every benchmark workload and every batch bucket it serves, the ensemble
is built with FS_TUNE=1, so the first pass of each bucket times every
candidate tile of every conv layer's kernel family (HIP events, two launches
after a warm-up) and keeps the fastest (a later candidate must win by 3 %).
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--summary", default=os.path.join(ROOT, "profiles", "conv_tile_choices.md"))
    ap.add_argument("--table", default=TABLE)
    args = ap.parse_args()
    os.environ["FS_TUNE"] = "1"
    sys.path.insert(0, ROOT)
    import workloads as wl
    from paper_2003_01538_amd import flexserve as fsb

    entries, seen = [], set()
    summary = ["# Conv tile choices per batch bucket (MI355X, HIP-event timing of every candidate)", "",
               "Command: `python -m paper_2003_01538_amd.make_tile_table` (repository root, on an MI355X).", "",
               "Per distinct layer shape and bucket (layers of one shape listed together; layers whose "
               "kernel family has a single tile omitted): the chosen tile and its time per launch, then the "
               "next-best candidate (a later candidate must win by 3 % to be chosen).", ""]
    for wname, max_batch, buckets in PLAN:
        w = wl.workload(wname)
        with fsb.Ensemble(w["models"], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, w["precision"],
                          max_batch=max_batch) as ens:
            for b in buckets:
                ens.infer(list(wl.images_uniform(w["image_seed"], b, *w["in_hw"])), want_logits=False)
                print(f"{wname}: bucket {b} timed", flush=True)
            log = fsb.fs_tuning_log(ens.handle)
        cands = {}
        for line in log.splitlines():
            m = CAND.match(line)
            if m:
                bk, gi, li = int(m.group(1)), int(m.group(2)), int(m.group(3))
                cands.setdefault((bk, gi, li), []).append((m.group(9), float(m.group(10)), m.groups()[3:8]))
        choices, chosen = [], {}
        for l in log.splitlines():
            if l.startswith("choice "):
                f = l.split()
                kv = dict(zip(f[1::2], f[2::2]))
                c = {k: int(kv[k]) for k in KEYS}
                c["tile"] = kv["tile"]
                choices.append(c)
                chosen[(c["bucket"], int(kv["group"]), int(kv["layer"]))] = c["tile"]
        summary += [f"## {wname} (max_batch {max_batch})", "",
                    "| bucket | group | layers | M x N x K (Z, split) | chosen | us | next best | us |",
                    "|---|---|---|---|---|---|---|---|"]
        rows = {}  # one row per distinct (bucket, shape): repeated layers of a network are alike
        for (bk, gi, li), cs in sorted(cands.items()):
            if len(cs) < 2:
                continue  # a kernel family with one tile: nothing was chosen
            M, N, K, Z, sp = cs[0][2]
            pick = [c for c in cs if c[0] == chosen[(bk, gi, li)]][0]
            alt = sorted((c for c in cs if c[0] != pick[0]), key=lambda c: c[1])
            key = (bk, M, N, K, Z, sp)
            if key in rows:
                rows[key][1].append(li)
                continue
            rows[key] = (gi, [li], pick, alt[0])
        for (bk, M, N, K, Z, sp), (gi, lis, pick, alt) in rows.items():
            summary.append(f"| {bk} | {gi} | {','.join(map(str, lis))} | {M} x {N} x {K} ({Z}, {sp}) | "
                           f"{pick[0].replace('bf16', '')} | {pick[1]:.1f} | {alt[0].replace('bf16', '')} | "
                           f"{alt[1]:.1f} |")
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
