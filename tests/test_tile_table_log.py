"""Host logic of the tile-table tool: parsing the runtime's tuning log into
table entries and evidence rows."""
from paper_2003_01538_amd.make_tile_table import KEYS, parse_log


def choice(layer, stride, cin, h, tile, proj_cin=0, proj_stride=0):
    return (f"choice bucket 32 group 0 layer {layer} prec 1 kh 3 kw 3 stride {stride} pad 1 cin {cin} "
            f"cout 128 h {h} w {h} z 5 proj_cin {proj_cin} proj_stride {proj_stride} tile {tile}")


def cand(layer, tile, us, k=1152):
    return f"bucket 32 group 0 layer {layer} M 25088 N 128 K {k} Z 5 split 1 tile {tile} us {us}"


# a stride-2 3x3 layer (56 -> 28) and stride-1 ones (28 -> 28) with equal
# M, N and K but different kernel families; a layer with a shortcut; a
# layer whose family has one tile
LOG = "\n".join([
    cand(13, "bf16dma2_128x128_w4_v8", 47.8), cand(13, "bf16dma2_96x128_w4m1_v8", 50.7),
    choice(13, 2, 128, 56, "bf16dma2_128x128_w4_v8"),
    cand(17, "bf16hs_128x128_w4_v8", 30.1), cand(17, "bf16hr_96x128_w4m1_v8", 31.0),
    choice(17, 1, 128, 28, "bf16hs_128x128_w4_v8"),
    cand(20, "bf16hs_128x128_w4_v8", 30.3), cand(20, "bf16hr_96x128_w4m1_v8", 30.9),
    choice(20, 1, 128, 28, "bf16hs_128x128_w4_v8"),
    cand(8, "bf16hr_160x128_w4m1_v8", 29.9, 1216), cand(8, "bf16hr_96x128_w4m1_v8", 35.1, 1216),
    choice(8, 1, 128, 28, "bf16hr_160x128_w4m1_v8", 64, 2),
    cand(2, "bf16halo_4x56_n64_v8", 30.0),
    choice(2, 1, 64, 56, "bf16halo_4x56_n64_v8"),
])


def test_layers_of_equal_gemm_shape_but_other_stride_get_their_own_row():
    choices, rows = parse_log(LOG)
    assert len(choices) == 5 and all(set(KEYS) <= set(c) for c in choices)
    assert [c["tile"] for c in choices if c["stride"] == 2] == ["bf16dma2_128x128_w4_v8"]
    by_layers = {r.split("|")[3].strip(): r for r in rows}
    assert set(by_layers) == {"13", "17,20", "8"}  # layer 2: one candidate, no row
    assert "| 3x3/2 |" in by_layers["13"] and "| dma2_128x128_w4_v8 | 47.8 | dma2_96x128_w4m1_v8 | 50.7 |" in by_layers["13"]
    assert "| 3x3/1 |" in by_layers["17,20"] and "| hs_128x128_w4_v8 | 30.1 | hr_96x128_w4m1_v8 | 31.0 |" in by_layers["17,20"]
    assert "| 3x3/1 + 1x1/2 shortcut |" in by_layers["8"] and "25088 x 128 x 1216 (5, 1)" in by_layers["8"]
