"""Host logic of the tile-counter summary: dispatches of a kernel trace and of
a counter run are mapped back to the (shape, bucket, tile) cases in launch
order, split-K completions are folded into their conv dispatch, counter
instances are summed, and the table's choice is marked."""
import csv

from paper_2003_01538_amd import tile_counters as tc

SHAPE = (14, 14, 256, 256, 3, 1, 1, 1, 0, 0, (14,))
CASES = [dict(workload="w", B=2, Z=3, shape=SHAPE, tile="bf16dma2_64x128_w4_v8"),
         dict(workload="w", B=2, Z=3, shape=SHAPE, tile="bf16dma2_96x128_w4m1_v8")]


def _write(path, fields, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        w.writerows(rows)


def test_summary_maps_dispatches_to_cases(tmp_path, monkeypatch):
    monkeypatch.setattr(tc, "cases", lambda: CASES)
    monkeypatch.setattr(tc, "read_table", lambda path=None: [dict(
        bucket=2, prec=1, kh=3, kw=3, stride=1, pad=1, cin=256, cout=256, h=14, w=14, z=3, proj_cin=0,
        proj_stride=0, tile="bf16dma2_96x128_w4m1_v8")])
    trace, pmc = [], []
    did, t = 0, 0
    per = tc.WARMUP + tc.ITERS
    for ci, (name, us) in enumerate([("k_conv_dma<64, 128, 2, 2, 2, false>", 10.0),
                                     ("k_conv_dma<96, 128, 1, 4, 2, false>", 7.0)]):
        did += 1  # a fill kernel between the cases
        trace.append(dict(Dispatch_Id=did, Kernel_Name="__amd_rocclr_fillBufferAligned", Start_Timestamp=t,
                          End_Timestamp=t + 500))
        for i in range(per):
            did += 1
            dur = 99.0 if i < tc.WARMUP else us  # the untimed launches must not count
            trace.append(dict(Dispatch_Id=did, Kernel_Name=name, Start_Timestamp=t, End_Timestamp=t + int(dur * 1e3)))
            for half in (0, 1):  # two counter instances of each counter, summed
                pmc += [dict(Dispatch_Id=did, Kernel_Name=name, Counter_Name="SQ_VALU_MFMA_BUSY_CYCLES",
                             Counter_Value=1024 * 100 * (ci + 1) / 2),
                        dict(Dispatch_Id=did, Kernel_Name=name, Counter_Name="GRBM_GUI_ACTIVE",
                             Counter_Value=8 * 1000 / 2),
                        dict(Dispatch_Id=did, Kernel_Name=name, Counter_Name="SQ_INSTS_MFMA", Counter_Value=1)]
            if ci == 1:  # a split-K completion after each conv of the second case
                did += 1
                trace.append(dict(Dispatch_Id=did, Kernel_Name="k_conv_splitk_reduce", Start_Timestamp=t,
                                  End_Timestamp=t + 2000))
                pmc.append(dict(Dispatch_Id=did, Kernel_Name="k_conv_splitk_reduce", Counter_Name="GRBM_GUI_ACTIVE",
                                Counter_Value=8))
            t += 100000
    _write(tmp_path / "t.csv", ["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"], trace)
    _write(tmp_path / "p.csv", ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], pmc)
    out = tmp_path / "s.md"
    tc.summarize(str(tmp_path / "t.csv"), str(tmp_path / "p.csv"), str(out), ["cmd"])
    text = out.read_text()
    rows = {l.split("|")[1].strip(): l.split("|") for l in text.splitlines() if l.startswith("| bf16")}
    r64 = rows["bf16dma2_64x128_w4_v8"]
    r96 = rows["bf16dma2_96x128_w4m1_v8 (fastest)"]
    assert r64[2].strip() == "10.0"  # the untimed launches do not count
    assert r96[2].strip() == "9.0"   # 7 us conv + its 2 us split-K completion
    assert r64[5].strip() == "0.100" and r96[5].strip() == "0.200"  # busy / (gui / 8 x 1024)
    assert r96[6].strip() == "*" and r64[6].strip() == ""
    assert "within 5 % of the fastest standalone candidate: 1 of 1" in text


def test_dispatch_count_mismatch_is_an_error(tmp_path, monkeypatch):
    monkeypatch.setattr(tc, "cases", lambda: CASES)
    rows = [dict(Dispatch_Id=i, Kernel_Name="k_conv_dma<64>", Start_Timestamp=0, End_Timestamp=1) for i in range(5)]
    try:
        tc.assign(CASES, tc.conv_dispatches(rows))
    except SystemExit as e:
        assert "conv dispatches" in str(e)
    else:
        raise AssertionError("a short trace must not map")
