"""The committed conv tile table covers every conv layer of the benchmark
workloads at every batch bucket they serve: with the default tile choice (the
table, timing only what it lacks) a pass at each bucket times nothing, so no
request waits for tile tuning, and every table entry names a tile that is a
candidate of its layer's kernel family (an entry that is not would fall back
to timing and show up here)."""
import re

import pytest

import workloads as wl
from paper_2003_01538_amd import flexserve as fsb
from paper_2003_01538_amd.make_tile_table import KEYS, PLAN, TABLE

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("wname,max_batch,buckets", PLAN, ids=[p[0] for p in PLAN])
def test_table_covers_every_bucket(monkeypatch, wname, max_batch, buckets):
    monkeypatch.setenv("FS_TUNE", "2")  # the default: the table, timing what it lacks
    w = wl.workload(wname)
    with fsb.Ensemble(w["models"], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, w["precision"],
                      max_batch=max_batch) as ens:
        for b in buckets:
            print(f"{wname}: bucket {b}", flush=True)
            ens.infer(list(wl.images_uniform(w["image_seed"], b, *w["in_hw"])), want_logits=False)
        log = fsb.fs_tuning_log(ens.handle)
    assert log == "", f"{wname}: layers without a usable table entry:\n{log[:2000]}"


def test_the_log_records_timing(monkeypatch):
    # the control: with every layer timed (FS_TUNE=1) the same pass fills the
    # log, so an empty log above means nothing was timed
    monkeypatch.setenv("FS_TUNE", "1")
    wname, max_batch, buckets = PLAN[1]
    w = wl.workload(wname)
    with fsb.Ensemble(w["models"], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, w["precision"],
                      max_batch=max_batch) as ens:
        ens.infer(list(wl.images_uniform(w["image_seed"], buckets[0], *w["in_hw"])), want_logits=False)
        log = fsb.fs_tuning_log(ens.handle)
    assert "choice bucket" in log


def test_retiming_times_the_table_tile_first(monkeypatch):
    # FS_TUNE=3 (how the table is re-timed): every layer is timed, and the
    # table's tile comes first, so another candidate must beat it by the
    # tuner's margin to replace it
    entries = {}
    for m in re.finditer(r'\{(\d+(?:, \d+){12}), "([^"]+)"\}', open(TABLE).read()):
        entries[tuple(int(x) for x in m.group(1).split(", "))] = m.group(2)
    monkeypatch.setenv("FS_TUNE", "3")
    wname, max_batch, buckets = PLAN[1]
    w = wl.workload(wname)
    with fsb.Ensemble(w["models"], w["out_hw"], wl.IMAGENET_MEAN, wl.IMAGENET_STD, w["precision"],
                      max_batch=max_batch) as ens:
        ens.infer(list(wl.images_uniform(w["image_seed"], 32, *w["in_hw"])), want_logits=False)
        log = fsb.fs_tuning_log(ens.handle)
    first, checked = {}, 0
    for line in log.splitlines():
        f = line.split()
        if line.startswith("bucket "):
            first.setdefault((f[3], f[5]), f[f.index("tile") + 1])
        elif line.startswith("choice "):
            kv = dict(zip(f[1::2], f[2::2]))
            key = tuple(int(kv[k]) for k in KEYS)
            if key in entries and (kv["group"], kv["layer"]) in first:
                assert first[(kv["group"], kv["layer"])] == entries[key], line
                checked += 1
    assert checked >= 10

