"""Host logic of bench.py: the HBM traffic it reports comes from the committed
rocprofv3 counter summary only while that summary was taken on the current
conv kernel sources."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_profile_counts_the_current_conv_sources():
    # the committed counters belong to the committed kernels; after a kernel
    # change the summary is re-taken (otherwise bench reports traffic: null)
    t = bench.counted_traffic()
    assert t is not None and t > 0


def test_traffic_is_withheld_when_the_sources_changed(monkeypatch):
    monkeypatch.setattr(bench, "conv_source_hash", lambda: "0" * 16)
    assert bench.counted_traffic() is None


def test_traffic_is_withheld_without_a_summary(monkeypatch, tmp_path):
    monkeypatch.setattr(bench, "PROFILE", str(tmp_path / "missing.md"))
    assert bench.counted_traffic() is None
