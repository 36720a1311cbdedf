"""Host-side helpers of bench.py (no GPU): the committed counter summary feeds
the traffic fields only of the workload it was measured on, its dedup phase
only for the dedup it was measured with, and only while the kernel sources it
names are unchanged."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402


def _workload_line(name):
    w = synth.workload(name)
    return f"{w.name}: {w.description}"


def test_counter_traffic_only_for_the_measured_workload():
    c3 = bench.counter_traffic(_workload_line("c3"), "emb_unique_ids")
    assert set(c3) == set(bench.PHASE_SOURCES)
    for name in ("c1", "c2", "c4", "c5"):
        other = bench.counter_traffic(_workload_line(name), "emb_unique_ids")
        assert other == {phase: None for phase in bench.PHASE_SOURCES}, name


def test_counter_traffic_follows_the_source_hashes(tmp_path, monkeypatch):
    wl = _workload_line("c3")
    src = tmp_path / "k.hip"
    src.write_text("kernel source\n")
    counters = tmp_path / "counters.txt"
    counters.write_text(f"Workload: {wl}\nDedup: emb_unique_ids_batched, groups of 4\n\nhbm_bytes_fwd = 123\n"
                        f"hbm_bytes_dedup = 45\nsha_k.hip = {bench.file_sha(str(src))}\n")
    monkeypatch.setattr(bench, "COUNTERS", str(counters))
    monkeypatch.setattr(bench, "PHASE_SOURCES", {"fwd": [str(src)], "dedup": [str(src)]})
    assert bench.counter_traffic(wl, "emb_unique_ids_batched, groups of 4") == {"fwd": 123.0, "dedup": 45.0}
    # the dedup phase only for the dedup the counters were taken with
    assert bench.counter_traffic(wl, "emb_unique_ids_batched, groups of 8") == {"fwd": 123.0, "dedup": None}
    assert bench.counter_traffic(wl, "emb_unique_ids") == {"fwd": 123.0, "dedup": None}
    src.write_text("kernel source, changed\n")
    assert bench.counter_traffic(wl, "emb_unique_ids_batched, groups of 4") == {"fwd": None, "dedup": None}
