"""bench.py's host-side logic (CPU): the one-GPU guard, the HBM-traffic record
built from counter runs, and the hash that ties a record to the code it was
measured on."""

from __future__ import annotations

import argparse
import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _counter_csv(path, counter, attn_kib, copy_kib):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value"])
        w.writeheader()
        d = 0
        for v in attn_kib:
            d += 1
            w.writerow({"Dispatch_Id": d, "Kernel_Name": "void tts::attn_kernel<128, 1, false>(tts::AttnParams)",
                        "Grid_Size": 65536, "Counter_Name": counter, "Counter_Value": v})
            d += 1  # the merge, not counted
            w.writerow({"Dispatch_Id": d, "Kernel_Name": "void tts::merge_row_kernel<128, true>(tts::MergeParams)",
                        "Grid_Size": 114688, "Counter_Name": counter, "Counter_Value": 999.0})
        for v in copy_kib:
            d += 1
            w.writerow({"Dispatch_Id": d, "Kernel_Name": "void at::native::bitwise_not_kernel(...)",
                        "Grid_Size": 268435456, "Counter_Name": counter, "Counter_Value": v})


def test_traffic_record_scales_by_the_copy(tmp_path, monkeypatch):
    """FETCH_SIZE reading half of a 256 MiB copy (factor 2) and WRITE_SIZE all of it (factor 1): an attention
    launch reading 1000 and 3000 KiB (mean 2000 -> 4000 KiB) and writing 500 KiB moves 4500 KiB."""
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    fetch, write = tmp_path / "fetch.csv", tmp_path / "write.csv"
    _counter_csv(fetch, "FETCH_SIZE", [1000.0, 3000.0], [131072.0, 131072.0])
    _counter_csv(write, "WRITE_SIZE", [500.0, 500.0], [262144.0])
    args = argparse.Namespace(copy_mib=256, ingest_traffic=[str(fetch), str(write)], config="7b64", variant="prefix")
    bench.ingest_traffic(args)
    rec = json.load(open(tmp_path / "traffic.json"))
    assert rec["kernel_sha"] == bench.kernel_sha()
    ent = rec["entries"]["7b64:prefix"]
    assert ent["fetch_size"]["factor"] == pytest.approx(2.0) and ent["write_size"]["factor"] == pytest.approx(1.0)
    assert ent["fetch_size"]["attn_dispatches"] == 2
    assert ent["bytes_per_launch"] == pytest.approx(4500.0 * 1024)
    # a second workload joins the same record; the first stays
    _counter_csv(fetch, "FETCH_SIZE", [10.0], [131072.0])
    bench.ingest_traffic(argparse.Namespace(copy_mib=256, ingest_traffic=[str(fetch), str(write)], config="tiny",
                                            variant="prefix"))
    rec = json.load(open(tmp_path / "traffic.json"))
    assert set(rec["entries"]) == {"7b64:prefix", "tiny:prefix"}


def test_traffic_record_needs_the_copy_size(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    with pytest.raises(SystemExit):
        bench.ingest_traffic(argparse.Namespace(copy_mib=0, ingest_traffic=["a", "b"], config="7b64",
                                                variant="prefix"))


def test_kernel_hash_covers_kernel_planner_and_flags(tmp_path, monkeypatch):
    base = bench.kernel_sha()
    for attr in ("KERNEL_SRC", "PLANNER_SRC"):
        src = getattr(bench, attr)
        copy = tmp_path / os.path.basename(src)
        copy.write_bytes(open(src, "rb").read() + b"\n")
        monkeypatch.setattr(bench, attr, str(copy))
        assert bench.kernel_sha() != base
        monkeypatch.setattr(bench, attr, src)
    assert bench.kernel_sha() == base
    import paper_2509_00195_amd.build as b

    monkeypatch.setattr(b, "DEVICE", [*b.DEVICE, "-O2"])
    assert bench.kernel_sha() != base
