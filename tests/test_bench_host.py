"""Host-side logic of bench.py: the HBM traffic record built from two counter
passes, and its invalidation when the kernel's sources change."""
import csv
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

FIELDS = ["Kernel_Name", "Counter_Name", "Counter_Value"]


def _csv(path, counter, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=FIELDS)
        w.writeheader()
        for name, v in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def test_record_traffic_calibrates_against_the_copy(tmp_path):
    kern = "void janus::index_scores_fp8_mfma<64, 2>(int const*)"
    copy = "__amd_rocclr_copyBuffer"
    # the 1 GiB copy reads 2^20 KiB but FETCH_SIZE shows half of it; small copies are ignored
    _csv(tmp_path / "f.csv", "FETCH_SIZE", [(copy, 12.0), (copy, 524288.0), (kern, 1000.0), (kern, 3000.0)])
    _csv(tmp_path / "w.csv", "WRITE_SIZE", [(copy, 4.0), (copy, 1048576.0), (kern, 500.0), (kern, 500.0)])
    out = tmp_path / "t.json"
    bench.record_traffic(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), str(out))
    rec = json.load(open(out))
    assert rec["fetch_scale"] == 2.0 and rec["write_scale"] == 1.0
    assert rec["bytes_per_launch"] == pytest.approx(2000.0 * 1024 * 2 + 500.0 * 1024)
    assert bench.measured_traffic(str(out)) == rec["bytes_per_launch"]
    rec["sources_sha256"] = "0" * 64
    json.dump(rec, open(out, "w"))
    assert bench.measured_traffic(str(out)) is None


def test_committed_traffic_record_matches_its_sources():
    """The committed record is either current (bytes) or reported as stale
    (None) - never an exception."""
    v = bench.measured_traffic(os.path.join(ROOT, "profiles", "index_scores_traffic.json"))
    assert v is None or v > 4.5e9  # at least the score matrix it writes
