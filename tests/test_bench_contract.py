"""Host-side parts of bench.py: the one-GPU guard and the lookup of the
measured HBM traffic (per workload, mode and kernel source)."""
import glob
import hashlib
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

TRAFFIC_FILES = sorted(glob.glob(os.path.join(ROOT, "profiles", "attention_*_hbm_traffic.json")))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_no_traffic_for_an_unprofiled_workload_or_mode():
    assert bench.measured_traffic("cross_ragged", "uos_pnq") is None
    assert bench.measured_traffic("video720p", "ocp_vanilla") is None


@pytest.mark.parametrize("path", TRAFFIC_FILES, ids=os.path.basename)
def test_traffic_record(path):
    with open(path) as f:
        rec = json.load(f)
    name = os.path.basename(path)[len("attention_"):-len("_hbm_traffic.json")]
    assert rec["workload_name"] == name
    cal = rec["copy_calibration"]
    # both counters scaled by what they read for the 1 GiB copy
    assert cal["fetch_factor"] == pytest.approx(1048576 / cal["fetch_size_kib"])
    assert cal["write_factor"] == pytest.approx(1048576 / cal["write_size_kib"])
    total = (rec["fetch_size_kib_per_launch"] * cal["fetch_factor"]
             + rec["write_size_kib_per_launch"] * cal["write_factor"]) * 1024
    assert rec["hbm_bytes_per_launch"] == pytest.approx(total)
    # reported only while the kernel source is the one the counters were taken on
    with open(bench.KERNEL_SOURCE, "rb") as f:
        current = hashlib.sha256(f.read()).hexdigest() == rec["kernel_source_sha256"]
    got = bench.measured_traffic(name, rec["mode"])
    assert got == (rec["hbm_bytes_per_launch"] if current else None)


def test_stratified_oracle_sample_covers_every_head_and_the_edges():
    """The bounded oracle sample of `bench.py --cpu-table`: every head gets
    its share, the first and the ragged last query tile and the sequence's
    end are in every head's rows, and each text row is in exactly one head."""
    N, heads, text = 3001, 5, 40
    rows = bench.stratified_rows(N, heads, 52, seed=3, text_tokens=text)
    assert sorted(rows) == list(range(heads))
    last = (N - 1) // 128 * 128
    for h, r in rows.items():
        assert r.size == 52 and r.dtype.kind == "i"
        assert len(set(r.tolist())) == r.size and r.min() >= 0 and r.max() < N
        assert {0, 1, 63, 127, last, last + 1, N - 2, N - 1} <= set(r.tolist())
    text_rows = [x for r in rows.values() for x in r.tolist() if x >= N - text]
    fixed = {N - 2, N - 1}  # in every head's rows anyway
    assert sorted(set(text_rows) - fixed) == sorted(set(range(N - text, N)) - fixed)
    # a sequence shorter than the sample takes every row
    assert bench.stratified_rows(100, 2, 300, seed=1)[1].tolist() == list(range(100))
