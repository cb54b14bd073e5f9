"""The committed counter summaries describe the committed kernels.

Each `profiles/*_pmc.md` that bench.py reads for `roofline.traffic` carries a
machine-readable record with the sha256 of the kernel source it was taken
with; bench.py reports `traffic: null` once the source changes.  These CPU
checks keep that from happening silently: every record parses, names its
workload, matches the current source, and its calibrated traffic is within
a plausible band of the algorithmic bytes it records.
"""
import json
import os
import re

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _record(name):
    text = open(os.path.join(ROOT, "profiles", name)).read()
    m = re.search(r"<!-- traffic-json (\{.*?\}) -->", text, re.S)
    assert m, f"{name}: no traffic record"
    return text, json.loads(m.group(1))


@pytest.mark.parametrize("workload", sorted(bench.PMC_SUMMARIES))
def test_counter_record_matches_source(workload):
    name, src = bench.PMC_SUMMARIES[workload]
    text, rec = _record(name)
    assert rec["workload"] == workload
    assert rec["source_sha256"] == bench.source_sha256(workload), (
        f"{name} was taken with another version of {src}: re-take the counters")
    # the copy calibration: FETCH_SIZE counts half the bytes read, WRITE_SIZE all
    assert abs(rec["fetch_factor"] - 2.0) < 0.01 and abs(rec["write_factor"] - 1.0) < 0.01
    b, note = bench.measured_traffic(workload)
    assert b is not None, note
    ratio = b / rec["algorithmic_bytes_per_launch"]
    assert 0.95 <= ratio <= 1.10, f"{workload}: traffic / algorithmic = {ratio:.3f}"
    # every command in the summary runs committed files (bench.py) only
    for line in text.splitlines():
        if "rocprofv3" in line and "--" in line:
            assert "_work" not in line and "python3 $REPO/bench.py" in line, line
