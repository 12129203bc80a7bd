"""The committed rocprofv3 summaries under profiles/ against the current sources
(host only): the HBM counters that bench.py reports as `roofline.traffic` must
have been taken on the decode kernel as it is now, and must describe traffic
close to the workload's algorithmic bytes (no tile read twice)."""
import glob
import json
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COUNTERS = sorted(glob.glob(os.path.join(ROOT, "profiles", "counters__decode_mfma_fused__*.md")))


def _record(path):
    m = re.search(r"TRAFFIC_JSON:\s*(\{.*\})", open(path).read())
    assert m, f"{path} has no TRAFFIC_JSON line"
    return json.loads(m.group(1))


def test_counter_summaries_exist_for_the_headline_workload():
    names = [os.path.basename(p) for p in COUNTERS]
    assert "counters__decode_mfma_fused__llama3.1-70b_b512_u256-4096.md" in names


@pytest.mark.parametrize("path", COUNTERS, ids=[os.path.basename(p) for p in COUNTERS])
def test_counters_were_taken_on_the_current_kernel(path):
    import bench
    rec = _record(path)
    assert rec["kernel_sha"] == bench.kernel_source_sha("mfma_fused"), (
        f"{os.path.basename(path)} was taken on other decode kernel sources; "
        "re-take the FETCH_SIZE / WRITE_SIZE runs")


@pytest.mark.parametrize("path", COUNTERS, ids=[os.path.basename(p) for p in COUNTERS])
def test_counted_traffic_is_close_to_the_algorithmic_bytes(path):
    rec = _record(path)
    ratio = rec["traffic_bytes_per_launch"] / rec["algorithmic_bytes_per_launch"]
    reads = rec["fetch_kib_per_launch"] * 1024 * rec["copy_factor_fetch"]
    assert 0.99 <= ratio <= 1.05, ratio
    assert reads <= 1.02 * rec["algorithmic_bytes_per_launch"]


TRACES = sorted(glob.glob(os.path.join(ROOT, "profiles", "decode_mfma_fused__*__kernel_trace.md")))


@pytest.mark.parametrize("path", TRACES, ids=[os.path.basename(p) for p in TRACES])
def test_trace_mean_agrees_with_the_bench_figure_of_the_same_run(path):
    # The decode kernel's mean duration over the timed region in rocprofv3's
    # kernel trace against bench.py's own event-timed kernel_ms of that run.
    text = open(path).read()
    bench_us = float(re.search(r"`roofline\.kernel_ms` =\s*([0-9.]+) us", text).group(1))
    trace_us = float(re.search(r"From the trace: [0-9.]+ MB / ([0-9.]+) us", text).group(1))
    assert abs(trace_us - bench_us) <= 0.015 * bench_us, (trace_us, bench_us)
    assert "rocprofv3 --kernel-trace --stats" in text
