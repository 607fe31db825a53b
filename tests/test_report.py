"""The result tables of README.md are generated from the committed run records
(paper_2608_15473_amd.report): a table that no longer matches its records fails here, and every
record carries the environment it was measured in and numbers consistent with each other."""

import glob
import json
import os

import pytest

from paper_2608_15473_amd import report

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_tables_match_the_run_records():
    assert report.main(["--check"]) == 0, "run: python -m paper_2608_15473_amd.report"


def _runs():
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "bench_*.json"))):
        with open(path) as f:
            rec = json.load(f)
        for r in rec["runs"]:
            yield os.path.basename(path), rec["workload"], r


@pytest.mark.parametrize("fname,workload,run", list(_runs()))
def test_records_are_complete_and_consistent(fname, workload, run):
    assert fname == f"bench_{workload}.json"
    assert run["config"]["workload"] == workload
    env = run["env"]
    for key in ("source_sha256", "rocm", "hip", "torch", "gpu", "cpu_model", "host_cores"):
        assert env.get(key), key
    if "kernels" in run:        # a decode-stage record: tokens/s, speedup and hidden share
        fused, serial = run["fused_ms_per_step"], run["serial_ms_per_step"]
        tps = run["config"]["batch"] / (fused / 1e3)
        assert abs(tps - run["value"]) <= tps * (1e-3 + 0.5e-4 / fused)
        assert abs(serial / fused - run["speedup_vs_serial"]) <= 2e-3 * serial / fused
        hidden = (serial - fused) / run["sweep_only_ms_per_step"]
        assert abs(hidden - run["sweep_hidden_frac"]) <= 2e-3
        roof = run["roofline"]
        assert roof["kernel"] in run["kernels"]
        assert abs(roof["achieved"] / roof["peak"] - roof["frac"]) <= 1e-3
        return
    # value = KV bytes per step / step time; the roofline fraction = achieved / peak
    ms = run["ms_per_step"]
    v = run["config"]["kv_bytes_per_step"] / (ms / 1e3) / 1e9
    assert abs(v - run["value"]) <= v * (1e-3 + 0.5e-4 / ms)     # ms printed to 4 decimals
    roof = run["roofline"]
    assert abs(roof["achieved"] / roof["peak"] - roof["frac"]) <= 1e-3
    ach = roof["algorithmic_bytes"] / (roof["launch_avg_us"] / 1e6) / 1e9
    assert abs(ach - roof["achieved"]) <= 2e-3 * ach
    if "cpu_baseline" in run:
        cb = run["cpu_baseline"]
        assert cb["kind"] == "oracle" and cb["cores"] >= 1 and cb.get("cpu_model")
