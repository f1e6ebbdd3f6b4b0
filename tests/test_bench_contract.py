"""The benchmark's command-line contract: one JSON line with the required fields.

The host test checks the refusal of more than one GPU (it exits before touching a
device); the GPU test runs a short benchmark and checks the line's fields and their
consistency.
"""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args, timeout=300):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT, capture_output=True,
                          text=True, timeout=timeout)


def test_more_than_one_gpu_is_refused():
    r = _bench("--gpus", "2", timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


@pytest.mark.gpu
def test_short_run_prints_one_complete_json_line():
    r = _bench("--steps", "3", "--warmup", "1", "--no-cpu-baseline", "--no-configs")
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
                "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1
    assert d["higher_is_better"] is True and d["value"] > 0 and d["ms_per_step"] > 0
    assert "workload" in d["config"]
    rf = d["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in rf, key
    assert rf["bound"] in ("hbm", "mfma", "alu") and rf["peak"] > 0
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    # value is the whole step's bytes over its time
    assert abs(d["value"] - d["config"]["bytes_per_step"] / (d["ms_per_step"] * 1e6)) / d["value"] < 0.01
    assert d["aux_bytes"] == 0
    # the reference rates beside the roofline: a device copy and an in-place pass over 1 GiB
    for ref in ("hbm_copy", "hbm_inplace"):
        assert d[ref]["GB_s"] > 0, ref


def test_cpu_baseline_reports_all_cores_and_one():
    """The oracle baseline on a tiny sample: an all-core figure with its worker count, and a
    one-core figure beside it."""
    sys.path.insert(0, ROOT)
    import bench
    from paper_2511_01385_amd import inputs

    ns = [64, 128]
    rows = {n: inputs.normal_rows(inputs.seed_for(2, salt=n), 32, n, "bf16") for n in ns}
    lay = dict(tokens=8, d=256, p=64, sigma=0.02)
    xcg = inputs.bca_problem(inputs.seed_for(4), 8, 256, 256, 64, 0.02, "bf16")
    r = bench.cpu_baseline(rows, xcg, ns=ns, bca=lay, min_seconds=0.05, max_workers=2)
    assert r["kind"] == "oracle" and r["unit"] == "GB/s" and r["value"] > 0
    assert 1 <= r["cores"] <= 2 and r["cores"] <= len(os.sched_getaffinity(0))
    assert r["single_core"]["cores"] == 1 and r["single_core"]["value"] > 0
    assert "sample" in r and "sample" in r["single_core"]
