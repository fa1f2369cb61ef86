"""The parts of bench.py's contract that need no GPU: the one-GPU guard, the oracle baseline
record, and the rule that a measured HBM traffic figure is reported only for the kernel source it
was measured on."""

import importlib.util
import json
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("n", [2, 8])
def test_more_than_one_gpu_is_refused(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert f"--gpus {n}" in r.stderr and r.stdout == ""


def test_cpu_baseline_record():
    """The oracle timed on a few query rows of a small workload: the record bench.py prints."""
    bench = _bench()
    from paper_2507_16697_amd import inputs

    w = inputs.WORKLOADS["shard_n16k_d64"]
    t = inputs.make_iid(1, 1, 4, w.Nk, w.d, seed=5, std=0.5, store="bf16", with_do=True)
    rec = bench.cpu_baseline(t, w, rows=4)
    assert rec["kind"] == "oracle" and rec["unit"] == "TFLOP/s"
    assert rec["value"] > 0 and rec["seconds"] > 0
    assert rec["cores"] == len(os.sched_getaffinity(0)) and 1 <= rec["blas_threads"]
    assert "queries 0..3" in rec["sample"] and str(w.Nk) in rec["sample"]
    # the same flop convention as the GPU figure: 12 * rows * Nk * d
    assert rec["value"] == pytest.approx(12.0 * 4 * w.Nk * w.d / rec["seconds"] / 1e12)
    # the whole step, extrapolated from the sample: every row of every head costs the same
    assert rec["step_seconds_extrapolated"] == pytest.approx(rec["seconds"] * w.H * w.Nq / 4)
    other = rec["other_configs"]
    c1 = other["exact_fp32_n1k"]
    assert c1["seconds"] > 0 and c1["seconds_1_core"] > 0 and c1["pass"] == "fwd"
    c2 = other["shard_n16k_d64"]
    assert c2["seconds_extrapolated"] == pytest.approx(16 * c2["seconds_head0"])


def test_input_hashes_identify_the_inputs():
    bench = _bench()
    from paper_2507_16697_amd import inputs

    t = inputs.make_iid(1, 2, 8, 16, 64, seed=9, store="bf16")
    a = bench.input_sha256(t)
    b = bench.input_sha256(inputs.make_iid(1, 2, 8, 16, 64, seed=9, store="bf16"))
    c = bench.input_sha256(inputs.make_iid(1, 2, 8, 16, 64, seed=10, store="bf16"))
    assert set(a) == {"q", "k", "v", "do"} and a == b
    assert all(a[n] != c[n] for n in a) and all(len(x) == 64 for x in a.values())


def test_traffic_is_reported_only_for_its_source():
    bench = _bench()
    path = os.path.join(ROOT, "profiles")
    recs = [f for f in os.listdir(path) if f.startswith("traffic_") and f.endswith(".json")]
    assert recs, "no measured traffic records"
    for f in recs:
        with open(os.path.join(path, f)) as fh:
            rec = json.load(fh)
        assert rec["bytes_per_launch"] > 0 and rec["commands"]
        # the calibrated counters add up to the reported bytes
        got = rec["fetch_size_kib"] * 1024 * rec["fetch_factor"] + \
            rec["write_size_kib"] * 1024 * rec["write_factor"]
        assert got == pytest.approx(rec["bytes_per_launch"], rel=1e-9)
        assert bench.load_traffic(rec["kernel"], rec["workload"], rec["source_hash"]) == \
            rec["bytes_per_launch"]
        assert bench.load_traffic(rec["kernel"], rec["workload"], "0" * 16) is None
    assert bench.load_traffic("no_such_kernel", "ring8_nk262k_d128", "0" * 16) is None


def test_source_hash_tracks_the_kernel_text():
    bench = _bench()
    a = bench.kernel_source_hash(["merge.hip", "ringx_device.h"])
    b = bench.kernel_source_hash(["merge.hip", "ringx_device.h"])
    c = bench.kernel_source_hash(["merge.hip"])
    assert a == b and a != c and len(a) == 16 and int(a, 16) >= 0
    assert np.isfinite(bench.PEAK_BF16_TFLOPS) and bench.PEAK_HBM_GBS == 8000.0
