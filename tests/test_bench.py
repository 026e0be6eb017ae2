"""The benchmark's contract on a host without the multi-GPU path or a GPU,
and its traffic records (counter-measured HBM bytes per launch, valid only
for the schedule and kernel source they were taken with)."""
import json
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=300)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_without_a_gpu_the_benchmark_fails_loudly():
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    r = _run("--steps", "1", "--warmup", "0")
    assert r.returncode == 1 and "needs a GPU" in r.stderr


def test_traffic_records_are_keyed_by_the_tuned_schedules():
    # Every workload has a counter record taken with its tuned schedule (a
    # kernel edit after the counters were taken makes the benchmark report
    # null traffic until they are re-taken; that is allowed, a stale schedule
    # key is not), and a record never answers for another schedule.
    import bench
    from paper_2506_01374_amd import workloads as W
    tuned = json.load(open(os.path.join(ROOT, "paper_2506_01374_amd", "tuned.json")))
    records = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    for name, text in tuned.items():
        op = W.workload_op(name)
        # (a knob added later takes its default in an older key)
        assert str(op.from_string(records[name]["key"])) == str(op.from_string(text)), name
        assert records[name]["bytes_per_launch"] > 0
        assert bench._load_traffic(name, op, op.default()) is None


def test_p0_speedup_records_answer_only_for_their_tuned_schedule():
    # Every workload has a P0 record taken with its tuned schedule; the
    # record never answers for another schedule or a missing workload.
    import bench
    from paper_2506_01374_amd import workloads as W
    tuned = json.load(open(os.path.join(ROOT, "paper_2506_01374_amd", "tuned.json")))
    for name, text in tuned.items():
        op = W.workload_op(name)
        rec = bench._p0_speedup(name, op, op.from_string(text))
        assert rec is not None and rec["value"] > 1.0, name
        assert min(rec["p0_us"]) > max(rec["tuned_us"]), name
        assert bench._p0_speedup(name, op, op.default()) is None
    assert bench._p0_speedup("no_such_workload", op, op.default()) is None
