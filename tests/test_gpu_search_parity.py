"""GPU parity for the schedules the search emits.

Every transformation is semantics-preserving (Sec. 2), so any schedule the
search can reach must match the oracle.  Two sources of such schedules:
seeded random legal transformation sequences of length 12 from P0 (the
rollouts of Sec. 3.2), 40 per operator at the small shapes, whole outputs
compared; and the best schedule of a short seeded UCT search per operator,
measured on the GPU with the timing call, then compared with the oracle.
The campaign evaluator's timing conditions (cold, warm, back-to-back
through input copies) are run on a real plan per operator, and the output
they leave is compared with the oracle too.
"""
import os

import numpy as np
import pytest

from paper_2506_01374_amd import rc
from paper_2506_01374_amd import workloads as W

import cases
from test_gpu_parity import assert_parity, run

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rc.set_cache_dir(os.path.join(ROOT, "paper_2506_01374_amd", "jit_cache"))
    torch.cuda.set_device(0)


def _walk_params():
    out = []
    for key in cases.WALK_KEYS:
        for i, s in enumerate(cases.random_walks(key)):
            out.append(pytest.param(key, s, id=f"{key}-walk{i}"))
    return out


@pytest.mark.parametrize("key,sched_text", _walk_params())
def test_random_walk_schedule(key, sched_text):
    op = cases.small_op(key)
    sched = op.from_string(sched_text)
    assert sched.validate() == ""
    host = W.host_inputs(op, seed=8)
    try:
        y, _ = run(op, sched, host)
    except rc.RCError as e:
        # a variant the compiler rejects (register spill) is no program
        assert e.status == rc.RC_ERR_ILLEGAL_SCHEDULE and "spill" in str(e), str(e)
        pytest.skip(f"rejected at compile time: {e}")
    assert_parity(op, y, host, label=f"{key} walk {sched_text}")


@pytest.mark.parametrize("key", cases.WALK_KEYS)
def test_short_uct_search_best_matches_oracle(key):
    from paper_2506_01374_amd import tune
    op = cases.small_op(key)
    ev = tune.GpuEvaluator(op, repeat=3, warmup=1)
    res = tune.run_search(op, ev, "uct", budget=6, seed=3)
    assert res["valid"] >= 1 and res["best"] is not None
    # every measured schedule, and the best one again after its timing
    for text, rec in ev.cache.items():
        if not rec.get("valid"):
            continue
        sched = op.from_string(text)
        host = W.host_inputs(op, seed=0)
        plan = rc.Plan(op, sched)
        dev = W.to_device(W.stored_inputs(op, sched, host))
        out = W.empty_output(op)
        ws = plan.workspace()
        plan.time(dev, out, ws, warmup=1, repeat=2, flush=True)
        torch.cuda.synchronize()
        assert_parity(op, W.output_to_f64(op, out), host, label=f"{key} searched {text}")


@pytest.mark.parametrize("key", cases.WALK_KEYS)
@pytest.mark.parametrize("mode", ["cold", "warm", "rotated"])
def test_campaign_timing_modes_time_a_real_plan_and_leave_its_output(key, mode):
    """The campaign evaluator's three timing conditions (cache flushed before
    each launch, warm, back-to-back steps through three input copies) time
    a real plan, and the output buffer then holds the oracle's result."""
    from paper_2506_01374_amd import tune
    op = cases.small_op(key)
    sched = op.default()
    print(f"[gpu] campaign timing {mode} kind={op.kind} dims={op.dims} sched={sched}", flush=True)
    # compile_fn: no worker pool; the plan compiles in this process
    ev = tune.ParallelGpuEvaluator(op, repeat=3, warmup=1, compile_fn=lambda job: 0,
                                   flush=(mode == "cold"), rotate=(3 if mode == "rotated" else 0))
    try:
        rec = ev.measure(sched)
    finally:
        ev.close()
    assert rec["valid"] and rec["ms"] > 0 and rec["reward"] > 0, rec
    if mode == "rotated":
        assert len(ev._copies) == 1 and len(next(iter(ev._copies.values()))) == 3
    torch.cuda.synchronize()
    assert_parity(op, W.output_to_f64(op, ev.inner.out), ev.inner.host, label=f"{key} {mode} timing")
