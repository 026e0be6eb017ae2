"""rc_launch_static (no allocation; workspace in the library's static
device array) against rc_launch with a caller workspace, through the C ABI.

Two calls in a row per operator, the second with a smaller input, each
compared bit for bit with rc_launch on the same inputs (same kernels, fixed
summation order).  A plan whose workspace exceeds the static array is
rejected before any GPU work.
"""
import os

import numpy as np
import pytest

from paper_2506_01374_amd import rc
from paper_2506_01374_amd import workloads as W

import cases

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

PAIRS = cases.NOALLOC_PAIRS


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rc.set_cache_dir(os.path.join(ROOT, "paper_2506_01374_amd", "jit_cache"))
    torch.cuda.set_device(0)


def _both(op, sched, seed):
    host = W.host_inputs(op, seed=seed)
    dev = W.to_device(W.stored_inputs(op, sched, host))
    plan = rc.Plan(op, sched)
    assert plan.workspace_bytes <= rc.lib().rc_static_scratch_bytes()
    ref = W.empty_output(op)
    plan.launch(dev, ref, plan.workspace())
    got = W.empty_output(op)
    plan.launch_static(dev, got)
    torch.cuda.synchronize()
    return W.output_to_f64(op, ref), W.output_to_f64(op, got)


@pytest.mark.parametrize("kind,big,small,flags,sched_text", PAIRS,
                         ids=[f"{k}-{i}" for i, (k, *_rest) in enumerate(PAIRS)])
def test_static_launch_matches_workspace_launch(kind, big, small, flags, sched_text):
    for dims, seed in ((big, 21), (small, 22)):
        op = rc.Op(kind, dims, flags)
        sched = op.from_string(sched_text)
        assert sched.validate() == "", sched.validate()
        print(f"[gpu] static kind={kind} dims={dims} sched={sched_text}", flush=True)
        ref, got = _both(op, sched, seed)
        assert np.all(np.isfinite(ref))
        assert np.array_equal(ref, got), f"dims {dims}: static launch differs"


def test_static_launch_rejects_oversized_workspace():
    name = "moe_t4096_h2048_e64_i1408_top6"
    op = W.workload_op(name)
    plan = rc.Plan(op, op.from_string(cases.TUNED[name]))
    assert plan.workspace_bytes > rc.lib().rc_static_scratch_bytes()
    out = W.empty_output(op)
    ins = [None] * 6
    with pytest.raises(rc.RCError) as e:
        plan.launch_static(ins, out)
    assert e.value.status == rc.RC_ERR_OUT_OF_MEMORY
    assert "static scratch" in str(e.value)
