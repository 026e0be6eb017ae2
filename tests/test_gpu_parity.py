"""GPU parity: every kernel path against the CPU oracle on the same seeded
inputs, through the C ABI.

Small shapes are compared element by element over the whole output; the
full-size workloads, in the schedules the benchmark times, are compared on
sampled outputs.  Outputs are NaN-filled before each launch so an unwritten
element fails.  Tolerances (see oracle.compare): 1e-4 for the fp32 GEMM,
2e-2 for bf16 inputs with fp32 accumulation, relative to max(|ref|, RMS).
"""
import os

import numpy as np
import pytest

import oracle
from paper_2506_01374_amd import inputs as gen
from paper_2506_01374_amd import rc
from paper_2506_01374_amd import workloads as W

import cases

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    rc.set_cache_dir(os.path.join(ROOT, "paper_2506_01374_amd", "jit_cache"))
    torch.cuda.set_device(0)


def run(op, sched, host):
    print(f"[gpu] kind={op.kind} dims={op.dims} sched={sched}", flush=True)
    dev = W.to_device(W.stored_inputs(op, sched, host))
    out = W.empty_output(op)
    plan = rc.Plan(op, sched)
    ws = plan.workspace()
    plan.launch(dev, out, ws)
    torch.cuda.synchronize()
    return W.output_to_f64(op, out), (plan, dev, out, ws)


def reference(op, host, rows=None):
    """Oracle output (fp64 values of the stored type) for the selected rows."""
    if op.kind == rc.RC_OP_GEMM_F32:
        return oracle.gemm_f32(host["A"], host["B"], rows=rows).astype(np.float64), oracle.TOL_F32
    if op.kind == rc.RC_OP_ATTENTION:
        o = oracle.attention_bf16(host["Q"], host["K"], host["V"], causal=bool(op.flags & 1), rows=rows)
    elif op.kind == rc.RC_OP_GATED_MLP:
        o = oracle.gated_mlp_bf16(host["X"], host["Wg"], host["Wu"], host["Wd"], rows=rows)
    elif op.kind == rc.RC_OP_MOE:
        o = oracle.moe_bf16(host["X"], host["ids"], host["w"], host["Wg"], host["Wu"], host["Wd"], rows=rows)
    else:
        o = oracle.conv2d_bf16(host["x"], host["w"], host["bias"], pad=op.dims[7], pixels=rows)
    return oracle.bf16_to_f64(o), oracle.TOL_BF16


def rows_of(op, y):
    """View the output as [independent rows][values]."""
    if op.kind == rc.RC_OP_ATTENTION:
        return y.reshape(-1, op.dims[3])
    if op.kind == rc.RC_OP_CONV2D:
        return y.reshape(-1, op.dims[4])
    return y.reshape(y.shape[0], -1)


def assert_parity(op, y, host, rows=None, label=""):
    ref, tol = reference(op, host, rows)
    got = rows_of(op, y)
    if rows is not None:
        got = got[np.asarray(rows)]
    ok, worst, rms = oracle.compare(got, ref, tol)
    print(f"[parity] {label} worst={worst:.3e} tol={tol:g} rms={rms:.3e}", flush=True)
    assert ok, f"{label}: worst scaled error {worst:.3e} > {tol:g}"
    return worst


# ---------------------------------------------------------------------------
# small shapes, many schedules, whole outputs
# ---------------------------------------------------------------------------

def _params():
    out = []
    for key, lst in cases.SCHEDULES.items():
        for i, s in enumerate(lst):
            out.append(pytest.param(key, s, id=f"{key}-{i}"))
    return out


@pytest.mark.parametrize("key,sched_text", _params())
def test_small_shapes(key, sched_text):
    op = cases.small_op(key)
    sched = op.from_string(sched_text)
    host = W.host_inputs(op, seed=1)
    y, _ = run(op, sched, host)
    assert_parity(op, y, host, label=f"{key} {sched_text}")


def test_gemm_sweep_has_18_legal_points():
    op = cases.small_op("gemm")
    legal = [s for s in cases.gemm_sweep() if op.from_string(s).validate() == ""]
    assert len(legal) == 18


@pytest.mark.parametrize("sched_text", [cases.SCHEDULES["gemm"][i] for i in (0, 7, 17, 18, 19, 20)])
def test_gemm_integer_inputs_bitwise(sched_text):
    # Integer inputs in [-4, 4]: every partial sum is an integer below 2^24,
    # exact in fp32 in any order, so every schedule must match bit for bit.
    op = cases.small_op("gemm")
    sched = op.from_string(sched_text)
    host = {"A": gen.int_valued_f32(3, 1, (128, 128), 4), "B": gen.int_valued_f32(3, 2, (128, 128), 4)}
    y, _ = run(op, sched, host)
    ref = oracle.gemm_f32(host["A"], host["B"]).astype(np.float64)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("sched_text", cases.SCHEDULES["gemm_skinny"][1:])
def test_gemm_skinny_integer_inputs_bitwise(sched_text):
    # The streaming stage adds the waves' and the K splits' partial sums in a
    # different order from the oracle; with integer inputs in [-4, 4] every
    # partial sum is an integer below 2^24, so the result is still exact.
    op = cases.small_op("gemm_skinny")
    M, N, K = op.dims
    sched = op.from_string(sched_text)
    host = {"A": gen.int_valued_f32(5, 1, (M, K), 4), "B": gen.int_valued_f32(5, 2, (K, N), 4)}
    y, _ = run(op, sched, host)
    ref = oracle.gemm_f32(host["A"], host["B"]).astype(np.float64)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("pattern", ["two_experts", "skewed", "one_expert_top1"])
def test_moe_edge_routing(pattern):
    # Routings with empty experts, a dominant expert and single-row groups.
    T, Hd, E, I, k = 256, 256, 8, 128, 2
    if pattern == "one_expert_top1":
        k = 1
    op = rc.Op(rc.RC_OP_MOE, (T, Hd, E, I, k))
    host = gen.moe_inputs(T, Hd, E, I, k, seed=4)
    if pattern == "two_experts":
        host["ids"] = np.tile(np.array([[1, 6]], dtype=np.int32), (T, 1))
        host["w"] = np.tile(np.array([[0.75, 0.25]], dtype=np.float32), (T, 1))
    elif pattern == "skewed":
        ids = np.tile(np.array([[0, 7]], dtype=np.int32), (T, 1))
        ids[5] = [3, 4]       # a single-row group for experts 3 and 4
        ids[200:] = [[2, 5]]
        host["ids"] = ids
    else:
        host["ids"] = np.full((T, 1), 3, dtype=np.int32)
        host["w"] = np.ones((T, 1), dtype=np.float32)
    for s in cases.SCHEDULES["moe"][:3]:
        y, _ = run(op, op.from_string(s), host)
        assert_parity(op, y, host, label=f"moe {pattern}")


@pytest.mark.parametrize("key", ["gemm", "attn_causal", "mlp", "moe", "conv"])
def test_repeat_launch_bitwise_deterministic(key):
    op = cases.small_op(key)
    sched = op.from_string(cases.SCHEDULES[key][1])
    host = W.host_inputs(op, seed=2)
    y1, (plan, dev, out, ws) = run(op, sched, host)
    out.fill_(float("nan"))
    plan.launch(dev, out, ws)
    torch.cuda.synchronize()
    y2 = W.output_to_f64(op, out)
    assert np.array_equal(y1, y2)


# ---------------------------------------------------------------------------
# full-size workloads in the benchmark's schedules, sampled outputs
# ---------------------------------------------------------------------------

def _sample_rows(op, n, seed=0):
    rng = np.random.default_rng(seed)
    d = op.dims
    if op.kind == rc.RC_OP_ATTENTION:
        B, H, S, _ = d
        fixed = [0, S - 1, S // 2, (H - 1) * S + S - 1, (B * H - 1) * S]
        total = B * H * S
    elif op.kind == rc.RC_OP_CONV2D:
        N, Hh, Ww, _, _, R, S, pad = d
        P, Q = Hh + 2 * pad - R + 1, Ww + 2 * pad - S + 1
        fixed = [0, Q - 1, (P - 1) * Q, P * Q - 1, P * Q + Q // 2, N * P * Q - 1]
        total = N * P * Q
    else:
        fixed = [0, d[0] - 1]
        total = d[0]
    extra = rng.choice(total, size=n, replace=False).tolist()
    return np.array(sorted(set(fixed + extra)), dtype=np.int64)


@pytest.mark.parametrize("name", list(W.WORKLOADS))
@pytest.mark.parametrize("which", ["tuned", "default"])
def test_full_size_sampled(name, which):
    op = W.workload_op(name)
    sched = op.from_string(cases.TUNED[name]) if which == "tuned" else op.default()
    host = W.host_inputs(op, seed=0)
    y, _ = run(op, sched, host)
    n = {rc.RC_OP_GEMM_F32: 128, rc.RC_OP_ATTENTION: 96, rc.RC_OP_GATED_MLP: 12,
         rc.RC_OP_MOE: 12, rc.RC_OP_CONV2D: 64}[op.kind]
    rows = None if op.kind == rc.RC_OP_GEMM_F32 else _sample_rows(op, n)
    assert_parity(op, y, host, rows=rows, label=f"{name} {which}")
    assert np.all(np.isfinite(y))


@pytest.mark.parametrize("name,sched_text", cases.FULL_ALT,
                         ids=[f"{n.split('_')[0]}-{i}" for i, (n, _) in enumerate(cases.FULL_ALT)])
def test_full_size_alternative_paths(name, sched_text):
    op = W.workload_op(name)
    sched = op.from_string(sched_text)
    assert sched.validate() == "", sched.validate()
    host = W.host_inputs(op, seed=0)
    y, _ = run(op, sched, host)
    n = {rc.RC_OP_ATTENTION: 96, rc.RC_OP_GATED_MLP: 12, rc.RC_OP_MOE: 12, rc.RC_OP_CONV2D: 64}[op.kind]
    assert_parity(op, y, host, rows=_sample_rows(op, n, seed=7), label=f"{name} {sched_text}")
    assert np.all(np.isfinite(y))


@pytest.mark.parametrize("name,dims,flags", cases.RAGGED_FULL,
                         ids=[f"{n.split('_')[0]}-{d[2] if len(d) > 3 else d[0]}" for n, d, _ in cases.RAGGED_FULL])
def test_ragged_near_full_size(name, dims, flags):
    kind = W.workload_op(name).kind
    op = rc.Op(kind, dims, flags)
    sched = op.from_string(cases.TUNED[name])
    assert sched.validate() == "", sched.validate()
    host = W.host_inputs(op, seed=3)
    y, _ = run(op, sched, host)
    n = {rc.RC_OP_GEMM_F32: 0, rc.RC_OP_ATTENTION: 96, rc.RC_OP_GATED_MLP: 12, rc.RC_OP_CONV2D: 64}[kind]
    rows = None if kind == rc.RC_OP_GEMM_F32 else _sample_rows(op, n, seed=11)
    assert_parity(op, y, host, rows=rows, label=f"{name} {dims}")
    assert np.all(np.isfinite(y))


@pytest.mark.parametrize("key", ["attn_causal", "mlp", "moe"])
def test_graph_replay_matches_eager(key):
    # The benchmark replays captured launches.  Capture one execution on a
    # side stream, replay it several times with eager work and host
    # synchronisation in between, and compare every replay with the eager
    # result bit for bit.
    op = cases.small_op(key)
    sched = op.from_string(cases.SCHEDULES[key][1])
    host = W.host_inputs(op, seed=5)
    eager, (plan, dev, out, ws) = run(op, sched, host)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        prep = plan.prepare(dev, out, ws, stream)
        prep.launch()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        prep.launch()
    torch.cuda.synchronize()
    scratch = torch.zeros(1 << 20, device="cuda")
    for rep in range(3):
        out.fill_(float("nan"))
        scratch.add_(1.0)                      # unrelated eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(W.output_to_f64(op, out), eager), f"replay {rep} differs"
