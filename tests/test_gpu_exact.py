"""GPU tests with exact expected values: the MoE routing preparation's
integer outputs, integer-valued inputs through the bf16 MFMA path, the
closed-form padding counts of the convolution, and the timing call.

Integer index work must match bit for bit; so must contractions of
integer-valued bf16 inputs, whose every partial sum is an integer below 2^24
and therefore exact in fp32 in any accumulation order (the schedules only
reorder the sums, Sec. 2).
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


def launch(op, sched, host):
    print(f"[gpu] kind={op.kind} dims={op.dims} flags={op.flags} sched={sched}", flush=True)
    dev = W.to_device(W.stored_inputs(op, sched, host))
    out = W.empty_output(op)
    plan = rc.Plan(op, sched)
    ws = plan.workspace()
    plan.launch(dev, out, ws)
    torch.cuda.synchronize()
    return plan, dev, out, ws


def ws_int32(plan, ws, name):
    off, n = plan.buffer(name)
    return ws[off:off + n].cpu().view(torch.int32).numpy().copy()


# ---------------------------------------------------------------------------
# MoE routing preparation: offsets, perm, pos and tile starts bit for bit
# ---------------------------------------------------------------------------

def _check_prep(op, sched, host, plan, ws):
    T, Hd, E, I, k = op.dims
    d = sched.as_dict()
    ref = oracle.moe_routing_prep(host["ids"], E, d["up.tile_m"], d["down.tile_m"])
    for name in ("offsets", "perm", "pos", "tile_up", "tile_down"):
        got = ws_int32(plan, ws, name)
        assert got.shape == ref[name].shape, name
        bad = np.flatnonzero(got != ref[name])
        assert bad.size == 0, f"{name}: {bad.size} entries differ, first at {bad[:5]}"


def _routing(pattern, T, E, k, seed):
    ids = None
    if pattern == "two_experts":
        ids = np.tile(np.array([[1, E - 2]], dtype=np.int32), (T, 1))
    elif pattern == "skewed":
        ids = np.tile(np.array([[0, E - 1]], dtype=np.int32), (T, 1))
        ids[5] = [3, 4]
        ids[T - 56:] = [[2, 5]]
    elif pattern == "one_expert_top1":
        ids = np.full((T, 1), 3, dtype=np.int32)
    return np.ascontiguousarray(ids)


@pytest.mark.parametrize("which", ["tuned", "default"])
def test_moe_prep_bitexact_full_size(which):
    name = "moe_t4096_h2048_e64_i1408_top6"
    op = W.workload_op(name)
    sched = op.from_string(cases.TUNED[name]) if which == "tuned" else op.default()
    host = W.host_inputs(op, seed=0)
    plan, dev, out, ws = launch(op, sched, host)
    _check_prep(op, sched, host, plan, ws)


@pytest.mark.parametrize("pattern", ["two_experts", "skewed", "one_expert_top1", "random_large"])
def test_moe_prep_bitexact_edge_routings(pattern):
    # empty experts, a dominant expert, single-row groups, top-1, and more
    # routed rows (49,152) than one LDS copy of the ids could hold
    if pattern == "random_large":
        T, Hd, E, I, k = 8192, 256, 64, 128, 6
    else:
        T, Hd, E, I, k = 256, 256, 8, 128, (1 if pattern == "one_expert_top1" else 2)
    op = rc.Op(rc.RC_OP_MOE, (T, Hd, E, I, k))
    host = gen.moe_inputs(T, Hd, E, I, k, seed=9)
    if pattern != "random_large":
        host["ids"] = _routing(pattern, T, E, k, 9)
        host["w"] = np.full((T, k), 1.0 / k, dtype=np.float32)
    for s in cases.SCHEDULES["moe"][:4]:
        sched = op.from_string(s)
        plan, dev, out, ws = launch(op, sched, host)
        _check_prep(op, sched, host, plan, ws)
        if pattern == "random_large":
            y = W.output_to_f64(op, out)
            rows = np.array([0, 1, T // 2, T - 1])
            ref = oracle.bf16_to_f64(oracle.moe_bf16(host["X"], host["ids"], host["w"], host["Wg"],
                                                     host["Wu"], host["Wd"], rows=rows))
            ok, worst, _ = oracle.compare(y[rows], ref, oracle.TOL_BF16)
            assert ok, worst


def test_moe_full_size_last_tile_of_every_expert():
    # Full-size MoE output on the tokens owning the first and last row of
    # every expert's last M tile in both expert GEMMs (the partially filled
    # tiles), in the benchmark's schedule.
    name = "moe_t4096_h2048_e64_i1408_top6"
    op = W.workload_op(name)
    T, Hd, E, I, k = op.dims
    sched = op.from_string(cases.TUNED[name])
    host = W.host_inputs(op, seed=0)
    plan, dev, out, ws = launch(op, sched, host)
    d = sched.as_dict()
    prep = oracle.moe_routing_prep(host["ids"], E, d["up.tile_m"], d["down.tile_m"])
    toks = set()
    for e in range(E):
        a, b = int(prep["offsets"][e]), int(prep["offsets"][e + 1])
        if b == a:
            continue
        for tm in (d["up.tile_m"], d["down.tile_m"]):
            first_of_last = a + ((b - a - 1) // tm) * tm
            toks.add(int(prep["perm"][first_of_last]) // k)
            toks.add(int(prep["perm"][b - 1]) // k)
    rows = np.array(sorted(toks), dtype=np.int64)
    assert len(rows) >= E
    y = W.output_to_f64(op, out)[rows]
    ref = oracle.bf16_to_f64(oracle.moe_bf16(host["X"], host["ids"], host["w"], host["Wg"], host["Wu"],
                                             host["Wd"], rows=rows))
    ok, worst, _ = oracle.compare(y, ref, oracle.TOL_BF16)
    print(f"[parity] moe last tiles: {len(rows)} tokens worst={worst:.3e}", flush=True)
    assert ok, worst


# ---------------------------------------------------------------------------
# Integer-valued inputs through the bf16 MFMA path (no activation): exact
# ---------------------------------------------------------------------------

def _int_conv_inputs(N, H, Wd, C, K, R, S, seed, a=8):
    return {"x": gen.int_valued_bf16(seed, 1, (N, H, Wd, C), a),
            "w": gen.int_valued_bf16(seed, 2, (K, R, S, C), a),
            "bias": gen.int_valued_f32(seed, 3, (K,), a)}


CONV_NOACT = [
    ("conv", (2, 16, 12, 64, 64, 3, 3, 1)),
    ("conv_ragged", (1, 10, 9, 64, 64, 3, 3, 1)),
    ("conv_k320", (1, 8, 8, 64, 320, 3, 3, 1)),
]


@pytest.mark.parametrize("key,dims", CONV_NOACT, ids=[k for k, _ in CONV_NOACT])
def test_conv_integer_inputs_bitwise(key, dims):
    # |x|, |w|, |bias| <= 8: every partial sum is an integer below 2^24, so
    # every schedule must reproduce the oracle bit for bit.
    op = rc.Op(rc.RC_OP_CONV2D, dims, rc.RC_FLAG_NO_ACT)
    host = _int_conv_inputs(*dims[:7], seed=11)
    ref = oracle.conv2d_bf16(host["x"], host["w"], host["bias"], pad=dims[7], act=False)
    ref = oracle.bf16_to_f64(ref)
    for s in cases.SCHEDULES[key]:
        sched = op.from_string(s)
        if sched.validate():
            continue
        _, _, out, _ = launch(op, sched, host)
        y = W.output_to_f64(op, out).reshape(ref.shape)
        bad = np.flatnonzero(y != ref)
        assert bad.size == 0, f"{s}: {bad.size} outputs differ"


@pytest.mark.parametrize("sched_text", cases.GEMM_1X1)
def test_bf16_gemm_integer_inputs_bitwise(sched_text):
    # A 1 x 1 convolution without padding is the plain bf16 GEMM
    # Y[M][K] = X[M][C] W^T + bias: integer inputs give exact outputs, and
    # ones give C in every output.
    N, H, Wd, C, K = 2, 16, 16, 256, 128
    op = rc.Op(rc.RC_OP_CONV2D, (N, H, Wd, C, K, 1, 1, 0), rc.RC_FLAG_NO_ACT)
    sched = op.from_string(sched_text)
    host = _int_conv_inputs(N, H, Wd, C, K, 1, 1, seed=13)
    _, _, out, _ = launch(op, sched, host)
    y = W.output_to_f64(op, out).reshape(-1, K)
    X = oracle.bf16_to_f64(host["x"]).reshape(-1, C)
    Wm = oracle.bf16_to_f64(host["w"]).reshape(K, C)
    exact = X @ Wm.T + host["bias"].astype(np.float64)[None, :]   # integers, exact in fp64
    assert np.array_equal(y, oracle.bf16_to_f64(oracle.bf16_from_f64(exact)).reshape(y.shape))
    ones = {"x": oracle.bf16_from_f64(np.ones((N, H, Wd, C))), "w": oracle.bf16_from_f64(np.ones((K, 1, 1, C))),
            "bias": np.zeros(K, dtype=np.float32)}
    _, _, out, _ = launch(op, sched, ones)
    assert np.all(W.output_to_f64(op, out) == C)


@pytest.mark.parametrize("sched_text", ["tuned", "default", cases.CONV_FULL_ALT])
def test_conv_full_size_ones_padding_counts(sched_text):
    # Ones input, ones filters, zero bias, no activation: interior outputs
    # count 9 x 320 = 2880 taps, edges 1920 and corners 1280, exactly.
    name = "conv3x3_n2_64x64_c320_k320"
    op = rc.Op(rc.RC_OP_CONV2D, W.workload_op(name).dims, rc.RC_FLAG_NO_ACT)
    N, H, Wd, C, K, R, S, pad = op.dims
    text = cases.TUNED[name] if sched_text == "tuned" else ("" if sched_text == "default" else sched_text)
    sched = op.from_string(text)
    host = {"x": oracle.bf16_from_f64(np.ones((N, H, Wd, C))),
            "w": oracle.bf16_from_f64(np.ones((K, R, S, C))), "bias": np.zeros(K, dtype=np.float32)}
    _, _, out, _ = launch(op, sched, host)
    v = W.output_to_f64(op, out).reshape(N, H, Wd, K)
    expect = np.full((H, Wd), 2880.0)
    expect[0, :] = expect[-1, :] = expect[:, 0] = expect[:, -1] = 1920.0
    for p, q in [(0, 0), (0, -1), (-1, 0), (-1, -1)]:
        expect[p, q] = 1280.0
    assert np.array_equal(v, np.broadcast_to(expect[None, :, :, None], v.shape))


def test_conv_full_size_integer_inputs_bitwise_sampled():
    name = "conv3x3_n2_64x64_c320_k320"
    op = rc.Op(rc.RC_OP_CONV2D, W.workload_op(name).dims, rc.RC_FLAG_NO_ACT)
    sched = op.from_string(cases.TUNED[name])
    host = _int_conv_inputs(*op.dims[:7], seed=17)
    _, _, out, _ = launch(op, sched, host)
    N, H, Wd, C, K, R, S, pad = op.dims
    rng = np.random.default_rng(3)
    pix = np.unique(np.concatenate([[0, Wd - 1, (H - 1) * Wd, H * Wd - 1, N * H * Wd - 1],
                                    rng.choice(N * H * Wd, 256, replace=False)]))
    ref = oracle.bf16_to_f64(oracle.conv2d_bf16(host["x"], host["w"], host["bias"], pad=pad, act=False,
                                                pixels=pix))
    y = W.output_to_f64(op, out).reshape(-1, K)[pix]
    assert np.array_equal(y, ref)


# ---------------------------------------------------------------------------
# Timing (time -> reward): ordered statistics, a reward consistent with the
# peaks, and outputs still right after the timed launches
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("key", ["gemm", "attn_causal", "mlp", "moe", "conv"])
def test_rc_time_flush_and_output(key):
    from paper_2506_01374_amd import tune
    op = cases.small_op(key)
    sched = op.from_string(cases.SCHEDULES[key][1])
    host = W.host_inputs(op, seed=6)
    dev = W.to_device(W.stored_inputs(op, sched, host))
    out = W.empty_output(op)
    plan = rc.Plan(op, sched)
    ws = plan.workspace()
    t = plan.time(dev, out, ws, warmup=2, repeat=9, flush=True)
    assert t.nkernels == plan.nkernels
    assert 0 < t.min_ms <= t.q1_ms <= t.median_ms <= t.q3_ms
    assert t.mean_ms >= t.min_ms
    assert all(t.kernel_ms[i] > 0 for i in range(min(8, t.nkernels)))
    assert sum(t.kernel_ms[:min(8, t.nkernels)]) <= t.q3_ms * 1.5 + 1e-3
    sec = t.median_ms * 1e-3
    assert abs(t.tflops - op.flops() / sec / 1e12) <= 1e-9 * max(1.0, t.tflops)
    assert abs(t.frac_flops - op.flops() / sec / op.peak_flops()) <= 1e-9
    assert abs(t.frac_bytes - op.bytes() / sec / 8.0e12) <= 1e-9
    r = tune.reward_of(op, t.median_ms)
    assert 0 < r < 1
    assert r == pytest.approx(t.frac_bytes if op.bound() == "hbm" else t.frac_flops, rel=1e-12)
    torch.cuda.synchronize()
    y = W.output_to_f64(op, out)
    from test_gpu_parity import assert_parity
    assert_parity(op, y, host, label=f"{key} after rc_time")
    # without flushing, and after releasing the flush buffer
    t2 = plan.time(dev, out, ws, warmup=1, repeat=3, flush=False)
    assert t2.median_ms > 0
    rc.time_release()
    t3 = plan.time(dev, out, ws, warmup=1, repeat=3, flush=True)
    assert t3.median_ms > 0
