"""CPU tests of the C ABI: the library loads and exports every entry point
the header declares; descriptors, knob tables, legality, transformations,
parsing and the FLOP / byte model.  No GPU work is done here."""
import ctypes
import math
import json
import os
import re
import subprocess

import pytest

from paper_2506_01374_amd import rc
from paper_2506_01374_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "rc.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = set(re.findall(r"\b(rc_[a-z0-9_]+)\s*\(", text))
    typedef_fns = set(re.findall(r"\(\s*\*\s*(rc_[a-z0-9_]+)\s*\)", text))
    return sorted(names - typedef_fns)


def test_library_exports_every_declared_symbol():
    declared = header_functions()
    assert len(declared) >= 35
    out = subprocess.check_output(["nm", "-D", "--defined-only", rc.LIB_PATH]).decode()
    exported = set(re.findall(r" T (rc_[a-z0-9_]+)", out))
    missing = [n for n in declared if n not in exported]
    assert not missing, missing
    lib = rc.lib()
    for n in declared:
        assert hasattr(lib, n)
    assert sorted(rc.EXPORTS) == declared


def test_status_strings_and_errors():
    L = rc.lib()
    assert L.rc_status_str(0) == b"RC_OK"
    assert L.rc_status_str(2) == b"RC_ERR_ILLEGAL_SCHEDULE"
    with pytest.raises(rc.RCError) as e:
        rc.Op(99, (1, 2, 3))
    assert "RC_ERR_UNSUPPORTED" in str(e.value)
    with pytest.raises(rc.RCError):
        rc.Op(rc.RC_OP_GEMM_F32, (128, 0, 128))
    with pytest.raises(rc.RCError):
        rc.Op(rc.RC_OP_GEMM_F32, (128, 128))
    with pytest.raises(rc.RCError):
        rc.Op(rc.RC_OP_MOE, (16, 8, 4, 8, 5))      # top-5 of 4 experts


def test_flops_and_bytes_model():
    g = W.workload_op("gemm_f32_128")
    assert g.flops() == 2 * 128 ** 3
    assert g.bytes() == 4 * 3 * 128 * 128
    a = W.workload_op("attention_causal_b1_h32_s1024_d128")
    assert a.flops() == 4 * 128 * 32 * 1024 * 1025 / 2 == 8_598_323_200
    assert a.bytes() == 2 * 4 * 32 * 1024 * 128
    m = W.workload_op("gated_mlp_t2048_h4096_i14336")
    assert m.flops() == 6 * 2048 * 4096 * 14336 == 721_554_505_728
    e = W.workload_op("moe_t4096_h2048_e64_i1408_top6")
    assert e.flops() == 6 * 4096 * 6 * 2048 * 1408 == 425_201_762_304
    c = W.workload_op("conv3x3_n2_64x64_c320_k320")
    assert c.flops() == 2 * 8192 * 320 * 2880 == 15_099_494_400
    f = W.workload_op("attention_noncausal_b1_h24_s4096_d128")
    assert f.flops() == 4 * 24 * 4096 * 4096 * 128 == 206_158_430_208
    assert f.bytes() == 4 * 2 * 24 * 4096 * 128
    assert g.peak_flops() == 157.3e12 and a.peak_flops() == 2516.6e12
    assert rc.lib().rc_peak_bytes_per_s() == 8.0e12


def test_knob_tables_and_default_is_legal():
    for name in W.WORKLOADS:
        op = W.workload_op(name)
        names = op.knob_names()
        assert len(names) == len(set(names)) and len(names) <= rc.MAX_KNOBS
        classes = {op.knob_class(i) for i in range(len(names))}
        assert classes <= {"TileSize", "Parallel", "Vectorize", "Unroll", "ComputeLocation", "Layout"}
        assert {"TileSize", "Parallel", "Unroll", "ComputeLocation"} <= classes
        d = op.default()
        assert d.validate() == ""
        for i in range(len(names)):
            assert d.raw.knob[i] == min(op.knob_values(i)) or names[i].endswith("vec")


def test_validate_rejects_with_reasons():
    g = W.workload_op("gemm_f32_128")
    s = g.schedule(tile_m=16, waves_m=2)
    assert "multiple of 16" in s.validate()
    s = g.schedule(tile_k=4, vec=4)
    assert "loads" in s.validate()
    # tiles may cross the edges of the fp32 GEMM (96 = 1.5 tiles of 64), but a
    # vector load may not cross the end of a row, and the streaming stage
    # needs whole column tiles
    odd = rc.Op(rc.RC_OP_GEMM_F32, (96, 100, 126))
    assert odd.schedule(tile_m=64).validate() == ""
    assert "rows of A" in odd.schedule(tile_k=16, vec=4).validate()
    assert "rows of B" in rc.Op(rc.RC_OP_GEMM_F32, (96, 102, 128)).schedule(tile_k=16, vec=4).validate()
    assert "does not divide N" in rc.Op(rc.RC_OP_GEMM_F32, (16, 100, 1024)).schedule(
        tile_n=64, tile_k=16, vec=4, stages=3).validate()
    conv = W.workload_op("conv3x3_n2_64x64_c320_k320")
    assert "filter tap" in conv.schedule(tile_k=128).validate()
    mlp = W.workload_op("gated_mlp_t2048_h4096_i14336")
    big = mlp.schedule(up__tile_m=256, up__tile_n=256, up__tile_k=128, up__waves_m=1, up__waves_n=1,
                       up__stages=2)
    assert "LDS" in big.validate() or "accumulators" in big.validate()
    att = W.workload_op("attention_causal_b1_h32_s1024_d128")
    assert "rows per wave" in att.schedule(block_m=64, waves=1, mfma=16).validate()
    s = g.default()
    s.raw.knob[0] = 48                      # not an allowed value
    assert "not an allowed value" in s.validate()


def test_moe_row_skip_and_pipelined_attention_splits_legality():
    # the MoE's partial-tile skip needs a staging path with a partial-tile
    # copy of its loop (not the ping-pong stage); the tile order knob has a
    # third value; the pipelined attention stage takes key splits while its
    # four ring slots per split fit the LDS
    moe = W.workload_op("moe_t4096_h2048_e64_i1408_top6")
    tuned = json.load(open(os.path.join(ROOT, "paper_2506_01374_amd", "tuned.json")))
    base = tuned["moe_t4096_h2048_e64_i1408_top6"]
    assert moe.from_string(base + ",up.skip=1,down.skip=1,up.grid=2,down.grid=2").validate() == ""
    names = moe.knob_names()
    assert "up.skip" in names and "down.skip" in names
    assert moe.knob_values(names.index("up.grid")) == [0, 1, 2]
    pp = moe.from_string("up.tile_m=128,up.tile_n=128,up.tile_k=64,up.waves_m=4,up.waves_n=2,up.stages=6,"
                         "up.vec=8,up.layout=1,up.occ=2,up.skip=1")
    assert "ping-pong" in pp.validate()
    assert "ping-pong" not in moe.from_string(str(pp).replace("up.skip=1", "up.skip=0")).validate()
    mlp = W.workload_op("gated_mlp_t2048_h4096_i14336")
    assert "up.skip" not in mlp.knob_names()
    att = W.workload_op("attention_causal_b1_h32_s1024_d128")
    two = att.schedule(block_m=64, block_n=32, waves=4, mfma=16, stages=5, vec=8, occ=2, order=1, splits=2)
    assert two.validate() == ""
    four = att.schedule(block_m=64, block_n=32, waves=4, mfma=16, stages=5, vec=8, occ=1, order=1, splits=4)
    assert "LDS" in four.validate()


def test_k_split_and_k_split_tail_legality_and_plans():
    # the MLP down projection's K split and the K-split tails: whole K tiles
    # per split, no tail split with a K split, the fused epilogue for a
    # K-split gate/up tail; the plans add the summing kernels and the
    # partial-sum workspace
    mlp = W.workload_op("gated_mlp_t2048_h4096_i14336")
    tuned = json.load(open(os.path.join(ROOT, "paper_2506_01374_amd", "tuned.json")))
    base = mlp.from_string(tuned["gated_mlp_t2048_h4096_i14336"]).as_dict()
    names = mlp.knob_names()
    assert mlp.knob_values(names.index("down.split")) == [1, 2, 4]
    assert mlp.knob_values(names.index("up.tail")) == [0, 1, 2]
    assert "down.split" not in W.workload_op("moe_t4096_h2048_e64_i1408_top6").knob_names()

    def sched(**kw):
        d = dict(base)
        d.update(kw)
        return mlp.schedule(**d)

    assert sched(**{"down.split": 2}).validate() == ""
    # a down GEMM whose tail split is legal on its own (1024 x 576 x 256)
    import cases
    tail_op = cases.small_op("mlp_tail_down")
    for text in cases.SCHEDULES["mlp_tail_down"][:1]:
        alone = tail_op.from_string(text)
        assert alone.validate() == ""
        for t in (1, 2):
            both = tail_op.schedule(**{**alone.as_dict(), "down.tail": t, "down.split": 2})
            assert "do not combine" in both.validate()
    # 14336 = 448 K tiles of 32: two or four whole halves/quarters; with 128-wide
    # K tiles 112 of them, 28 per quarter, an unroll of 2 divides them all
    assert sched(**{"down.split": 4}).validate() == ""
    odd = W.op_for(rc.RC_OP_GATED_MLP, (256, 256, 320))
    odd_s = odd.schedule(**{**odd.default().as_dict(), "down.tile_k": 32, "down.split": 4})
    assert "whole number" in odd_s.validate()          # 320 = 10 K tiles of 32, not 4 x whole
    assert "fused SwiGLU" in sched(**{"up.tail": 2, "fuse": 0}).validate()
    assert sched(**{"up.tail": 2}).validate() == ""
    plan_names = [k["name"] for k in rc.describe(mlp, sched(**{"up.tail": 2}))]
    assert plan_names == ["rc_gemm_bf16", "rc_gemm_bf16", "rc_splitk_swiglu_bf16", "rc_gemm_bf16",
                          "rc_splitk_sum_bf16"]
    grids = [k["grid"] for k in rc.describe(mlp, sched())]
    assert grids[2] == 2 * (2048 // 256) * (4096 // 256)     # two copies of the 128 down tiles


def test_apply_enumerate_and_illegal_transform():
    g = W.workload_op("gemm_f32_128")
    p0 = g.default()
    moves = p0.moves()
    assert moves
    for t in moves:
        nxt = p0.apply(t)
        assert nxt.validate() == ""
        assert nxt.raw.knob[t.knob] == t.value
    # every move differs from the current value and is unique
    assert len({(t.knob, t.value) for t in moves}) == len(moves)
    bad = rc.rc_transform(g.knob_names().index("vec"), 4)
    before = p0.copy()
    with pytest.raises(rc.RCError) as e:
        p0.apply(bad)
    assert "RC_ERR_ILLEGAL_SCHEDULE" in str(e.value)
    assert str(p0) == str(before)


def test_enumerate_matches_brute_force():
    op = W.workload_op("conv3x3_n2_64x64_c320_k320")
    s = op.default()
    expect = []
    for i in range(len(op.knob_names())):
        for v in op.knob_values(i):
            if v == s.raw.knob[i]:
                continue
            c = s.copy()
            c.raw.knob[i] = v
            if c.validate() == "":
                expect.append((i, v))
    assert sorted((t.knob, t.value) for t in s.moves()) == sorted(expect)


def test_parse_transform():
    op = W.workload_op("gated_mlp_t2048_h4096_i14336")
    t = op.parse("TileSize(up.tile_m=128)")
    assert op.knob_names()[t.knob] == "up.tile_m" and t.value == 128
    t = op.parse("  Unroll ( down.unroll = 2 ) ")
    assert op.knob_names()[t.knob] == "down.unroll" and t.value == 2
    for bad in ["TileSize(up.tile_m=100)", "Unroll(up.tile_m=128)", "Vectorise(up.vec=8)",
                "TileSize", "TileSize(up.tile_m=)", "TileSize(nope=1)", "Parallel(fuse=1)",
                "TileSize(up.tile_m=128) extra"]:
        with pytest.raises(rc.RCError):
            op.parse(bad)


def test_schedule_string_round_trip_and_hash():
    for name in W.WORKLOADS:
        op = W.workload_op(name)
        s = op.default()
        for t in s.moves()[:5]:
            s2 = s.apply(t)
            back = op.from_string(str(s2))
            assert str(back) == str(s2) and back.hash() == s2.hash()
            assert s2.hash() != s.hash()
    with pytest.raises(rc.RCError):
        W.workload_op("gemm_f32_128").from_string("tile_m=16,bogus=3")


def test_tuned_schedules_are_legal():
    import cases
    for name, text in cases.TUNED.items():
        op = W.workload_op(name)
        assert op.from_string(text).validate() == "", name
    for key, lst in cases.SCHEDULES.items():
        op = cases.small_op(key)
        for text in lst:
            assert op.from_string(text).validate() == "", (key, text)


def test_plan_create_rejects_illegal_before_gpu_work():
    g = W.workload_op("gemm_f32_128")
    s = g.schedule(tile_m=16, waves_m=2)
    h = ctypes.c_void_p()
    st = rc.lib().rc_plan_create(g.ref, ctypes.byref(s.raw), ctypes.byref(h))
    assert st == 2 and not h.value


def test_precompile_reports_illegal_and_compiles_legal(tmp_path):
    rc.set_cache_dir(str(tmp_path))
    try:
        g = W.workload_op("gemm_f32_128")
        st = rc.precompile(g, [g.default(), g.schedule(tile_m=16, waves_m=2)], nthreads=2)
        assert st == [0, 2]
        assert any(f.endswith(".hsaco") for f in os.listdir(tmp_path))
    finally:
        rc.set_cache_dir(os.path.join(ROOT, "paper_2506_01374_amd", "jit_cache"))


@pytest.mark.parametrize("kind,dims", [
    (rc.RC_OP_GEMM_F32, (0, 16, 16)),
    (rc.RC_OP_GEMM_F32, (16, 16, 0)),
    (rc.RC_OP_ATTENTION, (1, 2, 0, 128)),
    (rc.RC_OP_GATED_MLP, (0, 256, 512)),
    (rc.RC_OP_MOE, (0, 256, 8, 128, 2)),
    (rc.RC_OP_CONV2D, (1, 0, 4, 64, 64, 3, 3, 1)),
])
def test_empty_operators_are_rejected_when_described(kind, dims):
    # An operator with a zero extent has nothing to launch: the descriptor is
    # refused with RC_ERR_INVALID_ARGUMENT before any plan exists.
    with pytest.raises(rc.RCError) as e:
        rc.Op(kind, dims)
    assert e.value.status == rc.RC_ERR_INVALID_ARGUMENT
    assert "positive" in str(e.value)


def test_convolution_with_no_output_pixel_has_no_schedule():
    # a 3x3 filter over a 1x1 image without padding leaves no output pixel:
    # no schedule is legal, so not even P0 exists
    op = rc.Op(rc.RC_OP_CONV2D, (1, 1, 1, 64, 64, 3, 3, 0))
    with pytest.raises(rc.RCError) as e:
        op.default()
    assert e.value.status == rc.RC_ERR_UNSUPPORTED and "empty output" in str(e.value)
