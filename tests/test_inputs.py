"""The seeded input generator: published SplitMix64 outputs, C/numpy
agreement, distributions and the workload recipes' shapes."""
import numpy as np
from scipy import stats

from paper_2506_01374_amd import inputs as gen


def test_splitmix64_published_sequence():
    # SplitMix64 started from state 0 (Steele, Lea and Flood; the reference
    # sequence is 0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F).
    with np.errstate(over="ignore"):
        st = np.arange(1, 4, dtype=np.uint64) * gen.GAMMA
        out = gen._mix64(st)
    assert [int(v) for v in out] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_c_generator_matches_numpy_counters():
    for seed, tid, start in [(0, 1, 0), (7, 22, 12345), (2 ** 40, 3, 10 ** 9)]:
        assert np.array_equal(gen.raw_u64(seed, tid, start, 5000),
                              gen.raw_u64_numpy(seed, tid, start, 5000))


def test_distributions():
    u = gen.uniform_f32(0, 1, (200_000,))
    assert u.min() >= -1 and u.max() < 1
    assert stats.kstest(u, "uniform", args=(-1, 2)).pvalue > 1e-3
    z = gen.normal_f32(0, 2, (200_000,))
    assert stats.kstest(z, "norm").pvalue > 1e-3
    w = gen.bf16_bits_to_f32(gen.normal_bf16(0, 3, (200_000,), 0.02))
    assert abs(w.std() - 0.02) < 0.0005 and abs(w.mean()) < 0.0005
    iv = gen.bf16_bits_to_f32(gen.int_valued_bf16(0, 4, (100_000,), 8))
    assert set(np.unique(iv).tolist()) == set(range(-8, 9))


def test_streams_are_distinct_and_thread_independent():
    a = gen.normal_bf16(0, 1, (1000,))
    b = gen.normal_bf16(0, 2, (1000,))
    c = gen.normal_bf16(1, 1, (1000,))
    assert not np.array_equal(a, b) and not np.array_equal(a, c)
    big = gen.normal_bf16(0, 1, (3_000_000,))
    assert np.array_equal(big[:1000], a)


def test_recipes_shapes():
    d = gen.conv_inputs(2, 8, 8, 32, 16, 3, 3)
    assert d["x"].shape == (2, 8, 8, 32) and d["w"].shape == (16, 3, 3, 32)
    assert d["bias"].dtype == np.float32
    m = gen.moe_inputs(64, 16, 8, 4, 2)
    assert m["ids"].dtype == np.int32 and m["w"].dtype == np.float32
    w = gen.mlp_inputs(4, 8, 12)["Wg"]
    assert np.array_equal(gen.to_nk(w).T, w)
