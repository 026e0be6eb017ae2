"""Pins for the CPU oracle: each check comes from mathematics or a library
routine, not from retyping the oracle's own loops, and is chosen so that a
dropped term, a wrong index, a transposed operand or a wrong rounding in the
oracle fails at least one of them."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2506_01374_amd import inputs as gen

torch.set_num_threads(8)


def f32(x):
    return np.asarray(x, dtype=np.float32)


def bf(x):
    return orc.bf16_from_f64(np.asarray(x, dtype=np.float64))


# --------------------------------------------------------------------------
# bf16 rounding (storage rule of every bf16 output)
# --------------------------------------------------------------------------

def test_bf16_rounding_special_values():
    assert orc.bf16_from_f64(1.0)[0] == 0x3F80
    assert orc.bf16_from_f64(1.0 + 2.0 ** -8)[0] == 0x3F80          # tie -> even (down)
    assert orc.bf16_from_f64(1.0 + 3 * 2.0 ** -8)[0] == 0x3F82      # tie -> even (up)
    assert orc.bf16_from_f64(1.0 + 2.0 ** -8 + 2.0 ** -40)[0] == 0x3F81
    assert orc.bf16_from_f64(-2.5)[0] == 0xC020
    assert orc.bf16_from_f64(3.4e38)[0] == 0x7F80                    # overflow -> inf
    assert orc.bf16_from_f64(-3.4e38)[0] == 0xFF80
    assert orc.bf16_from_f64(3.3895e38)[0] == 0x7F7F                 # largest finite
    assert orc.bf16_from_f64(3.38e38)[0] == 0x7F7E                   # below the midpoint
    assert orc.bf16_from_f64(float("nan"))[0] == 0x7FC0
    assert orc.bf16_from_f64(-0.0)[0] == 0x8000
    assert orc.bf16_from_f64(2.0 ** -133)[0] == 0x0001               # smallest subnormal
    assert orc.bf16_from_f64(2.0 ** -134)[0] == 0x0000               # tie -> even zero
    assert orc.bf16_from_f64(3 * 2.0 ** -134)[0] == 0x0002


def test_bf16_rounding_matches_independent_bit_rounding():
    # The generator rounds fp32 -> bf16 with an integer bit trick; the oracle
    # rounds fp64 -> bf16 with frexp/rint.  On fp32-representable values the
    # two independent implementations must agree exactly.
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 2 ** 32, size=200_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x)]
    x = np.concatenate([x, f32([0.0, 1.0, 1.00390625, 1.01171875, 65504.0, 1e-40, -1e-39])])
    a = orc.bf16_from_f64(x.astype(np.float64))
    b = gen.f32_to_bf16_bits(x)
    assert np.array_equal(a, b)


def test_silu_pins():
    assert orc.silu(0.0) == 0.0
    assert abs(orc.silu(1.0) - 1.0 / (1.0 + math.exp(-1.0))) < 1e-16
    for x in np.linspace(-30, 30, 121):
        assert abs((orc.silu(x) - orc.silu(-x)) - x) < 1e-12 * max(1, abs(x))
    grid = torch.linspace(-30, 30, 601, dtype=torch.float64)
    ref = torch.nn.functional.silu(grid).numpy()
    got = np.array([orc.silu(float(v)) for v in grid])
    assert np.max(np.abs(got - ref)) < 1e-13
    assert orc.silu(-800.0) == 0.0 and orc.silu(800.0) == 800.0


# --------------------------------------------------------------------------
# fp32 GEMM
# --------------------------------------------------------------------------

def test_gemm_ones_gives_k():
    for (M, N, K) in [(3, 5, 7), (16, 16, 128), (128, 128, 128)]:
        C = orc.gemm_f32(np.ones((M, K)), np.ones((K, N)))
        assert np.all(C == K)


def test_gemm_identity_and_permutation():
    B = gen.uniform_f32(0, 2, (32, 24))
    assert np.array_equal(orc.gemm_f32(np.eye(32), B), B)
    perm = np.random.default_rng(1).permutation(32)
    P = np.eye(32)[perm]
    assert np.array_equal(orc.gemm_f32(P, B), B[perm])
    # a transposed operand would fail on a non-square B
    A = gen.uniform_f32(0, 1, (7, 32))
    assert orc.gemm_f32(A, B).shape == (7, 24)


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (2, 3, 5), (5, 7, 17), (3, 2, 7)])
def test_gemm_exact_fractions(M, N, K):
    A = gen.uniform_f32(5, 1, (M, K))
    B = gen.uniform_f32(5, 2, (K, N))
    C, C64 = orc.gemm_f32(A, B, want_f64=True)
    for m in range(M):
        for n in range(N):
            exact = sum(Fraction(float(A[m, k])) * Fraction(float(B[k, n])) for k in range(K))
            bound = K * 2.0 ** -52 * sum(abs(float(A[m, k]) * float(B[k, n])) for k in range(K))
            assert abs(Fraction(C64[m, n]) - exact) <= Fraction(bound)
            # fp32 output is the correctly rounded value (up to the fp64 sum error)
            ulp = abs(float(np.spacing(np.float32(float(exact)))))
            assert abs(float(C[m, n]) - float(exact)) <= 0.5 * ulp + bound


def test_gemm_full_size_vs_numpy_f64():
    A = gen.uniform_f32(0, 1, (128, 128))
    B = gen.uniform_f32(0, 2, (128, 128))
    C, C64 = orc.gemm_f32(A, B, want_f64=True)
    ref = A.astype(np.float64) @ B.astype(np.float64)
    assert np.max(np.abs(C64 - ref)) < 1e-11
    assert np.array_equal(C, ref.astype(np.float32))
    rows = np.array([0, 17, 127])
    assert np.array_equal(orc.gemm_f32(A, B, rows=rows), C[rows])


def test_gemm_integer_inputs_exact():
    A = gen.int_valued_f32(0, 1, (64, 96), 4)
    B = gen.int_valued_f32(0, 2, (96, 48), 4)
    ref = A.astype(np.int64) @ B.astype(np.int64)
    assert np.array_equal(orc.gemm_f32(A, B), ref.astype(np.float32))


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------

def _sdpa64(Q, K, V, causal):
    q, k, v = (torch.from_numpy(orc.bf16_to_f64(t)) for t in (Q, K, V))
    return torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=causal).numpy()


def test_attention_hand_case():
    # D = 1 (scale 1): q = [1, 1], k = [1, 2], v = [2, 4].
    Q = bf(np.array([1.0, 1.0]).reshape(1, 1, 2, 1))
    K = bf(np.array([1.0, 2.0]).reshape(1, 1, 2, 1))
    V = bf(np.array([2.0, 4.0]).reshape(1, 1, 2, 1))
    _, o = orc.attention_bf16(Q, K, V, causal=True, want_f64=True)
    e = math.e
    assert abs(o[0, 0] - 2.0) < 1e-15
    assert abs(o[1, 0] - (2.0 + 4.0 * e) / (1.0 + e)) < 1e-14
    _, o = orc.attention_bf16(Q, K, V, causal=False, want_f64=True)
    assert abs(o[0, 0] - (2.0 + 4.0 * e) / (1.0 + e)) < 1e-14


def test_attention_first_row_is_v0_and_zero_query_prefix_mean():
    B, H, S, D = 1, 2, 64, 32
    d = gen.attention_inputs(B, H, S, D, seed=3)
    O = orc.attention_bf16(d["Q"], d["K"], d["V"], causal=True)
    O = O.reshape(B, H, S, D)
    assert np.array_equal(O[:, :, 0, :], d["V"][:, :, 0, :])
    Qz = np.zeros_like(d["Q"])
    _, o64 = orc.attention_bf16(Qz, d["K"], d["V"], causal=True, want_f64=True)
    v = orc.bf16_to_f64(d["V"])
    prefix = np.cumsum(v, axis=2) / np.arange(1, S + 1)[None, None, :, None]
    assert np.max(np.abs(o64.reshape(B, H, S, D) - prefix)) < 1e-12


def test_attention_dominant_key():
    B, H, S, D = 1, 1, 16, 8
    K = np.zeros((B, H, S, D)); K[0, 0, 5, 0] = 64.0
    Q = np.zeros((B, H, S, D)); Q[0, 0, :, 0] = 64.0
    V = gen.normal_bf16(0, 9, (B, H, S, D))
    _, o = orc.attention_bf16(bf(Q), bf(K), V, causal=True, want_f64=True)
    v = orc.bf16_to_f64(V)[0, 0]
    for i in range(5, S):
        assert np.max(np.abs(o[i] - v[5])) < 1e-12


@pytest.mark.parametrize("causal", [True, False])
def test_attention_vs_torch_sdpa_f64(causal):
    B, H, S, D = 1, 4, 256, 128
    d = gen.attention_inputs(B, H, S, D, seed=1)
    O, o64 = orc.attention_bf16(d["Q"], d["K"], d["V"], causal=causal, want_f64=True)
    ref = _sdpa64(d["Q"], d["K"], d["V"], causal).reshape(-1, D)
    assert np.max(np.abs(o64 - ref)) < 1e-12
    assert np.array_equal(O, orc.bf16_from_f64(ref))


def test_attention_row_subset_and_head_permutation():
    B, H, S, D = 1, 4, 64, 32
    d = gen.attention_inputs(B, H, S, D, seed=2)
    full = orc.attention_bf16(d["Q"], d["K"], d["V"]).reshape(H, S, D)
    perm = [2, 0, 3, 1]
    pq, pk, pv = (t[:, perm] for t in (d["Q"], d["K"], d["V"]))
    permuted = orc.attention_bf16(pq, pk, pv).reshape(H, S, D)
    assert np.array_equal(permuted, full[perm])
    rows = np.array([0, 63, 64 + 10, 3 * 64 + 40])
    sub = orc.attention_bf16(d["Q"], d["K"], d["V"], rows=rows)
    assert np.array_equal(sub, full.reshape(-1, D)[rows])


# --------------------------------------------------------------------------
# gated MLP
# --------------------------------------------------------------------------

def _mlp_torch(X, Wg, Wu, Wd):
    x, g, u, d = (torch.from_numpy(orc.bf16_to_f64(t)) for t in (X, Wg, Wu, Wd))
    h = torch.nn.functional.silu(x @ g) * (x @ u)
    hb = torch.from_numpy(orc.bf16_to_f64(orc.bf16_from_f64(h.numpy())))
    return (hb @ d).numpy(), h.numpy()


def test_mlp_zero_cases():
    d = gen.mlp_inputs(8, 32, 48)
    assert np.all(orc.gated_mlp_bf16(np.zeros_like(d["X"]), d["Wg"], d["Wu"], d["Wd"]) & 0x7FFF == 0)
    assert np.all(orc.gated_mlp_bf16(d["X"], d["Wg"], np.zeros_like(d["Wu"]), d["Wd"]) & 0x7FFF == 0)


def test_mlp_vs_torch_composite():
    d = gen.mlp_inputs(16, 64, 96, seed=4, wsigma=0.1)
    out, o64, hid = orc.gated_mlp_bf16(d["X"], d["Wg"], d["Wu"], d["Wd"], want_f64=True,
                                       want_hidden=True)
    ref, h = _mlp_torch(d["X"], d["Wg"], d["Wu"], d["Wd"])
    assert np.max(np.abs(o64 - ref)) < 1e-10 * max(1.0, np.abs(ref).max())
    # the hidden activation is the bf16 rounding of SiLU(g) * u
    hb = orc.bf16_from_f64(h)
    assert np.mean(hb == hid) > 0.999
    assert np.max(np.abs(orc.bf16_to_f64(hid) - orc.bf16_to_f64(hb))) <= np.abs(h).max() * 2 ** -7


def test_mlp_identity_down_projection_returns_hidden():
    T, Hd = 8, 32
    d = gen.mlp_inputs(T, Hd, Hd, seed=6, wsigma=0.2)
    eye = bf(np.eye(Hd))
    out, hid = orc.gated_mlp_bf16(d["X"], d["Wg"], d["Wu"], eye, want_hidden=True)
    assert np.array_equal(out, hid)


def test_mlp_gate_saturation_gives_product():
    # A large positive gate makes SiLU(g) = g, so h = g * u exactly in fp64.
    T, Hd, I = 4, 16, 8
    X = bf(np.ones((T, Hd)))
    Wg = bf(np.full((Hd, I), 4.0))            # g = 64 for every unit
    Wu = gen.int_valued_bf16(0, 3, (Hd, I), 2)
    eye = bf(np.eye(I, Hd))
    out = orc.gated_mlp_bf16(X, Wg, Wu, eye[:, :Hd] if I == Hd else bf(np.eye(I, Hd)))
    u = orc.bf16_to_f64(Wu).sum(axis=0)
    expect = np.zeros((T, Hd)); expect[:, :I] = orc.silu(64.0) * u
    assert np.array_equal(out, orc.bf16_from_f64(expect))


# --------------------------------------------------------------------------
# MoE
# --------------------------------------------------------------------------

def test_routing_invariants():
    d = gen.moe_inputs(512, 16, 64, 8, 6)
    ids, w = d["ids"], d["w"]
    assert ids.shape == (512, 6)
    for t in range(512):
        assert len(set(ids[t].tolist())) == 6
        assert np.all(np.diff(w[t]) <= 0)
    counts = np.bincount(ids.ravel(), minlength=64)
    assert counts.sum() == 512 * 6
    # ties go to the lower expert index
    ids2, w2 = gen.moe_route(np.zeros((2, 8), dtype=np.float32), 3)
    assert ids2.tolist() == [[0, 1, 2], [0, 1, 2]]
    assert np.allclose(w2, 1.0 / 8)
    lg = np.array([[0.0, 2.0, 1.0, 2.0]], dtype=np.float32)
    ids3, w3 = gen.moe_route(lg, 2)
    assert ids3.tolist() == [[1, 3]]
    p = np.exp(lg[0] - 2.0) / np.exp(lg[0] - 2.0).sum()
    assert np.allclose(w3[0], [p[1], p[3]])


def test_routing_prep_brute_force_and_invariants():
    # Sorting the routed rows by expert, written out by hand: for each expert
    # in order, the rows routed to it in order of r = token * topk + slot.
    for seed, (T, E, k, tu, td) in enumerate([(37, 8, 2, 4, 3), (512, 64, 6, 256, 128),
                                              (5, 16, 3, 16, 16), (64, 3, 1, 1, 2)]):
        ids = gen.moe_inputs(T, 4, E, 4, k, seed=seed)["ids"]
        got = orc.moe_routing_prep(ids, E, tu, td)
        flat = ids.reshape(-1).tolist()
        perm = [r for e in range(E) for r in range(len(flat)) if flat[r] == e]
        assert got["perm"].tolist() == perm
        off, t_up, t_dn = [0], [0], [0]
        for e in range(E):
            c = flat.count(e)
            off.append(off[-1] + c)
            t_up.append(t_up[-1] + (c + tu - 1) // tu)
            t_dn.append(t_dn[-1] + (c + td - 1) // td)
        assert got["offsets"].tolist() == off
        assert got["tile_up"].tolist() == t_up and got["tile_down"].tolist() == t_dn
        # invariants: offsets monotone, perm a bijection, pos its inverse,
        # each expert's rows in its own range
        assert np.all(np.diff(got["offsets"]) >= 0) and got["offsets"][-1] == T * k
        assert sorted(got["perm"].tolist()) == list(range(T * k))
        assert np.array_equal(got["perm"][got["pos"]], np.arange(T * k))
        for e in range(E):
            rows = got["perm"][off[e]:off[e + 1]]
            assert all(flat[r] == e for r in rows) and np.all(np.diff(rows) > 0)
    # a planted mistake (an unstable order) is caught by the stability check
    ids = np.array([[1, 0], [1, 0]], dtype=np.int32)
    assert orc.moe_routing_prep(ids, 2, 1, 1)["perm"].tolist() == [1, 3, 0, 2]


def test_moe_forced_routing_equals_dense_mlp():
    T, Hd, E, I = 8, 32, 4, 16
    d = gen.moe_inputs(T, Hd, E, I, 1, seed=2, wsigma=0.2)
    for e in (0, 3):
        ids = np.full((T, 1), e, dtype=np.int32)
        w = np.ones((T, 1), dtype=np.float32)
        got = orc.moe_bf16(d["X"], ids, w, d["Wg"], d["Wu"], d["Wd"])
        ref = orc.gated_mlp_bf16(d["X"], d["Wg"][e], d["Wu"][e], d["Wd"][e])
        assert np.array_equal(got, ref)


def test_moe_weight_linearity():
    T, Hd, E, I, k = 6, 16, 4, 8, 2
    d = gen.moe_inputs(T, Hd, E, I, k, seed=3, wsigma=0.2)
    _, a = orc.moe_bf16(d["X"], d["ids"], d["w"], d["Wg"], d["Wu"], d["Wd"], want_f64=True)
    _, b = orc.moe_bf16(d["X"], d["ids"], d["w"] * 0.5, d["Wg"], d["Wu"], d["Wd"], want_f64=True)
    assert np.max(np.abs(b - 0.5 * a)) < 1e-14 * max(1, np.abs(a).max())
    # two slots on the same expert add their weights
    ids = np.repeat(d["ids"][:, :1], 2, axis=1)
    w = np.stack([d["w"][:, 0], d["w"][:, 1]], axis=1)
    _, two = orc.moe_bf16(d["X"], ids, w, d["Wg"], d["Wu"], d["Wd"], want_f64=True)
    _, one = orc.moe_bf16(d["X"], ids[:, :1], (w[:, :1] + w[:, 1:]).astype(np.float32),
                          d["Wg"], d["Wu"], d["Wd"], want_f64=True)
    assert np.max(np.abs(two - one)) < 1e-6 * max(1, np.abs(one).max())


def test_moe_tiny_brute_force_vs_torch():
    T, Hd, E, I, k = 5, 8, 4, 4, 2
    d = gen.moe_inputs(T, Hd, E, I, k, seed=7, wsigma=0.5)
    _, got = orc.moe_bf16(d["X"], d["ids"], d["w"], d["Wg"], d["Wu"], d["Wd"], want_f64=True)
    x = torch.from_numpy(orc.bf16_to_f64(d["X"]))
    ref = torch.zeros(T, Hd, dtype=torch.float64)
    for t in range(T):
        for s in range(k):
            e = int(d["ids"][t, s])
            g = x[t] @ torch.from_numpy(orc.bf16_to_f64(d["Wg"][e]))
            u = x[t] @ torch.from_numpy(orc.bf16_to_f64(d["Wu"][e]))
            h = torch.nn.functional.silu(g) * u
            h = torch.from_numpy(orc.bf16_to_f64(orc.bf16_from_f64(h.numpy())))
            ref[t] += float(d["w"][t, s]) * (h @ torch.from_numpy(orc.bf16_to_f64(d["Wd"][e])))
    assert np.max(np.abs(got - ref.numpy())) < 1e-12


# --------------------------------------------------------------------------
# convolution
# --------------------------------------------------------------------------

def test_conv_ones_pins_padding():
    N, H, W, C, K = 1, 8, 8, 320, 4
    x = bf(np.ones((N, H, W, C)))
    w = bf(np.ones((K, 3, 3, C)))
    y = orc.conv2d_bf16(x, w, None, pad=1, act=False).reshape(N, H, W, K)
    v = orc.bf16_to_f64(y)
    assert np.all(v[0, 1:-1, 1:-1] == 2880)
    assert np.all(v[0, 0, 1:-1] == 1920) and np.all(v[0, -1, 1:-1] == 1920)
    assert np.all(v[0, 1:-1, 0] == 1920) and np.all(v[0, 1:-1, -1] == 1920)
    for (p, q) in [(0, 0), (0, -1), (-1, 0), (-1, -1)]:
        assert np.all(v[0, p, q] == 1280)


def test_conv_delta_kernel_is_identity_plus_bias():
    N, H, W, C = 2, 6, 5, 8
    x = gen.normal_bf16(0, 1, (N, H, W, C))
    w = np.zeros((C, 3, 3, C)); w[np.arange(C), 1, 1, np.arange(C)] = 1.0
    bias = gen.normal_f32(0, 2, (C,))
    _, y64 = orc.conv2d_bf16(x, bf(w), bias, pad=1, act=False, want_f64=True)
    expect = orc.bf16_to_f64(x).reshape(-1, C) + bias.astype(np.float64)[None, :]
    assert np.array_equal(y64, expect)


def test_conv_vs_torch_conv2d_and_im2col():
    N, H, W, C, K = 2, 9, 7, 24, 16
    d = gen.conv_inputs(N, H, W, C, K, 3, 3, seed=5)
    y, y64 = orc.conv2d_bf16(d["x"], d["w"], d["bias"], pad=1, act=True, want_f64=True)
    x = torch.from_numpy(orc.bf16_to_f64(d["x"])).permute(0, 3, 1, 2)
    w = torch.from_numpy(orc.bf16_to_f64(d["w"])).permute(0, 3, 1, 2)
    pre = torch.nn.functional.conv2d(x, w, torch.from_numpy(d["bias"].astype(np.float64)),
                                     padding=1)
    ref = torch.nn.functional.silu(pre).permute(0, 2, 3, 1).reshape(-1, K).numpy()
    assert np.max(np.abs(y64 - ref)) < 1e-12
    # the same pre-activation as a GEMM over an explicitly built im2col matrix
    xp = np.pad(orc.bf16_to_f64(d["x"]), ((0, 0), (1, 1), (1, 1), (0, 0)))
    cols = np.stack([xp[:, r:r + H, s:s + W, :] for r in range(3) for s in range(3)], axis=3)
    A = cols.reshape(N * H * W, 9 * C)
    Bm = orc.bf16_to_f64(d["w"]).reshape(K, 9 * C).T
    _, pre64 = orc.conv2d_bf16(d["x"], d["w"], d["bias"], pad=1, act=False, want_f64=True)
    assert np.max(np.abs(pre64 - (A @ Bm + d["bias"].astype(np.float64)))) < 1e-12
    pix = np.array([0, 5, 62, N * H * W - 1])
    assert np.array_equal(orc.conv2d_bf16(d["x"], d["w"], d["bias"], pixels=pix), y[pix])


# --------------------------------------------------------------------------
# parity rule
# --------------------------------------------------------------------------

def test_compare_rule():
    r = np.array([1.0, -2.0, 0.0, 1e-6])
    ok, worst, s = orc.compare(r, r, 1e-4)
    assert ok and worst == 0.0
    s_exp = math.sqrt(np.mean(r * r))
    ok, worst, _ = orc.compare(r + np.array([0, 0, 1e-5 * s_exp, 0]), r, 1e-4)
    assert ok and abs(worst - 1e-5) < 1e-12
    assert not orc.compare(np.array([1.0, -2.0, np.nan, 0.0]), r, 1e-4)[0]
    assert not orc.compare(r * 1.01, r, 1e-4)[0]
