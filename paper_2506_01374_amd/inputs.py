"""Seeded synthetic inputs for every workload.

This module only draws numbers and moves bytes: it holds none of the
operators' arithmetic.  Both the HIP path and the CPU oracle read the buffers
it fills, so the two sides see bit-identical inputs by construction.

Generator: counter-based SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014).  Element ``i`` of tensor
``tid`` under ``seed`` is ``mix64(key(seed, tid) + (i + 1) * GAMMA)``.
Uniform doubles take the top 53 bits.  Normals use the Box-Muller transform
on two consecutive counters (2i, 2i+1).  Values are rounded fp64 -> fp32
(round to nearest even) and, for bf16 tensors, fp32 -> bf16 (round to
nearest even on the bit pattern).

MoE routing (softmax over router logits, top-k, ties to the lower expert
index, weights not renormalised) is input preparation: it decides which
expert rows each token visits, and both sides receive its result.
"""
from __future__ import annotations

import numpy as np

import ctypes
import os
import subprocess

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_SRC_PATH = os.path.join(_HERE, "csrc", "synth.c")
_lib = None


def build_synth() -> str:
    """Compile the generator library (plain C, OpenMP)."""
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", _LIB_PATH,
                           _SRC_PATH, "-lm"])
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build_synth()
        lib = ctypes.CDLL(_LIB_PATH)
        u64, i64, i32, dbl, vp = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_double, ctypes.c_void_p)
        lib.synth_u64.argtypes = [u64, u64, i64, i64, vp]
        lib.synth_uniform_f32.argtypes = [u64, u64, i64, dbl, dbl, vp]
        lib.synth_normal_f32.argtypes = [u64, u64, i64, dbl, vp]
        lib.synth_normal_bf16.argtypes = [u64, u64, i64, dbl, vp]
        lib.synth_int_bf16.argtypes = [u64, u64, i64, i32, vp]
        lib.synth_int_f32.argtypes = [u64, u64, i64, i32, vp]
        for f in (lib.synth_u64, lib.synth_uniform_f32, lib.synth_normal_f32,
                  lib.synth_normal_bf16, lib.synth_int_bf16, lib.synth_int_f32):
            f.restype = None
        _lib = lib
    return _lib


def _mix64(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def raw_u64_numpy(seed: int, tid: int, start: int, count: int) -> np.ndarray:
    """SplitMix64 outputs computed in numpy (used to cross-check the C side)."""
    with np.errstate(over="ignore"):
        key = _mix64(np.array([(seed * 0x100000001B3 + tid * 0x9E3779B1) & 0xFFFFFFFFFFFFFFFF],
                              dtype=np.uint64))[0]
        idx = np.arange(start + 1, start + count + 1, dtype=np.uint64)
        return _mix64(key + idx * GAMMA)


def raw_u64(seed: int, tid: int, start: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.uint64)
    _load().synth_u64(seed, tid, start, count, out.ctypes.data)
    return out


def uniform_f32(seed: int, tid: int, shape, lo: float = -1.0, hi: float = 1.0) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    _load().synth_uniform_f32(seed, tid, out.size, lo, hi, out.ctypes.data)
    return out


def normal_f32(seed: int, tid: int, shape, sigma: float = 1.0) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    _load().synth_normal_f32(seed, tid, out.size, sigma, out.ctypes.data)
    return out


def normal_bf16(seed: int, tid: int, shape, sigma: float = 1.0) -> np.ndarray:
    out = np.empty(shape, dtype=np.uint16)
    _load().synth_normal_bf16(seed, tid, out.size, sigma, out.ctypes.data)
    return out


def int_valued_bf16(seed: int, tid: int, shape, a: int) -> np.ndarray:
    """Integers uniform in [-a, a] as bf16 bits, for exact-arithmetic checks."""
    out = np.empty(shape, dtype=np.uint16)
    _load().synth_int_bf16(seed, tid, out.size, a, out.ctypes.data)
    return out


def int_valued_f32(seed: int, tid: int, shape, a: int) -> np.ndarray:
    out = np.empty(shape, dtype=np.float32)
    _load().synth_int_f32(seed, tid, out.size, a, out.ctypes.data)
    return out


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    r = r.astype(np.uint16)
    r[nan] = np.uint16(0x7FC0)
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def moe_route(logits: np.ndarray, topk: int):
    """Top-k experts per token from softmax(logits), ties to the lower index.

    Returns (ids int32 [T, k], weights fp32 [T, k]); weights are the softmax
    probabilities of the chosen experts, not renormalised.
    """
    lg = np.asarray(logits, dtype=np.float64)
    p = np.exp(lg - lg.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    order = np.argsort(-p, axis=1, kind="stable")[:, :topk]
    w = np.take_along_axis(p, order, axis=1)
    return order.astype(np.int32), w.astype(np.float32)


def to_nk(w_kn: np.ndarray) -> np.ndarray:
    """Store a logical [.., K, N] weight as [.., N, K] (K contiguous)."""
    return np.ascontiguousarray(np.swapaxes(w_kn, -1, -2))


# ---------------------------------------------------------------------------
# Workload recipes.  Tensor ids are fixed per workload so every consumer
# draws the same numbers.
# ---------------------------------------------------------------------------

def gemm_f32_inputs(M, N, K, seed=0):
    return {"A": uniform_f32(seed, 1, (M, K)), "B": uniform_f32(seed, 2, (K, N))}


def attention_inputs(B, H, S, D, seed=0):
    return {"Q": normal_bf16(seed, 11, (B, H, S, D)),
            "K": normal_bf16(seed, 12, (B, H, S, D)),
            "V": normal_bf16(seed, 13, (B, H, S, D))}


def mlp_inputs(T, Hd, I, seed=0, wsigma=0.02):
    return {"X": normal_bf16(seed, 21, (T, Hd)),
            "Wg": normal_bf16(seed, 22, (Hd, I), wsigma),
            "Wu": normal_bf16(seed, 23, (Hd, I), wsigma),
            "Wd": normal_bf16(seed, 24, (I, Hd), wsigma)}


def moe_inputs(T, Hd, E, I, topk, seed=0, wsigma=0.02):
    logits = normal_f32(seed, 35, (T, E))
    ids, w = moe_route(logits, topk)
    return {"X": normal_bf16(seed, 31, (T, Hd)),
            "Wg": normal_bf16(seed, 32, (E, Hd, I), wsigma),
            "Wu": normal_bf16(seed, 33, (E, Hd, I), wsigma),
            "Wd": normal_bf16(seed, 34, (E, I, Hd), wsigma),
            "ids": ids, "w": w}


def conv_inputs(N, H, W, C, K, R, S, seed=0):
    return {"x": normal_bf16(seed, 41, (N, H, W, C)),
            "w": normal_bf16(seed, 42, (K, R, S, C), 1.0 / np.sqrt(R * S * C)),
            "bias": normal_f32(seed, 43, (K,))}
