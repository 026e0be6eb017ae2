"""CPU oracle for the schedule-parameterised contractions.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline may import this package; the product path never does.  It shares no
code with the HIP path (its C source is ``oracle/oracle.c``, built with gcc).

Every schedule is a semantics-preserving rewrite of its operator (Sec. 2,
Eq. 1), so the oracle is each operator's plain definition evaluated in fp64,
rounded only at the stated storage points (see ``oracle.c``).

Parity rule used by every comparison (the reading of "relative error scaled
by sqrt(K)"): with s the RMS of the oracle output, an output y matches the
oracle value r when |y - r| / max(|r|, s) <= tol.  For zero-mean operands
s ~ sqrt(K) * rms(a) * rms(b), which is where the sqrt(K) scaling enters;
pure elementwise relative error is undefined near r = 0.  tol is 1e-4 for
the fp32 GEMM and 2e-2 for bf16 inputs with fp32 accumulation.  Any NaN,
infinity or unwritten output fails.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "oracle.c")
_lib = None

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def build() -> str:
    subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", _LIB, _SRC, "-lm"])
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        vp, i64, ci = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        lib.orc_bf16_from_f64.argtypes = [ctypes.c_double]
        lib.orc_bf16_from_f64.restype = ctypes.c_uint16
        lib.orc_bf16_round.argtypes = [vp, vp, i64]
        lib.orc_silu.argtypes = [ctypes.c_double]
        lib.orc_silu.restype = ctypes.c_double
        lib.orc_gemm_f32.argtypes = [vp, vp, vp, vp, i64, i64, i64, vp, i64]
        lib.orc_attention_bf16.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, ci, vp, i64]
        lib.orc_gated_mlp_bf16.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, vp, i64]
        lib.orc_moe_bf16.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i64, i64, i64, i64, i64,
                                     vp, i64]
        lib.orc_conv2d_bf16.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64, i64, i64, i64,
                                        i64, ci, vp, i64]
        lib.orc_num_threads.restype = ci
        for f in (lib.orc_bf16_round, lib.orc_gemm_f32, lib.orc_attention_bf16,
                  lib.orc_gated_mlp_bf16, lib.orc_moe_bf16, lib.orc_conv2d_bf16):
            f.restype = None
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dt):
    a = np.ascontiguousarray(a, dtype=dt)
    return a


def _sel(sel):
    if sel is None:
        return None, 0
    s = np.ascontiguousarray(sel, dtype=np.int64)
    return s, len(s)


def num_threads() -> int:
    return int(_load().orc_num_threads())


def bf16_from_f64(x) -> np.ndarray:
    x = _c(np.atleast_1d(x), np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    _load().orc_bf16_round(_p(x), _p(out), x.size)
    return out


def bf16_to_f64(b) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(
        np.float32).astype(np.float64)


def silu(x: float) -> float:
    return float(_load().orc_silu(float(x)))


def gemm_f32(A, B, rows=None, want_f64=False):
    """C = A B (fp32 in, fp64 sums, fp32 out) on the selected rows of A."""
    A, B = _c(A, np.float32), _c(B, np.float32)
    M, K = A.shape
    K2, N = B.shape
    assert K == K2
    sel, n = _sel(rows)
    n = M if sel is None else n
    C = np.empty((n, N), dtype=np.float32)
    C64 = np.empty((n, N), dtype=np.float64) if want_f64 else None
    _load().orc_gemm_f32(_p(A), _p(B), _p(C), _p(C64), M, N, K, _p(sel), n)
    return (C, C64) if want_f64 else C


def attention_bf16(Q, K, V, causal=True, rows=None, want_f64=False):
    """Softmax attention, scale 1/sqrt(D); rows are flat (b*H+h)*S+i indices."""
    Q, K, V = (_c(t, np.uint16) for t in (Q, K, V))
    B, H, S, D = Q.shape
    sel, n = _sel(rows)
    n = B * H * S if sel is None else n
    O = np.empty((n, D), dtype=np.uint16)
    O64 = np.empty((n, D), dtype=np.float64) if want_f64 else None
    _load().orc_attention_bf16(_p(Q), _p(K), _p(V), _p(O), _p(O64), B, H, S, D, int(causal),
                               _p(sel), n)
    return (O, O64) if want_f64 else O


def gated_mlp_bf16(X, Wg, Wu, Wd, rows=None, want_f64=False, want_hidden=False):
    """out = bf16(bf16(SiLU(X Wg) * (X Wu)) Wd) on the selected tokens."""
    X, Wg, Wu, Wd = (_c(t, np.uint16) for t in (X, Wg, Wu, Wd))
    T, Hd = X.shape
    I = Wg.shape[1]
    sel, n = _sel(rows)
    n = T if sel is None else n
    Out = np.empty((n, Hd), dtype=np.uint16)
    Out64 = np.empty((n, Hd), dtype=np.float64) if want_f64 else None
    Hm = np.empty((n, I), dtype=np.uint16) if want_hidden else None
    _load().orc_gated_mlp_bf16(_p(X), _p(Wg), _p(Wu), _p(Wd), _p(Out), _p(Out64), _p(Hm), T, Hd,
                               I, _p(sel), n)
    res = [Out]
    if want_f64:
        res.append(Out64)
    if want_hidden:
        res.append(Hm)
    return res[0] if len(res) == 1 else tuple(res)


def moe_bf16(X, ids, w, Wg, Wu, Wd, rows=None, want_f64=False):
    """Routed gated-MLP experts combined with the routing weights."""
    X, Wg, Wu, Wd = (_c(t, np.uint16) for t in (X, Wg, Wu, Wd))
    ids, w = _c(ids, np.int32), _c(w, np.float32)
    T, Hd = X.shape
    E, _, I = Wg.shape
    topk = ids.shape[1]
    sel, n = _sel(rows)
    n = T if sel is None else n
    Out = np.empty((n, Hd), dtype=np.uint16)
    Out64 = np.empty((n, Hd), dtype=np.float64) if want_f64 else None
    _load().orc_moe_bf16(_p(X), _p(ids), _p(w), _p(Wg), _p(Wu), _p(Wd), _p(Out), _p(Out64), T,
                         Hd, E, I, topk, _p(sel), n)
    return (Out, Out64) if want_f64 else Out


def conv2d_bf16(x, w, bias, pad=1, act=True, pixels=None, want_f64=False):
    """NHWC x, KRSC w, stride 1; pixels are flat (n*P+p)*Q+q output indices."""
    x, w = _c(x, np.uint16), _c(w, np.uint16)
    b = None if bias is None else _c(bias, np.float32)
    N, H, W, C = x.shape
    K, R, S, C2 = w.shape
    assert C == C2
    P, Q = H + 2 * pad - R + 1, W + 2 * pad - S + 1
    sel, n = _sel(pixels)
    n = N * P * Q if sel is None else n
    y = np.empty((n, K), dtype=np.uint16)
    y64 = np.empty((n, K), dtype=np.float64) if want_f64 else None
    _load().orc_conv2d_bf16(_p(x), _p(w), _p(b), _p(y), _p(y64), N, H, W, C, K, R, S, pad,
                            int(act), _p(sel), n)
    return (y, y64) if want_f64 else y


def moe_routing_prep(ids, E, tile_up, tile_down):
    """Routing preparation of the MoE layer (integer index work): the routed
    rows (token, slot), flattened as r = token * topk + slot, grouped by
    expert.

    Returns a dict of int32 arrays:
      offsets [E + 1]   offsets[e] = number of routed rows of experts < e
                        (the exclusive prefix sum of the expert histogram);
      perm [R]          the rows sorted by expert, rows of one expert in
                        increasing r (a stable sort by expert id);
      pos [R]           the inverse permutation: perm[pos[r]] = r;
      tile_up, tile_down [E + 1]
                        first M tile of each expert when each expert's rows
                        are cut into tiles of tile_up / tile_down rows: the
                        exclusive prefix sum of ceil(count_e / tile).
    ids must lie in [0, E).
    """
    ids = np.asarray(ids, dtype=np.int64).reshape(-1)
    assert ids.size == 0 or (ids.min() >= 0 and ids.max() < E)
    counts = np.bincount(ids, minlength=E)
    offsets = np.concatenate([[0], np.cumsum(counts)])
    perm = np.argsort(ids, kind="stable")
    pos = np.empty_like(perm)
    pos[perm] = np.arange(ids.size)
    tu = np.concatenate([[0], np.cumsum(-(-counts // tile_up))])
    td = np.concatenate([[0], np.cumsum(-(-counts // tile_down))])
    i32 = lambda a: np.asarray(a, dtype=np.int32)
    return {"offsets": i32(offsets), "perm": i32(perm), "pos": i32(pos),
            "tile_up": i32(tu), "tile_down": i32(td)}


def compare(y, r, tol):
    """Parity rule: max |y - r| / max(|r|, rms(r)) <= tol, all outputs finite.

    y and r are float arrays of the same shape.  Returns (ok, worst, rms).
    """
    y = np.asarray(y, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    if y.shape != r.shape:
        return False, float("inf"), 0.0
    if not np.all(np.isfinite(y)):
        return False, float("inf"), 0.0
    s = float(np.sqrt(np.mean(r * r))) if r.size else 0.0
    if r.size == 0:
        return True, 0.0, 0.0
    denom = np.maximum(np.abs(r), s if s > 0 else 1.0)
    worst = float(np.max(np.abs(y - r) / denom))
    return worst <= tol, worst, s
