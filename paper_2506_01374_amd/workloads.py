"""Named workloads (operator shapes of the paper's layer kinds) and the
placement of their seeded inputs on the device in a schedule's layout.

Shapes: fp32 GEMM 128^3 (the contraction of the App. A example module,
scaled down); Llama-3-8B-style causal attention 1 x 32 heads x 1024 x 128;
Llama-4-Scout-style gated MLP 2048 x 4096 x 14336; DeepSeek-style MoE with
4096 tokens, hidden 2048, 64 experts of intermediate 1408, top-6; FLUX-style
3x3 convolution 2 x 64 x 64 x 320 -> 320; FLUX-style bidirectional (no
mask) self-attention 1 x 24 heads x 4096 x 128, the image tokens of a
1024 x 1024 image (Sec. 4.1 names the layers; it prints no shapes, so these
are chosen stand-ins); and the App. A example module at its printed size,
C[1, 16, 2048] = A[1, 16, 7168] B[7168, 2048] in fp32 (one expert
projection of an MoE layer for 16 decode tokens).  All inputs are synthetic
and seeded (see ``inputs``).
"""
from __future__ import annotations

from typing import Dict, List, Tuple

import numpy as np

from . import inputs as gen
from . import rc

WORKLOADS: Dict[str, Tuple[int, Tuple[int, ...], int]] = {
    "gemm_f32_128": (rc.RC_OP_GEMM_F32, (128, 128, 128), 0),
    "attention_causal_b1_h32_s1024_d128": (rc.RC_OP_ATTENTION, (1, 32, 1024, 128), rc.RC_FLAG_CAUSAL),
    "gated_mlp_t2048_h4096_i14336": (rc.RC_OP_GATED_MLP, (2048, 4096, 14336), 0),
    "moe_t4096_h2048_e64_i1408_top6": (rc.RC_OP_MOE, (4096, 2048, 64, 1408, 6), 0),
    "conv3x3_n2_64x64_c320_k320": (rc.RC_OP_CONV2D, (2, 64, 64, 320, 320, 3, 3, 1), 0),
    "attention_noncausal_b1_h24_s4096_d128": (rc.RC_OP_ATTENTION, (1, 24, 4096, 128), 0),
    "gemm_f32_m16_n2048_k7168": (rc.RC_OP_GEMM_F32, (16, 2048, 7168), 0),
}


def op_for(kind: int, dims, flags: int = 0) -> rc.Op:
    return rc.Op(kind, dims, flags)


def workload_op(name: str) -> rc.Op:
    kind, dims, flags = WORKLOADS[name]
    return rc.Op(kind, dims, flags)


def host_inputs(op: rc.Op, seed: int = 0) -> Dict[str, np.ndarray]:
    """Seeded inputs in logical layouts (the oracle's layouts)."""
    d = op.dims
    if op.kind == rc.RC_OP_GEMM_F32:
        return gen.gemm_f32_inputs(d[0], d[1], d[2], seed)
    if op.kind == rc.RC_OP_ATTENTION:
        return gen.attention_inputs(*d, seed=seed)
    if op.kind == rc.RC_OP_GATED_MLP:
        return gen.mlp_inputs(*d, seed=seed)
    if op.kind == rc.RC_OP_MOE:
        return gen.moe_inputs(*d, seed=seed)
    if op.kind == rc.RC_OP_CONV2D:
        N, H, W, C, K, R, S, _ = d
        return gen.conv_inputs(N, H, W, C, K, R, S, seed)
    raise ValueError(op.kind)


def output_shape(op: rc.Op) -> Tuple[Tuple[int, ...], str]:
    d = op.dims
    if op.kind == rc.RC_OP_GEMM_F32:
        return (d[0], d[1]), "float32"
    if op.kind == rc.RC_OP_ATTENTION:
        return tuple(d), "bfloat16"
    if op.kind == rc.RC_OP_GATED_MLP:
        return (d[0], d[1]), "bfloat16"
    if op.kind == rc.RC_OP_MOE:
        return (d[0], d[1]), "bfloat16"
    N, H, W, C, K, R, S, pad = d
    return (N, H + 2 * pad - R + 1, W + 2 * pad - S + 1, K), "bfloat16"


def _stored(w: np.ndarray, layout: int) -> np.ndarray:
    """Weights are logically [..., K, N]; layout 1 stores them [..., N, K]."""
    return gen.to_nk(w) if layout == 1 else np.ascontiguousarray(w)


def stored_inputs(op: rc.Op, sched: rc.Schedule, host: Dict[str, np.ndarray]) -> List[np.ndarray]:
    """Host arrays in the order and storage layout rc_launch expects."""
    k = sched.as_dict()
    if op.kind == rc.RC_OP_GEMM_F32:
        return [host["A"], _stored(host["B"], k["layout"])]
    if op.kind == rc.RC_OP_ATTENTION:
        return [host["Q"], host["K"], host["V"]]
    if op.kind == rc.RC_OP_GATED_MLP:
        return [host["X"], _stored(host["Wg"], k["up.layout"]), _stored(host["Wu"], k["up.layout"]),
                _stored(host["Wd"], k["down.layout"])]
    if op.kind == rc.RC_OP_MOE:
        return [host["X"], host["ids"], host["w"], _stored(host["Wg"], k["up.layout"]),
                _stored(host["Wu"], k["up.layout"]), _stored(host["Wd"], k["down.layout"])]
    if op.kind == rc.RC_OP_CONV2D:
        w = host["w"]                     # [K][R][S][C] = logical [N][Kred]
        if k["layout"] == 0:
            w = np.ascontiguousarray(np.transpose(w, (1, 2, 3, 0)))   # [R][S][C][K]
        return [host["x"], w, host["bias"]]
    raise ValueError(op.kind)


def to_device(arrs: List[np.ndarray], device="cuda"):
    import torch
    out = []
    for a in arrs:
        t = torch.from_numpy(np.ascontiguousarray(a))
        if a.dtype == np.uint16:
            t = t.view(torch.bfloat16) if hasattr(torch, "bfloat16") else t
        out.append(t.to(device))
    return out


def empty_output(op: rc.Op, device="cuda", fill_nan=True):
    import torch
    shape, dt = output_shape(op)
    dtype = torch.float32 if dt == "float32" else torch.bfloat16
    t = torch.empty(shape, dtype=dtype, device=device)
    if fill_nan:
        t.fill_(float("nan"))
    return t


def output_to_f64(op: rc.Op, t) -> np.ndarray:
    import torch
    a = t.detach().cpu()
    if a.dtype == torch.bfloat16:
        return gen.bf16_bits_to_f32(a.view(torch.int16).numpy().view(np.uint16)).astype(np.float64)
    return a.numpy().astype(np.float64)
