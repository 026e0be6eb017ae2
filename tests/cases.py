"""Operator shapes and schedules exercised by the GPU parity tests.

Small shapes span several tiles (and ragged expert groups for the MoE) so
the oracle finishes in seconds; the full-size workloads are checked on
sampled outputs in the schedules the benchmark times.
"""
import json
import os

from paper_2506_01374_amd import rc, workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
TUNED = json.load(open(os.path.join(ROOT, "paper_2506_01374_amd", "tuned.json")))

SMALL = {
    "gemm": (rc.RC_OP_GEMM_F32, (128, 128, 128), 0),
    # decode-shaped fp32 contractions (streaming stage, K splits): a full
    # 16-row MFMA block, and 5 rows (padded inside the block)
    "gemm_skinny": (rc.RC_OP_GEMM_F32, (16, 256, 1024), 0),
    "gemm_skinny5": (rc.RC_OP_GEMM_F32, (5, 128, 512), 0),
    # ragged tails: no tile size divides M, N or K
    "gemm_ragged": (rc.RC_OP_GEMM_F32, (100, 72, 52), 0),
    "gemm_ragged_odd": (rc.RC_OP_GEMM_F32, (37, 50, 30), 0),
    "attn_causal": (rc.RC_OP_ATTENTION, (1, 2, 256, 128), rc.RC_FLAG_CAUSAL),
    "attn_full": (rc.RC_OP_ATTENTION, (1, 2, 256, 128), 0),
    "attn_d64": (rc.RC_OP_ATTENTION, (2, 1, 128, 64), rc.RC_FLAG_CAUSAL),
    # ragged sequences: no block divides S, so the last query and key tiles
    # are partial
    "attn_ragged_causal": (rc.RC_OP_ATTENTION, (1, 2, 200, 128), rc.RC_FLAG_CAUSAL),
    "attn_ragged_full": (rc.RC_OP_ATTENTION, (1, 2, 200, 128), 0),
    "attn_ragged_d64": (rc.RC_OP_ATTENTION, (2, 1, 77, 64), rc.RC_FLAG_CAUSAL),
    "mlp": (rc.RC_OP_GATED_MLP, (256, 256, 512), 0),
    # odd numbers of K tiles (3 for gate/up, 5 for down) for the ping-pong loop
    "mlp_odd": (rc.RC_OP_GATED_MLP, (256, 192, 320), 0),
    # ragged token count: no tile_m divides T = 200, so every schedule ends
    # in a partial M tile (both GEMMs)
    "mlp_ragged": (rc.RC_OP_GATED_MLP, (200, 256, 512), 0),
    "moe": (rc.RC_OP_MOE, (256, 256, 8, 128, 2), 0),
    "conv": (rc.RC_OP_CONV2D, (2, 16, 12, 64, 64, 3, 3, 1), 0),
    # 90 output pixels: a partial last M tile for every tile_m
    "conv_ragged": (rc.RC_OP_CONV2D, (1, 10, 9, 64, 64, 3, 3, 1), 0),
    # 320 output channels: the tile_n values 80, 160 and 320 that only
    # this channel count admits
    "conv_k320": (rc.RC_OP_CONV2D, (1, 8, 8, 64, 320, 3, 3, 1), 0),
    # 512 keys: work items of 8 key tiles
    "attn_causal_512": (rc.RC_OP_ATTENTION, (1, 2, 512, 128), rc.RC_FLAG_CAUSAL),
    # degenerate sizes: one row, one token, one key, one output pixel
    "gemm_one": (rc.RC_OP_GEMM_F32, (1, 1, 1), 0),
    "gemm_row": (rc.RC_OP_GEMM_F32, (1, 300, 77), 0),
    "attn_one_causal": (rc.RC_OP_ATTENTION, (1, 2, 1, 128), rc.RC_FLAG_CAUSAL),
    "attn_one_full": (rc.RC_OP_ATTENTION, (1, 2, 1, 128), 0),
    "mlp_one": (rc.RC_OP_GATED_MLP, (1, 256, 512), 0),
    # more workgroups than one round: the tail split of the gate/up GEMM
    # (I = 2304) and of the down GEMM (Hd = 576) runs a second launch
    "mlp_tail": (rc.RC_OP_GATED_MLP, (256, 256, 2304), 0),
    "mlp_tail_down": (rc.RC_OP_GATED_MLP, (1024, 576, 256), 0),
    "moe_one": (rc.RC_OP_MOE, (1, 256, 8, 128, 2), 0),
    "conv_one": (rc.RC_OP_CONV2D, (1, 1, 1, 64, 64, 3, 3, 1), 0),
}

_GEMM_BLOCK = ("tile_m", "tile_n", "tile_k", "waves_m", "waves_n", "mfma", "stages", "vec",
               "unroll", "layout", "grid", "occ")


def _block(prefix, tm, tn, tk, wm, wn, mf, st, vec, un, lay, grid, occ=1):
    vals = (tm, tn, tk, wm, wn, mf, st, vec, un, lay, grid, occ)
    return ",".join(f"{prefix}{k}={v}" for k, v in zip(_GEMM_BLOCK, vals))


def gemm_sweep():
    """The 18-point fp32 sweep: tile 16/32/64 (M and N) x vector width 1/4."""
    out = []
    for tm in (16, 32, 64):
        for tn in (16, 32, 64):
            for vec in (1, 4):
                out.append(f"tile_m={tm},tile_n={tn},tile_k=16,waves_m=1,waves_n=1,vec={vec},"
                           f"stages=2,unroll=1,layout=0")
    return out


SCHEDULES = {
    "gemm": gemm_sweep() + [
        "",   # P0
        "tile_m=64,tile_n=64,tile_k=32,waves_m=2,waves_n=2,vec=4,stages=2,unroll=2,layout=1",
        "tile_m=32,tile_n=64,tile_k=8,waves_m=2,waves_n=1,vec=1,stages=1,unroll=4,layout=1",
        "tile_m=64,tile_n=32,tile_k=4,waves_m=1,waves_n=2,vec=1,stages=2,unroll=1,layout=0",
    ],
    "gemm_ragged": [
        "",
        "tile_m=32,tile_n=32,tile_k=16,waves_m=1,waves_n=1,vec=4,stages=2,unroll=1,layout=0",
        "tile_m=64,tile_n=64,tile_k=32,waves_m=2,waves_n=2,vec=4,stages=2,unroll=2,layout=1",
        "tile_m=16,tile_n=16,tile_k=8,waves_m=1,waves_n=1,vec=1,stages=1,unroll=1,layout=0",
        "tile_m=64,tile_n=32,tile_k=4,waves_m=1,waves_n=2,vec=1,stages=2,unroll=1,layout=0",
    ],
    "gemm_ragged_odd": [
        "",
        "tile_m=16,tile_n=16,tile_k=16,waves_m=1,waves_n=1,vec=1,stages=2,unroll=1,layout=0",
        "tile_m=32,tile_n=64,tile_k=8,waves_m=2,waves_n=1,vec=1,stages=1,unroll=4,layout=0",
        "tile_m=64,tile_n=32,tile_k=16,waves_m=2,waves_n=2,vec=1,stages=2,unroll=1,layout=1",
    ],
    "gemm_skinny": [
        "",
        "tile_m=16,tile_n=64,tile_k=32,waves_m=2,waves_n=2,vec=4,stages=3,unroll=1,layout=0,splits=8",
        "tile_m=16,tile_n=64,tile_k=16,waves_m=1,waves_n=1,vec=4,stages=3,unroll=2,layout=0,splits=1",
        "tile_m=16,tile_n=64,tile_k=16,waves_m=1,waves_n=2,vec=4,stages=3,unroll=1,layout=0,splits=4",
        "tile_m=16,tile_n=64,tile_k=32,waves_m=2,waves_n=1,vec=4,stages=3,unroll=2,layout=0,splits=2",
        "tile_m=16,tile_n=64,tile_k=16,waves_m=2,waves_n=2,vec=4,stages=3,unroll=1,layout=0,splits=16",
        "tile_m=16,tile_n=64,tile_k=16,waves_m=1,waves_n=1,vec=4,stages=3,unroll=1,layout=0,splits=64",
    ],
    "gemm_skinny5": [
        "tile_m=16,tile_n=64,tile_k=16,waves_m=2,waves_n=2,vec=4,stages=3,unroll=1,layout=0,splits=8",
        "tile_m=16,tile_n=64,tile_k=32,waves_m=1,waves_n=2,vec=4,stages=3,unroll=1,layout=0,splits=1",
        "tile_m=16,tile_n=64,tile_k=16,waves_m=1,waves_n=1,vec=4,stages=3,unroll=2,layout=0,splits=2",
    ],
    "attn_causal": [
        "",
        "block_m=128,block_n=64,waves=4,mfma=32,stages=2,vec=8,unroll=1,order=1",
        "block_m=64,block_n=128,waves=4,mfma=16,stages=1,vec=4,unroll=2,order=0",
        "block_m=256,block_n=32,waves=8,mfma=32,stages=2,vec=8,unroll=1,order=1",
        "block_m=64,block_n=64,waves=2,mfma=32,stages=1,vec=8,unroll=1,order=0",
        "block_m=32,block_n=128,waves=2,mfma=16,stages=2,vec=2,unroll=1,order=1",
        "block_m=128,block_n=64,waves=4,mfma=16,stages=2,vec=8,unroll=1,order=2,occ=2",
        "block_m=64,block_n=64,waves=2,mfma=32,stages=2,vec=8,unroll=1,order=2,occ=1",
        "block_m=128,block_n=128,waves=8,mfma=16,stages=2,vec=8,unroll=2,order=2,occ=2",
        "block_m=64,block_n=64,waves=2,mfma=16,stages=1,vec=4,unroll=1,order=2,occ=2",
        "block_m=64,block_n=64,waves=4,mfma=16,stages=2,vec=8,unroll=1,order=2,occ=1,splits=2",
        "block_m=64,block_n=32,waves=2,mfma=32,stages=2,vec=8,unroll=1,order=1,occ=1,splits=4",
        "block_m=32,block_n=64,waves=2,mfma=16,stages=1,vec=8,unroll=2,order=0,occ=1,splits=4",
        "block_m=64,block_n=64,waves=4,mfma=16,stages=3,vec=8,unroll=1,order=2,occ=2",
        "block_m=64,block_n=32,waves=2,mfma=32,stages=3,vec=8,unroll=1,order=1,occ=1,splits=2",
        "block_m=128,block_n=64,waves=4,mfma=16,stages=3,vec=4,unroll=1,order=0,occ=1",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=2,occ=2",
        "block_m=32,block_n=64,waves=2,mfma=16,stages=4,vec=8,unroll=1,order=0,occ=1",
        "block_m=128,block_n=64,waves=8,mfma=16,stages=4,vec=8,unroll=1,order=1,occ=2",
        "block_m=64,block_n=64,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=2,occ=1",
        "block_m=64,block_n=32,waves=2,mfma=16,stages=4,vec=8,unroll=1,order=1,occ=1",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=2,occ=2,chunk=4",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=2,vec=8,unroll=1,order=1,chunk=4",
        "block_m=64,block_n=32,waves=2,mfma=32,stages=2,vec=8,unroll=1,order=0,splits=2,chunk=4",
        "block_m=256,block_n=32,waves=8,mfma=16,stages=2,vec=8,unroll=1,order=0,chunk=4",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=2,occ=2",
        "block_m=32,block_n=64,waves=2,mfma=16,stages=5,vec=8,unroll=1,order=0",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=2,occ=2,chunk=4",
        "block_m=128,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=1",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=2,occ=4,splits=2",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=4,vec=8,unroll=1,order=0,occ=2,splits=2",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=1,occ=4,splits=2,chunk=4",
        # four key splits sharing a ring of eight direct-to-LDS slots
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=1,occ=4,splits=4",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=4,vec=8,unroll=2,order=0,occ=2,splits=4",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=2,occ=4,splits=4,chunk=4",
        # the two-phase pipeline with key splits: four ring slots per split
        "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=1,occ=2,splits=2",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=5,vec=8,unroll=1,order=0,occ=1,splits=2",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=2,occ=2,splits=2,chunk=4",
    ],
    "attn_full": [
        "",
        "block_m=128,block_n=64,waves=4,mfma=32,stages=2,vec=8,unroll=1,order=1",
        "block_m=64,block_n=128,waves=4,mfma=16,stages=1,vec=4,unroll=2,order=0",
        "block_m=64,block_n=64,waves=4,mfma=16,stages=2,vec=8,unroll=1,order=0,splits=2",
        "block_m=64,block_n=64,waves=4,mfma=16,stages=3,vec=8,unroll=1,order=0,splits=2",
        "block_m=64,block_n=64,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=0",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=0,chunk=4",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=0",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=0,occ=4,splits=2",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=0,occ=4,splits=4",
        "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=0,occ=2,splits=2",
    ],
    "attn_d64": [
        "block_m=64,block_n=32,waves=2,mfma=32,stages=2,vec=8,unroll=1,order=0",
        "block_m=32,block_n=64,waves=2,mfma=16,stages=1,vec=4,unroll=1,order=1",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=4,vec=8,unroll=1,order=0",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=5,vec=8,unroll=1,order=0",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=4,vec=8,unroll=1,order=0,splits=2",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=4,vec=8,unroll=1,order=0,splits=4",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=5,vec=8,unroll=1,order=0,splits=2",
        "block_m=32,block_n=32,waves=2,mfma=16,stages=5,vec=8,unroll=1,order=2,splits=4",
    ],
    "mlp": [
        "",
        _block("up.", 128, 128, 64, 2, 2, 16, 5, 8, 1, 1, 1) + "," +
        _block("down.", 128, 64, 64, 2, 2, 32, 5, 8, 1, 1, 0) + ",fuse=1",
        _block("up.", 128, 128, 64, 2, 2, 32, 2, 8, 1, 1, 1) + "," +
        _block("down.", 128, 128, 64, 2, 2, 32, 2, 8, 1, 1, 1) + ",fuse=1",
        _block("up.", 64, 64, 32, 2, 2, 16, 1, 4, 2, 0, 0) + "," +
        _block("down.", 64, 128, 128, 1, 2, 16, 2, 8, 2, 0, 1) + ",fuse=0",
        _block("up.", 256, 64, 64, 4, 1, 32, 2, 8, 1, 1, 0) + "," +
        _block("down.", 32, 256, 32, 1, 4, 32, 1, 2, 1, 1, 0) + ",fuse=1",
        _block("up.", 32, 32, 128, 1, 1, 16, 2, 8, 2, 1, 1) + "," +
        _block("down.", 256, 256, 32, 4, 4, 16, 2, 8, 1, 0, 1) + ",fuse=0",
        _block("up.", 128, 128, 32, 2, 2, 32, 3, 8, 1, 1, 1, 2) + "," +
        _block("down.", 128, 128, 64, 2, 2, 16, 3, 8, 1, 1, 0, 2) + ",fuse=1",
        _block("up.", 128, 128, 64, 2, 2, 16, 4, 8, 1, 1, 1) + "," +
        _block("down.", 128, 128, 64, 2, 2, 16, 4, 8, 1, 1, 1) + ",fuse=1",
        _block("up.", 64, 128, 32, 2, 2, 32, 4, 8, 1, 1, 0) + "," +
        _block("down.", 256, 64, 32, 4, 1, 16, 4, 8, 1, 1, 0) + ",fuse=0",
        _block("up.", 192, 128, 64, 2, 4, 16, 3, 8, 1, 1, 1, 2) + "," +
        _block("down.", 192, 128, 64, 2, 4, 16, 4, 8, 1, 1, 1, 2) + ",fuse=1",
        # ping-pong staging
        _block("up.", 256, 128, 32, 4, 2, 32, 6, 8, 1, 1, 1, 2) + "," +
        _block("down.", 128, 256, 64, 2, 4, 32, 6, 8, 1, 1, 1, 2) + ",fuse=1",
        _block("up.", 128, 128, 32, 4, 2, 16, 6, 8, 1, 1, 0, 2) + "," +
        _block("down.", 256, 128, 32, 4, 2, 16, 6, 8, 1, 1, 0, 2) + ",fuse=0",
        # deep direct-to-LDS ring (buffer loads, zero-filled missing rows)
        _block("up.", 128, 128, 32, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
        _block("down.", 64, 128, 64, 2, 2, 16, 7, 8, 1, 1, 0, 2) + ",fuse=1",
        _block("up.", 256, 128, 32, 4, 2, 16, 7, 8, 1, 1, 1, 2) + "," +
        _block("down.", 128, 128, 64, 2, 2, 32, 7, 8, 1, 1, 1) + ",fuse=1",
        _block("up.", 64, 64, 64, 2, 2, 32, 7, 8, 1, 1, 0) + "," +
        _block("down.", 128, 256, 32, 2, 4, 16, 7, 8, 1, 1, 1, 2) + ",fuse=0",
        # XCD-major tile order, n fastest
        _block("up.", 128, 128, 32, 2, 2, 16, 7, 8, 1, 1, 2) + "," +
        _block("down.", 128, 64, 64, 2, 2, 16, 3, 8, 1, 1, 2) + ",fuse=1",
        # the down projection's K range cut over 2 or 4 workgroups per tile
        # (every staging path; weights stored N x K and K x N)
        _block("up.", 128, 128, 32, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
        _block("down.", 64, 64, 64, 2, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1,down.split=2",
        _block("up.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 0) + "," +
        _block("down.", 128, 128, 32, 2, 2, 16, 4, 8, 1, 1, 0) + ",fuse=1,down.split=4",
        _block("up.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 0) + "," +
        _block("down.", 64, 128, 64, 2, 2, 32, 3, 8, 2, 1, 2) + ",fuse=0,down.split=2",
        _block("up.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 0) + "," +
        _block("down.", 128, 128, 64, 2, 4, 16, 6, 8, 1, 1, 1, 2) + ",fuse=1,down.split=2",
        _block("up.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 0) + "," +
        _block("down.", 64, 64, 32, 2, 2, 16, 5, 4, 1, 0, 0) + ",fuse=1,down.split=4",
        _block("up.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 0) + "," +
        _block("down.", 32, 64, 64, 1, 2, 16, 1, 8, 2, 0, 2) + ",fuse=1,down.split=2",
    ],
    "mlp_odd": [
        _block("up.", 256, 64, 64, 4, 2, 16, 6, 8, 1, 1, 1, 2) + "," +
        _block("down.", 256, 64, 64, 4, 2, 16, 6, 8, 1, 1, 1, 2) + ",fuse=1",
        _block("up.", 256, 64, 64, 4, 2, 32, 6, 8, 1, 1, 0, 2) + "," +
        _block("down.", 128, 64, 64, 4, 2, 16, 6, 8, 1, 1, 0, 2) + ",fuse=1",
        _block("up.", 128, 64, 64, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
        _block("down.", 64, 64, 32, 2, 2, 16, 7, 8, 1, 1, 0) + ",fuse=1",
        # K split with an odd number of K tiles per split (320 = 2 x 5 x 32)
        _block("up.", 128, 64, 64, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
        _block("down.", 64, 64, 32, 2, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1,down.split=2",
    ],
    "moe": [
        "",
        _block("up.", 128, 128, 64, 2, 2, 16, 5, 8, 1, 1, 1) + "," +
        _block("down.", 64, 128, 64, 2, 2, 16, 5, 8, 1, 1, 1) + ",fuse=1",
        _block("up.", 128, 128, 64, 2, 2, 32, 2, 8, 1, 1, 1) + "," +
        _block("down.", 128, 128, 64, 2, 2, 32, 2, 8, 1, 1, 1) + ",fuse=1",
        _block("up.", 64, 64, 32, 2, 2, 16, 1, 4, 1, 0, 0) + "," +
        _block("down.", 32, 128, 128, 1, 2, 16, 2, 8, 1, 0, 1) + ",fuse=0",
        _block("up.", 32, 64, 32, 1, 2, 16, 2, 8, 2, 1, 0) + "," +
        _block("down.", 256, 64, 64, 4, 1, 32, 2, 8, 1, 1, 0) + ",fuse=1",
        _block("up.", 64, 128, 64, 2, 2, 32, 3, 8, 1, 1, 1, 2) + "," +
        _block("down.", 64, 128, 32, 2, 2, 16, 3, 8, 1, 1, 1, 2) + ",fuse=1",
        _block("up.", 128, 128, 64, 2, 2, 16, 4, 8, 1, 1, 1) + "," +
        _block("down.", 128, 128, 64, 2, 2, 16, 4, 8, 1, 1, 1) + ",fuse=1",
        _block("up.", 32, 128, 64, 1, 2, 16, 4, 8, 1, 1, 0) + "," +
        _block("down.", 64, 64, 64, 2, 1, 32, 4, 8, 1, 1, 0) + ",fuse=0",
        # 192-row tiles (three 64-row bands) on the register-staged and the
        # direct-to-LDS paths
        _block("up.", 192, 128, 64, 2, 4, 16, 3, 8, 1, 1, 1, 2) + "," +
        _block("down.", 192, 128, 64, 2, 4, 16, 4, 8, 1, 1, 1, 2) + ",fuse=1",
        _block("up.", 192, 64, 64, 4, 2, 16, 4, 8, 1, 1, 0) + "," +
        _block("down.", 192, 64, 32, 4, 1, 16, 2, 8, 1, 1, 0) + ",fuse=0",
        # ping-pong staging over gathered (gate/up) and grouped (down) rows
        _block("up.", 128, 128, 64, 4, 2, 16, 6, 8, 1, 1, 1, 2) + "," +
        _block("down.", 128, 256, 64, 2, 4, 16, 6, 8, 1, 1, 1, 2) + ",fuse=1",
        _block("up.", 128, 128, 32, 2, 4, 16, 6, 8, 1, 1, 0, 2) + "," +
        _block("down.", 128, 128, 32, 4, 2, 32, 6, 8, 1, 1, 0, 2) + ",fuse=0",
        # deep direct-to-LDS ring over gathered (gate/up) and grouped (down) rows
        _block("up.", 128, 128, 32, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
        _block("down.", 64, 128, 64, 2, 2, 16, 7, 8, 1, 1, 0, 2) + ",fuse=1",
        _block("up.", 64, 128, 64, 2, 2, 32, 7, 8, 1, 1, 0) + "," +
        _block("down.", 128, 256, 32, 2, 4, 16, 7, 8, 1, 1, 1, 2) + ",fuse=0",
        # XCD-major order over the routed tiles (n fastest); partial tiles
        # skip their empty row blocks on every staging path
        _block("up.", 256, 128, 32, 2, 4, 16, 7, 8, 1, 1, 2, 2) + "," +
        _block("down.", 128, 256, 64, 2, 4, 16, 4, 8, 1, 1, 2, 2) + ",fuse=1",
        _block("up.", 128, 64, 64, 4, 1, 16, 3, 8, 1, 1, 2) + "," +
        _block("down.", 128, 64, 32, 4, 1, 16, 1, 8, 1, 1, 2) + ",fuse=1",
        _block("up.", 64, 128, 64, 2, 2, 16, 5, 8, 1, 1, 2) + "," +
        _block("down.", 64, 128, 64, 4, 1, 16, 2, 8, 1, 1, 2) + ",fuse=0",
        # partial tiles skipping their empty row blocks, on each staging path
        _block("up.", 256, 128, 32, 2, 4, 16, 7, 8, 1, 1, 1, 2) + "," +
        _block("down.", 128, 128, 64, 2, 2, 16, 4, 8, 1, 1, 1) + ",fuse=1,up.skip=1,down.skip=1",
        _block("up.", 128, 64, 64, 4, 1, 16, 3, 8, 1, 1, 0) + "," +
        _block("down.", 128, 64, 32, 4, 1, 32, 1, 8, 1, 1, 2) + ",fuse=1,up.skip=1,down.skip=1",
        _block("up.", 128, 128, 64, 2, 2, 16, 5, 8, 1, 1, 2) + "," +
        _block("down.", 128, 64, 64, 2, 1, 16, 2, 8, 2, 1, 0) + ",fuse=0,up.skip=1,down.skip=1",
        _block("up.", 128, 128, 64, 4, 2, 16, 6, 8, 1, 1, 1, 2) + "," +
        _block("down.", 192, 64, 64, 4, 1, 16, 7, 8, 1, 1, 0) + ",fuse=1,up.skip=0,down.skip=1",
        # 256 x 256 down tiles on the ring, XCD-major, partial tiles skipping
        # their empty row blocks (groups of ~64 rows: mostly empty tiles)
        _block("up.", 64, 64, 32, 2, 2, 16, 7, 8, 1, 1, 2, 2) + "," +
        _block("down.", 256, 256, 32, 2, 4, 16, 7, 8, 1, 1, 2) + ",fuse=1,up.skip=1,down.skip=1",
    ],
    "conv": [
        "",
        _block("", 64, 64, 64, 2, 2, 32, 5, 8, 1, 1, 1) + ",fuse=1",
        _block("", 128, 64, 64, 2, 1, 16, 2, 8, 1, 1, 0) + ",fuse=1",
        _block("", 64, 32, 32, 2, 1, 16, 1, 4, 2, 0, 1) + ",fuse=0",
        _block("", 128, 64, 64, 2, 2, 32, 2, 8, 1, 1, 1) + ",fuse=1",
        _block("", 32, 64, 64, 1, 2, 16, 2, 2, 1, 0, 0) + ",fuse=1",
        _block("", 128, 64, 64, 2, 2, 16, 3, 8, 1, 1, 0, 2) + ",fuse=1",
        # deep direct-to-LDS ring: padded taps and missing pixels load zeros
        _block("", 64, 64, 64, 2, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1",
        _block("", 64, 64, 32, 2, 1, 32, 7, 8, 1, 1, 0, 2) + ",fuse=0",
        _block("", 128, 64, 64, 2, 2, 16, 7, 8, 1, 1, 1, 2) + ",fuse=1",
        _block("", 64, 64, 64, 2, 2, 16, 7, 8, 1, 1, 2) + ",fuse=1",
    ],
}

SCHEDULES["mlp_tail"] = [
    _block("up.", 64, 32, 64, 2, 2, 16, 2, 8, 1, 1, 1) + "," +
    _block("down.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 0) + ",fuse=1,up.tail=1",
    _block("up.", 64, 32, 64, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
    _block("down.", 64, 64, 64, 2, 2, 16, 3, 8, 1, 1, 0) + ",fuse=1,up.tail=1",
    _block("up.", 64, 32, 32, 2, 2, 16, 5, 4, 1, 1, 0) + "," +
    _block("down.", 32, 64, 64, 1, 2, 16, 2, 8, 1, 1, 0) + ",fuse=0,up.tail=1",
]
# the tail columns as full tiles with their K range cut in two (partial
# sums, then SwiGLU or the plain sum in a separate kernel)
SCHEDULES["mlp_tail"] += [
    _block("up.", 64, 32, 64, 2, 2, 16, 2, 8, 1, 1, 1) + "," +
    _block("down.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 0) + ",fuse=1,up.tail=2",
    _block("up.", 64, 32, 64, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
    _block("down.", 64, 64, 64, 2, 2, 16, 3, 8, 1, 1, 0) + ",fuse=1,up.tail=2",
]
SCHEDULES["mlp_tail_down"] = [
    _block("up.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 1) + "," +
    _block("down.", 64, 32, 64, 2, 2, 16, 2, 8, 1, 1, 1) + ",fuse=1,down.tail=1",
    _block("up.", 64, 64, 64, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
    _block("down.", 64, 32, 64, 2, 2, 16, 7, 8, 1, 1, 0) + ",fuse=1,down.tail=1",
    _block("up.", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 1) + "," +
    _block("down.", 64, 32, 64, 2, 2, 16, 2, 8, 1, 1, 1) + ",fuse=1,down.tail=2",
    _block("up.", 64, 64, 64, 2, 2, 16, 7, 8, 1, 1, 1) + "," +
    _block("down.", 64, 32, 64, 2, 2, 16, 7, 8, 1, 1, 0) + ",fuse=1,down.tail=2",
]
SCHEDULES["conv_k320"] = [
    _block("", 64, 80, 64, 1, 1, 16, 2, 8, 1, 1, 0) + ",fuse=1",
    _block("", 32, 160, 64, 1, 2, 16, 5, 8, 1, 1, 1) + ",fuse=1",
    _block("", 64, 320, 32, 2, 2, 16, 3, 8, 1, 1, 0) + ",fuse=0",
    _block("", 16, 320, 64, 1, 4, 16, 2, 4, 1, 0, 0) + ",fuse=1",
    _block("", 64, 320, 64, 2, 2, 32, 2, 8, 1, 1, 1) + ",fuse=1",
    _block("", 64, 160, 64, 2, 2, 16, 1, 8, 1, 1, 0, 2) + ",fuse=0",
    _block("", 64, 160, 64, 2, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1",
    _block("", 64, 320, 32, 2, 2, 16, 7, 8, 1, 1, 0) + ",fuse=1",
]
SCHEDULES["attn_causal_512"] = [
    "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=2,occ=2,chunk=8",
    "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=0,chunk=8",
    "block_m=32,block_n=32,waves=2,mfma=16,stages=2,vec=8,unroll=1,order=1,chunk=8",
    "block_m=64,block_n=32,waves=2,mfma=32,stages=2,vec=8,unroll=1,order=0,splits=4,chunk=8",
    "block_m=64,block_n=64,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=1,occ=1,splits=2,chunk=4",
    "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=2,occ=2,splits=2,chunk=8",
]
SCHEDULES["gemm_skinny"].append(
    "tile_m=16,tile_n=64,tile_k=16,waves_m=1,waves_n=2,vec=4,stages=3,unroll=1,layout=0,splits=32")

# the ragged shapes run every schedule of their full-tile counterparts that
# is legal for them (the paired order needs an even number of query tiles)
SCHEDULES["mlp_ragged"] = SCHEDULES["mlp"]
SCHEDULES["conv_ragged"] = SCHEDULES["conv"]


def _legal_for(key, scheds):
    kind, dims, flags = SMALL[key]
    op = rc.Op(kind, dims, flags)
    return [t for t in scheds if op.from_string(t).validate() == ""]


SCHEDULES["attn_ragged_causal"] = _legal_for("attn_ragged_causal", SCHEDULES["attn_causal"])
SCHEDULES["attn_ragged_full"] = _legal_for("attn_ragged_full", SCHEDULES["attn_full"])
SCHEDULES["attn_ragged_d64"] = _legal_for("attn_ragged_d64", SCHEDULES["attn_d64"])

# degenerate sizes: the smallest tiles, on every staging path they admit
_ONE_ATTN = [
    "",
    "block_m=16,block_n=32,waves=1,mfma=16,stages=1,vec=4,unroll=1,order=0",
    "block_m=16,block_n=32,waves=1,mfma=16,stages=3,vec=8,unroll=1,order=0",
    "block_m=16,block_n=32,waves=1,mfma=16,stages=4,vec=8,unroll=1,order=0,occ=1,splits=2",
    "block_m=16,block_n=32,waves=1,mfma=16,stages=4,vec=8,unroll=1,order=0,occ=1,splits=4",
]
_ONE_MLP = [
    "",
    _block("up.", 16, 64, 32, 1, 1, 16, 7, 8, 1, 1, 1) + "," +
    _block("down.", 16, 64, 32, 1, 1, 16, 7, 8, 1, 1, 1) + ",fuse=1",
    _block("up.", 16, 128, 64, 1, 2, 16, 4, 8, 1, 1, 1) + "," +
    _block("down.", 16, 128, 64, 1, 2, 16, 4, 8, 1, 1, 1) + ",fuse=1",
    _block("up.", 16, 64, 64, 1, 2, 16, 5, 8, 1, 1, 0) + "," +
    _block("down.", 16, 64, 64, 1, 2, 16, 3, 8, 1, 1, 0) + ",fuse=0",
]
SCHEDULES["gemm_one"] = [
    "", "tile_m=16,tile_n=16,tile_k=4,waves_m=1,waves_n=1,vec=1,stages=2,unroll=1,layout=1"]
SCHEDULES["gemm_row"] = [
    "",
    "tile_m=16,tile_n=64,tile_k=16,waves_m=1,waves_n=2,vec=1,stages=2,unroll=1,layout=0",
    "tile_m=16,tile_n=32,tile_k=8,waves_m=1,waves_n=1,vec=1,stages=1,unroll=2,layout=1",
    "tile_m=16,tile_n=64,tile_k=32,waves_m=1,waves_n=1,vec=1,stages=2,unroll=1,layout=1",
]
SCHEDULES["attn_one_causal"] = _legal_for("attn_one_causal", _ONE_ATTN)
SCHEDULES["attn_one_full"] = _legal_for("attn_one_full", _ONE_ATTN)
SCHEDULES["mlp_one"] = _ONE_MLP
SCHEDULES["moe_one"] = _ONE_MLP
SCHEDULES["conv_one"] = [
    "",
    _block("", 16, 64, 64, 1, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1",
    _block("", 16, 64, 64, 1, 2, 16, 5, 8, 1, 1, 1) + ",fuse=1",
    _block("", 16, 64, 32, 1, 1, 16, 2, 8, 1, 0, 0) + ",fuse=0",
]


def small_op(key):
    kind, dims, flags = SMALL[key]
    return rc.Op(kind, dims, flags)


# Full-size workloads in schedules that take the other code paths (pipelined
# and split direct-to-LDS attention, chunked work items, two-set register
# prefetch and direct-to-LDS GEMM staging), sampled outputs.
FULL_ALT = [
    ("attention_causal_b1_h32_s1024_d128",
     "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=2,order=2,occ=2"),
    ("attention_causal_b1_h32_s1024_d128",
     "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=2,occ=2"),
    ("attention_causal_b1_h32_s1024_d128",
     "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=1,occ=4,splits=2"),
    ("attention_causal_b1_h32_s1024_d128",
     "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=2,occ=2,chunk=16"),
    ("attention_causal_b1_h32_s1024_d128",
     "block_m=64,block_n=32,waves=4,mfma=16,stages=4,vec=8,unroll=1,order=1,occ=4,splits=4"),
    ("attention_causal_b1_h32_s1024_d128",
     "block_m=64,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=1,occ=2,splits=2"),
    ("attention_noncausal_b1_h24_s4096_d128",
     "block_m=128,block_n=32,waves=4,mfma=16,stages=5,vec=8,unroll=1,order=1,occ=2,splits=2"),
    ("gated_mlp_t2048_h4096_i14336",
     _block("up.", 128, 128, 64, 2, 2, 16, 5, 8, 1, 1, 1) + "," +
     _block("down.", 128, 256, 64, 2, 4, 16, 4, 8, 1, 1, 1) + ",fuse=1"),
    ("moe_t4096_h2048_e64_i1408_top6",
     _block("up.", 128, 128, 64, 2, 2, 16, 5, 8, 1, 1, 1) + "," +
     _block("down.", 128, 128, 64, 2, 2, 16, 3, 8, 1, 1, 0) + ",fuse=1"),
    ("conv3x3_n2_64x64_c320_k320",
     _block("", 64, 64, 64, 4, 2, 16, 2, 8, 1, 1, 1) + ",fuse=1"),
    # the gate/up GEMM's last half round as a second, half-height launch
    ("gated_mlp_t2048_h4096_i14336",
     _block("up.", 256, 128, 64, 4, 4, 16, 2, 8, 1, 1, 1, 2) + "," +
     _block("down.", 128, 128, 64, 2, 2, 16, 3, 8, 1, 1, 0) + ",fuse=1,up.tail=1"),
    ("gated_mlp_t2048_h4096_i14336",
     _block("up.", 256, 128, 32, 2, 4, 16, 7, 8, 1, 1, 1) + "," +
     _block("down.", 128, 128, 64, 2, 2, 16, 3, 8, 1, 1, 0) + ",fuse=1,up.tail=1"),
    # deep direct-to-LDS ring at full size
    ("gated_mlp_t2048_h4096_i14336",
     _block("up.", 256, 128, 32, 4, 2, 16, 7, 8, 1, 1, 1, 2) + "," +
     _block("down.", 128, 128, 64, 2, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1"),
    ("moe_t4096_h2048_e64_i1408_top6",
     _block("up.", 256, 128, 32, 4, 2, 16, 7, 8, 1, 1, 1, 2) + "," +
     _block("down.", 128, 128, 64, 2, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1"),
    ("moe_t4096_h2048_e64_i1408_top6",
     _block("up.", 256, 128, 32, 2, 4, 16, 7, 8, 1, 1, 2, 2) + "," +
     _block("down.", 128, 256, 64, 2, 4, 16, 7, 8, 1, 1, 2, 2) + ",fuse=1,up.skip=1,down.skip=1"),
    # both expert GEMMs on the ring in the XCD-major order, 256 x 256 down
    # tiles whose partial last tile per expert skips its empty row blocks
    ("moe_t4096_h2048_e64_i1408_top6",
     _block("up.", 256, 128, 32, 2, 4, 16, 7, 8, 1, 1, 2, 2) + "," +
     _block("down.", 256, 256, 32, 2, 4, 16, 7, 8, 1, 1, 2) + ",fuse=1,up.skip=1,down.skip=1"),
    ("conv3x3_n2_64x64_c320_k320",
     _block("", 64, 160, 64, 2, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1"),
    # the down projection on 256 x 256 tiles with its K range cut in two
    ("gated_mlp_t2048_h4096_i14336",
     _block("up.", 256, 128, 32, 2, 4, 16, 7, 8, 1, 1, 1) + "," +
     _block("down.", 256, 256, 32, 2, 4, 16, 7, 8, 1, 1, 1) + ",fuse=1,up.tail=1,down.split=2"),
    ("gated_mlp_t2048_h4096_i14336",
     _block("up.", 256, 128, 32, 2, 4, 16, 7, 8, 1, 1, 1) + "," +
     _block("down.", 128, 256, 64, 2, 4, 16, 4, 8, 1, 1, 2) + ",fuse=1,up.tail=1,down.split=4"),
    # the gate/up tail as full tiles with their K range cut in two
    ("gated_mlp_t2048_h4096_i14336",
     _block("up.", 256, 128, 32, 2, 4, 16, 7, 8, 1, 1, 1) + "," +
     _block("down.", 256, 256, 32, 2, 4, 16, 7, 8, 1, 1, 1) + ",fuse=1,up.tail=2,down.split=2"),
]


# Benchmark-sized operators whose row count no tile divides, run in the
# benchmark's tuned schedule (every tile but the last is full).
RAGGED_FULL = [
    ("attention_causal_b1_h32_s1024_d128", (1, 32, 1000, 128), rc.RC_FLAG_CAUSAL),
    ("attention_noncausal_b1_h24_s4096_d128", (1, 24, 4000, 128), 0),
    ("gated_mlp_t2048_h4096_i14336", (2000, 4096, 14336), 0),
    ("conv3x3_n2_64x64_c320_k320", (2, 63, 63, 320, 320, 3, 3, 1), 0),
    ("gemm_f32_128", (100, 120, 132), 0),
]


# Plain bf16 GEMMs (1 x 1 convolutions without padding or activation,
# M = 512 pixels, C = 256 -> K = 128) for integer-input bitwise checks.
GEMM_1X1 = [
    "",
    _block("", 64, 64, 64, 2, 2, 16, 2, 8, 1, 1, 1) + ",fuse=1",
    _block("", 128, 128, 32, 2, 2, 32, 3, 8, 1, 1, 0) + ",fuse=1",
    _block("", 32, 64, 128, 1, 2, 16, 5, 8, 2, 1, 1) + ",fuse=0",
    _block("", 64, 32, 64, 2, 1, 16, 1, 4, 1, 0, 0) + ",fuse=1",
    _block("", 256, 128, 64, 4, 2, 16, 2, 8, 1, 1, 1, 2) + ",fuse=1",
    _block("", 128, 128, 64, 2, 2, 16, 7, 8, 1, 1, 1) + ",fuse=1",
    _block("", 64, 128, 32, 2, 2, 32, 7, 8, 1, 1, 0, 2) + ",fuse=1",
]
GEMM_1X1_OP = (rc.RC_OP_CONV2D, (2, 16, 16, 256, 128, 1, 1, 0), rc.RC_FLAG_NO_ACT)
CONV_FULL_ALT = _block("", 64, 64, 64, 4, 2, 16, 2, 8, 1, 1, 1) + ",fuse=1"


# Schedules the search can emit: random legal transformation sequences of
# length 12 from P0 (the rollouts of Sec. 3.2), seeded, at the small shapes.
WALK_KEYS = ("gemm", "attn_causal", "mlp", "moe", "conv")
WALK_COUNT = 40


def random_walks(key, n=WALK_COUNT, seed=20260):
    from paper_2506_01374_amd import tune
    op = small_op(key)
    return [str(s) for s in tune.random_walk_space(op, n, seed + WALK_KEYS.index(key), horizon=12)]


# The no-allocation launch against the workspace launch: (kind, larger
# dims, smaller dims, flags, schedule) for every operator whose kernels use
# a workspace.
NOALLOC_PAIRS = [
    (rc.RC_OP_GATED_MLP, (256, 256, 512), (200, 256, 512), 0, SCHEDULES["mlp"][1]),
    (rc.RC_OP_GATED_MLP, (256, 256, 512), (40, 256, 512), 0, SCHEDULES["mlp"][3]),
    (rc.RC_OP_MOE, (256, 256, 8, 128, 2), (64, 256, 8, 128, 2), 0, SCHEDULES["moe"][1]),
    (rc.RC_OP_MOE, (256, 256, 8, 128, 2), (1, 256, 8, 128, 2), 0, SCHEDULES["moe"][3]),
    (rc.RC_OP_ATTENTION, (1, 2, 512, 128), (1, 2, 384, 128), rc.RC_FLAG_CAUSAL, SCHEDULES["attn_causal_512"][0]),
    (rc.RC_OP_GEMM_F32, (16, 256, 1024), (5, 128, 512), 0, SCHEDULES["gemm_skinny"][3]),
    (rc.RC_OP_CONV2D, (2, 16, 12, 64, 64, 3, 3, 1), (1, 10, 9, 64, 64, 3, 3, 1), 0, SCHEDULES["conv"][3]),
]


def walk_compile_jobs():
    """(op, [schedules]) of the random-walk cases; some may spill (rejected
    at compile time, which the tests accept)."""
    jobs = []
    for key in WALK_KEYS:
        op = small_op(key)
        jobs.append((op, [op.from_string(s) for s in random_walks(key)]))
    return jobs


def all_compile_jobs():
    """(op, [schedules]) pairs for ahead-of-time compilation."""
    jobs = []
    # the convolutions without activation (integer and closed-form checks)
    for key in ("conv", "conv_ragged", "conv_k320"):
        kind, dims, _ = SMALL[key]
        op = rc.Op(kind, dims, rc.RC_FLAG_NO_ACT)
        jobs.append((op, [op.from_string(t) for t in SCHEDULES[key] if op.from_string(t).validate() == ""]))
    op = rc.Op(*GEMM_1X1_OP)
    jobs.append((op, [op.from_string(t) for t in GEMM_1X1]))
    op = rc.Op(rc.RC_OP_CONV2D, W.workload_op("conv3x3_n2_64x64_c320_k320").dims, rc.RC_FLAG_NO_ACT)
    jobs.append((op, [op.from_string(TUNED["conv3x3_n2_64x64_c320_k320"]), op.default(),
                      op.from_string(CONV_FULL_ALT)]))
    for kind, big, small, flags, text in NOALLOC_PAIRS:
        for dims in (big, small):
            op = rc.Op(kind, dims, flags)
            jobs.append((op, [op.from_string(text)]))
    moe = W.workload_op("moe_t4096_h2048_e64_i1408_top6")
    for dims in ((256, 256, 8, 128, 2), (256, 256, 8, 128, 1), (8192, 256, 64, 128, 6)):
        op = rc.Op(rc.RC_OP_MOE, dims)
        jobs.append((op, [op.from_string(t) for t in SCHEDULES["moe"][:4]]))
    del moe
    for key, lst in SCHEDULES.items():
        op = small_op(key)
        jobs.append((op, [op.from_string(s) for s in lst]))
    for name, s in TUNED.items():
        op = W.workload_op(name)
        jobs.append((op, [op.from_string(s), op.default()]))
    for name, s in FULL_ALT:
        op = W.workload_op(name)
        jobs.append((op, [op.from_string(s)]))
    for name, dims, flags in RAGGED_FULL:
        op = rc.Op(W.workload_op(name).kind, dims, flags)
        jobs.append((op, [op.from_string(TUNED[name])]))
    return jobs
