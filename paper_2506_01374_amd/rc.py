"""ctypes binding of librc (include/rc.h), same names, marshalling only.

Every operator step runs in librc's HIP kernels; PyTorch is used only to
own device memory and to name the stream.  If ``librc.so`` is not built the
first call raises ``RuntimeError`` - there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Callable, Dict, Iterable, List, Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "librc.so")

RC_OK = 0
STATUS = {0: "RC_OK", 1: "RC_ERR_INVALID_ARGUMENT", 2: "RC_ERR_ILLEGAL_SCHEDULE",
          3: "RC_ERR_UNSUPPORTED", 4: "RC_ERR_COMPILE", 5: "RC_ERR_HIP",
          6: "RC_ERR_OUT_OF_MEMORY", 7: "RC_ERR_MISALIGNED", 8: "RC_ERR_BUDGET"}
(RC_ERR_INVALID_ARGUMENT, RC_ERR_ILLEGAL_SCHEDULE, RC_ERR_UNSUPPORTED, RC_ERR_COMPILE, RC_ERR_HIP,
 RC_ERR_OUT_OF_MEMORY, RC_ERR_MISALIGNED, RC_ERR_BUDGET) = range(1, 9)

RC_OP_GEMM_F32, RC_OP_ATTENTION, RC_OP_GATED_MLP, RC_OP_MOE, RC_OP_CONV2D = 1, 2, 3, 4, 5
RC_FLAG_CAUSAL = 1
RC_FLAG_NO_ACT = 2
RC_POLICY_RANDOM, RC_POLICY_UCT, RC_POLICY_EXHAUSTIVE = 0, 1, 2
MAX_DIMS, MAX_KNOBS = 8, 32


class rc_op_desc(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("kind", ctypes.c_int32),
                ("dim", ctypes.c_int64 * MAX_DIMS), ("flags", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class rc_schedule(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("nknobs", ctypes.c_int32),
                ("knob", ctypes.c_int32 * MAX_KNOBS)]


class rc_transform(ctypes.Structure):
    _fields_ = [("knob", ctypes.c_int32), ("value", ctypes.c_int32)]


class rc_kernel_info(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("name", ctypes.c_char * 48),
                ("grid", ctypes.c_int32), ("block", ctypes.c_int32), ("lds_bytes", ctypes.c_int32),
                ("vgprs", ctypes.c_int32), ("agprs", ctypes.c_int32), ("sgprs", ctypes.c_int32),
                ("scratch_bytes", ctypes.c_int32), ("waves_per_simd", ctypes.c_int32)]


class rc_args(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("in_", ctypes.c_void_p * 8),
                ("out", ctypes.c_void_p * 2)]


class rc_time_opts(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("warmup", ctypes.c_int32),
                ("repeat", ctypes.c_int32), ("flush", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class rc_timing(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("nkernels", ctypes.c_int32),
                ("median_ms", ctypes.c_double), ("min_ms", ctypes.c_double),
                ("mean_ms", ctypes.c_double), ("q1_ms", ctypes.c_double),
                ("q3_ms", ctypes.c_double), ("tflops", ctypes.c_double),
                ("gbps", ctypes.c_double), ("frac_flops", ctypes.c_double),
                ("frac_bytes", ctypes.c_double), ("kernel_ms", ctypes.c_double * 8)]


class rc_search_opts(ctypes.Structure):
    _fields_ = [("struct_size", ctypes.c_uint32), ("policy", ctypes.c_int32),
                ("budget", ctypes.c_int32), ("horizon", ctypes.c_int32),
                ("branching", ctypes.c_int32), ("c", ctypes.c_double),
                ("seed", ctypes.c_uint64), ("max_invalid", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


class rc_sample(ctypes.Structure):
    _fields_ = [("schedule", rc_schedule), ("reward", ctypes.c_double),
                ("valid", ctypes.c_int32), ("index", ctypes.c_int32),
                ("best_so_far", ctypes.c_double)]


EVAL_FN = ctypes.CFUNCTYPE(ctypes.c_int32, ctypes.c_void_p, ctypes.POINTER(rc_schedule),
                           ctypes.POINTER(ctypes.c_double))
PROPOSE_FN = ctypes.CFUNCTYPE(ctypes.c_int32, ctypes.c_void_p, ctypes.POINTER(rc_schedule),
                              ctypes.POINTER(rc_schedule), ctypes.POINTER(rc_schedule),
                              ctypes.c_void_p, ctypes.c_size_t)

# (name, restype, argtypes) of every exported entry point
_SIGS = [
    ("rc_status_str", ctypes.c_char_p, [ctypes.c_int]),
    ("rc_last_error", ctypes.c_char_p, []),
    ("rc_op_init", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.c_int32,
                                  ctypes.POINTER(ctypes.c_int64), ctypes.c_int32, ctypes.c_int32]),
    ("rc_op_flops", ctypes.c_double, [ctypes.POINTER(rc_op_desc)]),
    ("rc_op_bytes", ctypes.c_double, [ctypes.POINTER(rc_op_desc)]),
    ("rc_peak_flops", ctypes.c_double, [ctypes.POINTER(rc_op_desc)]),
    ("rc_peak_bytes_per_s", ctypes.c_double, []),
    ("rc_knob_count", ctypes.c_int32, [ctypes.POINTER(rc_op_desc)]),
    ("rc_knob_name", ctypes.c_char_p, [ctypes.POINTER(rc_op_desc), ctypes.c_int32]),
    ("rc_knob_class", ctypes.c_char_p, [ctypes.POINTER(rc_op_desc), ctypes.c_int32]),
    ("rc_knob_values", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.c_int32,
                                      ctypes.POINTER(ctypes.c_int32), ctypes.c_int32,
                                      ctypes.POINTER(ctypes.c_int32)]),
    ("rc_default_schedule", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_schedule)]),
    ("rc_validate", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_schedule),
                                   ctypes.c_char_p, ctypes.c_size_t]),
    ("rc_apply", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_schedule),
                                ctypes.POINTER(rc_transform), ctypes.POINTER(rc_schedule)]),
    ("rc_enumerate", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_schedule),
                                    ctypes.POINTER(rc_transform), ctypes.c_size_t,
                                    ctypes.POINTER(ctypes.c_size_t)]),
    ("rc_parse_transform", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.c_char_p,
                                          ctypes.POINTER(rc_transform)]),
    ("rc_schedule_to_string", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_schedule),
                                             ctypes.c_char_p, ctypes.c_size_t]),
    ("rc_schedule_from_string", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.c_char_p,
                                               ctypes.POINTER(rc_schedule)]),
    ("rc_schedule_hash", ctypes.c_uint64, [ctypes.POINTER(rc_schedule)]),
    ("rc_describe", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_schedule),
                                   ctypes.POINTER(rc_kernel_info), ctypes.c_int32,
                                   ctypes.POINTER(ctypes.c_int32)]),
    ("rc_plan_create", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_schedule),
                                      ctypes.POINTER(ctypes.c_void_p)]),
    ("rc_plan_destroy", None, [ctypes.c_void_p]),
    ("rc_precompile", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_schedule),
                                     ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(ctypes.c_int)]),
    ("rc_set_cache_dir", ctypes.c_int, [ctypes.c_char_p]),
    ("rc_plan_workspace", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_size_t)]),
    ("rc_plan_kernels", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32),
                                       ctypes.POINTER(ctypes.c_int32)]),
    ("rc_plan_kernel_flops", ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_double)]),
    ("rc_plan_buffer", ctypes.c_int, [ctypes.c_void_p, ctypes.c_char_p, ctypes.POINTER(ctypes.c_size_t),
                                      ctypes.POINTER(ctypes.c_size_t)]),
    ("rc_time_release", ctypes.c_int, []),
    ("rc_launch", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(rc_args), ctypes.c_void_p,
                                 ctypes.c_size_t, ctypes.c_void_p]),
    ("rc_launch_timed", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(rc_args), ctypes.c_void_p,
                                       ctypes.c_size_t, ctypes.c_void_p,
                                       ctypes.POINTER(ctypes.c_void_p), ctypes.c_int32]),
    ("rc_launch_static", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(rc_args), ctypes.c_void_p]),
    ("rc_static_scratch_bytes", ctypes.c_size_t, []),
    ("rc_time_opts_init", None, [ctypes.POINTER(rc_time_opts)]),
    ("rc_time", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(rc_args), ctypes.c_void_p,
                               ctypes.c_size_t, ctypes.c_void_p, ctypes.POINTER(rc_time_opts),
                               ctypes.POINTER(rc_timing)]),
    ("rc_search_opts_init", None, [ctypes.POINTER(rc_search_opts)]),
    ("rc_search_create", ctypes.c_int, [ctypes.POINTER(rc_op_desc), ctypes.POINTER(rc_search_opts),
                                        EVAL_FN, ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p)]),
    ("rc_search_set_proposer", ctypes.c_int, [ctypes.c_void_p, PROPOSE_FN, ctypes.c_void_p]),
    ("rc_search_step", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32)]),
    ("rc_search_run", ctypes.c_int, [ctypes.c_void_p]),
    ("rc_search_best", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(rc_schedule),
                                      ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int32)]),
    ("rc_search_history", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(rc_sample), ctypes.c_int32,
                                         ctypes.POINTER(ctypes.c_int32)]),
    ("rc_search_node_stats", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(rc_transform),
                                            ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                            ctypes.POINTER(ctypes.c_double)]),
    ("rc_search_fallbacks", ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32)]),
    ("rc_search_destroy", None, [ctypes.c_void_p]),
]

EXPORTS = [name for name, _, _ in _SIGS]
_lib = None


def _preload_torch_hip():
    """Bind librc to PyTorch's bundled HIP runtime and hipRTC.

    PyTorch-ROCm ships its own libamdhip64 / libhiprtc under the same sonames
    as /opt/rocm's.  Loading them (by path, without importing torch) before
    librc makes every HIP call in the process go through one runtime; two
    runtimes in one process cannot both see the GPU.  The code-object cache
    key names the hipRTC library actually loaded.
    """
    import importlib.util
    spec = importlib.util.find_spec("torch")
    if not spec or not spec.origin:
        return
    d = os.path.join(os.path.dirname(spec.origin), "lib")
    for name in ("libamdhip64.so", "libhiprtc.so"):
        path = os.path.join(d, name)
        if os.path.exists(path):
            ctypes.CDLL(path, mode=ctypes.RTLD_GLOBAL)


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"librc.so is not built ({LIB_PATH}); run __graft_entry__.build()")
        _preload_torch_hip()
        L = ctypes.CDLL(LIB_PATH)
        for name, res, args in _SIGS:
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


class RCError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        detail = lib().rc_last_error().decode(errors="replace")
        super().__init__(f"{where}: {STATUS.get(status, status)}: {detail}")


def _check(st: int, where: str) -> None:
    if st != RC_OK:
        raise RCError(st, where)


# ---------------------------------------------------------------------------
# Operators and schedules
# ---------------------------------------------------------------------------

class Op:
    """An operator descriptor (the input program P0)."""

    def __init__(self, kind: int, dims: Sequence[int], flags: int = 0):
        self.desc = rc_op_desc()
        arr = (ctypes.c_int64 * len(dims))(*dims)
        _check(lib().rc_op_init(ctypes.byref(self.desc), kind, arr, len(dims), flags), "rc_op_init")
        self.kind, self.dims, self.flags = kind, tuple(int(d) for d in dims), flags

    @property
    def ref(self):
        return ctypes.byref(self.desc)

    def flops(self) -> float:
        return lib().rc_op_flops(self.ref)

    def bytes(self) -> float:
        return lib().rc_op_bytes(self.ref)

    def peak_flops(self) -> float:
        return lib().rc_peak_flops(self.ref)

    def bound(self) -> str:
        """The roofline that binds: "hbm" when the algorithmic intensity
        (FLOPs per compulsory HBM byte) is below the ridge point peak FLOP/s
        / peak bytes/s of the operator's MFMA type, else "mfma"."""
        ridge = self.peak_flops() / lib().rc_peak_bytes_per_s()
        return "hbm" if self.flops() / self.bytes() < ridge else "mfma"

    def knob_names(self) -> List[str]:
        names = getattr(self, "_names", None)      # static per operator: read once
        if names is None:
            names = [lib().rc_knob_name(self.ref, i).decode() for i in range(lib().rc_knob_count(self.ref))]
            self._names = names
        return list(names)

    def knob_class(self, i: int) -> str:
        return lib().rc_knob_class(self.ref, i).decode()

    def knob_values(self, i: int) -> List[int]:
        n = ctypes.c_int32()
        buf = (ctypes.c_int32 * 64)()
        _check(lib().rc_knob_values(self.ref, i, buf, 64, ctypes.byref(n)), "rc_knob_values")
        return list(buf[: n.value])

    def default(self) -> "Schedule":
        s = rc_schedule()
        _check(lib().rc_default_schedule(self.ref, ctypes.byref(s)), "rc_default_schedule")
        return Schedule(self, s)

    def schedule(self, **knobs) -> "Schedule":
        s = self.default()
        names = self.knob_names()
        for k, v in knobs.items():
            s.raw.knob[names.index(k.replace("__", "."))] = int(v)
        return s

    def from_string(self, text: str) -> "Schedule":
        s = rc_schedule()
        _check(lib().rc_schedule_from_string(self.ref, text.encode(), ctypes.byref(s)),
               "rc_schedule_from_string")
        return Schedule(self, s)

    def parse(self, text: str) -> rc_transform:
        t = rc_transform()
        _check(lib().rc_parse_transform(self.ref, text.encode(), ctypes.byref(t)), "rc_parse_transform")
        return t


class Schedule:
    """A program variant: one value per knob."""

    def __init__(self, op: Op, raw: rc_schedule):
        self.op, self.raw = op, raw

    def copy(self) -> "Schedule":
        r = rc_schedule()
        ctypes.pointer(r)[0] = self.raw
        return Schedule(self.op, r)

    def __getitem__(self, name: str) -> int:
        return self.raw.knob[self.op.knob_names().index(name)]

    def as_dict(self) -> Dict[str, int]:
        return {n: self.raw.knob[i] for i, n in enumerate(self.op.knob_names())}

    def __str__(self) -> str:
        buf = ctypes.create_string_buffer(2048)
        _check(lib().rc_schedule_to_string(self.op.ref, ctypes.byref(self.raw), buf, 2048),
               "rc_schedule_to_string")
        return buf.value.decode()

    def validate(self) -> str:
        """'' when legal, else the first violated rule."""
        why = ctypes.create_string_buffer(512)
        st = lib().rc_validate(self.op.ref, ctypes.byref(self.raw), why, 512)
        if st == RC_OK:
            return ""
        if st == 2:
            return why.value.decode()
        raise RCError(st, "rc_validate")

    def apply(self, t: rc_transform) -> "Schedule":
        out = rc_schedule()
        _check(lib().rc_apply(self.op.ref, ctypes.byref(self.raw), ctypes.byref(t), ctypes.byref(out)),
               "rc_apply")
        return Schedule(self.op, out)

    def moves(self) -> List[rc_transform]:
        n = ctypes.c_size_t()
        _check(lib().rc_enumerate(self.op.ref, ctypes.byref(self.raw), None, 0, ctypes.byref(n)),
               "rc_enumerate")
        buf = (rc_transform * max(1, n.value))()
        _check(lib().rc_enumerate(self.op.ref, ctypes.byref(self.raw), buf, n.value, ctypes.byref(n)),
               "rc_enumerate")
        return list(buf[: n.value])

    def hash(self) -> int:
        return lib().rc_schedule_hash(ctypes.byref(self.raw))


def _precompile_worker(job):
    kind, dims, flags, texts, cache = job
    if cache:
        set_cache_dir(cache)
    op = Op(kind, dims, flags)
    return precompile(op, [op.from_string(t) for t in texts], nthreads=1)


def precompile_parallel(op: Op, schedules: Sequence[Schedule], nproc: int = 8,
                        cache_dir: Optional[str] = None) -> List[int]:
    """rc_precompile spread over worker processes: hipRTC serialises the
    compilations of one process, so parallel compilation needs processes."""
    import multiprocessing as mp
    texts = [str(s) for s in schedules]
    if nproc <= 1 or len(texts) <= 1:
        return precompile(op, schedules, 1)
    chunks = [texts[i::nproc] for i in range(nproc)]
    jobs = [(op.kind, op.dims, op.flags, c, cache_dir) for c in chunks if c]
    with mp.get_context("spawn").Pool(len(jobs)) as pool:
        res = pool.map(_precompile_worker, jobs)
    out = [0] * len(texts)
    for ci, r in enumerate(res):
        for j, st in enumerate(r):
            out[ci + j * nproc] = st
    return out


def precompile(op: Op, schedules: Sequence[Schedule], nthreads: int = 8) -> List[int]:
    n = len(schedules)
    arr = (rc_schedule * max(1, n))()
    for i, s in enumerate(schedules):
        arr[i] = s.raw
    st = (ctypes.c_int * max(1, n))()
    lib().rc_precompile(op.ref, arr, n, nthreads, st)
    return list(st[:n])


def describe(op: Op, sched: Schedule) -> List[dict]:
    """Launch shape and resources of each kernel of a schedule (no GPU)."""
    n = ctypes.c_int32()
    buf = (rc_kernel_info * 8)()
    _check(lib().rc_describe(op.ref, ctypes.byref(sched.raw), buf, 8, ctypes.byref(n)), "rc_describe")
    out = []
    for k in buf[: n.value]:
        out.append({f: (getattr(k, f).decode() if f == "name" else getattr(k, f))
                    for f, _ in rc_kernel_info._fields_ if f != "struct_size"})
    return out


def set_cache_dir(path: Optional[str]) -> None:
    _check(lib().rc_set_cache_dir(path.encode() if path else None), "rc_set_cache_dir")


# ---------------------------------------------------------------------------
# Plans (need a GPU)
# ---------------------------------------------------------------------------

def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream_ptr(stream) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


class Plan:
    """A compiled variant of an operator (rc_plan)."""

    def __init__(self, op: Op, sched: Schedule):
        h = ctypes.c_void_p()
        _check(lib().rc_plan_create(op.ref, ctypes.byref(sched.raw), ctypes.byref(h)), "rc_plan_create")
        self.op, self.sched, self.h = op, sched, h
        ws = ctypes.c_size_t()
        _check(lib().rc_plan_workspace(h, ctypes.byref(ws)), "rc_plan_workspace")
        self.workspace_bytes = ws.value
        nk, dom = ctypes.c_int32(), ctypes.c_int32()
        _check(lib().rc_plan_kernels(h, ctypes.byref(nk), ctypes.byref(dom)), "rc_plan_kernels")
        self.nkernels, self.dominant = nk.value, dom.value

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.rc_plan_destroy(self.h)
            self.h = None

    def kernel_flops(self, i: int) -> float:
        """Algorithmic FLOPs of kernel i of a launch."""
        f = ctypes.c_double()
        _check(lib().rc_plan_kernel_flops(self.h, i, ctypes.byref(f)), "rc_plan_kernel_flops")
        return f.value

    def buffer(self, name: str):
        """(byte offset, bytes) of a named part of the workspace."""
        off, n = ctypes.c_size_t(), ctypes.c_size_t()
        _check(lib().rc_plan_buffer(self.h, name.encode(), ctypes.byref(off), ctypes.byref(n)),
               "rc_plan_buffer")
        return off.value, n.value

    def workspace(self, device="cuda"):
        import torch
        if self.workspace_bytes == 0:
            return None
        return torch.empty(self.workspace_bytes, dtype=torch.uint8, device=device)

    @staticmethod
    def _args(inputs: Iterable, output) -> rc_args:
        a = rc_args()
        a.struct_size = ctypes.sizeof(rc_args)
        for i, t in enumerate(inputs):
            a.in_[i] = _ptr(t)
        a.out[0] = _ptr(output)
        return a

    class Prepared:
        """Argument block, workspace and stream of repeated launches, built once."""

        def __init__(self, plan, inputs, output, workspace, stream):
            self.plan = plan
            self.args = plan._args(inputs, output)
            self.keep = (list(inputs), output, workspace)       # keep tensors alive
            self.ws = _ptr(workspace)
            self.wsz = 0 if workspace is None else workspace.numel() * workspace.element_size()
            self.stream = _stream_ptr(stream)

        def events(self, events):
            handles = [int(e.cuda_event) for e in events]
            if not all(handles):
                raise ValueError("record each event once before use (torch creates events lazily)")
            return (ctypes.c_void_p * len(handles))(*handles)

        def launch(self) -> None:
            _check(lib().rc_launch(self.plan.h, ctypes.byref(self.args), self.ws, self.wsz, self.stream),
                   "rc_launch")

        def launch_timed(self, ev_array) -> None:
            _check(lib().rc_launch_timed(self.plan.h, ctypes.byref(self.args), self.ws, self.wsz,
                                         self.stream, ev_array, len(ev_array)), "rc_launch_timed")

    def prepare(self, inputs, output, workspace=None, stream=None) -> "Plan.Prepared":
        return Plan.Prepared(self, inputs, output, workspace, stream)

    def launch(self, inputs, output, workspace=None, stream=None) -> None:
        a = self._args(inputs, output)
        wsz = 0 if workspace is None else workspace.numel() * workspace.element_size()
        _check(lib().rc_launch(self.h, ctypes.byref(a), _ptr(workspace), wsz, _stream_ptr(stream)),
               "rc_launch")

    def launch_static(self, inputs, output, stream=None) -> None:
        """rc_launch_static: the workspace is the library's static array."""
        a = self._args(inputs, output)
        _check(lib().rc_launch_static(self.h, ctypes.byref(a), _stream_ptr(stream)), "rc_launch_static")

    def launch_timed(self, inputs, output, events, workspace=None, stream=None) -> None:
        """events: list of nkernels + 1 torch.cuda.Event(enable_timing=True),
        each already created (recorded once), since torch creates events lazily."""
        a = self._args(inputs, output)
        wsz = 0 if workspace is None else workspace.numel() * workspace.element_size()
        handles = [int(e.cuda_event) for e in events]
        if not all(handles):
            raise ValueError("launch_timed: record each event once before use (torch creates events lazily)")
        evs = (ctypes.c_void_p * len(events))(*handles)
        _check(lib().rc_launch_timed(self.h, ctypes.byref(a), _ptr(workspace), wsz,
                                     _stream_ptr(stream), evs, len(events)), "rc_launch_timed")

    def time(self, inputs, output, workspace=None, warmup=3, repeat=20, flush=True,
             stream=None) -> rc_timing:
        a = self._args(inputs, output)
        o = rc_time_opts()
        lib().rc_time_opts_init(ctypes.byref(o))
        o.warmup, o.repeat, o.flush = warmup, repeat, int(flush)
        t = rc_timing()
        wsz = 0 if workspace is None else workspace.numel() * workspace.element_size()
        _check(lib().rc_time(self.h, ctypes.byref(a), _ptr(workspace), wsz, _stream_ptr(stream),
                             ctypes.byref(o), ctypes.byref(t)), "rc_time")
        return t


def time_release() -> None:
    """Free rc_time's cache-flush buffers."""
    _check(lib().rc_time_release(), "rc_time_release")


# ---------------------------------------------------------------------------
# Search
# ---------------------------------------------------------------------------

class Search:
    """UCT / random / exhaustive search over schedules (rc_search_*).

    ``evaluate(schedule) -> reward`` returns a float >= 0, or None / raises to
    mark the schedule invalid.
    """

    def __init__(self, op: Op, evaluate: Callable[[Schedule], Optional[float]], policy=RC_POLICY_UCT,
                 budget=64, horizon=12, branching=2, c=math.sqrt(2.0), seed=0, max_invalid=-1,
                 propose: Optional[Callable[[Schedule, Optional[Schedule], Optional[Schedule]], str]] = None):
        self.op = op
        self._user_eval = evaluate
        self.errors: List[str] = []

        def _eval(_user, sp, rp):
            s = rc_schedule()
            ctypes.pointer(s)[0] = sp[0]
            try:
                r = self._user_eval(Schedule(op, s))
            except Exception as e:   # an evaluation failure marks the sample invalid
                self.errors.append(repr(e))
                return 1
            if r is None:
                return 1
            rp[0] = float(r)
            return 0

        self._cb = EVAL_FN(_eval)
        o = rc_search_opts()
        lib().rc_search_opts_init(ctypes.byref(o))
        o.policy, o.budget, o.horizon, o.branching, o.c, o.seed = policy, budget, horizon, branching, c, seed
        o.max_invalid = max_invalid
        h = ctypes.c_void_p()
        _check(lib().rc_search_create(op.ref, ctypes.byref(o), self._cb, None, ctypes.byref(h)),
               "rc_search_create")
        self.h = h
        self._pcb = None
        if propose is not None:
            def _prop(_user, at, par, gpar, buf, n):
                def mk(p):
                    if not p:
                        return None
                    s = rc_schedule()
                    ctypes.pointer(s)[0] = p[0]
                    return Schedule(op, s)
                try:
                    text = propose(mk(at), mk(par), mk(gpar)) or ""
                except Exception as e:
                    self.errors.append(repr(e))
                    text = ""
                data = text.encode()[: max(0, n - 1)] + b"\0"
                ctypes.memmove(buf, data, len(data))
                return 0
            self._pcb = PROPOSE_FN(_prop)
            _check(lib().rc_search_set_proposer(h, self._pcb, None), "rc_search_set_proposer")

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.rc_search_destroy(self.h)
            self.h = None

    def step(self) -> bool:
        done = ctypes.c_int32()
        _check(lib().rc_search_step(self.h, ctypes.byref(done)), "rc_search_step")
        return bool(done.value)

    def run(self) -> "Search":
        _check(lib().rc_search_run(self.h), "rc_search_run")
        return self

    def best(self):
        s, r, i = rc_schedule(), ctypes.c_double(), ctypes.c_int32()
        _check(lib().rc_search_best(self.h, ctypes.byref(s), ctypes.byref(r), ctypes.byref(i)),
               "rc_search_best")
        return Schedule(self.op, s), r.value, i.value

    def history(self) -> List[dict]:
        n = ctypes.c_int32()
        _check(lib().rc_search_history(self.h, None, 0, ctypes.byref(n)), "rc_search_history")
        buf = (rc_sample * max(1, n.value))()
        _check(lib().rc_search_history(self.h, buf, n.value, ctypes.byref(n)), "rc_search_history")
        out = []
        for smp in buf[: n.value]:
            s = rc_schedule()
            ctypes.pointer(s)[0] = smp.schedule
            out.append({"schedule": Schedule(self.op, s), "reward": smp.reward, "valid": bool(smp.valid),
                        "index": smp.index, "best_so_far": smp.best_so_far})
        return out

    def node_stats(self, path: Sequence[rc_transform]):
        arr = (rc_transform * max(1, len(path)))(*path)
        v, w = ctypes.c_int32(), ctypes.c_double()
        _check(lib().rc_search_node_stats(self.h, arr, len(path), ctypes.byref(v), ctypes.byref(w)),
               "rc_search_node_stats")
        return v.value, w.value

    def fallbacks(self) -> int:
        n = ctypes.c_int32()
        _check(lib().rc_search_fallbacks(self.h, ctypes.byref(n)), "rc_search_fallbacks")
        return n.value
