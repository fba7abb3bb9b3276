"""Python binding of libios (MI355X-native IOS: inter-operator scheduling and
stage execution of multi-branch CNN blocks).

Every function below has the name of the C entry point it wraps (see
``include/ios.h``) and only marshals arguments: graph building, the schedule
search and every kernel run inside ``libios.so``.  PyTorch is used by callers
for device memory and streams only.

The library must have been built (``python paper_2011_01302_amd/build.py``);
importing this package fails loudly when it is missing.
"""
from __future__ import annotations

import ctypes
import os
from typing import Callable, Dict, List, Optional, Sequence, Tuple

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libios.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python paper_2011_01302_amd/build.py`")

# One HIP runtime per process.  PyTorch-ROCm ships its own libamdhip64 and
# links it by the unversioned name; if libios.so were loaded first it would
# pull in the system runtime, torch would then load its copy as a second
# runtime, and the two would not share the GPU (the second reports "no
# ROCm-capable device").  Loading torch first makes libios bind to torch's
# runtime by soname.
try:
    import torch  # noqa: F401
except ImportError:   # no torch: libios uses the system HIP runtime
    pass

_lib = ctypes.CDLL(LIB_PATH)

# ------------------------------------------------------------------ constants
IOS_OK = 0
ERRORS = {-1: "IOS_E_ARG", -2: "IOS_E_SHAPE", -3: "IOS_E_STATE", -4: "IOS_E_NOT_MERGEABLE",
          -5: "IOS_E_BAD_STAGE", -6: "IOS_E_TOO_MANY_OPS", -7: "IOS_E_OOM", -8: "IOS_E_HIP",
          -9: "IOS_E_COST_FN", -10: "IOS_E_UNSUPPORTED", -11: "IOS_E_DEVICE"}
IOS_CONV, IOS_SEPCONV, IOS_POOL_MAX, IOS_POOL_AVG, IOS_ADD, IOS_MEAN, IOS_CONCAT, IOS_IDENTITY = range(8)
IOS_CONCURRENT, IOS_MERGE = 0, 1
IOS_SCHED_DP, IOS_SCHED_SEQUENTIAL, IOS_SCHED_GREEDY = 0, 1, 2
IOS_CONV_TILE_SHAPES = 12
INT64_MAX = (1 << 63) - 1

EXPORTED = ["ios_graph_create", "ios_graph_destroy", "ios_add_input", "ios_add_op",
            "ios_mark_output", "ios_graph_finalize", "ios_graph_blocks", "ios_block_units",
            "ios_stage_mergeable", "ios_profile_stage", "ios_get_conv_tile", "ios_set_conv_tile",
            "ios_get_unit_tiling", "ios_set_unit_tiling",
            "ios_sched_opts_default", "ios_schedule",
            "ios_schedule_from_stages", "ios_schedule_get", "ios_schedule_stats",
            "ios_schedule_tune_tiles", "ios_schedule_destroy", "ios_schedule_dump_costs", "ios_run", "ios_run_noalloc",
            "ios_run_timed",
            "ios_device_status", "ios_last_error"]


class IosError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code
        self.name = ERRORS.get(code, str(code))


class ios_op_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("kind", "cout", "kh", "kw", "stride_h", "stride_w", "pad_h", "pad_w",
                 "pre_relu", "post_relu", "block_id")]


class ios_sched_opts(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("mode", "r", "s", "strategies", "warmup", "reps", "repeats", "verify_reps")]


COST_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64,
                           ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.c_int32,
                           ctypes.POINTER(ctypes.c_int64))

_P = ctypes.c_void_p
_i32, _i64 = ctypes.c_int32, ctypes.c_int64
_pi32, _pi64 = ctypes.POINTER(_i32), ctypes.POINTER(_i64)
_pf = ctypes.POINTER(ctypes.c_float)

_sig = {
    "ios_graph_create": (ctypes.c_int, [_i32, ctypes.POINTER(_P)]),
    "ios_graph_destroy": (None, [_P]),
    "ios_add_input": (ctypes.c_int, [_P, _i32, _i32, _i32, _pi32]),
    "ios_add_op": (ctypes.c_int, [_P, ctypes.POINTER(ios_op_desc), _pi32, _i32, _pf, _pf, _pi32]),
    "ios_mark_output": (ctypes.c_int, [_P, _i32]),
    "ios_graph_finalize": (ctypes.c_int, [_P]),
    "ios_graph_blocks": (ctypes.c_int, [_P, _pi32]),
    "ios_block_units": (ctypes.c_int, [_P, _i32, _pi32, _pi32]),
    "ios_stage_mergeable": (ctypes.c_int, [_P, _pi32, _i32, _pi32]),
    "ios_profile_stage": (ctypes.c_int, [_P, _pi32, _i32, _i32, _i32, _i32, _i32, _pi64]),
    "ios_get_conv_tile": (ctypes.c_int, [_P, _i32, _pi32]),
    "ios_set_conv_tile": (ctypes.c_int, [_P, _i32, _i32]),
    "ios_get_unit_tiling": (ctypes.c_int, [_P, _i32, _pi32, _pi32]),
    "ios_set_unit_tiling": (ctypes.c_int, [_P, _i32, _i32, _i32]),
    "ios_sched_opts_default": (None, [ctypes.POINTER(ios_sched_opts)]),
    "ios_schedule": (ctypes.c_int, [_P, ctypes.POINTER(ios_sched_opts), COST_FN, _P,
                                    ctypes.POINTER(_P), _pi64]),
    "ios_schedule_from_stages": (ctypes.c_int, [_P, _i32, _pi32, _pi32, _pi32, ctypes.POINTER(_P)]),
    "ios_schedule_get": (ctypes.c_int, [_P, _pi32, ctypes.POINTER(_pi32), ctypes.POINTER(_pi32),
                                        ctypes.POINTER(_pi32)]),
    "ios_schedule_stats": (ctypes.c_int, [_P, _pi64, _pi64, _pi64]),
    "ios_schedule_tune_tiles": (ctypes.c_int, [_P, _P, ctypes.POINTER(ios_sched_opts), _pi64]),
    "ios_schedule_destroy": (None, [_P]),
    "ios_schedule_dump_costs": (ctypes.c_int, [_P, ctypes.c_char_p]),
    "ios_run": (ctypes.c_int, [_P, _P, ctypes.POINTER(_P), ctypes.POINTER(_P), _P]),
    "ios_run_noalloc": (ctypes.c_int, [_P, _P, ctypes.POINTER(_P), ctypes.POINTER(_P), _P]),
    "ios_run_timed": (ctypes.c_int, [_P, _P, ctypes.POINTER(_P), ctypes.POINTER(_P), _P, _pi64]),
    "ios_device_status": (ctypes.c_int, [_P, _P, _pi32]),
    "ios_last_error": (ctypes.c_char_p, []),
}
for _name, (_res, _args) in _sig.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def _check(rc: int):
    if rc != IOS_OK:
        raise IosError(rc, _lib.ios_last_error().decode())


def _i32arr(vals: Sequence[int]):
    return (_i32 * max(len(vals), 1))(*vals)


def _fptr(arr) -> Optional[ctypes.POINTER(ctypes.c_float)]:
    """Host float32 buffer (numpy array) -> float*; None stays NULL."""
    if arr is None:
        return None
    import numpy as np
    a = np.ascontiguousarray(arr, dtype=np.float32)
    _keep.append(a)
    return a.ctypes.data_as(_pf)


_keep: list = []


# ------------------------------------------------------------------ C calls

def ios_graph_create(batch: int) -> int:
    g = _P()
    _check(_lib.ios_graph_create(batch, ctypes.byref(g)))
    return g.value


def ios_graph_destroy(g: int) -> None:
    _lib.ios_graph_destroy(g)


def ios_add_input(g: int, c: int, h: int, w: int) -> int:
    t = _i32()
    _check(_lib.ios_add_input(g, c, h, w, ctypes.byref(t)))
    return t.value


def ios_add_op(g: int, desc: ios_op_desc, in_ids: Sequence[int], weights=None, bias=None) -> int:
    t = _i32()
    try:
        rc = _lib.ios_add_op(g, ctypes.byref(desc), _i32arr(in_ids), len(in_ids), _fptr(weights),
                             _fptr(bias), ctypes.byref(t))
    finally:
        _keep.clear()
    _check(rc)
    return t.value


def ios_mark_output(g: int, tensor_id: int) -> None:
    _check(_lib.ios_mark_output(g, tensor_id))


def ios_graph_finalize(g: int) -> None:
    _check(_lib.ios_graph_finalize(g))


def ios_graph_blocks(g: int) -> int:
    n = _i32()
    _check(_lib.ios_graph_blocks(g, ctypes.byref(n)))
    return n.value


def ios_block_units(g: int, block: int) -> List[int]:
    n = _i32()
    ids = (_i32 * 64)()
    _check(_lib.ios_block_units(g, block, ctypes.byref(n), ids))
    return list(ids[:n.value])


def ios_stage_mergeable(g: int, unit_ids: Sequence[int]) -> bool:
    ok = _i32()
    _check(_lib.ios_stage_mergeable(g, _i32arr(unit_ids), len(unit_ids), ctypes.byref(ok)))
    return bool(ok.value)


def ios_profile_stage(g: int, unit_ids: Sequence[int], strategy: int = IOS_CONCURRENT,
                      warmup: int = 3, reps: int = 20, repeats: int = 3) -> int:
    ns = _i64()
    _check(_lib.ios_profile_stage(g, _i32arr(unit_ids), len(unit_ids), strategy, warmup, reps,
                                  repeats, ctypes.byref(ns)))
    return ns.value


def ios_get_conv_tile(g: int, unit_id: int) -> int:
    v = _i32()
    _check(_lib.ios_get_conv_tile(g, unit_id, ctypes.byref(v)))
    return v.value


def ios_set_conv_tile(g: int, unit_id: int, shape: int) -> None:
    _check(_lib.ios_set_conv_tile(g, unit_id, shape))


def ios_get_unit_tiling(g: int, unit_id: int) -> Tuple[int, int]:
    t, x = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.ios_get_unit_tiling(g, unit_id, ctypes.byref(t), ctypes.byref(x)))
    return t.value, x.value


def ios_set_unit_tiling(g: int, unit_id: int, tile: int, xcd_lg: int) -> None:
    _check(_lib.ios_set_unit_tiling(g, unit_id, tile, xcd_lg))


def ios_sched_opts_default() -> ios_sched_opts:
    o = ios_sched_opts()
    _lib.ios_sched_opts_default(ctypes.byref(o))
    return o


def ios_schedule(g: int, opts: Optional[ios_sched_opts] = None,
                 cost: Optional[Callable[[int, int, List[int], int], int]] = None) -> Tuple[int, int]:
    """Returns (schedule handle, minimised cost in ns).  ``cost(block, mask,
    unit_ids, strategy) -> ns`` replaces the on-device profiler when given."""
    opts = opts or ios_sched_opts_default()
    err: list = []

    def tramp(ctx, block, mask, ids, n, strategy, out):
        try:
            v = cost(block, mask, [ids[i] for i in range(n)], strategy)
            out[0] = INT64_MAX if v is None or v == float("inf") else int(v)
            return 0
        except Exception as e:  # propagated as IOS_E_COST_FN
            err.append(e)
            return 1

    cb = COST_FN(tramp) if cost is not None else COST_FN()
    q = _P()
    c = _i64()
    rc = _lib.ios_schedule(g, ctypes.byref(opts), cb, None, ctypes.byref(q), ctypes.byref(c))
    if rc != IOS_OK and err:
        raise IosError(rc, f"cost callback raised {err[0]!r}") from err[0]
    _check(rc)
    return q.value, c.value


def ios_schedule_from_stages(g: int, stages: Sequence[Sequence[int]], strategies: Sequence[int]) -> int:
    offs, ids = [0], []
    for st in stages:
        ids += list(st)
        offs.append(len(ids))
    q = _P()
    _check(_lib.ios_schedule_from_stages(g, len(stages), _i32arr(offs), _i32arr(ids),
                                         _i32arr(strategies), ctypes.byref(q)))
    return q.value


def ios_schedule_get(q: int) -> List[Tuple[List[int], int]]:
    n = _i32()
    offs, ids, strat = _pi32(), _pi32(), _pi32()
    _check(_lib.ios_schedule_get(q, ctypes.byref(n), ctypes.byref(offs), ctypes.byref(ids),
                                 ctypes.byref(strat)))
    return [([ids[i] for i in range(offs[k], offs[k + 1])], strat[k]) for k in range(n.value)]


def ios_schedule_stats(q: int) -> Tuple[int, int, int]:
    a, b, c = _i64(), _i64(), _i64()
    _check(_lib.ios_schedule_stats(q, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
    return a.value, b.value, c.value


def ios_schedule_tune_tiles(g: int, q: int, opts: Optional[ios_sched_opts] = None) -> int:
    """Per-stage conv tile shapes for schedule q (kept on the graph); returns
    the sum of the stages' measured latencies in ns."""
    opts = opts or ios_sched_opts_default()
    c = _i64()
    _check(_lib.ios_schedule_tune_tiles(g, q, ctypes.byref(opts), ctypes.byref(c)))
    return c.value


def ios_schedule_destroy(q: int) -> None:
    _lib.ios_schedule_destroy(q)


def ios_schedule_dump_costs(g: int, path: str) -> None:
    _check(_lib.ios_schedule_dump_costs(g, path.encode()))


def _ptrs(vals: Sequence[int]):
    return (_P * max(len(vals), 1))(*vals)


def ios_run(g: int, q: int, d_inputs: Sequence[int], d_outputs: Sequence[int], stream: int = 0) -> None:
    """Device pointers (ints, e.g. ``tensor.data_ptr()``) and a hipStream_t
    (e.g. ``torch.cuda.current_stream().cuda_stream``)."""
    _check(_lib.ios_run(g, q, _ptrs(d_inputs), _ptrs(d_outputs), stream or None))


def ios_run_noalloc(g: int, q: int, d_inputs: Sequence[int], d_outputs: Sequence[int], stream: int = 0) -> None:
    _check(_lib.ios_run_noalloc(g, q, _ptrs(d_inputs), _ptrs(d_outputs), stream or None))


def ios_run_timed(g: int, q: int, d_inputs: Sequence[int], d_outputs: Sequence[int], stream: int = 0,
                  n_stages: Optional[int] = None) -> List[int]:
    n = n_stages if n_stages is not None else len(ios_schedule_get(q))
    out = (_i64 * max(n, 1))()
    _check(_lib.ios_run_timed(g, q, _ptrs(d_inputs), _ptrs(d_outputs), stream or None, out))
    return list(out[:n])


def ios_device_status(g: int, stream: int = 0) -> int:
    f = _i32()
    _check(_lib.ios_device_status(g, stream or None, ctypes.byref(f)))
    return f.value


def ios_last_error() -> str:
    return _lib.ios_last_error().decode()


# ------------------------------------------------------------------ graph from a description

_KIND = {"conv": IOS_CONV, "sepconv": IOS_SEPCONV, "maxpool": IOS_POOL_MAX, "avgpool": IOS_POOL_AVG,
         "add": IOS_ADD, "mean": IOS_MEAN, "concat": IOS_CONCAT, "identity": IOS_IDENTITY}


class Graph:
    """A finalized libios graph built from a workload description.

    ``spec`` lists inputs and operators in insertion order (see
    ``workloads``); ``tensors`` maps ``<op>.w`` / ``<op>.b`` / ``<op>.dw`` /
    ``<op>.pw`` to float32 arrays.  Names map to tensor ids in ``self.tid``."""

    def __init__(self, spec: dict, tensors: Dict[str, "object"], batch: Optional[int] = None):
        import numpy as np
        self.spec = spec
        self.batch = batch or spec["batch"]
        self.handle = ios_graph_create(self.batch)
        self.tid: Dict[str, int] = {}
        self.name_of: Dict[int, str] = {}
        try:
            for t in spec["inputs"]:
                self.tid[t["name"]] = ios_add_input(self.handle, t["c"], t["h"], t["w"])
            for op in spec["ops"]:
                d = ios_op_desc()
                d.kind = _KIND[op["kind"]]
                d.cout = op.get("cout", 0)
                d.kh, d.kw = op.get("kh", 1), op.get("kw", 1)
                d.stride_h, d.stride_w = op.get("sh", 1), op.get("sw", 1)
                d.pad_h, d.pad_w = op.get("ph", 0), op.get("pw", 0)
                d.pre_relu, d.post_relu = op.get("pre_relu", 0), op.get("post_relu", 0)
                d.block_id = op.get("block", -1)
                w = b = None
                nm = op["name"]
                if op["kind"] == "conv":
                    w, b = tensors[nm + ".w"], tensors.get(nm + ".b")
                elif op["kind"] == "sepconv":
                    w = np.concatenate([np.ravel(tensors[nm + ".dw"]), np.ravel(tensors[nm + ".pw"])])
                    b = tensors.get(nm + ".b")
                tid = ios_add_op(self.handle, d, [self.tid[i] for i in op["in"]], w, b)
                self.tid[nm] = tid
                self.name_of[tid] = nm
            for o in spec["outputs"]:
                ios_mark_output(self.handle, self.tid[o])
            ios_graph_finalize(self.handle)
        except Exception:
            ios_graph_destroy(self.handle)
            self.handle = None
            raise

    def close(self):
        if self.handle:
            ios_graph_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def blocks(self) -> List[List[int]]:
        return [ios_block_units(self.handle, b) for b in range(ios_graph_blocks(self.handle))]

    def names(self, ids: Sequence[int]) -> List[str]:
        return [self.name_of[i] for i in ids]
