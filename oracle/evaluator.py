"""Oracle DAG evaluator (TEST INFRASTRUCTURE ONLY).

Evaluates a workload description op by op, in insertion order (which is
topological, Sec. 3 "Computation Graph"), entirely in float64:

* conv      -> ``oracle_conv2d`` (C, direct loops)
* sepconv   -> sum of inputs, ReLU, ``oracle_depthwise``, then a 1x1
               ``oracle_conv2d`` ("Relu-SepConv", Table 2)
* pools     -> ``oracle_pool``
* add/mean  -> numpy sums of the inputs
* concat    -> channel concatenation; identity -> the input itself

Operator merge (Sec. 3, "Parallelization Strategy") is modelled separately
by ``merged_conv`` so that a test can check it against separate convs.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "evaluator.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_dp = ctypes.POINTER(ctypes.c_double)


def build(force: bool = False) -> str:
    """Compile evaluator.c with gcc into oracle/liboracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-ffp-contract=off", "-fno-fast-math", "-shared",
                               "-fPIC", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        i = ctypes.c_int
        lib.oracle_conv2d.argtypes = [_dp, i, i, i, i, _dp, i, i, i, i, i, i, i, _dp, i, i, _dp]
        lib.oracle_depthwise.argtypes = [_dp, i, i, i, i, _dp, i, i, i, i, _dp]
        lib.oracle_pool.argtypes = [_dp, i, i, i, i, i, i, i, i, _dp]
        for f in (lib.oracle_conv2d, lib.oracle_depthwise, lib.oracle_pool):
            f.restype = None
        _lib = lib
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(_dp)


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def conv2d(x, w, bias=None, stride=(1, 1), pad=(0, 0), pre_relu=False, post_relu=False):
    x, w = _f64(x), _f64(w)
    n, c, h, wd = x.shape
    cout, cin, kh, kw = w.shape
    assert cin == c, (cin, c)
    ho = (h + 2 * pad[0] - kh) // stride[0] + 1
    wo = (wd + 2 * pad[1] - kw) // stride[1] + 1
    y = np.empty((n, cout, ho, wo), dtype=np.float64)
    b = _f64(bias) if bias is not None else None
    _load().oracle_conv2d(_p(x), n, c, h, wd, _p(w), cout, kh, kw, stride[0], stride[1],
                          pad[0], pad[1], _p(b) if b is not None else None,
                          int(pre_relu), int(post_relu), _p(y))
    return y


def depthwise(x, w, pad):
    x, w = _f64(x), _f64(w)
    n, c, h, wd = x.shape
    assert w.shape[0] == c and w.shape[1] == 1
    kh, kw = w.shape[2], w.shape[3]
    ho, wo = h + 2 * pad[0] - kh + 1, wd + 2 * pad[1] - kw + 1
    y = np.empty((n, c, ho, wo), dtype=np.float64)
    _load().oracle_depthwise(_p(x), n, c, h, wd, _p(w), kh, kw, pad[0], pad[1], _p(y))
    return y


def pool(x, k, stride, pad, is_max):
    x = _f64(x)
    n, c, h, wd = x.shape
    ho = (h + 2 * pad - k) // stride + 1
    wo = (wd + 2 * pad - k) // stride + 1
    y = np.empty((n, c, ho, wo), dtype=np.float64)
    _load().oracle_pool(_p(x), n, c, h, wd, k, stride, pad, int(is_max), _p(y))
    return y


def sepconv(inputs: Sequence[np.ndarray], dw, pw, bias, pad, pre_relu=True):
    """Relu-SepConv unit: t = dw(ReLU(sum inputs)); y = pw(t) + bias."""
    s = _f64(inputs[0]).copy()
    for t in inputs[1:]:
        s = s + _f64(t)
    if pre_relu:
        s = np.maximum(s, 0.0)
    t = depthwise(s, dw, pad)
    return conv2d(t, pw, bias)


def eval_op(op: dict, env: Dict[str, np.ndarray], tensors: Dict[str, np.ndarray]) -> np.ndarray:
    """The output of one operator whose inputs are in ``env`` (float64)."""
    k = op["kind"]
    ins = [env[i] for i in op["in"]]
    nm = op["name"]
    if k == "conv":
        return conv2d(ins[0], tensors[nm + ".w"], tensors.get(nm + ".b"),
                      (op["sh"], op["sw"]), (op["ph"], op["pw"]),
                      op.get("pre_relu", 0), op.get("post_relu", 0))
    if k == "sepconv":
        return sepconv(ins, tensors[nm + ".dw"], tensors[nm + ".pw"],
                       tensors.get(nm + ".b"), (op["ph"], op["pw"]), op.get("pre_relu", 1))
    if k in ("maxpool", "avgpool"):
        assert op["kh"] == op["kw"] and op["sh"] == op["sw"] and op["ph"] == op["pw"]
        return pool(ins[0], op["kh"], op["sh"], op["ph"], k == "maxpool")
    if k == "add":
        s = ins[0].copy()
        for t in ins[1:]:
            s = s + t
        return s
    if k == "mean":
        s = ins[0].copy()
        for t in ins[1:]:
            s = s + t
        return s / float(len(ins))
    if k == "concat":
        return np.concatenate(ins, axis=1)
    if k == "identity":
        return ins[0]
    raise ValueError(k)


def evaluate(spec: dict, tensors: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    """Every named tensor of the block, as float64 arrays."""
    env = {t["name"]: _f64(tensors[t["name"]]) for t in spec["inputs"]}
    for op in spec["ops"]:
        env[op["name"]] = eval_op(op, env, tensors)
    return env


def outputs(spec: dict, tensors: Dict[str, np.ndarray]) -> List[np.ndarray]:
    env = evaluate(spec, tensors)
    return [env[o] for o in spec["outputs"]]


def merged_conv(x, convs: List[dict], stride=(1, 1)):
    """Operator merge (Sec. 3): stack the kernels of convs that read the same
    input along output channels, each zero-padded (centred) to the largest
    kernel size, run one conv, then split the output back per op.

    ``convs`` items: {"w": [Cout,Cin,kh,kw], "b": [Cout] or None,
    "pad": (ph, pw), "pre_relu", "post_relu"}.  All must share pre/post ReLU
    and give the same output size after centring.
    """
    KH = max(c["w"].shape[2] for c in convs)
    KW = max(c["w"].shape[3] for c in convs)
    cin = convs[0]["w"].shape[1]
    total = sum(c["w"].shape[0] for c in convs)
    wm = np.zeros((total, cin, KH, KW), dtype=np.float64)
    bm = np.zeros((total,), dtype=np.float64)
    pads = set()
    o = 0
    for c in convs:
        co, ci, kh, kw = c["w"].shape
        dh, dw = (KH - kh) // 2, (KW - kw) // 2
        assert 2 * dh == KH - kh and 2 * dw == KW - kw, "kernel cannot be centred"
        wm[o:o + co, :, dh:dh + kh, dw:dw + kw] = c["w"]
        if c.get("b") is not None:
            bm[o:o + co] = c["b"]
        pads.add((c["pad"][0] + dh, c["pad"][1] + dw))
        o += co
    assert len(pads) == 1, "merged convs must give the same output size"
    pad = pads.pop()
    y = conv2d(x, wm, bm, stride, pad, convs[0].get("pre_relu", 0), convs[0].get("post_relu", 0))
    parts, o = [], 0
    for c in convs:
        co = c["w"].shape[0]
        parts.append(y[:, o:o + co])
        o += co
    return parts
