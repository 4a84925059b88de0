"""CPU oracle for the forward pass of a CNN partition [begin, end).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the GPU library.  The arithmetic lives
in ``oracle.c`` (fp64 accumulation, NCHW); this module loads it and walks the
layer graph.  A partition spans layers ``begin`` to ``end`` exclusive and
receives exactly one feature map, the output of layer ``begin - 1`` (the
paper's MILP inputs: C_ldbij covers layers i to j exclusive, Y_bj transfers
the feature map of layer j - 1).
"""
import ctypes
import os
from typing import Dict, List, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
DTYPE_CODES = {"f32": 0, "f16": 1, "bf16": 2}
ACT_CODES = {"none": 0, "relu": 1, "relu6": 2}

_lib = None
_f = ctypes.POINTER(ctypes.c_float)
_d = ctypes.POINTER(ctypes.c_double)
_i = ctypes.c_int


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    lib.oracle_round.restype = ctypes.c_double
    lib.oracle_round.argtypes = [ctypes.c_double, _i]
    lib.oracle_round_array.argtypes = [_d, ctypes.c_int64, _i, _f]
    lib.oracle_num_threads.restype = _i
    lib.oracle_out_dim.restype = _i
    lib.oracle_out_dim.argtypes = [_i, _i, _i, _i]
    lib.oracle_conv2d.argtypes = [_f, _i, _i, _i, _i, _f, _i, _i, _i, _i, _i, _i,
                                  _f, _f, _f, _f, _f, ctypes.c_double, _f, _i, _i, _f]
    lib.oracle_maxpool2d.argtypes = [_f, _i, _i, _i, _i, _i, _i, _i, _i, _f]
    lib.oracle_global_avgpool.argtypes = [_f, _i, _i, _i, _i, _i, _f]
    lib.oracle_linear.argtypes = [_f, _i, _i, _f, _i, _f, _i, _i, _i, _f]
    _lib = lib
    return lib


def _p(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.dtype == np.float32 and a.flags.c_contiguous
    return a.ctypes.data_as(_f)


def _c32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float32)


def num_threads() -> int:
    return _load().oracle_num_threads()


def round_to(x, dtype: str) -> np.ndarray:
    """Round fp64 values to the storage dtype (RNE), returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    y = np.empty(x.shape, dtype=np.float32)
    _load().oracle_round_array(x.ctypes.data_as(_d), x.size, DTYPE_CODES[dtype], _p(y))
    return y


def out_dim(n: int, k: int, s: int, p: int) -> int:
    return _load().oracle_out_dim(n, k, s, p)


def conv2d(x, w, stride=1, pad=0, groups=1, bias=None, bn=None, eps=1e-5,
           res=None, act="none", dtype="f32") -> np.ndarray:
    """x: [N, C, H, W]; w: [Co, C/groups, KH, KW]; bn: (gamma, beta, mean, var)."""
    x, w = _c32(x), _c32(w)
    N, C, H, W = x.shape
    Co, cig, KH, KW = w.shape
    if C % groups or Co % groups or cig != C // groups:
        raise ValueError("inconsistent groups / channel counts")
    Ho, Wo = out_dim(H, KH, stride, pad), out_dim(W, KW, stride, pad)
    y = np.empty((N, Co, Ho, Wo), dtype=np.float32)
    g = b = m = v = None
    if bn is not None:
        g, b, m, v = (_c32(t) for t in bn)
    res = _c32(res)
    if res is not None and res.shape != y.shape:
        raise ValueError(f"residual shape {res.shape} != output {y.shape}")
    _load().oracle_conv2d(_p(x), N, C, H, W, _p(w), Co, KH, KW, stride, pad, groups,
                          _p(_c32(bias)), _p(g), _p(b), _p(m), _p(v), float(eps),
                          _p(res), ACT_CODES[act], DTYPE_CODES[dtype], _p(y))
    return y


def maxpool2d(x, k, stride, pad=0, dtype="f32") -> np.ndarray:
    x = _c32(x)
    N, C, H, W = x.shape
    y = np.empty((N, C, out_dim(H, k, stride, pad), out_dim(W, k, stride, pad)),
                 dtype=np.float32)
    _load().oracle_maxpool2d(_p(x), N, C, H, W, k, stride, pad, DTYPE_CODES[dtype], _p(y))
    return y


def global_avgpool(x, dtype="f32") -> np.ndarray:
    x = _c32(x)
    N, C, H, W = x.shape
    y = np.empty((N, C, 1, 1), dtype=np.float32)
    _load().oracle_global_avgpool(_p(x), N, C, H, W, DTYPE_CODES[dtype], _p(y))
    return y


def linear(x, w, bias=None, act="none", softmax=False, dtype="f32") -> np.ndarray:
    """x: [N, ...] flattened in C order (NCHW); w: [O, K]."""
    x = _c32(np.asarray(x).reshape(np.asarray(x).shape[0], -1))
    w = _c32(w)
    N, K = x.shape
    O = w.shape[0]
    if w.shape[1] != K:
        raise ValueError(f"fc expects {w.shape[1]} inputs, got {K}")
    y = np.empty((N, O), dtype=np.float32)
    _load().oracle_linear(_p(x), N, K, _p(w), O, _p(_c32(bias)), ACT_CODES[act],
                          1 if softmax else 0, DTYPE_CODES[dtype], _p(y))
    return y


def run_layer(L, p: Dict[str, np.ndarray], x: np.ndarray, res: Optional[np.ndarray],
              dtype: str) -> np.ndarray:
    """Forward of one fused layer; x and res are NCHW (or [N, K] for fc input)."""
    if L.op == "conv":
        bn = None
        if L.bn:
            bn = (p["bn_gamma"], p["bn_beta"], p["bn_mean"], p["bn_var"])
        return conv2d(x, p["weight"], L.stride, L.pad, L.groups, p.get("bias"), bn,
                      1e-5, res, L.act, dtype)
    if res is not None:
        raise ValueError(f"{L.name}: residual input on a {L.op} layer")
    if L.op == "maxpool":
        return maxpool2d(x, L.k, L.stride, L.pad, dtype)
    if L.op == "gap":
        return global_avgpool(x, dtype)
    if L.op in ("fc", "fc_softmax"):
        return linear(x, p["weight"], p.get("bias"), L.act, L.op == "fc_softmax", dtype)
    raise ValueError(f"unknown op {L.op!r}")


def forward(layers: List, params: Dict[int, Dict[str, np.ndarray]], begin: int, end: int,
            x: np.ndarray, dtype: str, keep: bool = False):
    """Run layers [begin, end) on x (NCHW, the output of layer begin-1 or the
    model input when begin == 0).  Returns the last layer's output, and with
    keep=True also the dict of every layer's output."""
    if not 0 <= begin < end <= len(layers):
        raise ValueError(f"bad range [{begin}, {end})")
    outs: Dict[int, np.ndarray] = {begin - 1: np.ascontiguousarray(x, dtype=np.float32)}

    def fetch(i: int, who: str) -> np.ndarray:
        if i not in outs:
            raise ValueError(f"{who} reads layer {i}, which is not available to "
                             f"partition [{begin}, {end})")
        return outs[i]

    for i in range(begin, end):
        L = layers[i]
        src = fetch(L.src, L.name)          # -1 names the model input
        res = fetch(L.res_src, L.name) if L.res_src >= 0 else None
        outs[i] = run_layer(L, params.get(i, {}), src, res, dtype)
        if not keep:
            # free what no later layer of the range reads
            for j in list(outs):
                if j == i:
                    continue
                if not any(layers[t].src == j or layers[t].res_src == j
                           for t in range(i + 1, end)):
                    del outs[j]
    return (outs[end - 1], outs) if keep else outs[end - 1]
