"""TEST INFRASTRUCTURE ONLY -- ctypes front end of the oracle's C arithmetic.

``oracle/carith.c`` holds the canonical fp32 operation sequence of the
scoring path (see that file's header).  This module compiles it with gcc
(``-O2 -ffp-contract=off``, no fast-math) into ``oracle/_carith.so`` and
exposes numpy-friendly wrappers.  Only tests, the smoke check and the
benchmark's CPU-baseline leg use it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "carith.c")
_LIB = os.path.join(_HERE, "_carith.so")
_lib = None

_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(dtype=np.int32, flags="C_CONTIGUOUS")


def build(force: bool = False) -> str:
    """Compile carith.c into _carith.so (always when force=True)."""
    if force or not os.path.exists(_LIB) or (
            os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call([
            "gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-fopenmp",
            "-ffp-contract=off", "-fno-fast-math", "-frounding-math",
            _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        L.orc_cexp.restype = ctypes.c_float
        L.orc_cexp.argtypes = [ctypes.c_float]
        L.orc_cexp_array.restype = None
        L.orc_cexp_array.argtypes = [_f32p, _f32p, ctypes.c_int64]
        L.orc_cdot.restype = ctypes.c_float
        L.orc_cdot.argtypes = [_f32p, _f32p, ctypes.c_int]
        L.orc_cdot_matrix.restype = None
        L.orc_cdot_matrix.argtypes = [_f32p, ctypes.c_int, _f32p,
                                      ctypes.c_int, ctypes.c_int, _f32p]
        L.orc_route.restype = None
        L.orc_route.argtypes = [_f32p, ctypes.c_int, ctypes.c_int, _f32p,
                                ctypes.c_void_p, ctypes.c_int, ctypes.c_int,
                                ctypes.c_int, _f32p, _i32p, _f32p]
        L.orc_predict.restype = None
        L.orc_predict.argtypes = [_f32p, ctypes.c_int, ctypes.c_int, _f32p,
                                  _f32p, ctypes.c_int, _i32p, _f32p, _f32p,
                                  ctypes.c_void_p]
        L.orc_aggregate.restype = None
        L.orc_aggregate.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    _i32p, _f32p, _f32p, _i32p]
        L.orc_gates.restype = None
        L.orc_gates.argtypes = [_f32p, _i32p, ctypes.c_int, ctypes.c_int,
                                ctypes.c_int, _i32p, ctypes.c_int,
                                ctypes.c_int, _f32p]
        _lib = L
    return _lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def cexp(x):
    x = _f32(np.atleast_1d(x))
    y = np.empty_like(x)
    lib().orc_cexp_array(x.ravel(), y.ravel(), x.size)
    return y


def cdot(p, q):
    p, q = _f32(p), _f32(q)
    assert p.shape == q.shape and p.ndim == 1 and p.size % 256 == 0
    return np.float32(lib().orc_cdot(p, q, p.size))


def cdot_matrix(P, Q):
    P, Q = _f32(P), _f32(Q)
    assert P.shape[1] == Q.shape[1] and P.shape[1] % 256 == 0
    out = np.empty((P.shape[0], Q.shape[0]), dtype=np.float32)
    lib().orc_cdot_matrix(P, P.shape[0], Q, Q.shape[0], P.shape[1], out)
    return out


def route(x, w_router, b_router, K, norm_topk=1):
    """Router logits [B,E], top-K ids [B,K] and weights [B,K] (fp32)."""
    x, W = _f32(x), _f32(w_router)
    B, d = x.shape
    E = W.shape[0]
    assert d % 256 == 0 and W.shape[1] == d and 1 <= K <= min(16, E)
    logits = np.empty((B, E), np.float32)
    ids = np.empty((B, K), np.int32)
    w = np.empty((B, K), np.float32)
    if b_router is None:
        bp = None
    else:
        b_router = _f32(b_router)
        bp = b_router.ctypes.data_as(ctypes.c_void_p)
    lib().orc_route(x, B, d, W, bp, E, K, int(norm_topk), logits, ids, w)
    return logits, ids, w


def predict(x, pred_a, pred_b, ids, w, return_inv=False):
    """Per routed pair cost w^2 * cexp(a_u . z_bar + b_u) [B,K] (fp32)."""
    x, A, b = _f32(x), _f32(pred_a), _f32(pred_b)
    ids, w = _i32(ids), _f32(w)
    B, d = x.shape
    K = ids.shape[1]
    cost = np.empty((B, K), np.float32)
    inv = np.empty(B, np.float32)
    lib().orc_predict(x, B, d, A, b, K, ids, w, cost,
                      inv.ctypes.data_as(ctypes.c_void_p))
    return (cost, inv) if return_inv else cost


def aggregate(ids, cost, E):
    """Batch scores D_hat [E] (fp32, fixed order) and route counts [E]."""
    ids, cost = _i32(ids), _f32(cost)
    B, K = ids.shape
    scores = np.empty(E, np.float32)
    counts = np.empty(E, np.int32)
    lib().orc_aggregate(B, K, E, ids, cost, scores, counts)
    return scores, counts


def gates(logits_t, ids_t, exec_t, norm_topk=1, renorm=False):
    lt, it, ex = _f32(logits_t), _i32(ids_t), _i32(exec_t)
    g = np.empty(max(1, ex.size), np.float32)
    lib().orc_gates(lt, it, lt.size, it.size, int(norm_topk), ex, ex.size,
                    int(renorm), g)
    return g[:ex.size]
