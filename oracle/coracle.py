"""ctypes front end of the C recurrent oracle (``mlstm_oracle.c``).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build_oracle

_lib = None


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("MLSTM_ORACLE_LIBRARY") or build_oracle.build(force=False)
        lib = ctypes.CDLL(path)
        dp = ctypes.POINTER(ctypes.c_double)
        lib.oracle_mlstm_recurrent_f64.argtypes = [dp, dp, dp, dp, dp, dp, dp, dp,
                                                   ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                                   ctypes.c_int64, dp, dp, dp, dp, ctypes.c_int]
        lib.oracle_mlstm_recurrent_f64.restype = ctypes.c_int
        lib.oracle_max_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def _p(x):
    if x is None:
        return None
    assert x.dtype == np.float64 and x.flags.c_contiguous
    return x.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def recurrent(q, k, v, ipre, fpre, C0=None, n0=None, m0=None, nthreads=None):
    """Recurrent fp64 oracle.  Arrays as in ``mlstm_ref`` (leading sequence axis S).

    Returns ``h [S,T,DV], C [S,DQK,DV], n [S,DQK], m [S]`` in fp64.
    """
    lib = _load()
    c = lambda a: None if a is None else np.ascontiguousarray(a, dtype=np.float64)
    q, k, v, ipre, fpre, C0, n0, m0 = map(c, (q, k, v, ipre, fpre, C0, n0, m0))
    S, T, DQK = q.shape
    DV = v.shape[2]
    assert k.shape == (S, T, DQK) and v.shape == (S, T, DV)
    assert ipre.shape == (S, T) and fpre.shape == (S, T)
    h = np.empty((S, T, DV))
    C = np.empty((S, DQK, DV))
    n = np.empty((S, DQK))
    m = np.empty((S,))
    rc = lib.oracle_mlstm_recurrent_f64(_p(q), _p(k), _p(v), _p(ipre), _p(fpre), _p(C0), _p(n0), _p(m0),
                                        S, T, DQK, DV, _p(h), _p(C), _p(n), _p(m),
                                        int(nthreads or default_threads()))
    if rc != 0:
        raise ValueError("oracle_mlstm_recurrent_f64 rejected its arguments")
    return h, C, n, m


def recurrent_inputs(inp, nthreads=None, T=None):
    """Run the C oracle on an ``Inputs`` batch (exact fp64 upcast of its arrays)."""
    B, NH = inp.q.shape[:2]
    S = B * NH
    Tn = inp.T if T is None else T
    f = lambda name, shape: None if getattr(inp, name) is None else inp.as_f64(name).reshape(shape)
    q = inp.as_f64("q")[:, :, :Tn].reshape(S, Tn, inp.DQK)
    k = inp.as_f64("k")[:, :, :Tn].reshape(S, Tn, inp.DQK)
    v = inp.as_f64("v")[:, :, :Tn].reshape(S, Tn, inp.DV)
    ipre = inp.as_f64("ipre")[:, :, :Tn].reshape(S, Tn)
    fpre = inp.as_f64("fpre")[:, :, :Tn].reshape(S, Tn)
    return recurrent(q, k, v, ipre, fpre, f("C0", (S, inp.DQK, inp.DV)), f("n0", (S, inp.DQK)),
                     f("m0", (S,)), nthreads=nthreads)
