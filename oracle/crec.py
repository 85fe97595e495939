"""ctypes front of oracle/recurrence.c, the plain-C fp64 twin of the oracle's
token-by-token recurrences (TEST INFRASTRUCTURE ONLY, like all of ``oracle``).

The C code evaluates one value head per call, single-threaded; this module
runs the heads of a segment on a pool of host threads (ctypes releases the
GIL during a foreign call).  ``build()`` compiles the shared library with
gcc; ``available()`` is False until it exists, and the oracle then uses its
numpy recurrences.  The two are pinned to each other in
tests/test_oracle_pins.py.
"""
from __future__ import annotations

import concurrent.futures
import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "recurrence.c")
LIB_PATH = os.path.join(HERE, "liboracle_rec.so")

_lib = None
_pool: Optional[concurrent.futures.ThreadPoolExecutor] = None


def build() -> str:
    """Compile recurrence.c with gcc (no fast-math: IEEE fp64 throughout)."""
    tmp = LIB_PATH + ".tmp"
    subprocess.run(["gcc", "-O2", "-std=c99", "-shared", "-fPIC", SRC, "-o", tmp], check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is None and os.path.exists(LIB_PATH):
        lib = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        common = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, P, ctypes.c_int64, P, ctypes.c_int64,
                  P, P, ctypes.c_int64, P]
        lib.oracle_gdn_head.argtypes = common + [P]
        lib.oracle_gdn_head.restype = None
        lib.oracle_decay_head.argtypes = common
        lib.oracle_decay_head.restype = None
        lib.oracle_gdn_head_out.argtypes = common + [P, P, ctypes.c_int64, P, ctypes.c_int64]
        lib.oracle_gdn_head_out.restype = None
        _lib = lib
    return _lib


def available() -> bool:
    return _load() is not None


def threads() -> int:
    """Host threads the C recurrence runs on (all cores the process may use)."""
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return max(1, os.cpu_count() or 1)


def _executor() -> concurrent.futures.ThreadPoolExecutor:
    global _pool
    if _pool is None:
        _pool = concurrent.futures.ThreadPoolExecutor(threads())
    return _pool


def recurrence(kind: str, k: np.ndarray, v: np.ndarray, alpha: np.ndarray, beta: np.ndarray,
               S0: Optional[np.ndarray] = None) -> np.ndarray:
    """Same contract as oracle.gated_delta_recurrence (kind "gdn") and
    oracle.decay_recurrence (kind "decay"): k [L, H, d_k], v [L, H, d_v],
    alpha/beta [L, H], S0 [H, d_v, d_k] or None; returns S_L [H, d_v, d_k]."""
    lib = _load()
    if lib is None:
        raise RuntimeError(f"{LIB_PATH} is not built (oracle.crec.build())")
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    beta = np.ascontiguousarray(beta, dtype=np.float64)
    L, H, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((H, dv, dk)) if S0 is None else np.array(S0, dtype=np.float64, order="C", copy=True)
    work = np.zeros((H, dv))
    f64 = 8

    def one(h: int):
        args = (L, dk, dv, k.ctypes.data + h * dk * f64, H * dk, v.ctypes.data + h * dv * f64, H * dv,
                alpha.ctypes.data + h * f64, beta.ctypes.data + h * f64, H, S[h].ctypes.data)
        if kind == "gdn":
            lib.oracle_gdn_head(*args, work[h].ctypes.data)
        elif kind == "decay":
            lib.oracle_decay_head(*args)
        else:
            raise ValueError(kind)

    if L > 0:
        list(_executor().map(one, range(H)))
    return S


def recurrence_with_outputs(k: np.ndarray, v: np.ndarray, q: np.ndarray, alpha: np.ndarray, beta: np.ndarray,
                            S0: Optional[np.ndarray] = None):
    """Same contract as oracle.block.gated_delta_outputs: returns (S_L
    [H, d_v, d_k], O [L, H, d_v]) with o_t = S_t q_t."""
    lib = _load()
    if lib is None:
        raise RuntimeError(f"{LIB_PATH} is not built (oracle.crec.build())")
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    q = np.ascontiguousarray(q, dtype=np.float64)
    alpha = np.ascontiguousarray(alpha, dtype=np.float64)
    beta = np.ascontiguousarray(beta, dtype=np.float64)
    L, H, dk = k.shape
    dv = v.shape[2]
    S = np.zeros((H, dv, dk)) if S0 is None else np.array(S0, dtype=np.float64, order="C", copy=True)
    O = np.zeros((L, H, dv))
    work = np.zeros((H, dv))
    f64 = 8

    def one(h: int):
        lib.oracle_gdn_head_out(L, dk, dv, k.ctypes.data + h * dk * f64, H * dk, v.ctypes.data + h * dv * f64, H * dv,
                                alpha.ctypes.data + h * f64, beta.ctypes.data + h * f64, H, S[h].ctypes.data,
                                work[h].ctypes.data, q.ctypes.data + h * dk * f64, H * dk,
                                O.ctypes.data + h * dv * f64, H * dv)

    if L > 0:
        list(_executor().map(one, range(H)))
    return S, O
