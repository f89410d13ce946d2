"""ctypes wrapper of the C oracle (``rotor_oracle.c``).

TEST INFRASTRUCTURE ONLY: loaded by the test suite, the smoke check and the
CPU-baseline leg of the benchmark, never by the GPU library or its binding.

The oracle's own table layout is the upper triangle stored s-major: the row
of the pair (s, t), 1 <= s <= t <= L, is ``oracle_row(L, s, t)`` and holds
the M+1 budgets m = 0..M.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "rotor_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")
INF = np.iinfo(np.int64).max
F_CK, F_NONE, F_ALL, B = 0, 1, 2, 3

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into ``oracle/liboracle.so``."""
    if force or not os.path.exists(LIB):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", "-O3", "-march=x86-64-v2", "-std=c11", "-Wall", "-Wextra",
                               "-shared", "-fPIC", SRC, "-o", tmp])
        os.replace(tmp, LIB)
    return LIB


def lib():
    """The oracle library: ``oracle/liboracle.so``, or the build named by the
    environment variable ROTOR_ORACLE_LIB (the sanitizer build of the tests)."""
    global _lib
    if _lib is None:
        path = os.environ.get("ROTOR_ORACLE_LIB")
        if not path:
            path = LIB
            if not os.path.exists(LIB):
                build(force=False)
        l = ctypes.CDLL(path)
        i64p = ctypes.POINTER(ctypes.c_int64)
        i16p = ctypes.POINTER(ctypes.c_int16)
        i32p = ctypes.POINTER(ctypes.c_int32)
        l.oracle_row.restype = ctypes.c_int64
        l.oracle_row.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
        l.oracle_m_all.restype = ctypes.c_int64
        l.oracle_m_all.argtypes = [ctypes.c_int, i64p, ctypes.c_int, ctypes.c_int]
        l.oracle_m_none.restype = ctypes.c_int64
        l.oracle_m_none.argtypes = [ctypes.c_int, i64p, ctypes.c_int, ctypes.c_int]
        l.oracle_check.restype = ctypes.c_int
        l.oracle_check.argtypes = [ctypes.c_int, ctypes.c_int64, i64p]
        l.oracle_cell.restype = ctypes.c_int64
        l.oracle_cell.argtypes = [ctypes.c_int, ctypes.c_int64, i64p, i64p, ctypes.c_int, ctypes.c_int,
                                  ctypes.c_int64, i16p]
        l.oracle_solve.restype = ctypes.c_int
        l.oracle_solve.argtypes = [ctypes.c_int, ctypes.c_int64, i64p, i64p, i16p]
        l.oracle_reconstruct.restype = ctypes.c_int64
        l.oracle_reconstruct.argtypes = [ctypes.c_int, ctypes.c_int64, i64p, i64p, ctypes.c_int64, i32p,
                                         ctypes.c_int64]
        l.oracle_slots.restype = ctypes.c_int64
        l.oracle_slots.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]
        l.oracle_discretize.restype = None
        l.oracle_discretize.argtypes = [ctypes.c_int, i64p, ctypes.c_int64, ctypes.c_int64, i64p]
        l.oracle_store_all_peak.restype = ctypes.c_int64
        l.oracle_store_all_peak.argtypes = [ctypes.c_int, i64p]
        _lib = l
    return _lib


def _p64(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))


def _chain(params):
    p = np.ascontiguousarray(params, dtype=np.int64)
    if p.ndim == 3:
        assert p.shape[0] == 1
        p = p[0]
    assert p.ndim == 2 and p.shape[0] == 6
    return np.ascontiguousarray(p)


def n_rows(L: int) -> int:
    return L * (L + 1) // 2


def row(L: int, s: int, t: int) -> int:
    return (s - 1) * (L + 1) - (s - 1) * s // 2 + (t - s)


def check(params, M: int) -> bool:
    p = _chain(params)
    return lib().oracle_check(p.shape[1], M, _p64(p)) == 0


def solve(params, M: int):
    """Return ``(C, D)`` of shapes ``[L(L+1)/2, M+1]`` (int64, int16)."""
    p = _chain(params)
    L = p.shape[1]
    C = np.empty((n_rows(L), M + 1), dtype=np.int64)
    D = np.empty((n_rows(L), M + 1), dtype=np.int16)
    rc = lib().oracle_solve(L, M, _p64(p), _p64(C), D.ctypes.data_as(ctypes.POINTER(ctypes.c_int16)))
    if rc != 0:
        raise ValueError("chain parameters outside the solver's domain")
    return C, D


def cell(params, M: int, C, s: int, t: int, m: int):
    """Theorem 1 at one cell, from a table holding all shorter sub-chains."""
    p = _chain(params)
    C = np.ascontiguousarray(C, dtype=np.int64)
    d = ctypes.c_int16(0)
    v = lib().oracle_cell(p.shape[1], M, _p64(p), _p64(C), s, t, m, ctypes.byref(d))
    return int(v), int(d.value)


def m_all(params, s: int, t: int) -> int:
    p = _chain(params)
    return int(lib().oracle_m_all(p.shape[1], _p64(p), s, t))


def m_none(params, s: int, t: int) -> int:
    p = _chain(params)
    return int(lib().oracle_m_none(p.shape[1], _p64(p), s, t))


def reconstruct(params, M: int, C, m: int):
    """Algorithm 2 from the cost table: list of (kind, stage), or None if
    C(1, L, m) is infinite."""
    p = _chain(params)
    L = p.shape[1]
    C = np.ascontiguousarray(C, dtype=np.int64)
    cap = L * (L + 1) // 2 + L + 1
    ops = np.zeros((cap, 2), dtype=np.int32)
    n = lib().oracle_reconstruct(L, M, _p64(p), _p64(C), m, ops.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                 cap)
    if n == -1:
        return None
    if n < 0:
        raise ValueError("bad arguments")
    assert n <= cap
    return [(int(k), int(s)) for k, s in ops[:n]]


def table_view(C, L: int):
    """Dict-free accessor: ``get(s, t)`` returns the row of (s, t)."""
    return lambda s, t: C[row(L, s, t)]


def slots(v: int, mem: int, S: int) -> int:
    """Slots of a size v for the limit mem split into S slots (Section 5.2)."""
    return lib().oracle_slots(v, mem, S)


def discretize(params, mem: int, S: int):
    """One chain [6, L] with its four size rows converted to slots."""
    p = _chain(params)
    out = np.empty_like(p)
    lib().oracle_discretize(p.shape[1], _p64(p), mem, S, _p64(out))
    return out


def store_all_peak(params) -> int:
    """Peak memory of F_all^1..F_all^L, B^L..B^1 (no recomputation)."""
    p = _chain(params)
    return lib().oracle_store_all_peak(p.shape[1], _p64(p))
