"""The pins are sensitive: plausible mistakes planted in a copy of the C
oracle (a dropped gate term, a wrong shift index, a transposed operand, a
flipped tie rule, an off-by-one sum) each make the brute-force comparison
fail.  Everything here runs on the CPU."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import model
from oracle import oracle as orc
from paper_1911_13214_amd import chaingen
from test_oracle_pins import TINY_M, tiny_chain, wide_chain

SRC = open(orc.SRC).read()

MUTATIONS = {
    "shift index s' instead of s'-1": ("int64_t w = wa(&c, sp - 1);", "int64_t w = wa(&c, sp);"),
    "transposed shifted operand": ("int64_t A = right[m - w], B = left[m];", "int64_t A = right[m], B = left[m - w];"),
    "prefix sum off by one": ("sum += uf(&c, sp - 1);", "sum += uf(&c, sp);"),
    "m_none drops o_f of the first step": ("int64_t g = wd(&c, t) + wa(&c, s) + of(&c, s);",
                                           "int64_t g = wd(&c, t) + wa(&c, s);"),
    "m_none drops the input of F_none": ("wd(&c, t) + wa(&c, j - 1) + wa(&c, j) + of(&c, j)",
                                         "wd(&c, t) + wa(&c, j) + of(&c, j)"),
    "m_all drops o_b": ("wd(&c, s) + wab(&c, s) + ob(&c, s)", "wd(&c, s) + wab(&c, s)"),
    "m_all uses omega_a for F_all": ("wd(&c, t) + wab(&c, s) + of(&c, s)", "wd(&c, t) + wa(&c, s) + of(&c, s)"),
    "C_2 shifted by omega_a": ("int64_t w = wab(&c, s);", "int64_t w = wa(&c, s);"),
    "C_2 drops u_b": ("int64_t v = uf(&c, s) + A + ub(&c, s);", "int64_t v = uf(&c, s) + A;"),
    "largest s' wins ties": ("if (v < best[m]) {\n                        best[m] = v;\n                        arg[m] = (int16_t)sp;",
                             "if (v <= best[m]) {\n                        best[m] = v;\n                        arg[m] = (int16_t)sp;"),
    "C_2 wins ties": ("if (v < best[m]) {\n                    best[m] = v;\n                    arg[m] = 0;",
                      "if (v <= best[m]) {\n                    best[m] = v;\n                    arg[m] = 0;"),
    "leaf gate off by one": ("row[m] = m >= g ? uf(&c, s) + ub(&c, s) : ORC_INF;",
                             "row[m] = m > g ? uf(&c, s) + ub(&c, s) : ORC_INF;"),
    "m_none ignores the last forward": ("for (int j = s + 1; j < t; ++j)", "for (int j = s + 1; j < t - 1; ++j)"),
}


def _build_mutant(tmp_path, name, old, new):
    assert SRC.count(old) >= 1, name
    src = tmp_path / f"m{abs(hash(name))}.c"
    src.write_text(SRC.replace(old, new))
    so = str(src)[:-2] + ".so"
    subprocess.check_call(["gcc", "-O1", "-std=c11", "-shared", "-fPIC", str(src), "-o", so])
    lib = ctypes.CDLL(so)
    i64p = ctypes.POINTER(ctypes.c_int64)
    lib.oracle_solve.argtypes = [ctypes.c_int, ctypes.c_int64, i64p, i64p, ctypes.POINTER(ctypes.c_int16)]
    lib.oracle_solve.restype = ctypes.c_int
    return lib


def _mutant_solve(lib, params, M):
    p = np.ascontiguousarray(params[0])
    L = p.shape[1]
    C = np.empty((orc.n_rows(L), M + 1), dtype=np.int64)
    D = np.empty((orc.n_rows(L), M + 1), dtype=np.int16)
    rc = lib.oracle_solve(L, M, p.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                          C.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                          D.ctypes.data_as(ctypes.POINTER(ctypes.c_int16)))
    assert rc == 0
    return C, D


def _cases():
    yield chaingen.homogeneous_chain(6), 100
    for s in range(4):
        yield chaingen.random_chains(1, 5, seed=s), 120
    for s in range(2):
        yield wide_chain(s), 120
    for s in range(300):
        yield tiny_chain(s), TINY_M


def _pins_pass(solve):
    for params, M in _cases():
        L = params.shape[-1]
        C, D = solve(params, M)
        for (s, t), (cost, dec) in model.brute_force(params, M).items():
            r = orc.row(L, s, t)
            if not (np.array_equal(C[r], cost) and np.array_equal(D[r], dec)):
                return False
    return True


def test_unmutated_oracle_passes():
    assert _pins_pass(orc.solve)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(tmp_path, name):
    old, new = MUTATIONS[name]
    lib = _build_mutant(tmp_path, name, old, new)
    assert not _pins_pass(lambda params, M: _mutant_solve(lib, params, M)), f"mutation '{name}' went unnoticed"


# the front end: a plausible mistake in the discretisation or in the
# store-everything memory is caught by the pins of test_frontend.py
FRONT_MUTATIONS = {
    "slots rounded down": ("if (q * (unsigned __int128)mem < need)\n        q += 1;", ""),
    "slots of the limit, not of S": ("(unsigned __int128)v * (unsigned __int128)S;", "(unsigned __int128)v;"),
    "store-all peak drops delta^L": ("int64_t stored = wd(&ch, L); /* delta^L */", "int64_t stored = 0;"),
    "store-all peak drops o_b": ("peak = max64(peak, stored + ob(&ch, j));", "peak = max64(peak, stored);"),
    "store-all peak keeps the freed gradient": ("stored -= wab(&ch, j) + wd(&ch, j);", "stored -= wab(&ch, j);"),
}


def _front_pins_pass(lib):
    import random
    i64p = ctypes.POINTER(ctypes.c_int64)
    lib.oracle_slots.restype = ctypes.c_int64
    lib.oracle_slots.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]
    lib.oracle_store_all_peak.restype = ctypes.c_int64
    lib.oracle_store_all_peak.argtypes = [ctypes.c_int, i64p]
    rng = random.Random(5)
    for _ in range(300):
        mem, S = rng.randint(1, 1 << 30), rng.choice([1, 500, rng.randint(1, 1 << 16)])
        v = rng.randint(0, 3 * mem)
        q = lib.oracle_slots(v, mem, S)
        if not (q * mem >= v * S and (q == 0 or (q - 1) * mem < v * S)):
            return False
    for seed in range(12):
        p = np.ascontiguousarray(chaingen.byte_sized_chain(1 + seed, seed=seed))
        if lib.oracle_store_all_peak(p.shape[1], p.ctypes.data_as(i64p)) != \
                model.all_fall_peak(model.Chain(p), 1, p.shape[1]):
            return False
    return True


def test_unmutated_front_end_passes(tmp_path):
    lib = _build_mutant(tmp_path, "none", "#include <stdint.h>", "#include <stdint.h>")
    assert _front_pins_pass(lib)


@pytest.mark.parametrize("name", sorted(FRONT_MUTATIONS))
def test_front_end_mutation_is_caught(tmp_path, name):
    old, new = FRONT_MUTATIONS[name]
    lib = _build_mutant(tmp_path, name, old, new)
    assert not _front_pins_pass(lib), f"mutation '{name}' went unnoticed"
