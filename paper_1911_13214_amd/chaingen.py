"""Seeded synthetic chains for the checkpointing dynamic program.

This module only draws numbers: it holds none of the dynamic program's
arithmetic, so both the GPU path and the CPU oracle can be fed from it.

A chain of ``L`` stages is described by six integer rows (Section 3.1 and
Table 1 of the paper): forward/backward times ``u_f``, ``u_b``, the size of
the stage output ``omega_a`` (also used as the size of the gradient
``delta``), the size of the full intermediate set ``omega_abar``, and the
forward/backward memory overheads ``o_f``, ``o_b``.  They are packed as an
``int64`` array of shape ``[n_chains, 6, L]`` in that row order; stage ``l``
(1-based in the paper) sits at column ``l - 1``.

Randomness comes from splitmix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014) with ``U{a..b} = a + x mod
(b - a + 1)``; the modulo bias is accepted.
"""
from __future__ import annotations

import numpy as np

UF, UB, WA, WABAR, OF, OB = range(6)
ROWS = ("uf", "ub", "wa", "wabar", "of", "ob")
_MASK = (1 << 64) - 1


class SplitMix64:
    """splitmix64: a Weyl sequence with increment 0x9E3779B97F4A7C15 followed
    by the two xor-shift-multiply finalisation rounds of the published
    generator."""

    def __init__(self, seed: int):
        self.state = seed & _MASK

    def next(self) -> int:
        self.state = (self.state + 0x9E3779B97F4A7C15) & _MASK
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK
        return z ^ (z >> 31)

    def uniform(self, lo: int, hi: int) -> int:
        """U{lo..hi}, both ends included."""
        return lo + self.next() % (hi - lo + 1)


def _random_stage(rng: SplitMix64, wa_hi: int):
    """One stage of the random heterogeneous recipe, drawn in the fixed order
    u_f, u_b, omega_a, omega_abar, o_f, o_b."""
    uf = rng.uniform(1, 100)
    ub = max(1, 2 * uf + rng.uniform(-5, 5))
    wa = rng.uniform(1, wa_hi)
    wabar = wa * rng.uniform(1, 4)
    of = rng.uniform(0, 3)
    ob = rng.uniform(0, 3)
    return uf, ub, wa, wabar, of, ob


def random_chains(n_chains: int, L: int, seed: int, wa_hi: int = 10) -> np.ndarray:
    """``n_chains`` random heterogeneous chains of length ``L`` from one
    splitmix64 stream, chains in order, stages in order."""
    rng = SplitMix64(seed)
    out = np.zeros((n_chains, 6, L), dtype=np.int64)
    for c in range(n_chains):
        for l in range(L):
            out[c, :, l] = _random_stage(rng, wa_hi)
    return out


def byte_sized_chain(L: int, seed: int) -> np.ndarray:
    """A chain [6, L] whose sizes are in bytes, as measured before the
    discretisation into slots: per stage u_f = U{1..100}, u_b = max(1, 2 u_f +
    U{-5..5}), omega_a = U{2^10..2^27} bytes, omega_abar = omega_a U{1..4},
    o_f, o_b = U{0..2^24} bytes (drawn in that order)."""
    rng = SplitMix64(seed)
    out = np.zeros((6, L), dtype=np.int64)
    for l in range(L):
        uf = rng.uniform(1, 100)
        ub = max(1, 2 * uf + rng.uniform(-5, 5))
        wa = rng.uniform(1 << 10, 1 << 27)
        wabar = wa * rng.uniform(1, 4)
        of = rng.uniform(0, 1 << 24)
        ob = rng.uniform(0, 1 << 24)
        out[:, l] = (uf, ub, wa, wabar, of, ob)
    return out


def homogeneous_chain(L: int, uf=10, ub=20, wa=5, wabar=15, of=0, ob=0) -> np.ndarray:
    out = np.zeros((1, 6, L), dtype=np.int64)
    for r, v in enumerate((uf, ub, wa, wabar, of, ob)):
        out[0, r, :] = v
    return out


def resnet_like_chain(seed: int = 3) -> np.ndarray:
    """L=100: four groups of 25 stages whose activation size halves from one
    group to the next (16, 8, 4, 2 slots), omega_abar = 3 omega_a, u_f = 40 +
    U{-4..4}, u_b = 2 u_f, no overheads; stage 1 is a heavy stem (u_f=200,
    u_b=400, omega_a=32, omega_abar=96)."""
    rng = SplitMix64(seed)
    L = 100
    out = np.zeros((1, 6, L), dtype=np.int64)
    for l in range(L):
        wa = (16, 8, 4, 2)[l // 25]
        uf = 40 + rng.uniform(-4, 4)
        out[0, :, l] = (uf, 2 * uf, wa, 3 * wa, 0, 0)
    out[0, :, 0] = (200, 400, 32, 96, 0, 0)
    return out


# The five workloads: (name, L, M, n_chains, builder).
CONFIGS = {
    1: dict(name="homogeneous L=10 M=100", L=10, M=100, n_chains=1),
    2: dict(name="random L=50 M=500", L=50, M=500, n_chains=1),
    3: dict(name="resnet-like L=100 M=1000", L=100, M=1000, n_chains=1),
    4: dict(name="batch 256 x random L=64 M=640", L=64, M=640, n_chains=256),
    5: dict(name="random L=500 M=5000", L=500, M=5000, n_chains=1),
}


def config_params(cfg: int) -> np.ndarray:
    """Packed ``[n_chains, 6, L]`` parameters of workload ``cfg`` (1..5)."""
    if cfg == 1:
        return homogeneous_chain(10)
    if cfg == 2:
        return random_chains(1, 50, seed=2)
    if cfg == 3:
        return resnet_like_chain(seed=3)
    if cfg == 4:
        return random_chains(256, 64, seed=4)
    if cfg == 5:
        return random_chains(1, 500, seed=5, wa_hi=20)
    raise ValueError(f"unknown workload {cfg}")


def config(cfg: int):
    """(params, L, M, n_chains, name) of workload ``cfg``."""
    c = CONFIGS[cfg]
    return config_params(cfg), c["L"], c["M"], c["n_chains"], c["name"]
