"""GPU parity on seeded chains of varied shape and value range: many equal
costs (ties between splits and between C_1 and C_2), zero sizes and
overheads, sizes beyond the budget, heavy overheads, and costs scaled onto
the 64-bit value path; batches of one to three chains; four fill orders
(edges by rounds beside the side stream, by rows, one stream, streamed).
Longer chains (8 to 13 blocks of 16 stages) at costs scaled by up to 2^18
put their block-diagonals on every side of the value-path thresholds (2-byte
copy of the diagonal blocks, packed middle keys, 4-byte or 64-bit values).
Chains with a cost scale of their own per stage, chains whose cost bound
sits near a value-path limit (2^15 - 1, 2^32 - 1, 2^38), and batches of
chains at different scales (block-diagonals of one launch on different
value paths) widen the mix.  Every cell of both tables must equal the oracle's."""
import numpy as np
import pytest

from gpu_util import solve_on_gpu
from paper_1911_13214_amd import chaingen
from test_gpu_parity import SCHEDULES, assert_same, say

pytestmark = pytest.mark.gpu

KINDS = ("ties", "zeros", "large", "wide")


def fuzz_stage(rng, kind):
    """One stage (u_f, u_b, w_a, w_abar, o_f, o_b) of the given kind."""
    u = rng.uniform
    if kind == "ties":
        return u(0, 2), u(0, 2), u(0, 3), u(0, 6), u(0, 2), u(0, 2)
    if kind == "zeros":
        return u(0, 50), u(0, 100), u(0, 1) * u(0, 8), u(0, 12), u(0, 1) * u(0, 5), u(0, 1) * u(0, 5)
    if kind == "large":
        return u(1, 1000), u(1, 2000), u(1, 90), u(1, 200), u(0, 40), u(0, 40)
    # wide: costs near 2^22 times the usual range push the cost bound past 2^32
    return u(1, 100) << 22, u(1, 200) << 22, u(1, 10), u(1, 30), u(0, 3), u(0, 3)


def fuzz_case(seed):
    rng = chaingen.SplitMix64(0xF022 + seed)
    kind = KINDS[seed % len(KINDS)]
    L = rng.uniform(1, 72)
    M = rng.uniform(0, 300)
    n = rng.uniform(1, 3)
    p = np.zeros((n, 6, L), dtype=np.int64)
    for c in range(n):
        for l in range(L):
            p[c, :, l] = fuzz_stage(rng, kind)
    return kind, p, M


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("seed", range(24))
def test_fuzz_parity(seed, schedule):
    kind, p, M = fuzz_case(seed)
    n, _, L = p.shape
    say(f"fuzz seed={seed} kind={kind} n={n} L={L} M={M} {schedule}")
    _, cost, dec = solve_on_gpu(p, M, schedule=schedule)
    for c in range(n):
        assert_same(p, M, cost, dec, c)


def long_case(seed):
    rng = chaingen.SplitMix64(0xB10C + seed)
    L = rng.uniform(120, 200)
    M = rng.uniform(40, 260)
    # from every block-diagonal narrow with the 2-byte copy (0), past the
    # copy's limit (1, 2), to every block-diagonal on the 64-bit path (18)
    shift = (0, 1, 2, 3, 5, 7, 9, 11, 13, 15, 16, 18)[seed]
    p = np.zeros((1, 6, L), dtype=np.int64)
    for l in range(L):
        uf = rng.uniform(1, 100)
        ub = max(1, 2 * uf + rng.uniform(-5, 5))
        wa = rng.uniform(1, 12)
        p[0, :, l] = (uf << shift, ub << shift, wa, wa * rng.uniform(1, 4), rng.uniform(0, 3), rng.uniform(0, 3))
    return p, M, shift


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("seed", range(12))
def test_fuzz_long_chains(seed, schedule):
    p, M, shift = long_case(seed)
    L = p.shape[-1]
    say(f"fuzz long seed={seed} L={L} M={M} shift={shift} {schedule}")
    _, cost, dec = solve_on_gpu(p, M, schedule=schedule)
    assert_same(p, M, cost, dec)


LIMITS = (32767, (1 << 32) - 1, 1 << 38)


def cost_bound(p):
    """sum_j (L - j + 1) u_f^j + sum u_b of one chain [6][L]."""
    return int(np.cumsum(p[0].astype(object)).sum() + p[1].astype(object).sum())


def plain_stage(rng):
    uf = rng.uniform(0, 100)
    return (uf, max(0, 2 * uf + rng.uniform(0, 10) - 5), rng.uniform(0, 12), rng.uniform(0, 30),
            rng.uniform(0, 4), rng.uniform(0, 4))


def mixed_case(seed):
    """One chain whose stages carry costs scaled by 2^0 .. 2^20 each."""
    rng = chaingen.SplitMix64(0x313D + seed)
    L, M = rng.uniform(20, 140), rng.uniform(0, 600)
    p = np.zeros((1, 6, L), dtype=np.int64)
    for l in range(L):
        p[0, :, l] = plain_stage(rng)
        p[0, :2, l] <<= rng.uniform(0, 20)
    return p, M


def near_case(seed):
    """One chain scaled so that its cost bound lies within 10% of a limit."""
    rng = chaingen.SplitMix64(0x4EA2 + seed)
    L, M = rng.uniform(16, 140), rng.uniform(0, 600)
    p = np.zeros((1, 6, L), dtype=np.int64)
    for l in range(L):
        p[0, :, l] = plain_stage(rng)
    target = LIMITS[seed % len(LIMITS)]
    num, den = target * rng.uniform(900, 1100), max(1, cost_bound(p[0])) * 1000
    p[0, :2] = p[0, :2] * num // den
    return p, M


def batch_case(seed):
    """8 to 24 chains, each with its own cost scale 2^0 .. 2^24."""
    rng = chaingen.SplitMix64(0xBA7C + seed)
    n, L, M = rng.uniform(8, 24), rng.uniform(16, 64), rng.uniform(0, 400)
    p = np.zeros((n, 6, L), dtype=np.int64)
    for c in range(n):
        for l in range(L):
            p[c, :, l] = plain_stage(rng)
        p[c, :2] <<= rng.uniform(0, 24)
    return p, M


@pytest.mark.parametrize("schedule", SCHEDULES)
@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("case", [mixed_case, near_case])
def test_fuzz_scales(case, seed, schedule):
    p, M = case(seed)
    L = p.shape[-1]
    say(f"fuzz {case.__name__} seed={seed} L={L} M={M} bound={cost_bound(p[0])} {schedule}")
    _, cost, dec = solve_on_gpu(p, M, schedule=schedule)
    assert_same(p, M, cost, dec)


@pytest.mark.parametrize("schedule", ["auto"] + SCHEDULES)
@pytest.mark.parametrize("seed", range(4))
def test_fuzz_batches_of_mixed_scales(seed, schedule):
    p, M = batch_case(seed)
    n, _, L = p.shape
    say(f"fuzz batch seed={seed} n={n} L={L} M={M} {schedule}")
    _, cost, dec = solve_on_gpu(p, M, schedule=schedule)
    for c in range(n):
        assert_same(p, M, cost, dec, c)
