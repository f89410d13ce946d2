"""GPU parity on seeded chains of varied shape and value range: many equal
costs (ties between splits and between C_1 and C_2), zero sizes and
overheads, sizes beyond the budget, heavy overheads, and costs scaled onto
the 64-bit value path; batches of one to three chains; both fill orders.
Every cell of both tables must equal the oracle's."""
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
    # wide: costs near 2^22 times the usual range push the cost bound past 2^30
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
