"""The seeded input generator that feeds both the oracle and the GPU path.

splitmix64 is pinned to the first outputs its authors' reference code
produces from state 0, so a slip in a constant or a shift would change every
input the tests draw without any parity test noticing."""
import numpy as np

from paper_1911_13214_amd import chaingen


def test_splitmix64_published_outputs_from_state_zero():
    rng = chaingen.SplitMix64(0)
    assert [rng.next() for _ in range(4)] == [
        0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC]


def test_uniform_stays_in_its_range_and_reaches_both_ends():
    rng = chaingen.SplitMix64(5)
    draws = [rng.uniform(-5, 5) for _ in range(2000)]
    assert min(draws) == -5 and max(draws) == 5


def test_random_chains_follow_the_recipe():
    p = chaingen.random_chains(3, 40, seed=9, wa_hi=20)
    assert p.shape == (3, 6, 40) and p.dtype == np.int64
    uf, ub, wa, wabar, of, ob = (p[:, r, :] for r in range(6))
    assert ((1 <= uf) & (uf <= 100)).all()
    assert (ub == np.maximum(1, ub)).all() and ((np.abs(ub - 2 * uf) <= 5) | (ub == 1)).all()
    assert ((1 <= wa) & (wa <= 20)).all()
    assert (wabar % wa == 0).all() and ((wabar >= wa) & (wabar <= 4 * wa)).all()
    assert ((0 <= of) & (of <= 3)).all() and ((0 <= ob) & (ob <= 3)).all()
    # one stream, chains then stages: a prefix of the batch is the smaller batch
    assert np.array_equal(chaingen.random_chains(2, 40, seed=9, wa_hi=20), p[:2])
