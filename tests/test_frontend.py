"""The front end around the solver: discretisation of byte sizes into slots
(Section 5.2), the memory of the store-everything schedule and equally spaced
budgets (Section 5.3).  Oracle pins and library-vs-oracle checks run on the
CPU (these entry points are host code); the whole pipeline through the GPU
is in test_gpu_parity.py."""
import random

import numpy as np
import pytest

import model
from oracle import oracle as orc
from paper_1911_13214_amd import chaingen, rotor

SIZE_ROWS = (chaingen.WA, chaingen.WABAR, chaingen.OF, chaingen.OB)


def _slot_cases():
    rng = random.Random(7)
    cases = [(0, 1, 1), (0, 10**12, 500), (7, 7, 3), (1, 3, 1), (10**12, 10**12, 500), (1, 10**12, 500),
             ((1 << 40) - 1, 1 << 40, (1 << 28) - 1), (1 << 45, 3, 5)]
    for _ in range(400):
        mem = rng.choice([rng.randint(1, 100), rng.randint(1, 1 << 40)])
        S = rng.choice([1, 2, 500, rng.randint(1, 1 << 20)])
        v = rng.choice([0, rng.randint(0, mem), rng.randint(0, 4 * mem), mem * rng.randint(0, 9)])
        cases.append((v, mem, S))
    return cases


def test_oracle_slots_is_the_rounded_up_slot_count():
    # Section 5.2: q slots of mem / S bytes hold v, q - 1 do not:
    # (q - 1) * mem / S < v <= q * mem / S, written without division
    for v, mem, S in _slot_cases():
        q = orc.slots(v, mem, S)
        assert q * mem >= v * S, (v, mem, S, q)
        assert q == 0 or (q - 1) * mem < v * S, (v, mem, S, q)


def test_oracle_slots_special_cases():
    assert orc.slots(0, 1000, 500) == 0
    assert orc.slots(1000, 1000, 500) == 500  # the whole limit is every slot
    assert orc.slots(6, 1000, 500) == 3       # exactly 3 slots of 2 bytes
    assert orc.slots(7, 1000, 500) == 4       # rounded up
    assert orc.slots(1, 1000, 500) == 1


def test_oracle_discretize_converts_only_sizes():
    p = chaingen.byte_sized_chain(17, seed=3)
    mem, S = int(p[chaingen.WA].sum()), 500
    q = orc.discretize(p, mem, S)
    for row in range(6):
        for l in range(17):
            want = orc.slots(int(p[row, l]), mem, S) if row in SIZE_ROWS else int(p[row, l])
            assert q[row, l] == want


@pytest.mark.parametrize("seed", range(12))
def test_oracle_store_all_peak_matches_the_simulator(seed):
    # model.all_fall_peak replays the schedule through the Table-1 simulator
    # helpers (pinned by brute force in test_oracle_pins.py)
    L = 1 + seed % 9
    p = chaingen.random_chains(1, L, seed=100 + seed)[0]
    assert orc.store_all_peak(p) == model.all_fall_peak(model.Chain(p), 1, L)
    p = chaingen.byte_sized_chain(L + 5, seed=seed)
    assert orc.store_all_peak(p) == model.all_fall_peak(model.Chain(p), 1, L + 5)


@pytest.mark.parametrize("seed", range(6))
def test_store_all_peak_is_where_recomputation_stops(seed):
    # u_f >= 1: only the schedule that stores everything avoids recomputation,
    # so C(1, L, m) = sum(u_f + u_b) exactly from its peak on
    L = 3 + seed
    p = chaingen.random_chains(1, L, seed=seed)[0]
    peak = orc.store_all_peak(p)
    M = peak + 20
    C, _ = orc.solve(p, M)
    top = orc.table_view(C, L)(1, L)
    base = int(p[chaingen.UF].sum() + p[chaingen.UB].sum())
    for m in range(M + 1):
        assert (top[m] == base) == (m >= peak), (m, peak, top[m], base)


def test_library_discretize_matches_oracle():
    rng = random.Random(11)
    for L, n in ((1, 1), (9, 3), (40, 10)):
        p = np.stack([chaingen.byte_sized_chain(L, seed=rng.randint(0, 1 << 30)) for _ in range(n)])
        mem = np.array([rng.randint(1 << 20, 1 << 36) for _ in range(n)], dtype=np.int64)
        for S in (1, 500, 4096):
            q = rotor.rotor_discretize(p, mem, S)
            for c in range(n):
                assert np.array_equal(q[c], orc.discretize(p[c], int(mem[c]), S))
    # in place, and one limit for the whole batch
    p = chaingen.byte_sized_chain(12, seed=5)[None].repeat(2, axis=0)
    assert np.array_equal(rotor.rotor_discretize(p, 1 << 30, 500)[1], orc.discretize(p[1], 1 << 30, 500))


def test_library_store_all_peak_and_budgets():
    for seed in range(8):
        p = chaingen.byte_sized_chain(1 + 7 * seed, seed=seed)
        assert rotor.rotor_store_all_peak(p) == orc.store_all_peak(p)
    for top, n in ((0, 1), (500, 10), (7, 3), (1 << 40, 10), (5, 10)):
        assert list(rotor.rotor_even_budgets(top, n)) == [top * i // n for i in range(1, n + 1)]


def test_front_end_rejects_bad_input():
    p = chaingen.byte_sized_chain(5, seed=1)
    for mem, S in ((0, 500), (-1, 500), (100, 0), (100, 1 << 28)):
        with pytest.raises(rotor.RotorError) as e:
            rotor.rotor_discretize(p, mem, S)
        assert e.value.status == rotor.ROTOR_EINVAL
    q = p.copy()
    q[chaingen.OB, 2] = -1
    with pytest.raises(rotor.RotorError) as e:
        rotor.rotor_discretize(q, 1 << 20, 500)
    assert e.value.status == rotor.ROTOR_EDOMAIN
    with pytest.raises(rotor.RotorError) as e:
        rotor.rotor_store_all_peak(q)
    assert e.value.status == rotor.ROTOR_EDOMAIN
    # a size of 2^30 slots or more is outside the solver's domain
    with pytest.raises(rotor.RotorError) as e:
        rotor.rotor_discretize(p, 1, (1 << 28) - 1)
    assert e.value.status == rotor.ROTOR_EDOMAIN
    for top, n in ((-1, 3), (5, 0), (5, (1 << 20) + 1)):
        with pytest.raises(rotor.RotorError):
            rotor.rotor_even_budgets(top, n)


# ---- the model's prediction for a sequence (Table 1, Theorem 1) -----------

def test_sequence_cost_matches_the_simulator_on_every_persistent_schedule():
    # model.simulate is the independent Table-1 replay the brute-force pins use
    rng = random.Random(3)
    for L in range(1, 7):
        for seed in range(4):
            p = chaingen.random_chains(1, L, seed=rng.randint(0, 1 << 20))[0]
            ch = model.Chain(p)
            for _, ops in model.persistent_schedules(1, L):
                assert rotor.rotor_sequence_cost(p, ops) == model.simulate(ch, 1, L, ops)


def test_sequence_cost_of_reconstructed_sequences_is_the_table():
    # the sequence Algorithm 2 rebuilds costs C(1, L, m) and fits in m
    for seed in range(5):
        L = 4 + seed
        p = chaingen.random_chains(1, L, seed=seed)[0]
        M = 60
        C, _ = orc.solve(p, M)
        top = orc.table_view(C, L)(1, L)
        for m in range(0, M + 1, 7):
            if top[m] == orc.INF:
                continue
            time, peak = rotor.rotor_sequence_cost(p, orc.reconstruct(p, M, C, m))
            assert time == top[m] and peak <= m


def test_sequence_cost_rejects_invalid_sequences():
    p = chaingen.random_chains(1, 3, seed=1)[0]
    F_CK, F_NONE, F_ALL, B = 0, 1, 2, 3
    good = [(F_ALL, 1), (F_ALL, 2), (F_ALL, 3), (B, 3), (B, 2), (B, 1)]
    assert rotor.rotor_sequence_cost(p, good) == model.simulate(model.Chain(p), 1, 3, good)
    bad = [
        good[:-1],                                                   # delta^1 left over
        [(F_ALL, 2)] + good[1:],                                     # forward without its input
        [(F_NONE, 1), (F_ALL, 1)] + good[1:],                        # a^0 consumed, then needed
        [(F_ALL, 1), (F_ALL, 1)] + good[1:],                         # abar^1 stored twice
        [(F_CK, 1), (F_ALL, 2), (F_ALL, 3), (B, 3), (B, 2), (B, 1)],  # B^1 without abar^1
    ]
    for ops in bad:
        with pytest.raises(model.InvalidSequence):
            model.simulate(model.Chain(p), 1, 3, ops)
        with pytest.raises(rotor.RotorError) as e:
            rotor.rotor_sequence_cost(p, ops)
        assert e.value.status == rotor.ROTOR_ESEQUENCE
    for ops in ([(4, 1)], [(F_ALL, 0)], [(F_ALL, 4)]):
        with pytest.raises(rotor.RotorError) as e:
            rotor.rotor_sequence_cost(p, ops)
        assert e.value.status == rotor.ROTOR_EINVAL


def test_kernel_code_digest_ignores_comments_only(tmp_path):
    import bench
    src = tmp_path / "k.hip"
    src.write_text("// header\nint f(int a) { return a + 1; } /* block\n comment */\n")
    d0 = bench.kernel_code_digest(str(src))
    src.write_text("// other header\nint f(int a)\n{\n    return a + 1;  // trailing\n}\n")
    assert bench.kernel_code_digest(str(src)) == d0
    src.write_text("int f(int a) { return a + 2; }\n")
    assert bench.kernel_code_digest(str(src)) != d0
