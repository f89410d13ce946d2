"""The bench's host side: the work it credits to one solve, the arithmetic
type it reports, and its refusal of more than one GPU.  No GPU needed."""
import subprocess
import sys

import numpy as np
import pytest

import bench
from paper_1911_13214_amd import chaingen


def brute_counts(n_chains, L, M):
    # one C_1 candidate per split s' in (s, t], one C_2 candidate per pair
    # s < t, one cell per pair s <= t; each per budget 0..M and per chain
    r_ck = sum(t - s for s in range(1, L + 1) for t in range(s, L + 1))
    r_all = sum(1 for s in range(1, L + 1) for t in range(s + 1, L + 1))
    cells = L * (L + 1) // 2
    W = (M + 1) * n_chains
    return r_ck * W, r_all * W, cells * W


@pytest.mark.parametrize("n,L,M", [(1, 1, 0), (1, 2, 3), (3, 17, 40), (2, 64, 640), (1, 100, 1000)])
def test_work_counts_match_the_enumerated_candidates(n, L, M):
    r_ck, r_all, cells, alg, diag = bench.work_counts(n, L, M)
    assert (r_ck, r_all, cells) == brute_counts(n, L, M)
    assert alg == 16 * r_ck + 8 * r_all + 10 * cells
    assert diag == alg - 10 * L * (M + 1) * n


def test_work_counts_of_the_large_and_batch_workloads():
    # the figures the roofline is priced on
    assert bench.work_counts(1, 500, 5000)[:3] == (104_187_083_250, 623_874_750, 626_375_250)
    assert bench.work_counts(256, 64, 640)[:3] == (7_167_713_280, 330_817_536, 341_319_680)
    alg = bench.work_counts(1, 500, 5000)[3]
    assert alg / 8e12 * 1e3 == pytest.approx(209.8, abs=0.05)  # ms at the 8 TB/s HBM peak


def test_arithmetic_type_follows_the_cost_bound():
    assert bench.arithmetic_type(chaingen.random_chains(1, 500, seed=5, wa_hi=20)) == "u32"
    p = chaingen.random_chains(1, 500, seed=5, wa_hi=20)
    p[:, chaingen.UF] <<= 10
    p[:, chaingen.UB] <<= 10
    # the whole chain's bound is past 2^32 - 1, the bounds of single blocks are not
    assert bench.arithmetic_type(p) == "u32+int64"
    p[:, chaingen.UF] <<= 14
    p[:, chaingen.UB] <<= 14
    assert bench.arithmetic_type(p) == "int64"
    # the bound sum_l P[l] + sum u_b just below and at 2^32 - 1
    L = 4
    p = np.zeros((1, 6, L), dtype=np.int64)
    p[0, chaingen.UF, 0] = ((1 << 32) - 2) // L
    assert bench.arithmetic_type(p) == "u32"
    p[0, chaingen.UB, 0] = (1 << 32) - 1 - L * p[0, chaingen.UF, 0]
    assert bench.arithmetic_type(p) == "int64"


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 2
    assert r.stdout == ""
    assert "one GPU" in r.stderr


@pytest.mark.parametrize("args", [["--profile-steps", "0"], ["--steps", "0"], ["--warmup", "-1"]])
def test_bad_counts_are_refused_before_any_device_work(args):
    r = subprocess.run([sys.executable, bench.__file__, *args], capture_output=True, text=True, timeout=60)
    assert r.returncode == 2 and r.stdout == ""
    assert "must be at least" in r.stderr


def test_cpu_baseline_times_the_whole_workload_on_one_pinned_thread():
    import os
    params = chaingen.random_chains(2, 12, seed=7)
    before = os.sched_getaffinity(0)
    rec, tables = bench.cpu_baseline(params, 60)
    assert os.sched_getaffinity(0) == before  # the pin is undone
    assert rec["cores"] == 1 and rec["kind"] == "oracle" and rec["solve_s"] >= 0
    assert rec["host_cpus"] >= 1 and rec["cpus_allowed"] >= 1 and rec["cpu_model"]
    r_ck, r_all = bench.work_counts(2, 12, 60)[:2]
    assert "whole workload" in rec["sample"] and f"{r_ck + r_all:.4e}" in rec["sample"]
    C, D = tables
    assert C.shape == (12 * 13 // 2, 61) and D.shape == C.shape
    rec, tables = bench.cpu_baseline(params, 60, stages=5)
    assert tables is None and "sub-chain [1,5]" in rec["sample"]


def _device_layout(C, D, L, M, pitch):
    import torch
    cost = torch.full((1, C.shape[0], pitch), -7, dtype=torch.int64)
    dec = torch.full((1, C.shape[0], pitch), -7, dtype=torch.int16)
    cost[0, :, :M + 1] = torch.from_numpy(C)
    dec[0, :, :M + 1] = torch.from_numpy(D)
    return cost, dec


def test_sampled_cells_check_compares_the_right_cells():
    from oracle import oracle
    L, M = 20, 90
    params = chaingen.random_chains(1, L, seed=11)
    C, D = oracle.solve(params, M)
    cost, dec = _device_layout(C, D, L, M, 96)
    assert bench.sampled_cells_equal(cost, dec, C, D, L, M, 5000, seed=55)
    # a wrong top-row decision, and a wrong cost in the middle of the table
    dec[0, L - 1, M // 2] += 1
    assert not bench.sampled_cells_equal(cost, dec, C, D, L, M, 0, seed=55)
    dec[0, L - 1, M // 2] -= 1
    r = oracle.row(L, 3, 9)
    cost[0, r, :M + 1] += 1
    assert not bench.sampled_cells_equal(cost, dec, C, D, L, M, 5000, seed=55)


def test_scaled_table_check_follows_homogeneity_in_the_times():
    from oracle import oracle
    L, M = 18, 70
    params = chaingen.random_chains(1, L, seed=12)
    p2 = params.copy()
    p2[:, :2] <<= 10
    C, D = oracle.solve(params, M)
    C2, D2 = oracle.solve(p2, M)
    a, b = _device_layout(C, D, L, M, 72)
    c, d = _device_layout(C2, D2, L, M, 72)
    assert bench.scaled_tables_equal(a, b, c, d, 10, M)
    d[0, 5, 3] = 99
    assert not bench.scaled_tables_equal(a, b, c, d, 10, M)


def test_class_rates_price_measured_bytes_and_valu_issue():
    k = {"avg_launch_us": 10.0}
    rec = {"bytes_per_launch": 40_000_000, "valu_insts_per_launch": 3_072_000}
    r = bench.class_rates(k, rec, copy_gbps=5000.0)
    assert r["measured_GBps"] == pytest.approx(4000.0)
    assert r["hbm_frac"] == pytest.approx(0.5) and r["copy_frac"] == pytest.approx(0.8)
    # 3.072e6 wave-instructions in 10 us: 307.2 G/s, half of 614.4
    assert r["valu_frac"] == pytest.approx(0.5)
    assert bench.class_rates(k, None, 5000.0) == {}
