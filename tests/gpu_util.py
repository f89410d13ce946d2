"""Helpers for the GPU tests: run the library through its binding and bring
its tables into the oracle's row order (s-major upper triangle)."""
import hashlib

import numpy as np

from oracle import oracle as orc


def gpu_rows_in_oracle_order(L: int) -> np.ndarray:
    """For each oracle row, the library's row of the same pair (s, t), from
    the layout the C ABI documents (both are s-major today; the mapping keeps
    the tests independent of that)."""
    from paper_1911_13214_amd import rotor

    idx = np.empty(L * (L + 1) // 2, dtype=np.int64)
    for s in range(1, L + 1):
        for t in range(s, L + 1):
            idx[orc.row(L, s, t)] = (s - 1) * L - (s - 1) * (s - 2) // 2 + (t - s)
    assert idx[-1] == rotor.rotor_row_index(L, L, L) and idx[0] == rotor.rotor_row_index(L, 1, 1)
    return idx


def solve_on_gpu(params, M, stream=None, schedule="auto"):
    import torch

    from paper_1911_13214_amd import rotor

    d_params, cost, dec = rotor.solve(params, M, device="cuda", stream=stream, schedule=schedule)
    torch.cuda.synchronize()
    return d_params, cost, dec


def chain_tables(cost, dec, c, L, M, order=None):
    """Host copies of chain c's tables in oracle row order, columns 0..M."""
    if order is None:
        order = gpu_rows_in_oracle_order(L)
    gc = cost[c].cpu().numpy()[order, :M + 1]
    gd = dec[c].cpu().numpy()[order, :M + 1]
    return gc, gd


def canonical_hashes(cost, dec, L, M):
    """blake2b of every chain's tables in canonical order (chain, s, t, m),
    matching tests/golden/make_golden.py.  Rows are gathered one s at a time."""
    order = gpu_rows_in_oracle_order(L)
    hc, hd = hashlib.blake2b(), hashlib.blake2b()
    n = cost.shape[0]
    for c in range(n):
        gc = cost[c].cpu().numpy()
        gd = dec[c].cpu().numpy()
        for s in range(1, L + 1):
            sel = order[orc.row(L, s, s):orc.row(L, s, L) + 1]
            hc.update(np.ascontiguousarray(gc[sel, :M + 1]).astype("<i8").tobytes())
            hd.update(np.ascontiguousarray(gd[sel, :M + 1]).astype("<i2").tobytes())
    return hc.hexdigest(), hd.hexdigest()
