"""Write the stored expected values of the two largest workloads.  Calls only
the C oracle (``oracle/``) and the seeded input generator.

  random L=500 M=5000 (seed 5):   top row C(1, 500, .) and D(1, 500, .),
                                  4096 seeded cells, blake2b hashes of the
                                  whole cost and decision tables
  random L=500 M=5000 (seed 5), u_f and u_b x 8:  the same records; at
                                  this cost scale some block-diagonals relax
                                  their middle splits in runs of 128
  batch 256 x random L=64 M=640:  blake2b hashes of both tables, all chains

Tables are hashed in canonical order: chain, then s, then t, then m = 0..M,
costs as little-endian int64 and decisions as little-endian int16.

Usage:  python tests/golden/make_golden.py [large|large_x8|batch ...]
        (all three: about 9 minutes, ~7 GB RAM)
"""
import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

from oracle import oracle  # noqa: E402
from paper_1911_13214_amd import chaingen  # noqa: E402

SAMPLE_SEED = 55
N_SAMPLES = 4096


def sample_cells(L, M, n, seed):
    """Seeded cells (s, t, m), uniform over pairs s <= t and budgets."""
    rng = np.random.default_rng(seed)
    out = np.empty((n, 3), dtype=np.int64)
    for k in range(n):
        s = int(rng.integers(1, L + 1))
        t = int(rng.integers(1, L + 1))
        s, t = min(s, t), max(s, t)
        out[k] = (s, t, int(rng.integers(0, M + 1)))
    return out


def write_large(name, shift):
    t0 = time.time()
    params, L, M, _, _ = chaingen.config(5)
    params[:, :2] <<= shift
    C, D = oracle.solve(params, M)
    print(f"{name}: oracle {time.time() - t0:.1f} s", flush=True)
    cells = sample_cells(L, M, N_SAMPLES, SAMPLE_SEED)
    rows = np.array([oracle.row(L, int(s), int(t)) for s, t, _ in cells])
    top = oracle.row(L, 1, L)
    np.savez_compressed(
        os.path.join(HERE, name + ".npz"),
        L=L, M=M, cost_shift=shift,
        top_cost=C[top], top_dec=D[top],
        cells=cells, cell_cost=C[rows, cells[:, 2]], cell_dec=D[rows, cells[:, 2]],
        hash_cost=hashlib.blake2b(C.astype("<i8").tobytes()).hexdigest(),
        hash_dec=hashlib.blake2b(D.astype("<i2").tobytes()).hexdigest(),
    )


def write_batch():
    t0 = time.time()
    params, L, M, n, _ = chaingen.config(4)
    hc, hd = hashlib.blake2b(), hashlib.blake2b()
    for c in range(n):
        C, D = oracle.solve(params[c:c + 1], M)
        hc.update(C.astype("<i8").tobytes())
        hd.update(D.astype("<i2").tobytes())
    print(f"batch: oracle {time.time() - t0:.1f} s", flush=True)
    np.savez_compressed(os.path.join(HERE, "batch256_L64_M640.npz"), L=L, M=M, n_chains=n,
                        hash_cost=hc.hexdigest(), hash_dec=hd.hexdigest())


WRITERS = {
    "large": lambda: write_large("random_L500_M5000", 0),
    "large_x8": lambda: write_large("random_L500_M5000_x8", 3),
    "batch": write_batch,
}


def main(names):
    for name in names or list(WRITERS):
        WRITERS[name]()


if __name__ == "__main__":
    main(sys.argv[1:])
