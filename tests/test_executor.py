"""The sequence executor (Section 5): every valid operation sequence computes
the same gradients as plain autograd, bit for bit, because each stage's
forward is recomputed identically and its backward runs exactly once.  CPU
tests here; the measured-versus-predicted check runs on the GPU in
test_gpu_executor.py."""
import numpy as np
import pytest

import model
from oracle import oracle as orc
from paper_1911_13214_amd import chaingen
from paper_1911_13214_amd import executor as ex

torch = pytest.importorskip("torch")


def plain_gradients(stages, x, dy):
    for f in stages:
        for q in f.parameters():
            q.grad = None
    xx = x.clone().requires_grad_()
    y = xx
    for f in stages:
        y = f(y)
    y.backward(dy)
    return xx.grad.clone(), [q.grad.clone() for f in stages for q in f.parameters()]


def executor_gradients(stages, x, dy, ops):
    for f in stages:
        for q in f.parameters():
            q.grad = None
    g = ex.run_sequence(stages, x, dy, ops)
    return g, [q.grad.clone() for f in stages for q in f.parameters()]


def same(a, b):
    return torch.equal(a[0], b[0]) and all(torch.equal(p, q) for p, q in zip(a[1], b[1]))


@pytest.mark.parametrize("L", [1, 2, 3, 4, 5])
def test_every_persistent_schedule_gives_the_plain_gradients(L):
    stages, dims = ex.synthetic_chain(L, seed=L, width=32)
    x = torch.randn(16, dims[0], generator=torch.Generator().manual_seed(1))
    dy = torch.randn(16, dims[-1], generator=torch.Generator().manual_seed(2))
    ref = plain_gradients(stages, x, dy)
    n = 0
    for _, ops in model.persistent_schedules(1, L):
        assert same(executor_gradients(stages, x, dy, ops), ref), ops
        n += 1
    assert n == model.schedule_count(L)


def test_optimal_sequences_give_the_plain_gradients():
    L = 9
    stages, dims = ex.synthetic_chain(L, seed=7, width=48)
    x = torch.randn(8, dims[0], generator=torch.Generator().manual_seed(3))
    dy = torch.randn(8, dims[-1], generator=torch.Generator().manual_seed(4))
    ref = plain_gradients(stages, x, dy)
    p = chaingen.random_chains(1, L, seed=7)[0]
    M = 80
    C, _ = orc.solve(p, M)
    seen = set()
    for m in range(M + 1):
        seq = orc.reconstruct(p, M, C, m)
        if seq is None or tuple(seq) in seen:
            continue
        seen.add(tuple(seq))
        assert same(executor_gradients(stages, x, dy, seq), ref), m
    assert len(seen) >= 5


def test_invalid_sequences_are_refused():
    stages, dims = ex.synthetic_chain(3, seed=1, width=16)
    x, dy = torch.randn(4, dims[0]), torch.randn(4, dims[-1])
    good = ex.store_all_sequence(3)
    for ops in (good[:-1], [(ex.F_ALL, 2)] + good[1:], [(ex.F_NONE, 1), (ex.F_ALL, 1)] + good[1:],
                [(ex.F_CK, 1)] + good[1:]):
        with pytest.raises(ValueError):
            ex.run_sequence(stages, x, dy, ops)
