"""Run an operation sequence on a PyTorch chain, and estimate the chain's
model parameters (Section 5 of Beaumont et al., arXiv 1911.13214).

A chain is a list of ``nn.Module`` stages applied one after the other (the
``nn.Sequential`` case the paper's tool handles).  The four operations of
Table 1 (Section 3.1) map onto autograd as follows:

- ``F_all^l``: the stage runs with autograd recording, on a detached leaf
  that shares the input's storage; abar^l is that leaf and the output with
  its graph (every tensor the backward step will need);
- ``F_ck^l``: the stage runs without recording; its output a^l is stored and
  the input kept;
- ``F_none^l``: the same, but the input a^{l-1} is dropped;
- ``B^l``: backward through the graph of abar^l with delta^l; the leaf's
  gradient is delta^{l-1}; the graph, delta^l and a plain input a^{l-1} are
  dropped.  Parameter gradients accumulate in the modules as in a plain
  backward pass: each stage's backward runs exactly once in a valid sequence.

Parameter estimation (Section 5.1) runs each stage once forward (with
recording) and once backward on a sample input, timing both and reading the
allocator's counters: u_f, u_b are times, w_a the output size, w_abar what
the recorded forward keeps, o_f and o_b the peaks beyond input and output.

This module uses PyTorch for the chain's own computation; the DP (solve,
discretise, reconstruct, sequence cost) runs in the library through
``rotor``.
"""
from __future__ import annotations


import numpy as np

F_CK, F_NONE, F_ALL, B = 0, 1, 2, 3


def run_sequence(stages, x, dy, ops):
    """Execute ``ops`` ((kind, stage) pairs, stages 1..L) on the chain for
    input ``x`` and output gradient ``dy``.  Returns the gradient with respect
    to ``x``.  Raises ValueError if an operation's input is missing."""
    import torch

    L = len(stages)
    a = {0: x.detach()}  # plain activations a^l
    abar = {}            # l -> (leaf input, output with its graph)
    delta = {L: dy}
    for kind, l in ops:
        if not 1 <= l <= L:
            raise ValueError(f"stage {l} outside 1..{L}")
        if kind == B:
            if l not in delta or l not in abar or not ((l - 1) in a or (l - 1) in abar):
                raise ValueError(f"B^{l} without its inputs")
            leaf, y = abar.pop(l)
            torch.autograd.backward(y, delta.pop(l))
            del y
            if (l - 1) not in abar:
                a.pop(l - 1, None)  # a plain input is consumed
            delta[l - 1] = leaf.grad
            del leaf
            continue
        if (l - 1) in a:
            inp = a[l - 1]
        elif kind != F_NONE and (l - 1) in abar:
            inp = abar[l - 1][1].detach()  # the value a^{l-1} inside abar^{l-1}
        else:
            raise ValueError(f"forward {l} without its input")
        if kind == F_ALL:
            leaf = inp.detach().requires_grad_()
            with torch.enable_grad():
                abar[l] = (leaf, stages[l - 1](leaf))
        else:
            with torch.no_grad():
                a[l] = stages[l - 1](inp)
            if kind == F_NONE:
                del a[l - 1]
        del inp
    if set(delta) != {0} or abar or any(k != 0 for k in a):
        raise ValueError("the sequence does not end with the input gradient alone")
    return delta[0]


def store_all_sequence(L):
    """F_all^1 .. F_all^L, B^L .. B^1: what plain autograd does."""
    return [(F_ALL, l) for l in range(1, L + 1)] + [(B, l) for l in range(L, 0, -1)]


def _sync(device):
    import torch
    if device.type == "cuda":
        torch.cuda.synchronize(device)


def estimate(stages, x, repeats=3, batch_runs=4):
    """Model parameters [6, L] of the chain for the sample input ``x``
    (Section 5.1).  Sizes and overheads in bytes from the allocator: one
    recorded forward and one backward per stage (the larger of the overheads
    of repeated passes).  Times in microseconds of device time: CUDA events
    around ``batch_runs`` back-to-back runs of the operation, so the host
    queues ahead as it does in a sequence, median of ``repeats``.  CUDA only."""
    import torch

    dev = x.device
    if dev.type != "cuda":
        raise ValueError("estimation reads the CUDA allocator: use a CUDA input")

    def device_us(fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        e1.synchronize()
        return e0.elapsed_time(e1) * 1e3 / batch_runs

    L = len(stages)
    p = np.zeros((6, L), dtype=np.int64)
    inp = x.detach()
    for l, f in enumerate(stages):
        of = ob = wab = 0
        for _ in range(2):  # the second pass finds the parameter gradients allocated
            leaf = inp.detach().requires_grad_()
            _sync(dev)
            base = torch.cuda.memory_allocated(dev)
            torch.cuda.reset_peak_memory_stats(dev)
            with torch.enable_grad():
                y = f(leaf)
            _sync(dev)
            after = torch.cuda.memory_allocated(dev)
            wab = max(wab, after - base)
            of = max(of, torch.cuda.max_memory_allocated(dev) - after)
            dy = torch.ones_like(y)
            _sync(dev)
            before_b = torch.cuda.memory_allocated(dev)
            torch.cuda.reset_peak_memory_stats(dev)
            torch.autograd.backward(y, dy)
            _sync(dev)
            ob = max(ob, torch.cuda.max_memory_allocated(dev) - before_b)
            del y, leaf
        with torch.no_grad():
            # F_ck / F_none keep only the output: their peak beyond input and output
            _sync(dev)
            base = torch.cuda.memory_allocated(dev)
            torch.cuda.reset_peak_memory_stats(dev)
            nxt = f(inp)
            _sync(dev)
            wa = nxt.numel() * nxt.element_size()
            of = max(of, torch.cuda.max_memory_allocated(dev) - base - wa)
        tf, tb = [], []
        for _ in range(repeats):
            with torch.no_grad():
                tf.append(device_us(lambda: [f(inp) for _ in range(batch_runs)]))
            leaves = [inp.detach().requires_grad_() for _ in range(batch_runs)]
            with torch.enable_grad():
                outs = [f(q) for q in leaves]
            _sync(dev)
            tb.append(device_us(lambda: [torch.autograd.backward(o, dy) for o in outs]))
            del outs, leaves
        for mod in f.modules():
            for q in mod.parameters(recurse=False):
                q.grad = None
        p[:, l] = (max(1, round(float(np.median(tf)))), max(1, round(float(np.median(tb)))), wa, max(wab, wa),
                   max(of, 0), max(ob, 0))
        inp = nxt
        del dy
    return p


def measure(stages, x, dy, ops, repeats=3):
    """Run ``ops`` ``repeats`` times after one warm-up; returns (median time
    in microseconds, from HIP events on the stream the sequence runs on,
    peak memory in bytes above what was allocated before the sequence
    started: parameters, their gradients, x and dy)."""
    import torch

    dev = x.device
    run_sequence(stages, x, dy, ops)  # warm-up: also allocates the parameter gradients
    times, peaks = [], []
    for _ in range(repeats):
        _sync(dev)
        base = torch.cuda.memory_allocated(dev)
        torch.cuda.reset_peak_memory_stats(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g = run_sequence(stages, x, dy, ops)
        e1.record()
        _sync(dev)
        times.append(e0.elapsed_time(e1) * 1e-3)
        peaks.append(torch.cuda.max_memory_allocated(dev) - base)
        del g
    return float(np.median(times) * 1e6), int(max(peaks))


def synthetic_chain(L, seed, width=1024, device="cpu", dtype=None):
    """A heterogeneous chain of L MLP stages: stage l maps d_{l-1} to d_l
    features (d drawn from {width/2, width, 2 width, 4 width}) through
    Linear, GELU and, every third stage, LayerNorm; seeded weights."""
    import torch
    from torch import nn

    from . import chaingen

    rng = chaingen.SplitMix64(seed)
    dims = [width] + [width * (1 << rng.uniform(0, 3)) // 2 for _ in range(L)]
    g = torch.Generator().manual_seed(seed)
    stages = []
    for l in range(L):
        layers = [nn.Linear(dims[l], dims[l + 1]), nn.GELU()]
        if l % 3 == 2:
            layers.append(nn.LayerNorm(dims[l + 1]))
        st = nn.Sequential(*layers)
        with torch.no_grad():
            for q in st.parameters():
                q.copy_(torch.randn(q.shape, generator=g) * (0.5 / q.shape[-1] ** 0.5))
        stages.append(st.to(device=device, dtype=dtype))
    return stages, dims


def validate(L=24, seed=1, width=1024, batch=4096, slots=500, n_budgets=10, repeats=3):
    """The paper's check of the model (Sections 5.3-5.4) on a synthetic chain
    on cuda:0: estimate the parameters, fill the table with the library at
    ``slots`` slots of the store-everything memory, rebuild the sequences of
    ``n_budgets`` equally spaced budgets in one call, run each, and compare
    the measured time and peak memory with what the model predicts for that
    sequence (rotor_sequence_cost on the byte-level parameters).  Every
    sequence's gradients are also compared, bit for bit, with plain autograd.
    Returns a dict with one row per budget and the mean absolute percentage
    errors."""
    import torch

    from . import rotor

    dev = torch.device("cuda:0")
    torch.manual_seed(seed)
    stages, dims = synthetic_chain(L, seed, width=width, device=dev)
    x = torch.randn(batch, dims[0], device=dev)
    dy = torch.randn(batch, dims[-1], device=dev)
    # a few passes of the whole chain first, so that the estimate does not
    # time a GPU still raising its clocks (the first work of a process)
    for _ in range(3):
        run_sequence(stages, x, dy, store_all_sequence(L))
    _sync(dev)
    for f in stages:
        for q in f.parameters():
            q.grad = None
    p = estimate(stages, x)
    ref = None
    plan = rotor.plan(p, slots=slots, n_budgets=n_budgets)
    top = plan["top_bytes"]
    rows = []
    for b, seq in zip(plan["budgets"], plan["sequences"]):
        if seq is None:
            rows.append({"budget_slots": b, "budget_bytes": top * b // slots, "feasible": False})
            continue
        pred_t, pred_m = rotor.rotor_sequence_cost(p, seq)
        t, m = measure(stages, x, dy, seq, repeats=repeats)
        m += dy.numel() * dy.element_size()  # the model counts delta^L, held here by the caller
        for f in stages:
            for q in f.parameters():
                q.grad = None
        g = run_sequence(stages, x, dy, seq)
        grads = [g] + [q.grad.clone() for f in stages for q in f.parameters()]
        if ref is None:
            for f in stages:
                for q in f.parameters():
                    q.grad = None
            g0 = run_sequence(stages, x, dy, store_all_sequence(L))
            ref = [g0] + [q.grad.clone() for f in stages for q in f.parameters()]
        same = all(torch.equal(u, v) for u, v in zip(grads, ref))
        rows.append({"budget_slots": b, "budget_bytes": top * b // slots, "feasible": True, "ops": len(seq),
                     "recomputed_forwards": sum(1 for k, _ in seq if k != B) - L,
                     "predicted_us": pred_t, "measured_us": round(t, 1), "predicted_bytes": pred_m,
                     "measured_bytes": m, "gradients_equal": same})
    ok = [r for r in rows if r["feasible"]]
    mape = lambda key_p, key_m: float(np.mean([abs(r[key_m] - r[key_p]) / r[key_m] for r in ok])) if ok else None
    return {"chain": {"L": L, "seed": seed, "width": width, "batch": batch, "dims": dims},
            "store_all_bytes": top, "slots": slots, "rows": rows,
            "mape_time": mape("predicted_us", "measured_us"), "mape_memory": mape("predicted_bytes", "measured_bytes"),
            "all_gradients_equal": all(r["gradients_equal"] for r in ok)}


if __name__ == "__main__":
    import argparse
    import json

    ap = argparse.ArgumentParser(description="measured versus predicted time and memory of optimal sequences")
    ap.add_argument("--L", type=int, default=24)
    ap.add_argument("--seed", type=int, default=1)
    ap.add_argument("--width", type=int, default=1024)
    ap.add_argument("--batch", type=int, default=4096)
    ap.add_argument("--slots", type=int, default=500)
    ap.add_argument("--budgets", type=int, default=10)
    a = ap.parse_args()
    print(json.dumps(validate(a.L, a.seed, a.width, a.batch, a.slots, a.budgets)))
