"""Independent checks of the checkpointing model, written from the paper's
operation semantics rather than from its recurrence.

- ``simulate``: replays a sequence of F_ck / F_none / F_all / B operations
  (Table 1 of the paper) and returns its time (sum of operation times) and
  its peak memory (max over operations of the live data plus the
  operation's own output and overhead, Section 3.1).  Memory accounting
  follows the conventions of the definition of C_BP (Section 4.2): the
  sub-chain input a^{s-1} (and the gradient delta^{s-1} it turns into) is not
  counted, delta^t is live from the start, and a backward step's peak is its
  live inputs plus o_b (the backward term of m_all does not count the
  output delta^{l-1}).
- ``persistent_schedules``: every memory persistent schedule of a sub-chain,
  following the structure established in the proof of Theorem 1: a
  schedule either starts with F_all^s (then solves [s+1, t] and ends with
  B^s), or starts with F_ck^s, runs F_none up to the next stored value
  a^{s'-1}, solves [s', t] and then [s, s'-1].
- ``brute_force``: the minimum time over all those schedules whose
  simulated peak fits each budget, and the root decision under the tie rule.
- ``feasibility_threshold``: the smallest budget with a finite cost, from a
  recurrence on thresholds (not on costs).
- ``all_fall_peak``: peak memory of the schedule with no recomputation.

None of this imports the oracle or the GPU library.
"""
from __future__ import annotations

from functools import lru_cache

import numpy as np

F_CK, F_NONE, F_ALL, B = 0, 1, 2, 3
UF, UB, WA, WABAR, OF, OB = range(6)
INF = np.iinfo(np.int64).max


class Chain:
    """1-based accessors over a packed [6, L] parameter array."""

    def __init__(self, params):
        p = np.asarray(params, dtype=np.int64)
        if p.ndim == 3:
            p = p[0]
        self.p = p
        self.L = p.shape[1]

    def uf(self, l): return int(self.p[UF, l - 1])
    def ub(self, l): return int(self.p[UB, l - 1])
    def wa(self, l): return int(self.p[WA, l - 1])
    def wd(self, l): return int(self.p[WA, l - 1])  # omega_delta = omega_a
    def wab(self, l): return int(self.p[WABAR, l - 1])
    def of(self, l): return int(self.p[OF, l - 1])
    def ob(self, l): return int(self.p[OB, l - 1])


class InvalidSequence(Exception):
    pass


def simulate(ch: Chain, s: int, t: int, ops):
    """Replay ``ops`` on sub-chain [s, t].  Returns (time, peak).  Raises
    InvalidSequence if an operation's input is missing or the sequence does
    not end with exactly delta^{s-1} (everything else freed)."""
    live = {}  # (kind, l) -> counted size

    def size(kind, l):
        if l == s - 1:
            return 0  # the sub-chain input and its gradient are not counted
        return {"a": ch.wa, "abar": ch.wab, "delta": ch.wd}[kind](l)

    def add(kind, l):
        if (kind, l) in live:
            raise InvalidSequence(f"{kind}^{l} stored twice")
        live[(kind, l)] = size(kind, l)

    live_input = {("a", s - 1)}  # uncounted: a^{s-1} is present at start
    add("delta", t)
    mem = lambda: sum(live.values())
    has = lambda kind, l: (kind, l) in live or (kind, l) in live_input
    time = 0
    peak = 0
    for kind, l in ops:
        if not (s <= l <= t):
            raise InvalidSequence(f"stage {l} outside [{s},{t}]")
        if kind in (F_CK, F_NONE, F_ALL):
            if not (has("a", l - 1) or (kind != F_NONE and has("abar", l - 1))):
                raise InvalidSequence(f"forward {l} without its input")
            out = ch.wab(l) if kind == F_ALL else ch.wa(l)
            peak = max(peak, mem() + out + ch.of(l))
            time += ch.uf(l)
            if kind == F_NONE:  # the input is replaced by the output
                if ("a", l - 1) in live:
                    del live[("a", l - 1)]
                else:
                    live_input.discard(("a", l - 1))
            add("abar" if kind == F_ALL else "a", l)
        elif kind == B:
            if not (has("delta", l) and has("abar", l) and (has("a", l - 1) or has("abar", l - 1))):
                raise InvalidSequence(f"backward {l} without its inputs")
            peak = max(peak, mem() + ch.ob(l))
            time += ch.ub(l)
            del live[("delta", l)]
            del live[("abar", l)]
            if not has("abar", l - 1):  # a plain a^{l-1} is consumed
                if ("a", l - 1) in live:
                    del live[("a", l - 1)]
                else:
                    live_input.discard(("a", l - 1))
            add("delta", l - 1)
        else:
            raise InvalidSequence(f"unknown op {kind}")
    if set(live) != {("delta", s - 1)}:
        raise InvalidSequence(f"left over at the end: {sorted(live)}")
    return time, peak


def persistent_schedules(s: int, t: int):
    """Yield (root, ops) for every persistent schedule of [s, t]; root is s'
    for a schedule starting with F_ck^s and storing a^{s'-1} next, 0 for one
    starting with F_all^s."""
    if s == t:
        yield 0, [(F_ALL, s), (B, s)]
        return
    for sp in range(s + 1, t + 1):
        head = [(F_CK, s)] + [(F_NONE, k) for k in range(s + 1, sp)]
        for _, right in persistent_schedules(sp, t):
            for _, left in persistent_schedules(s, sp - 1):
                yield sp, head + right + left
    for _, sub in persistent_schedules(s + 1, t):
        yield 0, [(F_ALL, s)] + sub + [(B, s)]


def brute_force(params, M: int):
    """For every pair (s, t) return arrays cost[m], dec[m] over m = 0..M: the
    minimum simulated time over persistent schedules with simulated peak <= m,
    and the root decision of a minimiser (smallest s' among F_ck roots, else
    0 for F_all), -1 / INF when none fits."""
    ch = Chain(params)
    L = ch.L
    out = {}
    for s in range(1, L + 1):
        for t in range(s, L + 1):
            sched = [(root,) + simulate(ch, s, t, ops) for root, ops in persistent_schedules(s, t)]
            roots = np.array([x[0] for x in sched])
            times = np.array([x[1] for x in sched], dtype=np.int64)
            peaks = np.array([x[2] for x in sched], dtype=np.int64)
            cost = np.full(M + 1, INF, dtype=np.int64)
            dec = np.full(M + 1, -1, dtype=np.int16)
            for m in range(M + 1):
                ok = peaks <= m
                if not ok.any():
                    continue
                best = times[ok].min()
                cost[m] = best
                winners = roots[ok & (times == best)]
                ck = winners[winners > 0]
                dec[m] = ck.min() if ck.size else 0
            out[(s, t)] = (cost, dec)
    return out


def schedule_count(n: int) -> int:
    """Number of persistent schedules of a chain of n stages."""
    @lru_cache(None)
    def f(k):
        if k == 1:
            return 1
        return sum(f(k - j) * f(j) for j in range(1, k)) + f(k - 1)
    return f(n)


def all_fall_peak(ch: Chain, s: int, t: int) -> int:
    """Peak of F_all^s .. F_all^t, B^t .. B^s (no recomputation): during
    F_all^j the data abar^s..abar^{j-1} and delta^t are live; during B^j the
    data abar^s..abar^j and delta^j are."""
    peak = 0
    acc = 0
    for j in range(s, t + 1):
        peak = max(peak, ch.wd(t) + acc + ch.wab(j) + ch.of(j))
        acc += ch.wab(j)
        peak = max(peak, ch.wd(j) + acc + ch.ob(j))
    return peak


def feasibility_threshold(params):
    """Smallest feasible budget of every pair, from a recurrence on
    thresholds.  A schedule that starts with F_ck^s and stores a^{s'-1} next
    fits in m iff its forward prefix does (each F_none^j, j < s', and F_ck^s
    with delta^t live), the right part fits in m - omega_a^{s'-1} and the
    left part fits in m.  One that starts with F_all^s fits iff F_all^s and
    B^s do and the rest fits in m - omega_abar^s."""
    ch = Chain(params)
    L = ch.L
    th = {}
    for d in range(L):
        for s in range(1, L - d + 1):
            t = s + d
            opt_all = max(ch.wd(t) + ch.wab(s) + ch.of(s), ch.wd(s) + ch.wab(s) + ch.ob(s))
            if s == t:
                th[(s, t)] = opt_all
                continue
            opt_all = max(opt_all, th[(s + 1, t)] + ch.wab(s))
            best_ck = None
            prefix = ch.wd(t) + ch.wa(s) + ch.of(s)
            for sp in range(s + 1, t + 1):
                if sp - 1 > s:
                    j = sp - 1
                    prefix = max(prefix, ch.wd(t) + ch.wa(j - 1) + ch.wa(j) + ch.of(j))
                v = max(prefix, th[(sp, t)] + ch.wa(sp - 1), th[(s, sp - 1)])
                best_ck = v if best_ck is None else min(best_ck, v)
            th[(s, t)] = min(opt_all, best_ck)
    return th
