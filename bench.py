"""Benchmark: one step = one rotor_solve, the whole table fill of the
checkpointing dynamic program (every sub-chain, every budget) for one
synthetic workload, inputs already resident in device memory.

Prints ONE JSON line on stdout.  Everything else goes to stderr.

  python bench.py [--steps K] [--warmup W] [--workload 1..5] [--no-cpu-baseline]
  python bench.py --shape L,M[,N] [--cost-shift B]   # N seeded random chains of any size

Only one GPU is supported: --gpus N with N > 1 exits with a message.
"""
import argparse
import hashlib
import re
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DP candidate relaxations/sec (G/s) and solve ms at L=500,M=5000; % of BW roofline"
HBM_PEAK_GBS = 8000.0
FILL_SOURCE = os.path.join(ROOT, "paper_1911_13214_amd", "csrc", "rotor_fill.hip")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def work_counts(n_chains, L, M):
    """Candidate relaxations and algorithmic bytes of one full solve.

    R_ck  = sum over pairs s < t of (t - s) C_1 candidates per budget,
    R_all = one C_2 candidate per budget of every pair s < t,
    cells = every (s, t, m).  Each C_1 candidate reads two int64 cells, each
    C_2 candidate one, each cell writes 8 + 2 bytes."""
    W = M + 1
    r_ck = (L ** 3 - L) // 6 * W * n_chains
    r_all = L * (L - 1) // 2 * W * n_chains
    cells = L * (L + 1) // 2 * W * n_chains
    alg_bytes = 16 * r_ck + 8 * r_all + 10 * cells
    # the diagonal kernels (d >= 1) carry all but the single-stage cells
    diag_bytes = alg_bytes - 10 * L * W * n_chains
    return r_ck, r_all, cells, alg_bytes, diag_bytes


def cpu_baseline(params, M, stages):
    """The C oracle, single-threaded, on the sub-chain [1, stages] of the
    workload with every budget."""
    from oracle import oracle

    sub = params[:, :, :stages].copy()
    r_ck, r_all, _, _, _ = work_counts(1, stages, M)
    t0 = time.perf_counter()
    oracle.solve(sub, M)
    dt = time.perf_counter() - t0
    return {
        "value": round((r_ck + r_all) / dt / 1e9, 4),
        "unit": "G relaxations/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"sub-chain [1,{stages}] of the workload chain, all {M + 1} budgets "
                  f"({r_ck + r_all:.3e} candidates, {dt:.1f} s, single thread, {platform.processor() or 'cpu'})",
    }


def arithmetic_type(params):
    """The integer types the fill computes in.  The library takes uint32 with
    saturation for the pairs whose block-diagonal of 16-stage blocks has a cost
    bound below 2^30 (the bound of a sub-chain [s, t] is
    sum_{j=s}^{t} (t - j + 1) u_f^j + sum_{j=s}^{t} u_b^j, and it grows with the
    sub-chain), int64 for the others: "u32" when that holds for the whole
    chain, "int64" when not even for one block, else "u32+int64"."""
    import numpy as np
    p = params if params.ndim == 3 else params[None]

    def bound(c, lo, hi):
        return int(np.cumsum(c[0, lo:hi].astype(object)).sum() + c[1, lo:hi].astype(object).sum())

    L = p.shape[-1]
    whole = max(bound(c, 0, L) for c in p)
    block = max(bound(c, b, min(b + 16, L)) for c in p for b in range(0, L, 16))
    if whole < (1 << 30):
        return "u32"
    return "int64" if block >= (1 << 30) else "u32+int64"


def kernel_code_digest(path=None):
    """sha256 of the fill kernels' source with comments and whitespace
    removed: it changes when the code changes, not when a comment does."""
    text = open(path or FILL_SOURCE).read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return hashlib.sha256("".join(text.split()).encode()).hexdigest()


def traffic_if_current(kernel_class, workload):
    """Measured HBM bytes per launch of a kernel class from the committed
    counter summary, if it was taken on this workload and on the current
    kernel code."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_class}_kernel.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("fill_code_digest") != kernel_code_digest() or rec.get("bench_workload") != workload:
        return None
    return rec.get("bytes_per_launch")


def copy_bandwidth(dev, mib=1024, reps=5):
    """What the part delivers to a plain stream: GB/s (read + write) of a
    device-to-device copy of ``mib`` MiB, HIP events around ``reps`` copies."""
    import torch
    src = torch.ones(mib << 17, dtype=torch.int64, device=dev)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    b.synchronize()
    gbps = 2 * (mib << 20) * reps / (a.elapsed_time(b) * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return round(gbps, 1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=5)
    ap.add_argument("--shape", default=None, metavar="L,M[,N]",
                    help="instead of a preset workload: N (default 1) random chains of L stages, budgets 0..M")
    ap.add_argument("--cost-shift", type=int, default=0, metavar="B",
                    help="with --shape: multiply u_f and u_b by 2^B (B = 10 puts L=500 on the 64-bit path)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-stages", type=int, default=300)
    ap.add_argument("--profile-steps", type=int, default=2)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="before timing, run one plain device-to-device copy of this many MiB so that a "
                         "counter run can scale FETCH_SIZE / WRITE_SIZE by a kernel of known traffic")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0:
        ap.error("--steps must be at least 1 and --warmup at least 0")
    if args.profile_steps < 1:
        ap.error("--profile-steps must be at least 1: the roofline is priced on the kernel times it measures")
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the solver has no multi-GPU path (a batch of chains would "
              "shard by chain, a single chain over its budget range)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1911_13214_amd import chaingen, rotor

    if args.shape:
        dims = [int(v) for v in args.shape.split(",")]
        L, M = dims[0], dims[1]
        n_chains = dims[2] if len(dims) > 2 else 1
        params = chaingen.random_chains(n_chains, L, seed=L + M)
        params[:, :2] <<= args.cost_shift
        name = f"random L={L} M={M}" + (f" x {n_chains}" if n_chains > 1 else "") + \
            (f" costs x 2^{args.cost_shift}" if args.cost_shift else "")
        args.workload = 0
    else:
        params, L, M, n_chains, name = chaingen.config(args.workload)
    r_ck, r_all, cells, alg_bytes, diag_bytes = work_counts(n_chains, L, M)
    R = r_ck + r_all
    dev = torch.device("cuda:0")
    d_params = rotor.upload_params(params, M, dev)
    cost, dec = rotor.alloc_tables(n_chains, L, M, dev)
    work = rotor.alloc_workspace(n_chains, L, M, dev)
    stream = torch.cuda.current_stream(dev)
    log(f"workload {name}: L={L} M={M} chains={n_chains} candidates={R:.4e} alg bytes={alg_bytes:.4e}")

    if args.calibrate_copy:
        src = torch.ones(args.calibrate_copy << 17, dtype=torch.int64, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {args.calibrate_copy} MiB read, {args.calibrate_copy} MiB written")
        del src, dst

    for _ in range(args.warmup):
        rotor.rotor_solve(d_params, n_chains, L, M, cost, dec, work, stream)
    torch.cuda.synchronize()

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        rotor.rotor_solve(d_params, n_chains, L, M, cost, dec, work, stream)
        ends[k].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    ms = float(np.mean(ev_ms))
    log(f"per-step ms (events): {[round(x, 3) for x in ev_ms]}; wall {wall * 1e3 / args.steps:.3f} ms/step")

    # parity spot check of the timed output against the stored oracle values
    check = None
    golden = os.path.join(ROOT, "tests", "golden", "random_L500_M5000.npz")
    if args.workload == 5 and os.path.exists(golden):
        g = np.load(golden)
        top = rotor.rotor_row_index(L, 1, L)
        ok = np.array_equal(cost[0, top, :M + 1].cpu().numpy(), g["top_cost"]) and \
            np.array_equal(dec[0, top, :M + 1].cpu().numpy(), g["top_dec"])
        check = "top row equals oracle" if ok else "TOP ROW DIFFERS FROM ORACLE"
        log(check)

    # per-kernel-class breakdown, HIP events around every launch on the same
    # stream (separate steps, after the timed region)
    classes = None
    for _ in range(args.profile_steps):
        st = rotor.rotor_solve_timed(d_params, n_chains, L, M, cost, dec, work, stream)
        if classes is None:
            classes = st
        else:
            for k in classes:
                classes[k]["ms"] += st[k]["ms"]
    for k in classes:
        classes[k]["ms"] /= args.profile_steps
    assert sum(c["split_candidates"] for c in classes.values()) == r_ck
    assert sum(c["all_candidates"] for c in classes.values()) == r_all
    kernels = {}
    for k, c in classes.items():
        if c["launches"] == 0:
            continue
        alg = 16 * c["split_candidates"] + 8 * c["all_candidates"] + 10 * c["cells"]
        kernels[k] = {"launches": c["launches"], "ms": round(c["ms"], 3),
                      "avg_launch_us": round(c["ms"] * 1e3 / c["launches"], 2),
                      "candidates": c["split_candidates"] + c["all_candidates"], "alg_bytes": alg,
                      "alg_GBps": round(alg / (c["ms"] * 1e-3) / 1e9, 1)}
    dom = max(kernels, key=lambda k: kernels[k]["ms"])
    kd = kernels[dom]
    # achieved = algorithmic bytes per launch / average launch duration
    achieved = kd["alg_bytes"] / kd["launches"] / (kd["ms"] * 1e-3 / kd["launches"]) / 1e9
    log("kernel classes: " + json.dumps(kernels))
    out = {
        "metric": METRIC,
        "value": round(R / (ms * 1e-3) / 1e9, 3),
        "unit": "G relaxations/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": arithmetic_type(params),
        "data": "synthetic",
        "config": {"workload": name, "L": L, "M": M, "n_chains": n_chains, "candidates_per_step": R,
                   "alg_bytes_per_step": alg_bytes},
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic_if_current(dom, name),
                     "kernel": f"{dom}_kernel", "launches_per_step": kd["launches"],
                     "avg_launch_us": kd["avg_launch_us"]},
        "kernels": kernels,
        "solve_alg_GBps": round(alg_bytes / (ms * 1e-3) / 1e9, 1),
        "check": check,
    }
    # the same kernel against what a plain copy reaches on this part, on the
    # measured traffic (when the committed counter record is current)
    copy = copy_bandwidth(dev)
    traffic = out["roofline"]["traffic"]
    measured = round(traffic / (kd["avg_launch_us"] * 1e-6) / 1e9, 1) if traffic else None
    out["copy_roofline"] = {"kernel": f"{dom}_kernel", "copy_GBps": copy, "measured_GBps": measured,
                            "frac": round(measured / copy, 4) if measured else None,
                            "copy": "device-to-device copy of 1 GiB, read + write, HIP events, mean of 5"}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(params, M, min(args.cpu_stages, L)) if n_chains == 1 else None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
