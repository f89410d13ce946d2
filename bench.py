"""Benchmark: one step = one rotor_solve, the whole table fill of the
checkpointing dynamic program (every sub-chain, every budget) for one
synthetic workload, inputs already resident in device memory.

Prints ONE JSON line on stdout.  Everything else goes to stderr.

  python bench.py [--steps K] [--warmup W] [--workload 1..5] [--no-cpu-baseline] [--int64-shift B]
  python bench.py --shape L,M[,N] [--cost-shift B]   # N seeded random chains of any size

The line carries the throughput of the timed solves, a per-kernel-class
breakdown, the roofline of the dominant class against the resource that
binds it (measured HBM traffic or VALU issue, from the committed counter
records of the current kernel code), the oracle's time on the same workload
on one host core, and, for the large workload, the same chain solved on the
int64 path (costs times 2^B).  A failed parity check exits with status 1
after the line is printed.

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
# VALU issue peak of MI355X: 256 CUs, each issuing one wave-wide VALU
# instruction per cycle (four SIMDs, a 64-lane instruction every four
# cycles on each), at 2.4 GHz: 614.4 G wave-instructions/s (39.3 T
# lane-instructions/s).
VALU_PEAK_GWIS = 256 * 2.4
CSRC = os.path.join(ROOT, "paper_1911_13214_amd", "csrc")
# the sources of the fill kernels, whose digest the counter records carry
FILL_SOURCES = [os.path.join(CSRC, f) for f in ("rotor_paths.h", "rotor_fill.hip", "rotor_rows.h", "rotor_rows_0.hip",
                                                "rotor_rows_1.hip", "rotor_rows_2.hip", "rotor_rows_3.hip")]


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


def host_cpu():
    """(model name, logical CPUs this process may run on, logical CPUs of the host)."""
    model = platform.processor() or "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0)), os.cpu_count()


def cpu_baseline(params, M, stages=None):
    """The C oracle on the workload (every chain, or the sub-chain [1, stages]
    of each when given), single-threaded, with the calling thread pinned to
    one CPU.  Returns the baseline record and the oracle's tables of the
    last chain (or None for a sub-chain)."""
    from oracle import oracle

    n, _, L = params.shape
    Ls = min(stages, L) if stages else L
    r_ck, r_all, _, _, _ = work_counts(n, Ls, M)
    allowed = os.sched_getaffinity(0)
    cpu = min(allowed)
    os.sched_setaffinity(0, {cpu})  # pid 0: this thread only
    try:
        t0 = time.perf_counter()
        for c in range(n):
            C, D = oracle.solve(params[c:c + 1, :, :Ls].copy(), M)
        dt = time.perf_counter() - t0
    finally:
        os.sched_setaffinity(0, allowed)
    model, usable, host = host_cpu()
    what = "the whole workload" if Ls == L else f"sub-chain [1,{Ls}] of each chain"
    rec = {
        "value": round((r_ck + r_all) / dt / 1e9, 4),
        "unit": "G relaxations/s",
        "cores": 1,
        "kind": "oracle",
        "solve_s": round(dt, 2),
        "sample": f"{what}: {n} chain(s) of L={Ls}, all {M + 1} budgets, {r_ck + r_all:.4e} candidates "
                  f"in {dt:.1f} s, one thread pinned to CPU {cpu}",
        "cpu_model": model,
        "host_cpus": host,
        "cpus_allowed": usable,
    }
    return rec, ((C, D) if Ls == L else None)


def arithmetic_type(params):
    """The integer types the fill computes in.  The library takes uint32 with
    saturation for the pairs whose block-diagonal of 16-stage blocks has a cost
    bound below 2^32 - 1 (the bound of a sub-chain [s, t] is
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
    narrow = (1 << 32) - 1
    if whole < narrow:
        return "u32"
    return "int64" if block >= narrow else "u32+int64"


def kernel_code_digest(path=None):
    """sha256 of the fill kernels' sources (or of the file `path`) with
    comments and whitespace removed: it changes when the code changes, not
    when a comment does."""
    text = "\n".join(open(p).read() for p in ([path] if path else FILL_SOURCES))
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return hashlib.sha256("".join(text.split()).encode()).hexdigest()


def counter_record(kernel_class, workload):
    """The committed counter record of a kernel class (HBM bytes and VALU
    wave-instructions per launch, from rocprofv3), if it was taken on this
    workload and on the current kernel code."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel_class}_kernel.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("fill_code_digest") != kernel_code_digest() or rec.get("bench_workload") != workload:
        return None
    return rec


def class_rates(k, rec, copy_gbps):
    """Measured rates of one kernel class from its counter record and its
    average launch time: HBM bytes/s against the 8 TB/s peak and against the
    copy timed in the same run, VALU wave-instructions/s against the issue
    peak."""
    t = k["avg_launch_us"] * 1e-6
    out = {}
    if rec and rec.get("bytes_per_launch"):
        gbps = rec["bytes_per_launch"] / t / 1e9
        out.update({"traffic_per_launch": rec["bytes_per_launch"], "measured_GBps": round(gbps, 1),
                    "hbm_frac": round(gbps / HBM_PEAK_GBS, 4),
                    "copy_frac": round(gbps / copy_gbps, 4) if copy_gbps else None})
    if rec and rec.get("valu_insts_per_launch"):
        gw = rec["valu_insts_per_launch"] / t / 1e9
        out.update({"valu_insts_per_launch": rec["valu_insts_per_launch"], "valu_GWIps": round(gw, 1),
                    "valu_frac": round(gw / VALU_PEAK_GWIS, 4)})
    return out


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


def timed_solves(rotor, d_params, n_chains, L, M, cost, dec, work, stream, steps, warmup):
    """Mean ms per solve over `steps` solves after `warmup` untimed ones, HIP
    events on the solve's stream around each."""
    import numpy as np
    import torch
    for _ in range(warmup):
        rotor.rotor_solve(d_params, n_chains, L, M, cost, dec, work, stream)
    torch.cuda.synchronize()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    t0 = time.perf_counter()
    for k in range(steps):
        starts[k].record(stream)
        rotor.rotor_solve(d_params, n_chains, L, M, cost, dec, work, stream)
        ends[k].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ev_ms = [a.elapsed_time(b) for a, b in zip(starts, ends)]
    log(f"per-step ms (events): {[round(x, 3) for x in ev_ms]}; wall {wall * 1e3 / steps:.3f} ms/step")
    return float(np.mean(ev_ms))


def class_breakdown(rotor, d_params, n_chains, L, M, cost, dec, work, stream, reps, r_ck, r_all):
    """Per kernel class: launches, mean ms per solve (HIP events around each
    run of launches of the class, `reps` solves after the timed region),
    candidates and algorithmic bytes (16 per C_1 candidate, 8 per C_2
    candidate, 10 per cell written)."""
    classes = None
    for _ in range(reps):
        st = rotor.rotor_solve_timed(d_params, n_chains, L, M, cost, dec, work, stream)
        if classes is None:
            classes = st
        else:
            for k in classes:
                classes[k]["ms"] += st[k]["ms"]
    for k in classes:
        classes[k]["ms"] /= reps
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
    return kernels


def sampled_cells_equal(cost, dec, C, D, L, M, n_samples, seed):
    """The device tables of chain 0 against the oracle's at the full top row
    and `n_samples` seeded uniform cells (s <= t, 0 <= m <= M)."""
    import numpy as np
    import torch
    rng = np.random.default_rng(seed)
    s = rng.integers(1, L + 1, n_samples)
    t = rng.integers(1, L + 1, n_samples)
    s, t = np.minimum(s, t), np.maximum(s, t)
    m = rng.integers(0, M + 1, n_samples)
    row = (s - 1) * L - (s - 1) * (s - 2) // 2 + (t - s)
    top = L - 1  # row of (1, L)
    row = np.concatenate([row, np.full(M + 1, top)])
    m = np.concatenate([m, np.arange(M + 1)])
    pitch = cost.shape[-1]
    flat = torch.from_numpy(row * pitch + m).to(cost.device)
    gc = cost.reshape(-1)[flat].cpu().numpy()
    gd = dec.reshape(-1)[flat].cpu().numpy()
    return bool(np.array_equal(gc, C[row, m]) and np.array_equal(gd, D[row, m]))


def scaled_tables_equal(cost, dec, cost2, dec2, shift, M):
    """Costs scaled by 2^shift scale every finite cell by 2^shift and leave
    every decision unchanged (the recurrence is positively homogeneous in
    the times): compared over the whole table, a few rows at a time."""
    import torch
    inf = torch.iinfo(torch.int64).max
    n = cost.shape[1]
    for r0 in range(0, n, 4096):
        a, b = cost[:, r0:r0 + 4096, :M + 1], cost2[:, r0:r0 + 4096, :M + 1]
        fin = a != inf
        if not torch.equal(fin, b != inf) or not torch.equal(a[fin] << shift, b[fin]):
            return False
        if not torch.equal(dec[:, r0:r0 + 4096, :M + 1], dec2[:, r0:r0 + 4096, :M + 1]):
            return False
    return True


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
    ap.add_argument("--int64-shift", type=int, default=10, metavar="B",
                    help="large workload: also time the chain with costs times 2^B, which takes the int64 "
                         "path (0: skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-stages", type=int, default=0,
                    help="time the oracle on the sub-chain [1, N] of each chain only (0: the whole workload)")
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

    ms = timed_solves(rotor, d_params, n_chains, L, M, cost, dec, work, stream, args.steps, args.warmup)
    st, per = rotor.rotor_solve_status(work, n_chains, L, M, stream)
    checks = {"domain": "ok" if st == rotor.ROTOR_OK else f"status {st}"}

    # per-kernel-class breakdown (separate solves, after the timed region)
    kernels = class_breakdown(rotor, d_params, n_chains, L, M, cost, dec, work, stream, args.profile_steps,
                              r_ck, r_all)
    log("kernel classes: " + json.dumps(kernels))
    copy = copy_bandwidth(dev)
    records = {k: counter_record(k, name) for k in kernels}
    for k in kernels:
        kernels[k].update(class_rates(kernels[k], records[k], copy))
    dom = max(kernels, key=lambda k: kernels[k]["ms"])
    kd = kernels[dom]
    # The roofline of the dominant class against the resource that binds it.
    # Its tiled kernels reuse operands, so the 16 bytes per candidate of the
    # plain wavefront overstate what they move; the measured bytes (FETCH_SIZE
    # + WRITE_SIZE per launch) and VALU wave-instructions per launch of the
    # committed counter records, over the launch time measured here, are the
    # rates that can reach a peak.  Without a current record the algorithmic
    # rate is all there is, and the line says so.
    alg_achieved = kd["alg_bytes"] / (kd["ms"] * 1e-3) / 1e9
    # the class's kernels as the counter record names them (else the class)
    kernel_names = "+".join(records[dom]["kernels"]) if records[dom] and records[dom].get("kernels") else dom
    roof = {"kernel": kernel_names, "kernel_class": dom, "launches_per_step": kd["launches"],
            "avg_launch_us": kd["avg_launch_us"],
            "alg_GBps": round(alg_achieved, 1), "alg_frac": round(alg_achieved / HBM_PEAK_GBS, 4),
            "alg_basis": "16 B per C_1 candidate, 8 per C_2 candidate, 10 per cell written"}
    if "hbm_frac" in kd:
        hbm = kd["hbm_frac"]
        valu = kd.get("valu_frac", 0.0)
        if valu > hbm:
            roof = {"bound": "alu", "achieved": kd["valu_GWIps"], "peak": VALU_PEAK_GWIS,
                    "unit": "G VALU wave-instructions/s", "frac": valu, **roof}
        else:
            roof = {"bound": "hbm", "achieved": kd["measured_GBps"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": hbm, **roof}
        roof.update({"traffic": records[dom]["bytes_per_launch"], "hbm_frac": hbm, "valu_frac": valu,
                     "copy_frac": kd.get("copy_frac"),
                     "basis": "measured FETCH_SIZE + WRITE_SIZE (and SQ_INSTS_VALU) per launch from "
                              f"profiles/traffic_{dom}_kernel.json over the launch time measured here"})
    else:
        roof = {"bound": "hbm", "achieved": round(alg_achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(alg_achieved / HBM_PEAK_GBS, 4), "traffic": None, **roof,
                "basis": "algorithmic bytes: no counter record of the current kernel code for this workload"}
    solve_traffic = None
    if all(records[k] and records[k].get("bytes_per_launch") for k in kernels):
        tb = sum(records[k]["bytes_per_launch"] * kernels[k]["launches"] for k in kernels)
        solve_traffic = {"bytes": tb, "GBps": round(tb / (ms * 1e-3) / 1e9, 1),
                         "hbm_frac": round(tb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                         "copy_frac": round(tb / (ms * 1e-3) / 1e9 / copy, 4)}

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
        "roofline": roof,
        "solve_traffic": solve_traffic,
        "copy_GBps": copy,
        "copy": "device-to-device copy of 1 GiB, read + write, HIP events, mean of 5",
        "kernels": kernels,
        "solve_alg_GBps": round(alg_bytes / (ms * 1e-3) / 1e9, 1),
    }

    # the same chain on the int64 path: costs times 2^B scale every finite
    # cell by 2^B and keep every decision, which the whole table must show
    if args.workload == 5 and args.int64_shift:
        B = args.int64_shift
        p64 = params.copy()
        p64[:, :2] <<= B
        d_p64 = rotor.upload_params(p64, M, dev)
        cost2, dec2 = rotor.alloc_tables(n_chains, L, M, dev)
        log(f"int64 path: costs x 2^{B}")
        ms64 = timed_solves(rotor, d_p64, n_chains, L, M, cost2, dec2, work, stream, args.steps, args.warmup)
        k64 = class_breakdown(rotor, d_p64, n_chains, L, M, cost2, dec2, work, stream, args.profile_steps,
                              r_ck, r_all)
        same = scaled_tables_equal(cost, dec, cost2, dec2, B, M)
        checks["int64_path_scaled_table"] = "equal" if same else "DIFFERS"
        out["int64_path"] = {"workload": f"{name} costs x 2^{B}", "dtype": arithmetic_type(p64),
                             "ms_per_step": round(ms64, 4), "value": round(R / (ms64 * 1e-3) / 1e9, 3),
                             "unit": "G relaxations/s",
                             "kernels": {k: {f: v[f] for f in ("launches", "ms", "avg_launch_us")}
                                         for k, v in k64.items()}}
        del cost2, dec2, d_p64
        torch.cuda.empty_cache()

    oracle_tables = None
    if not args.no_cpu_baseline:
        log("oracle on the host ...")
        out["cpu_baseline"], oracle_tables = cpu_baseline(params, M, args.cpu_stages or None)
        log(f"oracle: {out['cpu_baseline']['sample']}")
    if oracle_tables is not None:
        C, D = oracle_tables
        ok = sampled_cells_equal(cost[n_chains - 1:], dec[n_chains - 1:], C, D, L, M, 100000, seed=55)
        checks["oracle"] = ("top row and 1e5 sampled cells of chain %d equal the oracle" % (n_chains - 1)) if ok \
            else "DIFFERS FROM ORACLE"
    else:
        golden = os.path.join(ROOT, "tests", "golden", "random_L500_M5000.npz")
        if args.workload == 5 and os.path.exists(golden):
            g = np.load(golden)
            top = rotor.rotor_row_index(L, 1, L)
            ok = np.array_equal(cost[0, top, :M + 1].cpu().numpy(), g["top_cost"]) and \
                np.array_equal(dec[0, top, :M + 1].cpu().numpy(), g["top_dec"])
            checks["oracle"] = "top row equals the stored oracle values" if ok else "TOP ROW DIFFERS FROM ORACLE"
    out["check"] = checks
    log(f"checks: {checks}")
    print(json.dumps(out), flush=True)
    if any("DIFFER" in v or v.startswith("status") for v in checks.values()):
        sys.exit(1)


if __name__ == "__main__":
    main()
