"""Python binding of the C ABI in include/rotor.h (``librotor.so``).

Argument marshalling only: every step of the solve and of the sequence walk
runs in the library's HIP kernels.  PyTorch provides device memory and the
stream.  If the library has not been built, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librotor.so")

ROTOR_OK = 0
ROTOR_EINVAL = -1
ROTOR_EDOMAIN = -2
ROTOR_EDEVICE = -3
ROTOR_INFEASIBLE = -4
ROTOR_ECAPACITY = -5
ROTOR_ECORRUPT = -6
ROTOR_ESEQUENCE = -7
ROTOR_INF = np.iinfo(np.int64).max
F_CK, F_NONE, F_ALL, B = 0, 1, 2, 3
N_ROWS = 6
MAX_L = 32767
MAX_L_RECONSTRUCT = 8191

# name -> (restype, argtypes) of every function include/rotor.h declares
_i32, _i64, _u64, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_void_p
_P = ctypes.POINTER
SIGNATURES = {
    "rotor_version": (_i32, []),
    "rotor_status_string": (ctypes.c_char_p, [_i32]),
    "rotor_layout": (_i32, [_i32, _i32, _i64, _P(_i64), _P(_i64), _P(_u64), _P(_u64)]),
    "rotor_row_index": (_i64, [_i32, _i32, _i32]),
    "rotor_check_params": (_i32, [_vp, _i32, _i32, _i64]),
    "rotor_workspace_bytes": (_i32, [_i32, _i32, _i64, _P(_u64)]),
    "rotor_solve": (_i32, [_vp, _i32, _i32, _i64, _vp, _vp, _vp, _u64, _vp]),
    "rotor_solve_schedule": (_i32, [_vp, _i32, _i32, _i64, _vp, _vp, _vp, _u64, _vp, _i32]),
    "rotor_reconstruct": (_i32, [_vp, _i32, _i32, _i64, _vp, _i32, _i32, _vp, _i64, _vp, _vp, _vp, _vp]),
    "rotor_solve_noalloc": (_i32, [_vp, _i32, _i32, _i64, _vp, _vp, _vp]),
    "rotor_solve_status": (_i32, [_vp, _u64, _i32, _i32, _i64, _vp, _vp]),
    "rotor_solve_timed": (_i32, [_vp, _i32, _i32, _i64, _vp, _vp, _vp, _u64, _vp, _vp]),
    "rotor_discretize": (_i32, [_vp, _i32, _i32, _vp, _i64, _vp]),
    "rotor_store_all_peak": (_i32, [_vp, _i32, _P(_i64)]),
    "rotor_even_budgets": (_i32, [_i64, _i32, _vp]),
    "rotor_sequence_cost": (_i32, [_vp, _i32, _vp, _i64, _P(_i64), _P(_i64)]),
}

KERNEL_CLASSES = ("leaf", "diag", "middle", "edge", "prep")
SCHEDULES = {"auto": 0, "blocked": 1, "diagonal": 2, "rows": 3, "rounds": 4, "serial": 5}


class KernelStats(ctypes.Structure):
    _fields_ = [("launches", ctypes.c_int32), ("ms", ctypes.c_double), ("split_candidates", ctypes.c_uint64),
                ("all_candidates", ctypes.c_uint64), ("cells", ctypes.c_uint64)]

_lib = None


class RotorError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


def lib():
    """The loaded library (``librotor.so`` beside this file, or the build
    named by the environment variable ROTOR_LIB).  Raises if it has not been
    built.  A host-only build (the sanitizer build of the CPU tests) lacks
    the device entry points: they stay unbound, and calling one raises."""
    global _lib
    if _lib is None:
        override = os.environ.get("ROTOR_LIB")
        # torch ships its own HIP runtime under the same soname as the
        # system's (libamdhip64.so.7).  Loaded after torch, the library binds
        # to torch's runtime; loaded first, it would pull in the system copy
        # and torch would then load a second runtime, whose memory and
        # streams the library's launches would not know.  So torch comes
        # first.
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
        path = override or LIB_PATH
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `python -c 'import __graft_entry__ as g; "
                               "g.build()'` (hipcc, gfx950)")
        l = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            if override and not hasattr(l, name):
                continue
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def status_string(status: int) -> str:
    return lib().rotor_status_string(status).decode()


def _check(status: int, what: str):
    if status != ROTOR_OK:
        raise RotorError(status, what)


def rotor_version() -> int:
    return lib().rotor_version()


def rotor_layout(n_chains: int, L: int, M: int):
    """(pitch, rows_per_chain, cost_bytes, dec_bytes) of the tables."""
    pitch, rows = ctypes.c_int64(), ctypes.c_int64()
    cb, db = ctypes.c_uint64(), ctypes.c_uint64()
    _check(lib().rotor_layout(n_chains, L, M, ctypes.byref(pitch), ctypes.byref(rows), ctypes.byref(cb),
                              ctypes.byref(db)), "rotor_layout")
    return pitch.value, rows.value, cb.value, db.value


def rotor_workspace_bytes(n_chains: int, L: int, M: int) -> int:
    b = ctypes.c_uint64()
    _check(lib().rotor_workspace_bytes(n_chains, L, M, ctypes.byref(b)), "rotor_workspace_bytes")
    return b.value


def rotor_row_index(L: int, s: int, t: int) -> int:
    return lib().rotor_row_index(L, s, t)


def rotor_check_params(params: np.ndarray, M: int) -> int:
    """Status of the host parameter array [n_chains, 6, L] (ROTOR_OK,
    ROTOR_EINVAL or ROTOR_EDOMAIN)."""
    p = np.ascontiguousarray(params, dtype=np.int64)
    if p.ndim == 2:
        p = p[None]
    if p.ndim != 3 or p.shape[1] != N_ROWS:
        return ROTOR_EINVAL
    return lib().rotor_check_params(p.ctypes.data, p.shape[0], p.shape[2], M)


def _stream_ptr(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _dev_ptr(t, dtype, what):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda or t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous {dtype} CUDA tensor")
    return t.data_ptr()


def _solve_ptrs(d_params, n_chains, L, M, d_cost, d_dec, d_work):
    import torch
    _, _, cb, db = rotor_layout(n_chains, L, M)
    if d_params.numel() < n_chains * N_ROWS * L or d_cost.numel() * 8 < cb or d_dec.numel() * 2 < db:
        raise ValueError("buffer smaller than the layout requires")
    if not isinstance(d_work, torch.Tensor) or not d_work.is_cuda or not d_work.is_contiguous():
        raise ValueError("workspace must be a contiguous CUDA tensor")
    return (_dev_ptr(d_params, torch.int64, "params"), _dev_ptr(d_cost, torch.int64, "cost"),
            _dev_ptr(d_dec, torch.int16, "dec"), d_work.data_ptr(), d_work.numel() * d_work.element_size())


def rotor_solve(d_params, n_chains: int, L: int, M: int, d_cost, d_dec, d_work, stream=None):
    """Enqueue the table fill (asynchronous).  ``d_params``: int64 device
    tensor [n_chains, 6, L]; ``d_cost`` / ``d_dec``: int64 / int16 device
    tensors with at least rotor_layout's element counts; ``d_work``: device
    tensor of at least rotor_workspace_bytes."""
    p, c, d, w, wb = _solve_ptrs(d_params, n_chains, L, M, d_cost, d_dec, d_work)
    _check(lib().rotor_solve(p, n_chains, L, M, c, d, w, wb, _stream_ptr(stream)), "rotor_solve")


def rotor_solve_schedule(d_params, n_chains: int, L: int, M: int, d_cost, d_dec, d_work, schedule: str,
                         stream=None):
    """rotor_solve with an explicit fill order, a key of SCHEDULES: "auto",
    "blocked" (edges by rounds or rows, chosen per block-diagonal), "rows",
    "rounds", "serial" (blocked, every middle product on the caller's
    stream) or "diagonal" (same tables, different speed)."""
    p, c, d, w, wb = _solve_ptrs(d_params, n_chains, L, M, d_cost, d_dec, d_work)
    _check(lib().rotor_solve_schedule(p, n_chains, L, M, c, d, w, wb, _stream_ptr(stream), SCHEDULES[schedule]),
           "rotor_solve_schedule")


def rotor_solve_timed(d_params, n_chains: int, L: int, M: int, d_cost, d_dec, d_work, stream=None):
    """rotor_solve with a per-kernel-class breakdown (synchronous).  Returns
    {class: {launches, ms, split_candidates, all_candidates, cells}}."""
    p, c, d, w, wb = _solve_ptrs(d_params, n_chains, L, M, d_cost, d_dec, d_work)
    stats = (KernelStats * len(KERNEL_CLASSES))()
    _check(lib().rotor_solve_timed(p, n_chains, L, M, c, d, w, wb, _stream_ptr(stream),
                                   ctypes.cast(stats, ctypes.c_void_p)), "rotor_solve_timed")
    return {name: {f: getattr(st, f) for f, _ in KernelStats._fields_} for name, st in zip(KERNEL_CLASSES, stats)}


NOALLOC_WORK_BYTES = 128 << 20


def rotor_solve_noalloc(d_params, n_chains: int, L: int, M: int, d_cost, d_dec, stream=None):
    """rotor_solve with the library's static device workspace instead of a
    caller buffer (asynchronous; calls on one device must not overlap)."""
    import torch
    _, _, cb, db = rotor_layout(n_chains, L, M)
    if d_params.numel() < n_chains * N_ROWS * L or d_cost.numel() * 8 < cb or d_dec.numel() * 2 < db:
        raise ValueError("buffer smaller than the layout requires")
    _check(lib().rotor_solve_noalloc(_dev_ptr(d_params, torch.int64, "params"), n_chains, L, M,
                                     _dev_ptr(d_cost, torch.int64, "cost"), _dev_ptr(d_dec, torch.int16, "dec"),
                                     _stream_ptr(stream)), "rotor_solve_noalloc")


def rotor_solve_status(d_work, n_chains: int, L: int, M: int, stream=None):
    """Domain report of the solve that last used ``d_work`` (synchronises the
    stream): (status, per-chain statuses), status ROTOR_OK or
    ROTOR_EDOMAIN."""
    if not hasattr(d_work, "is_cuda") or not d_work.is_cuda or not d_work.is_contiguous():
        raise ValueError("workspace must be a contiguous CUDA tensor")
    per = np.zeros(n_chains, dtype=np.int32)
    st = lib().rotor_solve_status(d_work.data_ptr(), d_work.numel() * d_work.element_size(), n_chains, L, M,
                                  per.ctypes.data, _stream_ptr(stream))
    if st not in (ROTOR_OK, ROTOR_EDOMAIN):
        raise RotorError(st, "rotor_solve_status")
    return st, per


def rotor_reconstruct(d_params, n_chains: int, L: int, M: int, d_dec, chain: int, d_budgets, cap: int, d_ops,
                      d_count, d_status, stream=None):
    """Enqueue the sequence walk (asynchronous).  ``d_budgets``: int64 device
    tensor [n]; ``d_ops``: int32 device tensor [n, cap, 2] (kind, stage);
    ``d_count``: int64 [n]; ``d_status``: int32 [n]."""
    import torch
    n = d_budgets.numel()
    if d_ops.numel() < n * cap * 2 or d_count.numel() < n or d_status.numel() < n:
        raise ValueError("output buffer too small")
    ops_ptr = _dev_ptr(d_ops, torch.int32, "ops") if cap > 0 else None
    _check(lib().rotor_reconstruct(_dev_ptr(d_params, torch.int64, "params"), n_chains, L, M,
                                   _dev_ptr(d_dec, torch.int16, "dec"), chain, n,
                                   _dev_ptr(d_budgets, torch.int64, "budgets"), cap, ops_ptr,
                                   _dev_ptr(d_count, torch.int64, "count"), _dev_ptr(d_status, torch.int32, "status"),
                                   _stream_ptr(stream)), "rotor_reconstruct")


def rotor_discretize(params: np.ndarray, mem_bytes, slots: int) -> np.ndarray:
    """Sizes in bytes -> slots of mem_bytes / slots each, rounded up
    (Section 5.2).  ``params`` [n_chains, 6, L] (or [6, L]); ``mem_bytes`` one
    limit or one per chain.  Returns the converted array (same shape)."""
    p = np.ascontiguousarray(params, dtype=np.int64)
    squeeze = p.ndim == 2
    if squeeze:
        p = p[None]
    if p.ndim != 3 or p.shape[1] != N_ROWS:
        raise ValueError("params must be [n_chains, 6, L]")
    mem = np.ascontiguousarray(np.broadcast_to(np.asarray(mem_bytes, dtype=np.int64), (p.shape[0],)))
    out = np.empty_like(p)
    _check(lib().rotor_discretize(p.ctypes.data, p.shape[0], p.shape[2], mem.ctypes.data, slots, out.ctypes.data),
           "rotor_discretize")
    return out[0] if squeeze else out


def rotor_store_all_peak(params: np.ndarray) -> int:
    """Memory of the schedule that recomputes nothing, for one chain [6, L]."""
    p = np.ascontiguousarray(params, dtype=np.int64)
    if p.ndim == 3 and p.shape[0] == 1:
        p = p[0]
    if p.ndim != 2 or p.shape[0] != N_ROWS:
        raise ValueError("params must be one chain [6, L]")
    peak = ctypes.c_int64()
    _check(lib().rotor_store_all_peak(p.ctypes.data, p.shape[1], ctypes.byref(peak)), "rotor_store_all_peak")
    return peak.value


def rotor_even_budgets(top: int, n: int) -> np.ndarray:
    """floor(i * top / n) for i = 1..n."""
    out = np.empty(n, dtype=np.int64) if n > 0 else np.empty(1, dtype=np.int64)
    _check(lib().rotor_even_budgets(top, n, out.ctypes.data), "rotor_even_budgets")
    return out


def rotor_sequence_cost(params: np.ndarray, ops) -> tuple:
    """(time, peak memory) the model predicts for the sequence ``ops`` (a list
    of (kind, stage)) on one chain [6, L]."""
    p = np.ascontiguousarray(params, dtype=np.int64)
    if p.ndim == 3 and p.shape[0] == 1:
        p = p[0]
    if p.ndim != 2 or p.shape[0] != N_ROWS:
        raise ValueError("params must be one chain [6, L]")
    o = np.ascontiguousarray(np.asarray(ops, dtype=np.int32).reshape(-1, 2))
    t, pk = ctypes.c_int64(), ctypes.c_int64()
    _check(lib().rotor_sequence_cost(p.ctypes.data, p.shape[1], o.ctypes.data, o.shape[0], ctypes.byref(t),
                                     ctypes.byref(pk)), "rotor_sequence_cost")
    return t.value, pk.value


# ---- conveniences (allocation and host copies only) -------------------------

def upload_params(params: np.ndarray, M: int, device="cuda"):
    """Check the host parameters against the domain, then copy them to the
    device as an int64 tensor [n_chains, 6, L]."""
    import torch
    p = np.ascontiguousarray(params, dtype=np.int64)
    if p.ndim == 2:
        p = p[None]
    _check(rotor_check_params(p, M), "rotor_check_params")
    return torch.from_numpy(p).to(device)


def alloc_tables(n_chains: int, L: int, M: int, device="cuda"):
    """Uninitialised cost (int64) and decision (int16) tables shaped
    [n_chains, rows, pitch]."""
    import torch
    pitch, rows, _, _ = rotor_layout(n_chains, L, M)
    cost = torch.empty((n_chains, rows, pitch), dtype=torch.int64, device=device)
    dec = torch.empty((n_chains, rows, pitch), dtype=torch.int16, device=device)
    return cost, dec


def alloc_workspace(n_chains: int, L: int, M: int, device="cuda"):
    """Uninitialised device workspace of rotor_workspace_bytes (int64 words)."""
    import torch
    return torch.empty(((rotor_workspace_bytes(n_chains, L, M) + 7) // 8,), dtype=torch.int64, device=device)


def solve(params: np.ndarray, M: int, device="cuda", stream=None, schedule: str = "auto"):
    """Upload, allocate and fill.  Returns (d_params, cost, dec) device
    tensors; the fill is enqueued on ``stream`` (the workspace is released to
    torch's caching allocator on that stream)."""
    p = np.asarray(params)
    if p.ndim == 2:
        p = p[None]
    n_chains, _, L = p.shape
    d_params = upload_params(p, M, device)
    cost, dec = alloc_tables(n_chains, L, M, device)
    work = alloc_workspace(n_chains, L, M, device)
    rotor_solve_schedule(d_params, n_chains, L, M, cost, dec, work, schedule, stream)
    if stream is not None:
        work.record_stream(stream)
    return d_params, cost, dec


def reconstruct(d_params, n_chains: int, L: int, M: int, d_dec, chain: int, budgets, stream=None):
    """Sequences of chain ``chain`` at each budget, as lists of (kind, stage);
    None where no sequence fits.  Synchronises the stream."""
    import torch
    device = d_dec.device
    budgets = torch.as_tensor(np.asarray(budgets, dtype=np.int64), device=device)
    n = budgets.numel()
    cap = L * (L + 1) // 2 + L
    ops = torch.empty((n, cap, 2), dtype=torch.int32, device=device)
    count = torch.empty(n, dtype=torch.int64, device=device)
    status = torch.empty(n, dtype=torch.int32, device=device)
    rotor_reconstruct(d_params, n_chains, L, M, d_dec, chain, budgets, cap, ops, count, status, stream)
    if stream is None:
        torch.cuda.current_stream().synchronize()
    else:
        stream.synchronize()
    count, status = count.cpu().numpy(), status.cpu().numpy()
    ops = ops.cpu().numpy()
    out = []
    for b in range(n):
        if status[b] == ROTOR_INFEASIBLE:
            out.append(None)
            continue
        _check(int(status[b]), "rotor_reconstruct")
        out.append([(int(k), int(s)) for k, s in ops[b, :count[b]]])
    return out


def plan(params_bytes: np.ndarray, slots: int = 500, n_budgets: int = 10, top_bytes=None, device="cuda"):
    """The paper's use of the solver (Sections 5.2 and 5.3) for one chain
    whose sizes are in bytes: discretise with respect to ``top_bytes``
    (default: the memory of the store-everything schedule) into ``slots``
    slots, fill one table with M = slots, and walk it at ``n_budgets``
    budgets equally spaced up to the top in one call.  Returns a dict with
    the slot parameters, the budgets (slots), their times C(1, L, budget)
    (None where infeasible) and the sequences."""
    p = np.ascontiguousarray(params_bytes, dtype=np.int64)
    if p.ndim == 3:
        p = p[0]
    L = p.shape[1]
    top = rotor_store_all_peak(p) if top_bytes is None else int(top_bytes)
    ps = rotor_discretize(p, max(top, 1), slots)
    d_params, cost, dec = solve(ps, slots, device=device)
    budgets = rotor_even_budgets(slots, n_budgets)
    seqs = reconstruct(d_params, 1, L, slots, dec, 0, budgets)
    top_row = cost[0, rotor_row_index(L, 1, L)].cpu().numpy()
    times = [None if top_row[b] == ROTOR_INF else int(top_row[b]) for b in budgets]
    return {"params_slots": ps, "top_bytes": top, "budgets": [int(b) for b in budgets], "times": times,
            "sequences": seqs}
