"""ctypes wrapper of the multithreaded C oracle (test infrastructure).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg
may import this module.  It loads ``oracle/liboracle.so``, which is built
from ``oracle/oracle.c`` with plain gcc (see :func:`build`).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no HIP, no shared headers); without
    force, only when the library is missing or older than its source."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-Wno-unused-parameter",
                        "-shared", "-fPIC", "-pthread", SRC, "-o", tmp], check=True)
        os.replace(tmp, LIB)
    return LIB


class _Problem(C.Structure):
    _fields_ = [("L", C.c_uint32), ("S", C.c_uint32), ("M", C.c_uint32), ("T", C.c_uint32),
                ("fwd", C.c_void_p), ("bwd", C.c_void_p), ("cf", C.c_void_p), ("cb", C.c_void_p),
                ("mem", C.c_void_p), ("cap", C.c_void_p), ("assign", C.c_void_p),
                ("A", C.c_uint64), ("allreduce", C.c_void_p), ("schedule", C.c_uint32), ("V", C.c_uint32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        build(force=False)
        _lib = C.CDLL(LIB)
        _lib.oc_eval.restype = C.c_int
        _lib.oc_eval.argtypes = [C.POINTER(_Problem), C.c_uint64, C.c_uint64, C.c_void_p,
                                 C.c_void_p, C.c_void_p, C.c_void_p, C.c_int]
        _lib.oc_bounded.restype = C.c_int
        _lib.oc_bounded.argtypes = [C.POINTER(_Problem), C.c_uint64, C.c_uint64, C.c_void_p,
                                    C.c_void_p, C.c_uint32, C.c_uint64, C.c_int,
                                    C.POINTER(C.c_uint64), C.POINTER(C.c_uint32),
                                    C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                    C.POINTER(C.c_uint64), C.c_int]
        _lib.oc_search.restype = C.c_int
        _lib.oc_search.argtypes = [C.POINTER(_Problem), C.c_uint64, C.c_uint64, C.c_uint32, C.c_uint64,
                                   C.c_uint32, C.POINTER(C.c_uint64), C.POINTER(C.c_uint32),
                                   C.POINTER(C.c_uint64), C.c_int]
        _lib.oc_finish_times.restype = C.c_int64
        _lib.oc_finish_times.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int] + [C.c_void_p] * 7
        _lib.oc_dag_counts.restype = C.c_int
        _lib.oc_dag_counts.argtypes = [C.c_int, C.c_int] + [C.POINTER(C.c_int)] * 5
    return _lib


def default_threads() -> int:
    try:
        return max(1, len(os.sched_getaffinity(0)))
    except AttributeError:  # pragma: no cover
        return os.cpu_count() or 1


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _problem(prob):
    keep = []

    def arr(x, dt):
        if x is None:
            return None
        a = np.ascontiguousarray(np.asarray(x, dtype=dt))
        keep.append(a)
        return a

    st = _Problem(prob.L, prob.S, prob.M, prob.T,
                  _ptr(arr(prob.fwd, np.uint32)), _ptr(arr(prob.bwd, np.uint32)),
                  _ptr(arr(prob.comm_fwd if prob.S > 1 else np.zeros(1), np.uint32)),
                  _ptr(arr(prob.comm_bwd if prob.S > 1 else np.zeros(1), np.uint32)),
                  _ptr(arr(prob.mem, np.uint32)), _ptr(arr(prob.cap, np.uint32)),
                  _ptr(arr(prob.assign, np.uint8)), prob.A,
                  _ptr(arr(getattr(prob, "allreduce", None), np.uint32)),
                  int(getattr(prob, "schedule", 0)), int(getattr(prob, "V", 1)))
    return st, keep


def evaluate(prob, cands, nthreads: Optional[int] = None, lo: int = 0, hi: Optional[int] = None):
    """Makespans (uint32) and feasibility (bool) of candidates [lo, hi)."""
    st, keep = _problem(prob)
    n = len(cands)
    hi = n if hi is None else hi
    cnt = hi - lo
    out_T = np.zeros(cnt, dtype=np.uint32)
    out_f = np.zeros(cnt, dtype=np.uint8)
    if cands.is_list:
        rank = np.ascontiguousarray(cands.comp_rank[lo:hi], dtype=np.uint64)
        aidx = None if cands.assign_idx is None else np.ascontiguousarray(cands.assign_idx[lo:hi], dtype=np.uint32)
        rc = lib().oc_eval(C.byref(st), 0, cnt, _ptr(rank), _ptr(aidx), _ptr(out_T), _ptr(out_f),
                           nthreads or default_threads())
    else:
        rc = lib().oc_eval(C.byref(st), cands.first + lo, cnt, None, None, _ptr(out_T), _ptr(out_f),
                           nthreads or default_threads())
    if rc != 0:
        raise RuntimeError(f"oracle oc_eval failed: {rc}")
    del keep
    return out_T, out_f.astype(bool)


def bounded(prob, cands, bound: int, chunk: int = 0, nthreads: Optional[int] = None, ramp: bool = False):
    """Early-stop pass (chunks of `chunk` candidates, or with ramp chunk,
    2 chunk, 4 chunk, ...); returns (best (idx, T) or None, evaluated,
    pruned, infeasible)."""
    st, keep = _problem(prob)
    n = len(cands)
    bi, bt = C.c_uint64(), C.c_uint32()
    ev, pr, inf = C.c_uint64(), C.c_uint64(), C.c_uint64()
    if cands.is_list:
        rank = np.ascontiguousarray(cands.comp_rank, dtype=np.uint64)
        aidx = None if cands.assign_idx is None else np.ascontiguousarray(cands.assign_idx, dtype=np.uint32)
        rc = lib().oc_bounded(C.byref(st), 0, n, _ptr(rank), _ptr(aidx), bound, chunk, int(ramp),
                              C.byref(bi), C.byref(bt), C.byref(ev), C.byref(pr), C.byref(inf),
                              nthreads or default_threads())
    else:
        rc = lib().oc_bounded(C.byref(st), cands.first, n, None, None, bound, chunk, int(ramp),
                              C.byref(bi), C.byref(bt), C.byref(ev), C.byref(pr), C.byref(inf),
                              nthreads or default_threads())
    if rc != 0:
        raise RuntimeError(f"oracle oc_bounded failed: {rc}")
    del keep
    best = None if bi.value == 2**64 - 1 else (int(bi.value), int(bt.value))
    return best, int(ev.value), int(pr.value), int(inf.value)


SEARCH_RIDGE, SEARCH_NO_STAGE_PRUNING, SEARCH_RAMP = 1, 2, 4
SEARCH_COUNTERS = ("visited", "evaluated", "pruned_memory", "pruned_ridge", "pruned_bound")


def search(prob, bound: int, first_row: int = 0, n_rows: Optional[int] = None, rows_per_chunk: int = 0,
           ridge: bool = False, stage_pruning: bool = True, ramp: bool = False, nthreads: Optional[int] = None):
    """Pruned search (same semantics and counters as oracle.search.stage_search)."""
    st, keep = _problem(prob)
    n_rows = prob.A - first_row if n_rows is None else n_rows
    bi, bt = C.c_uint64(), C.c_uint32()
    cnt = (C.c_uint64 * 5)()
    flags = (SEARCH_RIDGE if ridge else 0) | (0 if stage_pruning else SEARCH_NO_STAGE_PRUNING) | \
        (SEARCH_RAMP if ramp else 0)
    rc = lib().oc_search(C.byref(st), first_row, n_rows, bound, rows_per_chunk, flags, C.byref(bi), C.byref(bt),
                         cnt, nthreads or default_threads())
    if rc != 0:
        raise RuntimeError(f"oracle oc_search failed: {rc}")
    del keep
    out = {k: int(v) for k, v in zip(SEARCH_COUNTERS, cnt)}
    out["best"] = None if bi.value == 2**64 - 1 else (int(bi.value), int(bt.value))
    return out


def finish_times(S: int, M: int, F, B, cf, cb, d=None, schedule: int = 0, V: int = 1):
    """(T, fin_F, fin_B): the makespan and the finish time of every compute
    node, fin_F[s-1, m-1] = finish(F_{s,m}) (likewise fin_B), for one
    candidate's stage weights; d is the per-stage (per-device under
    Interleaved 1F1B) all-reduce weight, or None."""
    f = np.ascontiguousarray(F, dtype=np.uint64)
    b = np.ascontiguousarray(B, dtype=np.uint64)
    dd = None if d is None else np.ascontiguousarray(d, dtype=np.uint64)
    tf = np.ascontiguousarray(cf if S > 1 else [0], dtype=np.uint32)
    tb = np.ascontiguousarray(cb if S > 1 else [0], dtype=np.uint32)
    fin_f = np.zeros((S, M), dtype=np.uint64)
    fin_b = np.zeros((S, M), dtype=np.uint64)
    T = lib().oc_finish_times(S, M, schedule, V, _ptr(f), _ptr(b), _ptr(dd), _ptr(tf), _ptr(tb),
                              _ptr(fin_f), _ptr(fin_b))
    if T < 0:
        raise RuntimeError("oc_finish_times failed")
    return int(T), fin_f, fin_b


def dag_counts(S: int, M: int):
    vals = [C.c_int() for _ in range(5)]
    rc = lib().oc_dag_counts(S, M, *[C.byref(v) for v in vals])
    if rc != 0:
        raise RuntimeError("oc_dag_counts failed")
    n, f, b, intra, other = (v.value for v in vals)
    return dict(nodes=n, fwd=f, bwd=b, intra=intra, other=other)


def argmin(makespans: np.ndarray, feasible: np.ndarray):
    """Smallest (makespan, index) over feasible entries (vectorised scan)."""
    if not feasible.any():
        return None
    t = np.where(feasible, makespans.astype(np.uint64), np.uint64(2**63))
    i = int(np.argmin(t))          # numpy returns the first occurrence on ties
    return i, int(makespans[i])
