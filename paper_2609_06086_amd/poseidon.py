"""ctypes binding of the C-ABI in ``include/poseidon.h`` (argument marshalling only).

Every step of the evaluation runs in the HIP library ``libposeidon.so``
built next to this file; importing this module fails loudly if it is not
there.  Host tables are numpy arrays; device buffers are torch tensors (or
raw integer device addresses); streams are ``torch.cuda.Stream`` objects or
raw ``hipStream_t`` integers.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libposeidon.so")

POSEIDON_OK = 0
POSEIDON_NO_FEASIBLE = 1
POSEIDON_E_INVAL = -1
POSEIDON_E_RANGE = -2
POSEIDON_E_DEVICE = -3
POSEIDON_E_NOMEM = -4
SCHEDULE_1F1B, SCHEDULE_EAGER_1F1B, SCHEDULE_INTERLEAVED_1F1B = 0, 1, 2
SEARCH_RIDGE, SEARCH_NO_STAGE_PRUNING, SEARCH_RAMP = 1, 2, 4
BOUNDED_RAMP = 1
S_MAX, L_MAX, T_MAX, M_MAX = 16, 256, 8, 1 << 20


class PoseidonError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {strerror(status)} (status {status})")
        self.status = status


class _Problem(C.Structure):
    _fields_ = [("L", C.c_uint32), ("S", C.c_uint32), ("M", C.c_uint32), ("T", C.c_uint32),
                ("fwd_us", C.c_void_p), ("bwd_us", C.c_void_p),
                ("comm_fwd_us", C.c_void_p), ("comm_bwd_us", C.c_void_p),
                ("mem_mb", C.c_void_p), ("cap_mb", C.c_void_p),
                ("assign", C.c_void_p), ("A", C.c_uint64), ("allreduce_us", C.c_void_p),
                ("schedule", C.c_uint32), ("V", C.c_uint32)]


class _Cands(C.Structure):
    _fields_ = [("first", C.c_uint64), ("count", C.c_uint64),
                ("comp_rank", C.c_void_p), ("assign_idx", C.c_void_p)]


class _Best(C.Structure):
    _fields_ = [("index", C.c_uint64), ("makespan", C.c_uint32), ("feasible", C.c_uint32)]


class _SearchStats(C.Structure):
    _fields_ = [("visited", C.c_uint64), ("evaluated", C.c_uint64), ("pruned_memory", C.c_uint64),
                ("pruned_ridge", C.c_uint64), ("pruned_bound", C.c_uint64)]


class _Stats(C.Structure):
    _fields_ = [("evaluated", C.c_uint64), ("pruned", C.c_uint64), ("infeasible", C.c_uint64)]


@dataclass
class Best:
    index: Optional[int]     # None when nothing qualified
    makespan: Optional[int]
    status: int


@dataclass
class PruneStats:
    evaluated: int
    pruned: int
    infeasible: int


@dataclass
class SearchStats:
    visited: int
    evaluated: int
    pruned_memory: int
    pruned_ridge: int
    pruned_bound: int


EXPORTS = ("poseidon_validate", "poseidon_load_costs", "poseidon_eval_candidates",
           "poseidon_eval_candidates_noalloc", "poseidon_last_best", "poseidon_eval_candidates_bounded",
           "poseidon_argmin", "poseidon_search", "poseidon_free", "poseidon_strerror")

_lib = None


def lib():
    """The loaded HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        L.poseidon_validate.argtypes = [C.POINTER(_Problem), C.POINTER(C.c_uint64)]
        L.poseidon_validate.restype = C.c_int
        L.poseidon_load_costs.argtypes = [C.POINTER(_Problem), C.c_int, C.POINTER(C.c_void_p)]
        L.poseidon_load_costs.restype = C.c_int
        L.poseidon_eval_candidates.argtypes = [C.c_void_p, C.POINTER(_Cands), C.c_void_p, C.c_void_p,
                                               C.POINTER(_Best), C.c_void_p]
        L.poseidon_eval_candidates.restype = C.c_int
        L.poseidon_eval_candidates_noalloc.argtypes = L.poseidon_eval_candidates.argtypes
        L.poseidon_eval_candidates_noalloc.restype = C.c_int
        L.poseidon_last_best.argtypes = [C.c_void_p, C.POINTER(_Best), C.c_void_p]
        L.poseidon_last_best.restype = C.c_int
        L.poseidon_eval_candidates_bounded.argtypes = [C.c_void_p, C.POINTER(_Cands), C.c_uint32, C.c_uint64,
                                                       C.c_uint32, C.POINTER(_Best), C.POINTER(_Stats),
                                                       C.c_void_p]
        L.poseidon_eval_candidates_bounded.restype = C.c_int
        L.poseidon_argmin.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_uint64, C.c_uint64,
                                      C.POINTER(_Best), C.c_void_p]
        L.poseidon_argmin.restype = C.c_int
        L.poseidon_search.argtypes = [C.c_void_p, C.c_uint64, C.c_uint64, C.c_uint32, C.c_uint64, C.c_uint32,
                                      C.POINTER(_Best), C.POINTER(_SearchStats), C.c_void_p]
        L.poseidon_search.restype = C.c_int
        L.poseidon_free.argtypes = [C.c_void_p]
        L.poseidon_free.restype = None
        L.poseidon_strerror.argtypes = [C.c_int]
        L.poseidon_strerror.restype = C.c_char_p
        _lib = L
    return _lib


def strerror(status: int) -> str:
    return lib().poseidon_strerror(int(status)).decode()


def _addr(x) -> Optional[int]:
    """Device address of a torch tensor / int, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def _problem_struct(prob):
    keep = []

    def host(a, dt):
        if a is None:
            return None
        arr = np.ascontiguousarray(np.asarray(a, dtype=dt))
        keep.append(arr)
        return arr.ctypes.data

    S = int(prob.S)
    st = _Problem(int(prob.L), S, int(prob.M), int(prob.T),
                  host(prob.fwd, np.uint32), host(prob.bwd, np.uint32),
                  host(prob.comm_fwd, np.uint32) if S > 1 else None,
                  host(prob.comm_bwd, np.uint32) if S > 1 else None,
                  host(prob.mem, np.uint32), host(prob.cap, np.uint32),
                  host(prob.assign, np.uint8),
                  int(prob.assign.shape[0]) if prob.assign is not None else 0,
                  host(getattr(prob, "allreduce", None), np.uint32),
                  int(getattr(prob, "schedule", 0)), int(getattr(prob, "V", 1)))
    return st, keep


def poseidon_validate(prob) -> int:
    """Number of candidates C(L-1, S-1) * A; raises PoseidonError if invalid."""
    st, keep = _problem_struct(prob)
    n = C.c_uint64()
    rc = lib().poseidon_validate(C.byref(st), C.byref(n))
    if rc != POSEIDON_OK:
        raise PoseidonError(rc, "poseidon_validate")
    return int(n.value)


class Context:
    """Owns a ``poseidon_ctx*``; freed on close() / garbage collection."""

    def __init__(self, handle: int, prob):
        self.handle = handle
        self.S, self.M, self.L, self.T = prob.S, prob.M, prob.L, prob.T
        self.A = int(prob.A)

    def close(self):
        if self.handle:
            lib().poseidon_free(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def poseidon_load_costs(prob, device: int = 0) -> Context:
    st, keep = _problem_struct(prob)
    h = C.c_void_p()
    rc = lib().poseidon_load_costs(C.byref(st), int(device), C.byref(h))
    if rc != POSEIDON_OK:
        raise PoseidonError(rc, "poseidon_load_costs")
    return Context(h.value, prob)


def _cands(first=0, count=0, comp_rank=None, assign_idx=None):
    cr = _addr(comp_rank)
    ai = _addr(assign_idx)
    if comp_rank is not None and not isinstance(comp_rank, int):
        count = int(comp_rank.numel())
    return _Cands(int(first), int(count), cr, ai)


def _best(rc: int, b: _Best) -> Best:
    if rc == POSEIDON_NO_FEASIBLE:
        return Best(None, None, rc)
    return Best(int(b.index), int(b.makespan), rc)


def poseidon_eval_candidates(ctx: Context, *, first: int = 0, count: int = 0, comp_rank=None,
                             assign_idx=None, makespan_out=None, feasible_bits_out=None,
                             want_best: bool = True, stream=None) -> Optional[Best]:
    """Range mode (first, count) or list mode (comp_rank[, assign_idx]
    device tensors).  Returns the best (synchronising) if want_best; its
    index is the joint index first + i in range mode, the position i in
    list mode."""
    c = _cands(first, count, comp_rank, assign_idx)
    b = _Best()
    rc = lib().poseidon_eval_candidates(ctx.handle, C.byref(c), _addr(makespan_out), _addr(feasible_bits_out),
                                        C.byref(b) if want_best else None, _stream(stream))
    if rc < 0:
        raise PoseidonError(rc, "poseidon_eval_candidates")
    return _best(rc, b) if want_best else None


def poseidon_eval_candidates_noalloc(ctx: Context, *, first: int = 0, count: int = 0, comp_rank=None,
                                     assign_idx=None, makespan_out=None, feasible_bits_out=None,
                                     want_best: bool = True, stream=None) -> Optional[Best]:
    """poseidon_eval_candidates on the library's fixed per-GPU scratch (no
    device allocation during the call); same arguments and results."""
    c = _cands(first, count, comp_rank, assign_idx)
    b = _Best()
    rc = lib().poseidon_eval_candidates_noalloc(ctx.handle, C.byref(c), _addr(makespan_out),
                                                _addr(feasible_bits_out), C.byref(b) if want_best else None,
                                                _stream(stream))
    if rc < 0:
        raise PoseidonError(rc, "poseidon_eval_candidates_noalloc")
    return _best(rc, b) if want_best else None


def poseidon_last_best(ctx: Context, stream=None) -> Best:
    b = _Best()
    rc = lib().poseidon_last_best(ctx.handle, C.byref(b), _stream(stream))
    if rc < 0:
        raise PoseidonError(rc, "poseidon_last_best")
    return _best(rc, b)


def poseidon_eval_candidates_bounded(ctx: Context, bound: int, *, chunk: int = 0, first: int = 0,
                                     count: int = 0, comp_rank=None, assign_idx=None, ramp: bool = False,
                                     stream=None):
    """Early-stop pass (chunks of `chunk`, or with ramp chunk, 2 chunk,
    4 chunk, ...); returns (Best, PruneStats)."""
    c = _cands(first, count, comp_rank, assign_idx)
    b, s = _Best(), _Stats()
    rc = lib().poseidon_eval_candidates_bounded(ctx.handle, C.byref(c), int(bound), int(chunk),
                                                BOUNDED_RAMP if ramp else 0, C.byref(b), C.byref(s),
                                                _stream(stream))
    if rc < 0:
        raise PoseidonError(rc, "poseidon_eval_candidates_bounded")
    return _best(rc, b), PruneStats(int(s.evaluated), int(s.pruned), int(s.infeasible))


def poseidon_argmin(ctx: Context, makespan, feasible_bits=None, *, count: Optional[int] = None,
                    index_base: int = 0, stream=None) -> Best:
    n = int(makespan.numel()) if count is None else int(count)
    b = _Best()
    rc = lib().poseidon_argmin(ctx.handle, _addr(makespan), _addr(feasible_bits), n, int(index_base),
                               C.byref(b), _stream(stream))
    if rc < 0:
        raise PoseidonError(rc, "poseidon_argmin")
    return _best(rc, b)


def poseidon_search(ctx: Context, bound: int = 2 ** 31 - 1, *, first_row: int = 0, n_rows: Optional[int] = None,
                    rows_per_chunk: int = 0, ridge: bool = False, stage_pruning: bool = True, ramp: bool = False,
                    stream=None):
    """Pruned configuration search over assignment rows; returns (Best, SearchStats).
    Best.index is the joint index rank * A + row.  With ramp the chunks grow
    1, 2, 4, ... rows up to rows_per_chunk."""
    n = ctx.A - first_row if n_rows is None else n_rows
    flags = (SEARCH_RIDGE if ridge else 0) | (0 if stage_pruning else SEARCH_NO_STAGE_PRUNING) | \
        (SEARCH_RAMP if ramp else 0)
    b, s = _Best(), _SearchStats()
    rc = lib().poseidon_search(ctx.handle, int(first_row), int(n), int(bound), int(rows_per_chunk), flags,
                               C.byref(b), C.byref(s), _stream(stream))
    if rc < 0:
        raise PoseidonError(rc, "poseidon_search")
    return _best(rc, b), SearchStats(int(s.visited), int(s.evaluated), int(s.pruned_memory),
                                     int(s.pruned_ridge), int(s.pruned_bound))


def poseidon_free(ctx: Context) -> None:
    ctx.close()
