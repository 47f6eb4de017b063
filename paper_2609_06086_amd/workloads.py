"""Seeded synthetic inputs for the batched 1F1B-DAG cost evaluation.

This module only draws numbers.  It holds none of the cost model's
arithmetic (no stage sums, no DAG, no longest path, no unranking), so the
HIP path and the CPU oracle can both consume what it produces without
sharing any of the method's code.

A *problem* is the per-layer profile of one model on T device types, in the
form the paper's simulator consumes (Sec. 4.1.3: per-layer forward/backward
time per device type, activation-transfer time per stage boundary, per-layer
memory footprint and a per-device memory cap).  A *candidate set* is either
an index range over all (composition, assignment) pairs or an explicit list
of sampled (composition rank, assignment index) pairs.

The five named workloads bracket the scale of the paper's search (Sec. 6.1, 6.2.3:
tens of layers, up to 16 stages, 2-4 device types with speed ratios up to
about 3x and memory caps of tens of GB).  There is no profiled data in the
paper's text, so these synthetic tables stand in for the profiling module's
output.  Integer rounding is round-half-up throughout.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = ["Problem", "Candidates", "Workload", "workload", "random_problem",
           "random_candidates", "interleaved_variant", "WORKLOAD_IDS"]


@dataclass
class Problem:
    """Per-layer profile tables (all integer microseconds / MB)."""
    L: int
    S: int
    M: int
    T: int
    fwd: np.ndarray          # uint32 [T][L]
    bwd: np.ndarray          # uint32 [T][L]
    comm_fwd: np.ndarray     # uint32 [S-1], F_{b,m} -> F_{b+1,m}
    comm_bwd: np.ndarray     # uint32 [S-1], B_{b+1,m} -> B_{b,m}
    mem: np.ndarray          # uint32 [L]
    cap: np.ndarray          # uint32 [T]
    assign: Optional[np.ndarray] = None   # uint8 [A][devices]; None => all T^devices rows
    seed: Optional[int] = None
    allreduce: Optional[np.ndarray] = None  # uint32 [T][L] DP all-reduce time per layer, or None
    schedule: int = 0                       # 0 = 1F1B, 1 = Eager 1F1B, 2 = Interleaved 1F1B
    V: int = 1                              # model chunks per device (Interleaved 1F1B)

    @property
    def devices(self) -> int:
        """Pipeline devices: S, or S / V virtual stages under Interleaved 1F1B."""
        return self.S // self.V if self.schedule == 2 else self.S

    @property
    def A(self) -> int:
        return int(self.assign.shape[0]) if self.assign is not None else self.T ** self.devices

    @property
    def n_compositions(self) -> int:
        return math.comb(self.L - 1, self.S - 1)

    @property
    def n_candidates(self) -> int:
        return self.n_compositions * self.A


@dataclass
class Candidates:
    """Range mode (first, count) or list mode (comp_rank[, assign_idx])."""
    first: int = 0
    count: int = 0
    comp_rank: Optional[np.ndarray] = None    # uint64 [count]
    assign_idx: Optional[np.ndarray] = None   # uint32 [count] or None (=> 0)

    @property
    def is_list(self) -> bool:
        return self.comp_rank is not None

    def __len__(self) -> int:
        return int(self.comp_rank.shape[0]) if self.is_list else int(self.count)


@dataclass
class Workload:
    name: str
    description: str
    problem: Problem
    cands: Candidates
    extra: dict = field(default_factory=dict)


def _rhu_scale(x: np.ndarray, p: int, q: int) -> np.ndarray:
    """round-half-up of x * p / q on non-negative integers."""
    x = x.astype(np.int64)
    return ((2 * x * p + q) // (2 * q)).astype(np.int64)


def _lognormal_base(rng, L):
    v = rng.lognormal(mean=math.log(1000.0), sigma=0.1, size=L)
    return np.maximum(np.floor(v + 0.5).astype(np.int64), 1)


def _u32(a) -> np.ndarray:
    a = np.asarray(a, dtype=np.int64)
    assert (a >= 0).all() and (a < 2**32).all()
    return np.ascontiguousarray(a.astype(np.uint32))


WORKLOAD_IDS = (1, 2, 3, 4, 5, 6)


def workload(cfg: int, n_samples: Optional[int] = None) -> Workload:
    """Build one of the five named synthetic workloads.

    ``n_samples`` overrides the sample count of the list-mode workloads
    (4 and 5); the first n entries of a shorter list equal the first n
    entries of the full list only if drawn with the same count, so tests
    that want a sub-sample should slice the full list instead.
    """
    seed = 1000 + cfg
    rng = np.random.Generator(np.random.PCG64(seed))
    if cfg == 1:
        L, S, M, T = 8, 2, 4, 2
        base = rng.integers(900, 1101, size=L)
        comm = np.full(S - 1, 50)
        mem = rng.integers(1024, 2049, size=L)
        fwd = np.stack([base, 2 * base])
        cap = [16384, 16384]
        prob = Problem(L, S, M, T, _u32(fwd), _u32(2 * fwd), _u32(comm), _u32(comm),
                       _u32(mem), _u32(cap), None, seed)
        cands = Candidates(first=0, count=prob.n_candidates)
        desc = "L=8 S=2 M=4 T=2, exhaustive 7 compositions x 4 assignments"
    elif cfg in (2, 3):
        L, S, M = (32, 4, 16) if cfg == 2 else (48, 8, 32)
        T = 2
        base = rng.integers(800, 1201, size=L)
        base[0] = (3 * base[0] + 1) // 2
        base[L - 1] = (3 * base[L - 1] + 1) // 2
        comm = rng.integers(30, 81, size=S - 1)
        mem = rng.integers(1024, 2049, size=L)
        if cfg == 2:
            fwd = np.stack([base, _rhu_scale(base, 16, 10)])
            cap = [40960, 81920]
            assign = None
            desc = "L=32 S=4 M=16 T=2, exhaustive 4,495 compositions x 16 assignments"
        else:
            fwd = np.stack([base, 2 * base])
            cap = [32768, 98304]
            assign = np.array([[0, 0, 0, 0, 1, 1, 1, 1]], dtype=np.uint8)
            desc = "L=48 S=8 M=32 T=2, fixed AAAABBBB, exhaustive C(47,7) compositions"
        prob = Problem(L, S, M, T, _u32(fwd), _u32(2 * fwd), _u32(comm), _u32(comm),
                       _u32(mem), _u32(cap), assign, seed)
        cands = Candidates(first=0, count=prob.n_candidates)
    elif cfg in (4, 5, 6):
        if cfg in (4, 6):
            L, S, M, T = 80, 8, 64, 3
            speeds, cap, comm_hi = (10, 17, 26), [65536, 81920, 196608], 120
            n = 1 << 26 if cfg == 4 else 1 << 24
        else:
            L, S, M, T = 126, 16, 128, 4
            speeds, cap, comm_hi = (10, 14, 20, 30), [49152, 65536, 98304, 196608], 160
            n = 1 << 24
        if n_samples is not None:
            n = int(n_samples)
        base = _lognormal_base(rng, L)
        base[L - 1] = 2 * base[L - 1]
        comm = rng.integers(40, comm_hi + 1, size=S - 1)
        mem = rng.integers(1024, 2049, size=L)
        # cost_t = round(base * 10 / speed_t): a faster device takes less time
        fwd = np.stack([_rhu_scale(base, 10, sp) for sp in speeds])
        if cfg == 5:
            perm = rng.permutation(np.repeat(np.arange(T), S // T))
            assign = perm.astype(np.uint8)[None, :]
        else:
            assign = None
        ar = None
        if cfg == 6:
            # gradient all-reduce per layer (data parallelism, Sec. 4.1.3): a
            # per-layer base time, slower on the device types with slower links
            ar_base = rng.integers(20000, 60001, size=L)
            ar = np.stack([_rhu_scale(ar_base, 10, sp) for sp in speeds])
        prob = Problem(L, S, M, T, _u32(fwd), _u32(2 * fwd), _u32(comm), _u32(comm),
                       _u32(mem), _u32(cap), assign, seed, None if ar is None else _u32(ar))
        ncomp = prob.n_compositions
        ranks = rng.integers(0, ncomp, size=n, dtype=np.uint64)
        if assign is None:
            aidx = rng.integers(0, prob.A, size=n, dtype=np.uint32)
        else:
            aidx = None
        cands = Candidates(comp_rank=np.ascontiguousarray(ranks),
                           assign_idx=None if aidx is None else np.ascontiguousarray(aidx))
        if cfg == 6:
            desc = "L=80 S=8 M=64 T=3 with DP all-reduce, 2^24 sampled (composition, assignment) pairs"
        elif cfg == 4:
            desc = "L=80 S=8 M=64 T=3, 2^26 sampled (composition, assignment) pairs"
        else:
            desc = "L=126 S=16 M=128 T=4, fixed 4x4 type permutation, 2^24 sampled compositions"
    else:
        raise ValueError(f"unknown workload {cfg}")
    return Workload(f"cfg{cfg}", desc, prob, cands)


def random_problem(rng: np.random.Generator, L: int, S: int, M: int, T: int, *,
                   cost_lo: int = 1, cost_hi: int = 1000, comm_hi: int = 100,
                   mem_lo: int = 1, mem_hi: int = 100, cap=None,
                   assign_rows: Optional[int] = None) -> Problem:
    """Small random problem for tests: independent uniform integer tables."""
    fwd = rng.integers(cost_lo, cost_hi + 1, size=(T, L))
    bwd = rng.integers(cost_lo, cost_hi + 1, size=(T, L))
    cf = rng.integers(0, comm_hi + 1, size=max(S - 1, 0))
    cb = rng.integers(0, comm_hi + 1, size=max(S - 1, 0))
    mem = rng.integers(mem_lo, mem_hi + 1, size=L)
    if cap is None:
        cap = rng.integers(mem_hi, mem_hi * L + 1, size=T)
    assign = None
    if assign_rows is not None:
        assign = rng.integers(0, T, size=(assign_rows, S)).astype(np.uint8)
    return Problem(L, S, M, T, _u32(fwd), _u32(bwd), _u32(cf), _u32(cb), _u32(mem),
                   _u32(np.broadcast_to(cap, (T,))), assign)


def random_candidates(rng: np.random.Generator, prob: Problem, n: int,
                      with_assign: bool = True) -> Candidates:
    """n uniform (composition rank, assignment index) samples, with repeats."""
    ranks = rng.integers(0, prob.n_compositions, size=n, dtype=np.uint64)
    aidx = None
    if with_assign and prob.A > 1:
        aidx = rng.integers(0, prob.A, size=n, dtype=np.uint32)
    return Candidates(comp_rank=np.ascontiguousarray(ranks),
                      assign_idx=None if aidx is None else np.ascontiguousarray(aidx))


def interleaved_variant(wl: "Workload", V: int = 2) -> "Workload":
    """The same tables and samples under Interleaved 1F1B: the S stages
    become virtual stages on S / V devices (V chunks each), and the stage
    type row keeps its first S / V entries as the device types.  Needs a
    fixed type row (A = 1) and M a multiple of S / V."""
    prob = wl.problem
    N = prob.S // V
    if prob.assign is None or prob.assign.shape[0] != 1 or prob.S % V or prob.M % N:
        raise ValueError("interleaved variant needs one fixed type row and M a multiple of S / V")
    prob.schedule = 2
    prob.V = V
    prob.assign = np.ascontiguousarray(prob.assign[:, :N])
    wl.description = wl.description + f", Interleaved 1F1B with {N} devices x {V} chunks"
    return wl
