"""CPU oracle of Poseidon's pruned configuration search (test infrastructure).

Only the test-suite, the smoke check and the CPU-baseline leg of the
benchmark may import this module.  It shares no code with the HIP library.

The search (Sec. 4.2.3) walks the device-to-stage assignments in order and,
for each, allocates layers to stages recursively, stage 1 first, trying the
smaller layer counts first.  A partial configuration S_x (stages 1..x
fixed) is discarded with all its extensions when

* stage x does not fit the memory of its device type (Sec. 4.2.3: only
  allocations that satisfy the memory constraints are explored),
* with layer-level pruning on, the layer counts of the stages of some device
  type can no longer be ridge-like (Sec. 4.2.2, Theorem 2), or
* with stage-level pruning on, g(S_x) of Eq. 2 exceeds the current bound
  (Theorem 1).

Complete configurations that pass are evaluated on the DAG.  Readings (the
numbering continues that of ``oracle/dag.py``):

* R16 (ridge-like, Sec. 4.2.2 and Theorem 2): "first increases and then
  decreases" is read as unimodal with plateaus: non-decreasing up to some
  stage, non-increasing after it; either part may be empty.
* R17 (bound updates, Sec. 4.2.3 "updates T_min when a shorter time is
  found"): the assignments are processed in consecutive chunks of rows; a
  chunk prunes against b = min(bound, best makespan of the earlier chunks),
  fixed within the chunk, so every counter is deterministic for a given
  chunk size.  A chunk of one row updates the bound after every assignment.
  With ``ramp`` the chunks grow: chunk k (k = 0, 1, ...) holds
  min(2^k, rows_per_chunk) rows, so the bound tightens after the first row,
  then after every doubling, while the later chunks stay large.
* R18 (result and ties): the result is, among feasible (and, with the
  ridge filter, ridge-like) candidates whose makespan is <= bound, the
  one with the smallest makespan that comes first in the search's order
  (assignment row, then composition rank), reported as the joint index
  rank * A + row.  Theorem 1 makes this the exhaustive optimum: an optimal
  configuration has g(S_x) <= T_opt <= b for every prefix.
* R19 (what is counted): `visited` = partial or complete configurations
  accepted at some stage; `evaluated` = complete ones evaluated on the DAG;
  `pruned_*` = branches cut by each rule, one per stage choice that failed
  (the rules are checked in the order memory, ridge, bound, and a failed
  choice also rules out every larger layer count for that stage, since the
  memory sum and g(S_x) only grow with it and, once a type's counts are
  falling, so does the ridge test).
"""
from __future__ import annotations

import math
from typing import Optional, Sequence, Tuple

from . import dag as D


def ridge_like(seq: Sequence[int]) -> bool:
    """Unimodal with plateaus (reading R16): non-decreasing, then
    non-increasing."""
    i, n = 0, len(seq)
    while i + 1 < n and seq[i] <= seq[i + 1]:
        i += 1
    while i + 1 < n and seq[i] >= seq[i + 1]:
        i += 1
    return i >= n - 1


def layer_counts(L: int, cuts: Sequence[int]) -> Tuple[int, ...]:
    b = [0] + list(cuts) + [L]
    return tuple(b[i + 1] - b[i] for i in range(len(b) - 1))


def ridge_candidate(L: int, cuts: Sequence[int], types: Sequence[int]) -> bool:
    """Every device type's subsequence of stage layer counts is ridge-like
    (Theorem 2's property)."""
    counts = layer_counts(L, cuts)
    for t in set(types):
        if not ridge_like([counts[s] for s in range(len(types)) if types[s] == t]):
            return False
    return True


def rank_composition(L: int, S: int, cuts: Sequence[int]) -> int:
    """Lexicographic rank of a cut tuple (inverse of dag.unrank_composition,
    reading R8): for every cut, count the tuples that agree before it and
    have a smaller value there."""
    k = S - 1
    r = 0
    prev = 0
    for j, c in enumerate(cuts, start=1):
        for v in range(prev + 1, c):
            r += math.comb(L - 1 - v, k - j)
        prev = c
    return r


class _Ridge:
    """Per-type state of the prefix ridge test: last count, falling yet."""

    def __init__(self, T: int):
        self.last = [None] * T
        self.falling = [False] * T

    def admits(self, t: int, l: int) -> bool:
        return not (self.last[t] is not None and self.falling[t] and l > self.last[t])

    def push(self, t: int, l: int):
        saved = (self.last[t], self.falling[t])
        if self.last[t] is not None and l < self.last[t]:
            self.falling[t] = True
        self.last[t] = l
        return saved

    def pop(self, t: int, saved):
        self.last[t], self.falling[t] = saved


def chunk_bounds(n_rows: int, chunk: int, ramp: bool):
    """Row ranges [c0, c1) of the consecutive chunks (R17): `chunk` rows
    each, or with `ramp` 1, 2, 4, ... rows until the size reaches `chunk`."""
    out, c0, size = [], 0, 1
    while c0 < n_rows:
        step = min(size, chunk) if ramp else chunk
        out.append((c0, min(n_rows, c0 + step)))
        c0 += step
        size *= 2
    return out


def stage_search(prob, bound: int, first_row: int = 0, n_rows: Optional[int] = None,
                 rows_per_chunk: int = 0, ridge: bool = False, stage_pruning: bool = True,
                 ramp: bool = False):
    """The pruned search of Sec. 4.2.3 over assignment rows
    [first_row, first_row + n_rows) (readings R16-R19).  Returns a dict with
    `best` = (joint index, makespan) or None and the counters."""
    if getattr(prob, "schedule", 0) == D.SCHEDULE_INTERLEAVED:
        raise ValueError("Eq. 2 is stated for one stage per device; no search under Interleaved 1F1B")
    L, S, M = prob.L, prob.S, prob.M
    A = prob.A
    n_rows = A - first_row if n_rows is None else n_rows
    allreduce = getattr(prob, "allreduce", None)
    g_dag = D.dag_for(S, M, getattr(prob, "schedule", 0))
    cnt = dict(visited=0, evaluated=0, pruned_memory=0, pruned_ridge=0, pruned_bound=0)
    chunk = n_rows if rows_per_chunk <= 0 else rows_per_chunk
    best = None            # (makespan, row, rank)

    for c0, c1 in chunk_bounds(n_rows, chunk, ramp):
        b = bound if best is None else min(bound, best[0])
        chunk_best = None
        for a in range(first_row + c0, first_row + c1):
            types = D.assignment_row(prob, a)
            rs = _Ridge(prob.T)
            cuts = []

            def weights(lo, hi, t):
                f = sum(int(prob.fwd[t][k]) for k in range(lo, hi))
                bw = sum(int(prob.bwd[t][k]) for k in range(lo, hi))
                mm = sum(int(prob.mem[k]) for k in range(lo, hi))
                dd = sum(int(allreduce[t][k]) for k in range(lo, hi)) if allreduce is not None else 0
                return f, bw, mm, dd

            def rec(x, lo, pre_f, inner, Fs, Bs, Ds):
                # choose stage x (1-based) = layers [lo, hi)
                nonlocal chunk_best
                t = types[x - 1]
                last = x == S
                his = [L] if last else range(lo + 1, L - (S - x) + 1)
                for hi in his:
                    f, bw, mm, dd = weights(lo, hi, t)
                    if mm > int(prob.cap[t]):
                        cnt["pruned_memory"] += 1
                        break
                    l = hi - lo
                    if ridge and not rs.admits(t, l):
                        cnt["pruned_ridge"] += 1
                        break
                    # Eq. 2: inner_x = max_{i<=x} (B_i + ... + B_{x-1} + d_i)
                    inn = dd if x == 1 else max(inner + Bs[-1], dd)
                    g = pre_f + M * (f + bw) + inn
                    if stage_pruning and g > b:
                        cnt["pruned_bound"] += 1
                        break
                    cnt["visited"] += 1
                    saved = rs.push(t, l)
                    if last:
                        cnt["evaluated"] += 1
                        F, B, Dd = Fs + [f], Bs + [bw], Ds + [dd]
                        T = D.longest_path(g_dag, F, B, prob.comm_fwd, prob.comm_bwd,
                                           Dd if allreduce is not None else None)
                        r = rank_composition(L, S, cuts)
                        if T <= b and (chunk_best is None or T < chunk_best[0]):
                            chunk_best = (T, a, r)
                    else:
                        cuts.append(hi)
                        rec(x + 1, hi, pre_f + f, inn, Fs + [f], Bs + [bw], Ds + [dd])
                        cuts.pop()
                    rs.pop(t, saved)

            rec(1, 0, 0, 0, [], [], [])
        if chunk_best is not None and (best is None or chunk_best[0] < best[0]):
            best = chunk_best
    out = dict(cnt)
    out["best"] = None if best is None else (best[2] * A + best[1], best[0])
    return out


def exhaustive_best(prob, bound: int = 2 ** 31, first_row: int = 0, n_rows: Optional[int] = None,
                    ridge: bool = False):
    """The same result by brute force: every composition of every row in the
    range, in search order (row, then rank), no pruning."""
    L, S = prob.L, prob.S
    A = prob.A
    n_rows = A - first_row if n_rows is None else n_rows
    allreduce = getattr(prob, "allreduce", None)
    g_dag = D.dag_for(S, prob.M, getattr(prob, "schedule", 0))
    best = None
    import itertools
    for a in range(first_row, first_row + n_rows):
        types = D.assignment_row(prob, a)
        for r, cuts in enumerate(itertools.combinations(range(1, L), S - 1)):
            F, B, _, Dd, ok = D.stage_weights(prob, cuts, types, allreduce)
            if not ok or (ridge and not ridge_candidate(L, cuts, types)):
                continue
            T = D.longest_path(g_dag, F, B, prob.comm_fwd, prob.comm_bwd, Dd if allreduce is not None else None)
            if T <= bound and (best is None or T < best[0]):
                best = (T, a, r)
    return None if best is None else (best[2] * A + best[1], best[0])
