"""CPU oracle for Poseidon's DAG-based training-time model (test infrastructure).

This package is test infrastructure.  Only the test-suite, the smoke check
and the CPU-baseline leg of the benchmark may import it.  It shares no code
with the HIP library: it builds the paper's DAG explicitly and takes the
longest path in topological order, slowly and in the most literal form.

Every function cites the passage of the paper (Poseidon, arXiv 2609.06086)
it follows.  Where the paper is silent the reading is named in the
docstring; the list of readings:

* R1 (1F1B order, Sec. 4.1.2 "Intra-stage edges"): the paper does not state
  the warm-up length of plain 1F1B.  Stage s of S runs w_s = min(S - s, M)
  forward passes, then alternates (F_{w+i}, B_i) for i = 1..M-w, then runs
  the remaining M - (M - w) backward passes (the PipeDream-Flush order).
* R2 (auxiliary edges, Sec. 4.1.2): one zero-weight edge from the start node
  to F_{1,1} per pipeline.  Further zero-weight edges from the start node to
  F_{1,m} would change nothing.
* R3 (inter-stage weights, Sec. 4.1.3): one activation-transfer time per
  stage boundary and direction, independent of the layer cut.
* R4 (path weight, Def. "critical path" in App. B.1): the sum over the
  path's nodes and edges; the start node begins at time 0.
* R5 (DP all-reduce, Sec. 4.1.1/4.1.3): one pipeline (D = 1); R_s carries
  the per-layer all-reduce time summed over the stage (zero by default), so
  T = finish(E) = finish(B_{1,M}) when all-reduce times are zero.
* R6 (node weights, Sec. 4.1.3): "per-layer time x #layers" generalised to
  the sum of the per-layer times of the stage's layers on its device type.
* R7 (memory, Sec. 3.2 and Sec. 4.2.2): a stage is feasible iff the sum of its
  layers' memory footprints is <= the cap of its device type.
* R8 (candidate order): compositions in lexicographic order of the sorted
  cut tuple (itertools.combinations order), assignments in base-T order
  with stage 1 most significant; joint index = comp_rank * A + a.
* R9 (ties): the argmin returns the smallest index among equal makespans;
  infeasible candidates still get their raw DAG makespan but never win.
* R10 (stage-level bound, Eq. 2): g(S_x) as printed, with f_i, b_i the
  stage totals and d_i the stage all-reduce time; a candidate is discarded
  iff some stage exceeds its device's memory or max_x g(S_x) > bound
  (strict, as in Theorem 1).  A discarded candidate is classified as the
  search of Sec. 4.2.3 discards a partial configuration, stage by stage in
  pipeline order: the first stage x that exceeds memory (infeasible) or has
  g(S_x) > bound (pruned) decides, memory first at the same stage.
* R11 (Eager 1F1B, App. B.1): stage s runs w = min(2(S-s)+1, M) forward
  passes, then M - w groups of one backward and one forward pass, then the
  remaining backward passes.
* R20 (Interleaved 1F1B, Sec. 4.1.4; the paper gives only node and edge
  counts): N devices each hold V >= 2 model chunks; virtual stage j
  (1-based, j = 1..VN) is chunk (j-1) div N of device (j-1) mod N + 1, so
  the L layers are split into VN consecutive parts and consecutive parts
  sit on consecutive devices, wrapping from device N to device 1.  M must be
  a multiple of N.  Device p (0-based) runs the interleaved order of
  Megatron-LM (the paper's reference for the schedule): forward step k
  (k = 0..VM-1) runs chunk (k mod VN) div N on micro-batch
  (k div VN) N + k mod N + 1, backward step k runs chunk V-1 - (k mod VN) div N
  on the same micro-batch; a warm-up of min(2(N-p-1) + (V-1) N, VM) forward
  steps (all VM of them if M = N), then pairs (forward step w+i, backward
  step i), then the remaining backward steps.  For M >= 2N that warm-up is
  the one that keeps the device busy until its first backward can start and
  starts it at once (with unit weights and no transfer time); with M = N no
  warm-up can, and every forward runs first.  The intra-stage edges follow
  each device's order; one all-reduce node per device follows its last node
  and weighs the device's summed per-layer all-reduce time; a device fits
  when the summed memory of all its chunks' layers fits its cap.
"""
from __future__ import annotations

import itertools
import math
from collections import deque
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

Node = Tuple[str, int, int]      # ('F'|'B', stage s in 1..S, micro-batch m in 1..M), or ('S',0,0)...

START: Node = ("S", 0, 0)
END: Node = ("E", 0, 0)


def one_f_one_b_order(S: int, M: int, s: int) -> List[Tuple[str, int]]:
    """Execution order of stage s under 1F1B (Sec. 4.1.2, reading R1)."""
    w = min(S - s, M)
    order = [("F", m) for m in range(1, w + 1)]
    for i in range(1, M - w + 1):
        order.append(("F", w + i))
        order.append(("B", i))
    order += [("B", m) for m in range(M - w + 1, M + 1)]
    return order


def eager_1f1b_order(S: int, M: int, s: int) -> List[Tuple[str, int]]:
    """Execution order of stage s under Eager 1F1B (App. B.1, reading R11):
    a warm-up of 2(S-s)+1 forwards, steady groups of (backward, forward),
    a cool-down of the remaining backwards."""
    w = min(2 * (S - s) + 1, M)
    order = [("F", m) for m in range(1, w + 1)]
    for k in range(1, M - w + 1):
        order.append(("B", k))
        order.append(("F", w + k))
    order += [("B", m) for m in range(M - w + 1, M + 1)]
    return order


SCHEDULES = {0: one_f_one_b_order, 1: eager_1f1b_order}
SCHEDULE_INTERLEAVED = 2


def interleaved_order(N: int, V: int, M: int, p: int) -> List[Tuple[str, int, int]]:
    """Execution order of device p (1-based) under Interleaved 1F1B (Sec.
    4.1.4, reading R20) as (kind, virtual stage 1..VN, micro-batch)."""
    q = p - 1
    total = V * M
    w = total if M == N else min(2 * (N - q - 1) + (V - 1) * N, total)

    def mb(k):
        return (k // (N * V)) * N + k % N + 1

    def fwd(k):
        c = (k % (N * V)) // N
        return ("F", c * N + q + 1, mb(k))

    def bwd(k):
        c = V - 1 - (k % (N * V)) // N
        return ("B", c * N + q + 1, mb(k))

    order = [fwd(k) for k in range(w)]
    for i in range(total - w):
        order.append(fwd(w + i))
        order.append(bwd(i))
    order += [bwd(k) for k in range(total - w, total)]
    return order


def build_interleaved_dag(N: int, V: int, M: int) -> "Dag":
    """Sec. 4.1.4: 2VNM compute nodes; inter-stage edges along the VN
    virtual stages (2(NV-1)M); intra-stage edges along each device's order
    (N(2VM-1)); one all-reduce node per device after its last node; start ->
    F_{1,1}; all-reduce nodes -> end (reading R20)."""
    S = N * V
    nodes: List[Node] = [START]
    for j in range(1, S + 1):
        for m in range(1, M + 1):
            nodes.append(("F", j, m))
            nodes.append(("B", j, m))
    for p in range(1, N + 1):
        nodes.append(("R", p, 0))
    nodes.append(END)
    edges: List[Tuple[Node, Node, str]] = []
    for m in range(1, M + 1):
        for j in range(1, S):
            edges.append((("F", j, m), ("F", j + 1, m), "fwd"))
            edges.append((("B", j + 1, m), ("B", j, m), "bwd"))
    for p in range(1, N + 1):
        seq = interleaved_order(N, V, M, p)
        for a, b in zip(seq, seq[1:]):
            edges.append((a, b, "intra"))
        edges.append((seq[-1], ("R", p, 0), "allreduce"))
    edges.append((START, ("F", 1, 1), "aux"))
    for p in range(1, N + 1):
        edges.append((("R", p, 0), END, "aux"))
    return _finish_dag(S, M, nodes, edges)


@dataclass
class Dag:
    """The explicit DAG of Sec. 4.1.1-4.1.2 for one pipeline (D = 1)."""
    S: int
    M: int
    nodes: List[Node]
    # edges as (u, v, kind): kind in {'intra', 'fwd', 'bwd', 'allreduce', 'aux'}
    edges: List[Tuple[Node, Node, str]]
    topo: List[Node]
    preds: Dict[Node, List[Tuple[Node, str]]]

    def counts(self) -> Dict[str, int]:
        c: Dict[str, int] = {}
        for _, _, k in self.edges:
            c[k] = c.get(k, 0) + 1
        c["compute_nodes"] = sum(1 for n in self.nodes if n[0] in ("F", "B"))
        c["allreduce_nodes"] = sum(1 for n in self.nodes if n[0] == "R")
        return c


def build_dag(S: int, M: int, order=one_f_one_b_order) -> Dag:
    """Node and edge construction of Sec. 4.1.1-4.1.2 plus Kahn's order.

    Compute nodes F_{s,m}, B_{s,m} (2SM); all-reduce nodes R_s (S); the
    control nodes S and E.  Edges: inter-stage F_{s,m}->F_{s+1,m} and
    B_{s+1,m}->B_{s,m} (2(S-1)M); intra-stage edges along the schedule
    order (S(2M-1)); B_{s,M}->R_s (S); auxiliary S->F_{1,1} and R_s->E.
    """
    nodes: List[Node] = [START]
    for s in range(1, S + 1):
        for m in range(1, M + 1):
            nodes.append(("F", s, m))
            nodes.append(("B", s, m))
    for s in range(1, S + 1):
        nodes.append(("R", s, 0))
    nodes.append(END)
    edges: List[Tuple[Node, Node, str]] = []
    for m in range(1, M + 1):
        for s in range(1, S):
            edges.append((("F", s, m), ("F", s + 1, m), "fwd"))
            edges.append((("B", s + 1, m), ("B", s, m), "bwd"))
    for s in range(1, S + 1):
        seq = order(S, M, s)
        for (t0, m0), (t1, m1) in zip(seq, seq[1:]):
            edges.append(((t0, s, m0), (t1, s, m1), "intra"))
    for s in range(1, S + 1):
        edges.append((("B", s, M), ("R", s, 0), "allreduce"))
    edges.append((START, ("F", 1, 1), "aux"))
    for s in range(1, S + 1):
        edges.append((("R", s, 0), END, "aux"))

    return _finish_dag(S, M, nodes, edges)


def _finish_dag(S: int, M: int, nodes: List[Node], edges: List[Tuple[Node, Node, str]]) -> "Dag":
    """Predecessor lists and Kahn's topological order."""
    preds: Dict[Node, List[Tuple[Node, str]]] = {n: [] for n in nodes}
    succs: Dict[Node, List[Node]] = {n: [] for n in nodes}
    indeg: Dict[Node, int] = {n: 0 for n in nodes}
    for u, v, k in edges:
        preds[v].append((u, k))
        succs[u].append(v)
        indeg[v] += 1
    # Kahn's algorithm
    ready = deque(n for n in nodes if indeg[n] == 0)
    topo: List[Node] = []
    while ready:
        u = ready.popleft()
        topo.append(u)
        for v in succs[u]:
            indeg[v] -= 1
            if indeg[v] == 0:
                ready.append(v)
    if len(topo) != len(nodes):
        raise ValueError("schedule order produced a cycle")
    return Dag(S, M, nodes, edges, topo, preds)


_DAG_CACHE: Dict[Tuple[int, int, int, int], Dag] = {}


def dag_for(S: int, M: int, schedule: int = 0, V: int = 1) -> Dag:
    """The topology depends only on (S, M), the schedule and V; reuse it
    (Sec. 5, simulator design).  Under Interleaved 1F1B S counts virtual
    stages and the devices are N = S / V."""
    key = (S, M, schedule, V)
    if key not in _DAG_CACHE:
        if schedule == SCHEDULE_INTERLEAVED:
            _DAG_CACHE[key] = build_interleaved_dag(S // V, V, M)
        else:
            _DAG_CACHE[key] = build_dag(S, M, order=SCHEDULES[schedule])
    return _DAG_CACHE[key]


def longest_path(dag: Dag, F: Sequence[int], B: Sequence[int], cf: Sequence[int],
                 cb: Sequence[int], d: Optional[Sequence[int]] = None,
                 return_finish: bool = False):
    """Critical-path length by DP in topological order (Sec. 4.1, reading R4).

    Weights (Sec. 4.1.3): node F_{s,m} -> F[s-1], B_{s,m} -> B[s-1],
    R_s -> d[s-1] (0 if absent); edge F_{s,m}->F_{s+1,m} -> cf[s-1],
    B_{s+1,m}->B_{s,m} -> cb[s-1]; intra-stage, all-reduce and auxiliary
    edges -> 0.  finish(v) = w(v) + max(0, max over preds u of
    finish(u) + w(u, v)); T = finish(E).
    """
    finish: Dict[Node, int] = {}
    for v in dag.topo:
        kind, s, _ = v
        if kind == "F":
            wv = int(F[s - 1])
        elif kind == "B":
            wv = int(B[s - 1])
        elif kind == "R":
            wv = int(d[s - 1]) if d is not None else 0
        else:
            wv = 0
        best = 0
        for u, ek in dag.preds[v]:
            if ek == "fwd":
                we = int(cf[u[1] - 1])           # boundary u.s -> u.s + 1
            elif ek == "bwd":
                we = int(cb[v[1] - 1])           # boundary v.s <- v.s + 1
            else:
                we = 0
            best = max(best, finish[u] + we)
        finish[v] = wv + best
    if return_finish:
        return finish[END], finish
    return finish[END]


# ---------------------------------------------------------------------------
# candidates: compositions x assignments (reading R8)
# ---------------------------------------------------------------------------

def unrank_composition(L: int, S: int, r: int) -> Tuple[int, ...]:
    """Cut tuple (c_1 < ... < c_{S-1}) of lexicographic rank r among all
    (S-1)-subsets of {1..L-1}: count, for each candidate value of the next
    cut, how many subsets start with it (a Pascal-table count), skip whole
    blocks until r falls inside one."""
    k = S - 1
    if not 0 <= r < math.comb(L - 1, k):
        raise ValueError("rank out of range")
    cuts = []
    v = 0
    for j in range(1, k + 1):
        v += 1
        while True:
            cnt = math.comb(L - 1 - v, k - j)
            if r < cnt:
                cuts.append(v)
                break
            r -= cnt
            v += 1
    return tuple(cuts)


def assignment_row(prob, a: int) -> Tuple[int, ...]:
    """Stage -> device-type row a: explicit table row, or base-T digits of a
    with stage 1 the most significant digit (itertools.product order)."""
    if prob.assign is not None:
        return tuple(int(x) for x in prob.assign[a])
    digits = []
    for _ in range(n_devices(prob)):
        digits.append(a % prob.T)
        a //= prob.T
    return tuple(reversed(digits))


def n_devices(prob) -> int:
    """Devices of the pipeline: S, or S / V under Interleaved 1F1B (R20)."""
    if getattr(prob, "schedule", 0) == SCHEDULE_INTERLEAVED:
        return prob.S // prob.V
    return prob.S


def all_assignments(prob):
    if prob.assign is not None:
        return [tuple(int(x) for x in row) for row in prob.assign]
    return list(itertools.product(range(prob.T), repeat=n_devices(prob)))


def enumerate_all(prob):
    """(index, cuts, types) over every candidate, composition-major."""
    idx = 0
    rows = all_assignments(prob)
    for cuts in itertools.combinations(range(1, prob.L), prob.S - 1):
        for types in rows:
            yield idx, cuts, types
            idx += 1


def stage_weights(prob, cuts: Sequence[int], types: Sequence[int],
                  allreduce: Optional[np.ndarray] = None):
    """Per-stage F_s, B_s, memory, R_s weight and feasibility (Sec. 4.1.3,
    readings R6/R7): plain sums over each stage's layers."""
    bounds = [0] + list(cuts) + [prob.L]
    F, B, MEM, D = [], [], [], []
    feasible = True
    for s in range(prob.S):
        lo, hi = bounds[s], bounds[s + 1]
        t = types[s]
        f = sum(int(prob.fwd[t][k]) for k in range(lo, hi))
        b = sum(int(prob.bwd[t][k]) for k in range(lo, hi))
        mm = sum(int(prob.mem[k]) for k in range(lo, hi))
        dd = sum(int(allreduce[t][k]) for k in range(lo, hi)) if allreduce is not None else 0
        F.append(f)
        B.append(b)
        MEM.append(mm)
        D.append(dd)
        if mm > int(prob.cap[t]):
            feasible = False
    return F, B, MEM, D, feasible


def interleaved_weights(prob, cuts: Sequence[int], dev_types: Sequence[int],
                        allreduce: Optional[np.ndarray] = None):
    """Interleaved 1F1B (reading R20): F_j, B_j of every virtual stage on its
    device's type; memory and all-reduce weight per device, summed over the
    layers of all its chunks; feasible iff every device fits its cap."""
    N = len(dev_types)
    types = [dev_types[j % N] for j in range(prob.S)]
    F, B, MEM, D, _ = stage_weights(prob, cuts, types, allreduce)
    mem_dev = [sum(MEM[j] for j in range(prob.S) if j % N == q) for q in range(N)]
    d_dev = [sum(D[j] for j in range(prob.S) if j % N == q) for q in range(N)]
    ok = all(mem_dev[q] <= int(prob.cap[dev_types[q]]) for q in range(N))
    return F, B, mem_dev, d_dev, ok


def weights(prob, cuts, types, allreduce=None):
    """Stage weights for the problem's schedule (see stage_weights and
    interleaved_weights)."""
    if getattr(prob, "schedule", 0) == SCHEDULE_INTERLEAVED:
        return interleaved_weights(prob, cuts, types, allreduce)
    return stage_weights(prob, cuts, types, allreduce)


def candidate_list(prob, cands):
    """(index, cuts, types) for a Candidates object (range or list mode)."""
    if cands.is_list:
        out = []
        for i in range(len(cands)):
            r = int(cands.comp_rank[i])
            a = int(cands.assign_idx[i]) if cands.assign_idx is not None else 0
            out.append((i, unrank_composition(prob.L, prob.S, r), assignment_row(prob, a)))
        return out
    out = []
    lo, hi = cands.first, cands.first + cands.count
    for idx, cuts, types in enumerate_all(prob):
        if idx >= hi:
            break
        if idx >= lo:
            out.append((idx - lo, cuts, types))
    return out


def evaluate(prob, cands, allreduce=None):
    """Makespan of every candidate and its feasibility (uint32 / bool arrays).
    The all-reduce table defaults to the problem's own (``prob.allreduce``)."""
    if allreduce is None:
        allreduce = getattr(prob, "allreduce", None)
    dag = dag_for(prob.S, prob.M, getattr(prob, "schedule", 0), getattr(prob, "V", 1))
    lst = candidate_list(prob, cands)
    T = np.zeros(len(lst), dtype=np.int64)
    feas = np.zeros(len(lst), dtype=bool)
    for i, cuts, types in lst:
        F, B, _, D, ok = weights(prob, cuts, types, allreduce)
        T[i] = longest_path(dag, F, B, prob.comm_fwd, prob.comm_bwd,
                            D if allreduce is not None else None)
        feas[i] = ok
    return T, feas


def argmin(makespans, feasible):
    """Smallest makespan over feasible candidates, smallest index on ties
    (reading R9).  Returns (index, makespan) or None if nothing is feasible."""
    best = None
    for i in range(len(makespans)):
        if not feasible[i]:
            continue
        t = int(makespans[i])
        if best is None or t < best[1]:
            best = (i, t)
    return best


def eq2_terms(F: Sequence[int], B: Sequence[int], M: int,
              d: Optional[Sequence[int]] = None) -> List[int]:
    """[g(S_1), ..., g(S_S)] of Eq. 2:
    g(S_x) = sum_{i<x} f_i + M (f_x + b_x) + max_{1<=i<=x} (sum_{j=i}^{x-1} b_j + d_i)."""
    S = len(F)
    dd = d if d is not None else [0] * S
    out = []
    for x in range(1, S + 1):
        g = sum(F[i - 1] for i in range(1, x)) + M * (F[x - 1] + B[x - 1])
        inner = max(sum(B[j - 1] for j in range(i, x)) + dd[i - 1] for i in range(1, x + 1))
        out.append(g + inner)
    return out


def eq2_bound(F: Sequence[int], B: Sequence[int], M: int,
              d: Optional[Sequence[int]] = None) -> int:
    """max over x of g(S_x), Eq. 2."""
    return max(eq2_terms(F, B, M, d))


def classify(prob, cuts: Sequence[int], types: Sequence[int], bound: int, allreduce=None) -> str:
    """Reading R10's classification of one candidate against `bound`:
    'infeasible' or 'pruned' by the first stage (in pipeline order) that
    exceeds its device's memory or has g(S_x) > bound, memory first;
    'evaluated' if no stage does."""
    F, B, MEM, D, _ = stage_weights(prob, cuts, types, allreduce)
    g = eq2_terms(F, B, prob.M, D if allreduce is not None else None)
    for x in range(prob.S):
        if MEM[x] > int(prob.cap[types[x]]):
            return "infeasible"
        if g[x] > bound:
            return "pruned"
    return "evaluated"


def bounded_search(prob, cands, bound: int, chunk: int = 0, ramp: bool = False):
    """Early-stop pass (Thm. 1, reading R10) over a candidate list.

    The list is cut into consecutive chunks of `chunk` entries (0 = one
    chunk), or with ramp into chunks of chunk, 2 chunk, 4 chunk, ...
    entries.  Each chunk classifies against b = min(bound, best makespan
    found in earlier chunks) (see classify); the candidates it does not
    discard are evaluated exactly.  The result is the
    (makespan, index)-smallest evaluated candidate if its makespan is
    <= bound, else None.  Returns (best, evaluated, pruned, infeasible)."""
    if getattr(prob, "schedule", 0) == SCHEDULE_INTERLEAVED:
        raise ValueError("Eq. 2 is stated for one stage per device; no early stop under Interleaved 1F1B")
    allreduce = getattr(prob, "allreduce", None)
    dag = dag_for(prob.S, prob.M, getattr(prob, "schedule", 0))
    lst = candidate_list(prob, cands)
    n = len(lst)
    size = n if chunk <= 0 else chunk
    best = None
    evaluated = pruned = infeasible = 0
    c0 = 0
    while c0 < n:
        c1 = min(n, c0 + size)
        if ramp:
            size *= 2
        b = bound if best is None else min(bound, best[1])
        for i, cuts, types in lst[c0:c1]:
            cls = classify(prob, cuts, types, b, allreduce)
            if cls == "infeasible":
                infeasible += 1
                continue
            if cls == "pruned":
                pruned += 1
                continue
            evaluated += 1
            F, B, _, D, _ = stage_weights(prob, cuts, types, allreduce)
            t = longest_path(dag, F, B, prob.comm_fwd, prob.comm_bwd, D if allreduce is not None else None)
            if best is None or (t, i) < best[::-1]:
                best = (i, t)
        c0 = c1
    if best is not None and best[1] > bound:
        best = None
    return best, evaluated, pruned, infeasible
