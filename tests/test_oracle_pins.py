"""Pins of the CPU oracle against facts that do not come from the oracle.

Each test checks the oracle (Python and C) against something fixed by the
paper or by mathematics: the node/edge counts of Sec. 4.1.1-4.1.2, closed
forms of uniform pipelines, hand-derived worked examples, an independent
event-driven simulation, brute-force path enumeration, symmetry and
monotonicity of longest paths, Eq. 2's lower bound and Theorem 1.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

from oracle import coracle, dag, des
from paper_2609_06086_amd import workloads as W

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def T_of(S, M, F, B, cf, cb):
    return dag.longest_path(dag.dag_for(S, M), F, B, cf, cb)


# ---------------------------------------------------------------- DAG shape

@pytest.mark.parametrize("S,M", [(1, 1), (2, 4), (3, 2), (4, 8), (4, 3), (8, 32), (5, 1)])
def test_dag_counts_sec_4_1(S, M):
    """Sec. 4.1.1-4.1.2: 2SM compute nodes, 2(S-1)M inter-stage edges,
    S(2M-1) intra-stage edges, S all-reduce nodes and edges, D + S auxiliary
    edges (D = 1)."""
    c = dag.build_dag(S, M).counts()
    assert c["compute_nodes"] == 2 * S * M
    assert c.get("fwd", 0) + c.get("bwd", 0) == 2 * (S - 1) * M
    assert c["intra"] == S * (2 * M - 1)
    assert c["allreduce_nodes"] == S and c["allreduce"] == S
    assert c["aux"] == 1 + S
    cc = coracle.dag_counts(S, M)
    assert cc["nodes"] == 2 * S * M + S + 2
    assert cc["fwd"] + cc["bwd"] == 2 * (S - 1) * M
    assert cc["intra"] == S * (2 * M - 1)
    assert cc["other"] == S + 1 + S


def test_1f1b_order_is_a_permutation_with_f_before_b():
    for S in range(1, 7):
        for M in range(1, 9):
            for s in range(1, S + 1):
                o = dag.one_f_one_b_order(S, M, s)
                assert sorted(o) == sorted([("F", m) for m in range(1, M + 1)] +
                                           [("B", m) for m in range(1, M + 1)])
                pos = {x: i for i, x in enumerate(o)}
                assert all(pos[("F", m)] < pos[("B", m)] for m in range(1, M + 1))
                # forward passes run in micro-batch order, as do backward passes
                assert [m for k, m in o if k == "F"] == list(range(1, M + 1))
                assert [m for k, m in o if k == "B"] == list(range(1, M + 1))
                # in-flight forwards never exceed the warm-up depth + 1
                infl, peak = 0, 0
                for k, _ in o:
                    infl += 1 if k == "F" else -1
                    peak = max(peak, infl)
                assert peak == min(S - s + 1, M)


# ------------------------------------------------------------ closed forms

@pytest.mark.parametrize("S", range(1, 7))
@pytest.mark.parametrize("M", range(1, 12))
def test_uniform_zero_comm_closed_form(S, M):
    """Uniform stages, no transfer time: T = (M + S - 1)(t_f + t_b)."""
    tf, tb = 7, 13
    assert T_of(S, M, [tf] * S, [tb] * S, [0] * (S - 1), [0] * (S - 1)) == (M + S - 1) * (tf + tb)


def test_uniform_closed_form_c_oracle_large():
    """Same closed form through the C oracle at the workloads' (S, M) shapes."""
    for S, M in [(2, 4), (4, 16), (8, 32), (8, 64), (16, 128), (16, 3), (9, 20)]:
        L = S * 3
        prob = W.Problem(L, S, M, 1, np.full((1, L), 5, np.uint32), np.full((1, L), 11, np.uint32),
                         np.zeros(S - 1, np.uint32), np.zeros(S - 1, np.uint32),
                         np.ones(L, np.uint32), np.array([10**6], np.uint32),
                         np.full((1, S), 0, np.uint8))
        # the composition with 3 layers on every stage
        cuts = tuple(range(3, L, 3))
        r = list(itertools.combinations(range(1, L), S - 1)).index(cuts) if L <= 24 else None
        if r is None:
            # rank of the all-3 composition by direct counting of smaller tuples
            r = 0
            prev = 0
            for j, c in enumerate(cuts, start=1):
                for v in range(prev + 1, c):
                    r += math.comb(L - 1 - v, S - 1 - j)
                prev = c
        cands = W.Candidates(comp_rank=np.array([r], np.uint64))
        T, f = coracle.evaluate(prob, cands)
        assert int(T[0]) == (M + S - 1) * 3 * (5 + 11)


@pytest.mark.parametrize("M", [1, 2, 5, 9])
def test_single_stage(M):
    """S = 1: the stage runs F, B alternately with nothing else: T = M(F + B)."""
    assert T_of(1, M, [17], [29], [], []) == M * (17 + 29)


@pytest.mark.parametrize("S", [1, 2, 3, 6])
def test_single_microbatch(S):
    """M = 1: the DAG is one chain F_1..F_S, B_S..B_1: T = sum(F+B) + sum(cf+cb)."""
    rng = np.random.default_rng(S)
    F, B = rng.integers(1, 100, S), rng.integers(1, 100, S)
    cf, cb = rng.integers(0, 50, S - 1), rng.integers(0, 50, S - 1)
    assert T_of(S, 1, F, B, cf, cb) == int(F.sum() + B.sum() + cf.sum() + cb.sum())


def test_worked_examples_golden():
    """Hand-derived per-node finish times (tests/golden/worked_examples.json)."""
    ex = json.load(open(os.path.join(GOLD, "worked_examples.json")))["examples"]
    for e in ex:
        T, fin = dag.longest_path(dag.build_dag(e["S"], e["M"]), e["F"], e["B"], e["cf"], e["cb"],
                                  return_finish=True)
        assert T == e["T"], e["name"]
        for key, val in e["finish"].items():
            k, s, m = key.split(",")
            assert fin[(k, int(s), int(m))] == val, (e["name"], key)
        # the same value through the C oracle: one composition with one layer per stage
        S = e["S"]
        prob = W.Problem(S, S, e["M"], 1, np.array([e["F"]], np.uint32), np.array([e["B"]], np.uint32),
                         np.array(e["cf"], np.uint32), np.array(e["cb"], np.uint32),
                         np.ones(S, np.uint32), np.array([S], np.uint32), np.zeros((1, S), np.uint8))
        Tc, fc = coracle.evaluate(prob, W.Candidates(first=0, count=1))
        assert int(Tc[0]) == e["T"] and bool(fc[0])


# ----------------------------------------------------- independent models

def _rand_case(rng, S, M, hi=60):
    return (rng.integers(1, hi, S), rng.integers(1, hi, S),
            rng.integers(0, hi, S - 1), rng.integers(0, hi, S - 1))


def test_event_driven_simulation_matches_dag():
    """An event-queue simulation of the 1F1B schedule gives the DAG's T."""
    rng = np.random.default_rng(7)
    for _ in range(250):
        S, M = int(rng.integers(1, 7)), int(rng.integers(1, 9))
        F, B, cf, cb = _rand_case(rng, S, M)
        assert des.simulate_1f1b(S, M, F, B, cf, cb, dag.one_f_one_b_order) == T_of(S, M, F, B, cf, cb)


def test_brute_force_paths_match_dp():
    """Every start->end path enumerated; the heaviest equals the DP value."""
    rng = np.random.default_rng(8)
    for S, M in [(1, 3), (2, 2), (2, 4), (3, 2), (3, 3), (4, 2)]:
        d = dag.build_dag(S, M)
        for _ in range(20):
            F, B, cf, cb = _rand_case(rng, S, M)
            assert des.all_paths_longest(d, F, B, cf, cb) == dag.longest_path(d, F, B, cf, cb)


def test_allreduce_nodes_extend_the_sink():
    """With per-stage all-reduce weights d_s the end node takes
    max_s(finish(B_{s,M}) + d_s) (Sec. 4.1.1/4.1.3); with d = 0 it is finish(B_{1,M})."""
    rng = np.random.default_rng(9)
    for _ in range(50):
        S, M = int(rng.integers(1, 6)), int(rng.integers(1, 7))
        F, B, cf, cb = _rand_case(rng, S, M)
        d = rng.integers(0, 500, S)
        g = dag.build_dag(S, M)
        T0, fin = dag.longest_path(g, F, B, cf, cb, return_finish=True)
        assert T0 == fin[("B", 1, M)]
        assert all(fin[("B", s, M)] <= T0 for s in range(1, S + 1))
        T1 = dag.longest_path(g, F, B, cf, cb, d)
        assert T1 == max(fin[("B", s, M)] + int(d[s - 1]) for s in range(1, S + 1))
        assert des.all_paths_longest(g, F, B, cf, cb, d) == T1 if S * M <= 6 else True


# ----------------------------------------------------------- invariants

def test_reversal_symmetry():
    """Reversing every edge maps the 1F1B DAG onto itself with F<->B and
    cf<->cb swapped (F_{s,m} <-> B_{s,M+1-m}), so T is unchanged."""
    rng = np.random.default_rng(10)
    for _ in range(200):
        S, M = int(rng.integers(1, 7)), int(rng.integers(1, 9))
        F, B, cf, cb = _rand_case(rng, S, M)
        assert T_of(S, M, F, B, cf, cb) == T_of(S, M, B, F, cb, cf)


def test_monotone_and_homogeneous():
    rng = np.random.default_rng(11)
    for _ in range(150):
        S, M = int(rng.integers(1, 6)), int(rng.integers(1, 8))
        F, B, cf, cb = _rand_case(rng, S, M)
        T = T_of(S, M, F, B, cf, cb)
        assert T_of(S, M, 3 * F, 3 * B, 3 * cf, 3 * cb) == 3 * T
        assert T_of(S, M + 1, F, B, cf, cb) >= T
        which = int(rng.integers(0, 4))
        arrs = [F.copy(), B.copy(), cf.copy(), cb.copy()]
        if len(arrs[which]):
            arrs[which][int(rng.integers(0, len(arrs[which])))] += int(rng.integers(1, 40))
            assert T_of(S, M, *arrs) >= T
        # upper bound: every node and edge weight counted once
        assert T <= M * int(F.sum() + B.sum()) + M * int(cf.sum() + cb.sum())
        # the busiest stage must run all its work
        assert T >= M * int((F + B).max())


def test_eq2_lower_bound_holds():
    """Theorem 1 needs g(S_x) <= T for every completion: check T >= max_x g(S_x)."""
    rng = np.random.default_rng(12)
    for _ in range(300):
        S, M = int(rng.integers(1, 7)), int(rng.integers(1, 10))
        F, B, cf, cb = _rand_case(rng, S, M)
        assert dag.eq2_bound(list(F), list(B), M) <= T_of(S, M, F, B, cf, cb)


def test_eq2_bound_is_a_real_path_when_uniform():
    """Uniform stages, no comm: g(S_S) = (S-1)(f+b) + M(f+b) = T, the bound is tight."""
    for S in range(1, 6):
        for M in range(1, 8):
            assert dag.eq2_bound([3] * S, [5] * S, M) == (M + S - 1) * 8 == T_of(S, M, [3] * S, [5] * S,
                                                                                 [0] * (S - 1), [0] * (S - 1))


def test_static_model_eq1_differs():
    """Sec. 2.2: the static model sum t_s + (B-1) max t_j is not the DAG's
    T; it overestimates when communication overlaps with computation."""
    S, M, F, B, c = 2, 2, [10, 10], [20, 20], [3]
    t = [F[0] + B[0] + c[0], F[1] + B[1] + c[0]]
    eq1 = sum(t) + (M - 1) * max(t)
    assert eq1 != T_of(S, M, F, B, c, c)


# ---------------------------------------------------------- enumeration

def test_candidate_counts():
    assert W.workload(1).problem.n_candidates == 28
    assert W.workload(2).problem.n_candidates == 71920
    assert W.workload(3).problem.n_candidates == 62891499
    assert math.comb(79, 7) == 2898753715 and math.comb(125, 15) < 2 ** 63


@pytest.mark.parametrize("L,S", [(8, 2), (9, 4), (10, 10), (12, 1), (13, 6)])
def test_unrank_is_lexicographic(L, S):
    allc = list(itertools.combinations(range(1, L), S - 1))
    assert len(allc) == math.comb(L - 1, S - 1)
    for r, c in enumerate(allc):
        assert dag.unrank_composition(L, S, r) == c


def test_c_oracle_matches_python_oracle_random():
    rng = np.random.default_rng(13)
    for trial in range(25):
        S = int(rng.integers(1, 6))
        L = int(rng.integers(S, S + 6))
        M = int(rng.integers(1, 9))
        T = int(rng.integers(1, 4))
        rows = None if trial % 2 else int(rng.integers(1, 5))
        prob = W.random_problem(rng, L, S, M, T, assign_rows=rows, mem_hi=30, cap=int(rng.integers(30, 120)))
        full = W.Candidates(first=0, count=prob.n_candidates)
        Tp, fp = dag.evaluate(prob, full)
        Tc, fc = coracle.evaluate(prob, full, nthreads=3)
        assert (Tp == Tc).all() and (fp == fc).all()
        lst = W.random_candidates(rng, prob, 40)
        Tp, fp = dag.evaluate(prob, lst)
        Tc, fc = coracle.evaluate(prob, lst, nthreads=2)
        assert (Tp == Tc).all() and (fp == fc).all()


def test_c_oracle_matches_python_oracle_cfg1_cfg2():
    wl = W.workload(1)
    Tp, fp = dag.evaluate(wl.problem, wl.cands)
    Tc, fc = coracle.evaluate(wl.problem, wl.cands)
    assert (Tp == Tc).all() and (fp == fc).all()
    wl = W.workload(2)
    # a strided sample of config 2 through the Python enumeration
    sub = W.Candidates(first=0, count=wl.problem.n_candidates)
    Tc, fc = coracle.evaluate(wl.problem, sub)
    picks = list(range(0, wl.problem.n_candidates, 997))
    full = {i: (c, t) for i, c, t in dag.enumerate_all(wl.problem) if i % 997 == 0}
    g = dag.dag_for(wl.problem.S, wl.problem.M)
    for i in picks:
        cuts, types = full[i]
        F, B, _, _, ok = dag.stage_weights(wl.problem, cuts, types)
        assert dag.longest_path(g, F, B, wl.problem.comm_fwd, wl.problem.comm_bwd) == int(Tc[i])
        assert ok == bool(fc[i])


# ---------------------------------------------------- argmin, feasibility

def test_argmin_tie_break_and_no_feasible():
    T = np.array([5, 3, 3, 7, 3], np.uint32)
    f = np.array([True, False, True, True, True])
    assert dag.argmin(T, f) == (2, 3)
    assert coracle.argmin(T, f) == (2, 3)
    assert dag.argmin(T, np.zeros(5, bool)) is None
    assert coracle.argmin(T, np.zeros(5, bool)) is None


def test_cap_equality_is_feasible():
    prob = W.Problem(2, 2, 2, 1, np.ones((1, 2), np.uint32), np.ones((1, 2), np.uint32),
                     np.zeros(1, np.uint32), np.zeros(1, np.uint32), np.array([7, 9], np.uint32),
                     np.array([9], np.uint32), None)
    _, fc = coracle.evaluate(prob, W.Candidates(first=0, count=1))
    assert bool(fc[0])
    prob.cap = np.array([8], np.uint32)
    _, fc = coracle.evaluate(prob, W.Candidates(first=0, count=1))
    assert not bool(fc[0])
    _, _, _, _, ok = dag.stage_weights(prob, (1,), (0, 0))
    assert not ok


def test_duplicate_candidates_tie_to_first():
    wl = W.workload(2)
    prob = wl.problem
    rng = np.random.default_rng(3)
    lst = W.random_candidates(rng, prob, 300)
    lst.comp_rank[250] = lst.comp_rank[40]
    lst.assign_idx[250] = lst.assign_idx[40]
    T, f = coracle.evaluate(prob, lst)
    assert T[250] == T[40] and f[250] == f[40]
    best = coracle.argmin(T, f)
    assert best[0] != 250


# ------------------------------------------------------------ early stop

def test_bounded_search_theorem1():
    """Pruning with g(S_x) > bound never loses the optimum (Theorem 1); the
    pruned candidates all have T > bound; Python and C agree on counts."""
    rng = np.random.default_rng(14)
    for trial in range(12):
        S = int(rng.integers(2, 6))
        L = int(rng.integers(S + 2, S + 9))
        M = int(rng.integers(1, 12))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=20, cap=int(rng.integers(40, 120)))
        lst = W.random_candidates(rng, prob, 150)
        Tx, fx = dag.evaluate(prob, lst)
        exact = dag.argmin(Tx, fx)
        if exact is None:
            continue
        warm = dag.argmin(Tx[:20], fx[:20])
        bound = warm[1] if warm else 2 ** 32 - 1
        for chunk, ramp in ((0, False), (17, False), (64, False), (1, True), (9, True)):
            best, ev, pr, inf = dag.bounded_search(prob, lst, bound, chunk, ramp=ramp)
            assert best == exact
            bc = coracle.bounded(prob, lst, bound, chunk, nthreads=3, ramp=ramp)
            assert bc == (best, ev, pr, inf)
            assert ev + pr + inf == len(lst) and inf <= int((~fx).sum())
            # the evaluated candidates are exactly the feasible ones within the bound
            if chunk == 0:
                assert ev == sum(1 for i, cuts, types in dag.candidate_list(prob, lst)
                                 if fx[i] and dag.eq2_bound(*dag.stage_weights(prob, cuts, types)[:2], M) <= bound)
        # every candidate pruned against the fixed bound is strictly worse than it
        for i, cuts, types in dag.candidate_list(prob, lst):
            F, B, _, _, ok = dag.stage_weights(prob, cuts, types)
            if ok and dag.eq2_bound(F, B, M) > bound:
                assert Tx[i] > bound


def test_bounded_classification_in_stage_order():
    """A discarded candidate is classified by its first failing stage, memory
    first.  With bound 0 every g(S_1) > 0 fails at stage 1, so exactly the
    candidates whose first stage exceeds memory are infeasible, whatever
    their later stages do; with no bound the infeasible ones are exactly
    those with some stage over memory."""
    rng = np.random.default_rng(17)
    for trial in range(6):
        prob = W.random_problem(rng, 14, 4, int(rng.integers(1, 6)), 2, mem_hi=20, cap=int(rng.integers(35, 70)))
        lst = W.random_candidates(rng, prob, 300)
        Tx, fx = dag.evaluate(prob, lst)
        first_over = later_over = 0
        for i, cuts, types in dag.candidate_list(prob, lst):
            mem0 = sum(int(prob.mem[k]) for k in range(0, cuts[0]))
            if mem0 > int(prob.cap[types[0]]):
                first_over += 1
            elif not fx[i]:
                later_over += 1
        assert later_over > 0   # the case that tells the two orders apart
        for impl in (dag.bounded_search, coracle.bounded):
            best, ev, pr, inf = impl(prob, lst, 0)
            assert (best, ev, pr, inf) == (None, 0, len(lst) - first_over, first_over)
            best, ev, pr, inf = impl(prob, lst, 2 ** 32 - 1)
            assert (pr, inf, ev) == (0, int((~fx).sum()), int(fx.sum()))


def test_bounded_ramp_chunks_double():
    """With ramp the chunks are [0, c), [c, 3c), [3c, 7c), ...: running the
    fixed-chunk pass on each piece in turn, the bound of each piece being the
    best makespan of the pieces before it, gives the same counts."""
    rng = np.random.default_rng(16)
    for trial in range(6):
        prob = W.random_problem(rng, 12, 4, int(rng.integers(2, 9)), 2, mem_hi=15, cap=90)
        n = int(rng.integers(40, 130))
        cands = W.random_candidates(rng, prob, n)
        bound = 2 ** 32 - 1
        c = int(rng.integers(1, 6))
        lo, size, best, tot = 0, c, None, [0, 0, 0]
        while lo < n:
            hi = min(n, lo + size)
            size *= 2
            piece = W.Candidates(comp_rank=cands.comp_rank[lo:hi],
                                 assign_idx=None if cands.assign_idx is None else cands.assign_idx[lo:hi])
            b = bound if best is None else min(bound, best[1])
            pb, ev, pr, inf = dag.bounded_search(prob, piece, b)
            tot = [tot[0] + ev, tot[1] + pr, tot[2] + inf]
            if pb is not None and (best is None or (pb[1], pb[0] + lo) < (best[1], best[0])):
                best = (pb[0] + lo, pb[1])
            lo = hi
        assert dag.bounded_search(prob, cands, bound, c, ramp=True) == (best, *tot)
        assert coracle.bounded(prob, cands, bound, c, ramp=True) == (best, *tot)


def test_bounded_search_no_candidate_under_bound():
    rng = np.random.default_rng(15)
    prob = W.random_problem(rng, 8, 3, 4, 2, mem_hi=10, cap=200)
    lst = W.random_candidates(rng, prob, 50)
    Tx, fx = dag.evaluate(prob, lst)
    lo = int(Tx[fx].min())
    assert dag.bounded_search(prob, lst, lo - 1)[0] is None
    assert coracle.bounded(prob, lst, lo - 1)[0] is None
    assert dag.bounded_search(prob, lst, lo)[0][1] == lo


# -------------------------------------------------- planted mistakes

def _wrong_warmup(S, M, s):
    w = min(S - s + 1, M)
    o = [("F", m) for m in range(1, w + 1)]
    for i in range(1, M - w + 1):
        o += [("F", w + i), ("B", i)]
    return o + [("B", m) for m in range(M - w + 1, M + 1)]


def _gpipe(S, M, s):
    return [("F", m) for m in range(1, M + 1)] + [("B", m) for m in range(1, M + 1)]


@pytest.mark.parametrize("mutant", [_wrong_warmup, _gpipe])
def test_planted_schedule_mistakes_are_caught(mutant):
    """A wrong intra-stage order must fail the worked examples."""
    ex = json.load(open(os.path.join(GOLD, "worked_examples.json")))["examples"]
    fails = 0
    for e in ex:
        g = dag.build_dag(e["S"], e["M"], order=mutant)
        fails += dag.longest_path(g, e["F"], e["B"], e["cf"], e["cb"]) != e["T"]
    assert fails > 0


def test_planted_weight_mistakes_are_caught():
    """Weight mix-ups planted in the DP's inputs (a boundary index reversed,
    an edge weight dropped) are caught by the event-driven simulation on
    random cases.  (Swapping F with B, or cf with cb, leaves T unchanged on
    every random case tried, so such a swap is harmless to the makespan;
    the per-node finish times of the worked examples still catch it.)"""
    rng = np.random.default_rng(16)
    mutants = {
        "cb_reversed": lambda F, B, cf, cb: (F, B, cf, cb[::-1]),
        "cf_reversed": lambda F, B, cf, cb: (F, B, cf[::-1], cb),
        "cb_dropped": lambda F, B, cf, cb: (F, B, cf, 0 * cb),
    }
    caught = {k: False for k in mutants}
    for _ in range(300):
        S, M = int(rng.integers(3, 6)), int(rng.integers(2, 7))
        F, B, cf, cb = _rand_case(rng, S, M)
        ref = des.simulate_1f1b(S, M, F, B, cf, cb, dag.one_f_one_b_order)
        assert T_of(S, M, F, B, cf, cb) == ref
        for k, mut in mutants.items():
            if T_of(S, M, *mut(F, B, cf, cb)) != ref:
                caught[k] = True
    assert all(caught.values()), caught


def test_stage_weights_cover_exactly_the_stage_layers():
    """With fwd[t][k] = 2^k + t * 2^40 a stage's sum spells out which layers
    and which type it took: F_s = 2^{c_s} - 2^{c_{s-1}} + n_s t_s 2^40."""
    L, S, T = 12, 4, 3
    fwd = np.array([[2 ** k + t * 2 ** 40 for k in range(L)] for t in range(T)], dtype=object)
    prob = W.Problem(L, S, 2, T, fwd, fwd, np.zeros(S - 1, np.uint32), np.zeros(S - 1, np.uint32),
                     np.arange(1, L + 1, dtype=np.uint32), np.full(T, 10 ** 6, np.uint32), None)
    rng = np.random.default_rng(17)
    for _ in range(40):
        r = int(rng.integers(0, math.comb(L - 1, S - 1)))
        a = int(rng.integers(0, T ** S))
        cuts, types = dag.unrank_composition(L, S, r), dag.assignment_row(prob, a)
        assert a == sum(t * T ** (S - 1 - s) for s, t in enumerate(types))
        F, B, MEM, _, _ = dag.stage_weights(prob, cuts, types)
        b = [0] + list(cuts) + [L]
        for s in range(S):
            n = b[s + 1] - b[s]
            assert F[s] == 2 ** b[s + 1] - 2 ** b[s] + n * types[s] * 2 ** 40
            assert MEM[s] == sum(range(b[s] + 1, b[s + 1] + 1))


# ------------------------------------------------------- DP all-reduce

def test_c_oracle_allreduce_matches_python():
    """R_s weights (per-layer all-reduce summed over the stage, Sec. 4.1.3)
    and the d_i term of Eq. 2, Python vs C, exhaustive and early stop."""
    rng = np.random.default_rng(18)
    for trial in range(12):
        S = int(rng.integers(1, 6))
        L = S + int(rng.integers(0, 6))
        M = int(rng.integers(1, 9))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=30, cap=int(rng.integers(30, 150)),
                                assign_rows=None if trial % 2 else 3)
        prob.allreduce = rng.integers(0, 800, size=(2, L)).astype(np.uint32)
        full = W.Candidates(first=0, count=prob.n_candidates)
        Tp, fp = dag.evaluate(prob, full)
        Tc, fc = coracle.evaluate(prob, full, nthreads=3)
        assert (Tp == Tc).all() and (fp == fc).all()
        Tx, fx = Tp, fp
        ex = dag.argmin(Tx, fx)
        if ex is None:
            continue
        bound = int(Tx[fx].max())
        for chunk in (0, 7):
            best, ev, pr, inf = dag.bounded_search(prob, full, bound, chunk)
            assert best == ex
            assert coracle.bounded(prob, full, bound, chunk, nthreads=2) == (best, ev, pr, inf)


def test_allreduce_event_simulation():
    """The event-driven run extended with a gradient all-reduce that each
    stage starts after its last backward pass: iteration end = max over
    stages of (last backward finish + d_s); equals the DAG's finish(E)."""
    rng = np.random.default_rng(19)
    for _ in range(100):
        S, M = int(rng.integers(1, 6)), int(rng.integers(1, 8))
        F, B, cf, cb = _rand_case(rng, S, M)
        d = rng.integers(0, 400, S)
        t_end = des.simulate_1f1b(S, M, F, B, cf, cb, dag.one_f_one_b_order, allreduce=d)
        assert t_end == dag.longest_path(dag.dag_for(S, M), F, B, cf, cb, d)


def test_eq2_with_allreduce_is_a_lower_bound():
    rng = np.random.default_rng(20)
    for _ in range(300):
        S, M = int(rng.integers(1, 7)), int(rng.integers(1, 10))
        F, B, cf, cb = _rand_case(rng, S, M)
        d = rng.integers(0, 500, S)
        assert dag.eq2_bound(list(F), list(B), M, list(d)) <= dag.longest_path(dag.dag_for(S, M), F, B, cf, cb, d)


# ------------------------------------------------------- Eager 1F1B

def _kxyw_cost(N, M, F, B, tf, tb, x, y, w):
    """Cost of the canonical path K(x, y, w) (App. B.2, Eq. formula.cost)."""
    c = sum(F[i] + B[i] + tf[i] + tb[i] for i in range(x - 1)) + F[x - 1] + B[x - 1]
    c += 2 * (N - x) * F[w - 1] + 2 * (N - y) * B[w - 1]
    c += (M - 2 * (N - y) - 1) * (F[y - 1] + B[y - 1])
    return c


def _kxyw_max(N, M, F, B, tf, tb):
    best = 0
    for x in range(1, N + 1):
        for y in range(1, x + 1):
            if F[y - 1] != max(F[y - 1:x]):
                continue
            for w in range(1, y + 1):
                if F[w - 1] == max(F[:x]):
                    best = max(best, _kxyw_cost(N, M, F, B, tf, tb, x, y, w))
    return best


def _assumption_case(rng):
    """Random Eager-1F1B instance satisfying Assumptions 1-4 of App. B.1:
    b_i = r f_i (r > 1), t <= (r-1)/2 F_min, M >= 2N, F_min >= alpha F_max."""
    N = int(rng.integers(1, 6))
    M = int(rng.integers(2 * N, 2 * N + 12))
    p, q = int(rng.integers(12, 31)), 10          # r = p / q in [1.2, 3.0]
    r = p / q
    alpha = max(2 / 3, r / (1 + r))
    fmax = int(rng.integers(50, 200))
    F = [q * int(rng.integers(int(np.ceil(alpha * fmax)), fmax + 1)) for _ in range(N)]
    B = [f * p // q for f in F]
    tmax = int((r - 1) / 2 * min(F))
    tf = [int(rng.integers(0, tmax + 1)) for _ in range(N - 1)]
    tb = [int(rng.integers(0, tmax + 1)) for _ in range(N - 1)]
    return N, M, F, B, tf, tb


def test_eager_matches_the_papers_critical_path_theorem():
    """Under Assumptions 1-4 some K(x, y, w) is a critical path of the
    Eager-1F1B DAG (App. B.2), so the DAG's longest path equals the largest
    C(K(x, y, w)) over the admissible (x, y, w) of Def. 4."""
    rng = np.random.default_rng(21)
    for _ in range(300):
        N, M, F, B, tf, tb = _assumption_case(rng)
        g = dag.dag_for(N, M, 1)
        assert dag.longest_path(g, F, B, tf, tb) == _kxyw_max(N, M, F, B, tf + [0], tb + [0])


def test_eager_planted_order_mistakes_fail_the_theorem():
    """Reading the warm-up as 2(N-i) forwards, or the steady groups as
    (forward, backward), breaks the equality with C(K(x, y, w))."""
    def wrong_warmup(S, M, s):
        w = min(2 * (S - s), M)
        o = [("F", m) for m in range(1, w + 1)]
        for k in range(1, M - w + 1):
            o += [("B", k), ("F", w + k)]
        return o + [("B", m) for m in range(M - w + 1, M + 1)]

    def wrong_group(S, M, s):
        w = min(2 * (S - s) + 1, M)
        o = [("F", m) for m in range(1, w + 1)]
        for k in range(1, M - w + 1):
            o += [("F", w + k), ("B", k)]
        return o + [("B", m) for m in range(M - w + 1, M + 1)]

    rng = np.random.default_rng(22)
    for mutant in (wrong_warmup, wrong_group, dag.one_f_one_b_order):
        caught = False
        for _ in range(200):
            N, M, F, B, tf, tb = _assumption_case(rng)
            try:
                g = dag.build_dag(N, M, order=mutant)
            except ValueError:
                caught = True
                break
            if dag.longest_path(g, F, B, tf, tb) != _kxyw_max(N, M, F, B, tf + [0], tb + [0]):
                caught = True
                break
        assert caught, mutant.__name__


def test_eager_event_simulation_and_c_oracle():
    rng = np.random.default_rng(23)
    for _ in range(150):
        S, M = int(rng.integers(1, 7)), int(rng.integers(1, 12))
        F, B, cf, cb = _rand_case(rng, S, M)
        assert des.simulate_1f1b(S, M, F, B, cf, cb, dag.eager_1f1b_order) == \
            dag.longest_path(dag.dag_for(S, M, 1), F, B, cf, cb)
    for trial in range(10):
        S = int(rng.integers(1, 6))
        L = S + int(rng.integers(0, 6))
        M = int(rng.integers(1, 14))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=30, cap=int(rng.integers(30, 150)))
        prob.schedule = 1
        if trial % 2:
            prob.allreduce = rng.integers(0, 500, size=(2, L)).astype(np.uint32)
        full = W.Candidates(first=0, count=prob.n_candidates)
        Tp, fp = dag.evaluate(prob, full)
        Tc, fc = coracle.evaluate(prob, full, nthreads=2)
        assert (Tp == Tc).all() and (fp == fc).all()
        ex = dag.argmin(Tp, fp)
        if ex is not None:
            bound = int(Tp[fp].max())
            best = dag.bounded_search(prob, full, bound, 9)
            assert best[0] == ex
            assert coracle.bounded(prob, full, bound, 9, nthreads=2) == best


def test_eager_same_uniform_closed_form_and_dag_shape():
    """Eager 1F1B has the same nodes and edge counts (Sec. 4.1.2) and, with
    uniform stages and no transfer time, the same (M+S-1)(f+b)."""
    for S in range(1, 6):
        for M in range(1, 10):
            c = dag.dag_for(S, M, 1).counts()
            assert c["compute_nodes"] == 2 * S * M and c["intra"] == S * (2 * M - 1)
            assert dag.longest_path(dag.dag_for(S, M, 1), [3] * S, [5] * S, [0] * (S - 1), [0] * (S - 1)) == \
                (M + S - 1) * 8


def test_eq2_lower_bound_holds_under_eager():
    """Eq. 2 only uses that a stage runs its 2M nodes one after another, so it
    bounds the Eager 1F1B critical path too (with and without R_s)."""
    rng = np.random.default_rng(24)
    for trial in range(300):
        S, M = int(rng.integers(1, 7)), int(rng.integers(1, 12))
        F, B, cf, cb = _rand_case(rng, S, M)
        d = list(rng.integers(0, 500, S)) if trial % 2 else None
        T = dag.longest_path(dag.dag_for(S, M, 1), F, B, cf, cb, d)
        assert dag.eq2_bound(list(F), list(B), M, d) <= T


# ------------------------------------------------------- Interleaved 1F1B

def test_interleaved_dag_counts_match_sec_4_1_4():
    """Sec. 4.1.4: 2VNM compute nodes, 2(NV-1)M inter-stage edges and
    N(2VM-1) intra-stage edges."""
    for N in range(2, 6):
        for V in range(2, 5):
            for M in (N, 2 * N, 3 * N):
                c = dag.dag_for(N * V, M, 2, V).counts()
                assert c["compute_nodes"] == 2 * V * N * M
                assert c["fwd"] + c["bwd"] == 2 * (N * V - 1) * M
                assert c["intra"] == N * (2 * V * M - 1)
                assert c["allreduce_nodes"] == N


def test_interleaved_uniform_closed_form():
    """Equal chunks, no transfer time: T = (VM + N - 1)(f + b), the
    interleaved pipeline's bubble of N - 1 chunk slots."""
    for N in range(2, 6):
        for V in range(2, 5):
            for M in (N, 2 * N, 4 * N):
                S = N * V
                T = dag.longest_path(dag.dag_for(S, M, 2, V), [3] * S, [5] * S, [0] * (S - 1), [0] * (S - 1))
                assert T == (V * M + N - 1) * 8


def test_interleaved_orders_are_device_permutations():
    for N in range(2, 5):
        for V in range(2, 4):
            for M in (N, 2 * N):
                seen = set()
                for p in range(1, N + 1):
                    o = dag.interleaved_order(N, V, M, p)
                    assert len(o) == len(set(o)) == 2 * V * M
                    assert all((j - 1) % N == p - 1 for _, j, _ in o)
                    pos = {x: i for i, x in enumerate(o)}
                    assert all(pos[("F", j, m)] < pos[("B", j, m)] for _, j, m in o)
                    seen |= set(o)
                assert len(seen) == 2 * N * V * M


def test_interleaved_event_simulation_and_c_oracle():
    """The DAG's T equals an event-driven run of the device task lists
    (with per-device all-reduce); the C oracle equals the Python one."""
    rng = np.random.default_rng(40)
    for trial in range(150):
        N, V = int(rng.integers(2, 5)), int(rng.integers(2, 4))
        M, S = N * int(rng.integers(1, 4)), N * V
        F, B, cf, cb = (list(rng.integers(1, 100, S)), list(rng.integers(1, 200, S)),
                        list(rng.integers(0, 50, S - 1)), list(rng.integers(0, 50, S - 1)))
        d = list(rng.integers(0, 300, N)) if trial % 2 else None
        tasks = {p: dag.interleaved_order(N, V, M, p) for p in range(1, N + 1)}
        assert des.simulate_devices(S, N, M, F, B, cf, cb, tasks, d) == \
            dag.longest_path(dag.dag_for(S, M, 2, V), F, B, cf, cb, d)
    for trial in range(12):
        N, V = int(rng.integers(2, 5)), int(rng.integers(2, 4))
        S, M = N * V, N * int(rng.integers(1, 3))
        T = int(rng.integers(1, 3))
        L = S + int(rng.integers(0, 5))
        prob = W.random_problem(rng, L, S, M, T, mem_hi=30, cap=int(rng.integers(60, 300)))
        prob.schedule, prob.V = 2, V
        if trial % 3 == 0:
            prob.assign = rng.integers(0, T, size=(5, N)).astype(np.uint8)
        if trial % 2:
            prob.allreduce = rng.integers(0, 400, size=(T, L)).astype(np.uint32)
        cands = W.random_candidates(rng, prob, 150)
        Tp, fp = dag.evaluate(prob, cands)
        Tc, fc = coracle.evaluate(prob, cands, nthreads=2)
        assert (Tp == Tc).all() and (fp == fc).all()


def test_interleaved_weights_per_device():
    """Virtual stage j runs on device (j-1) mod N; a device's memory and
    all-reduce weight sum over all its chunks (powers of two spell out which
    layers were summed)."""
    L, N, V = 6, 2, 3
    prob = W.random_problem(np.random.default_rng(41), L, N * V, N, 2)
    prob.schedule, prob.V = 2, V
    prob.fwd = np.array([[1 << k for k in range(L)], [1 << (k + 8) for k in range(L)]], dtype=np.uint32)
    prob.bwd = 2 * prob.fwd
    prob.mem = np.array([1 << k for k in range(L)], dtype=np.uint32)
    prob.cap = np.array([0b010101, 0b101010], dtype=np.uint32)
    ar = np.array([[1 << k for k in range(L)], [1 << (k + 8) for k in range(L)]], dtype=np.uint32)
    F, B, mem, d, ok = dag.interleaved_weights(prob, (1, 2, 3, 4, 5), (0, 1), ar)
    assert F == [1, 2 << 8, 4, 8 << 8, 16, 32 << 8] and B == [2 * x for x in F]
    assert mem == [0b010101, 0b101010] and d == [0b010101, 0b101010 << 8] and ok


# ---------------------------- Interleaved 1F1B warm-up: the fill property

def _python_finish_arrays(S, M, schedule, V, F, B):
    T, fin = dag.longest_path(dag.dag_for(S, M, schedule, V), F, B, [0] * (S - 1), [0] * (S - 1),
                              return_finish=True)
    fF = np.array([[fin[("F", s, m)] for m in range(1, M + 1)] for s in range(1, S + 1)])
    fB = np.array([[fin[("B", s, m)] for m in range(1, M + 1)] for s in range(1, S + 1)])
    return T, fF, fB


def _fill_violations(fin_F, fin_B, N, V, M):
    """Devices (0-based) that break the interleaved warm-up's defining
    property under unit node weights and no transfer time.

    Every node then takes one time unit and a device runs one node at a
    time, so the finish times of a device's nodes, sorted, are its order.
    The warm-up of the interleaved schedule (Narayanan et al., the paper's
    reference for it) is sized so that the device stays busy until its
    first backward can start and starts that backward the moment its input
    exists.  The earliest finish of B on virtual stage j (1-based) is the
    chain F_{1,1} .. F_{S,1}, B_{S,1} .. B_{j,1}: S + (S - j + 1) nodes.
    So: (a) the device's nodes up to its first backward finish at
    consecutive times, and (b) that backward finishes at 2S - j + 1.
    A warm-up one forward shorter leaves an idle unit before the first
    backward (a fails); one forward longer delays it (b fails)."""
    S = N * V
    bad = []
    for q in range(N):
        stages = [j for j in range(S) if j % N == q]
        tb, jb = min((int(fin_B[j, m]), j) for j in stages for m in range(M))
        times = sorted(int(fin_F[j, m]) for j in stages for m in range(M))
        times = sorted(times + [int(fin_B[j, m]) for j in stages for m in range(M)])
        upto = [t for t in times if t <= tb]
        if upto != list(range(upto[0], upto[0] + len(upto))) or tb != 2 * S - (jb + 1) + 1:
            bad.append(q)
    return bad


_FILL_CASES = [(N, V, M) for N in range(2, 7) for V in range(2, 5) if N * V <= 18 for M in (2 * N, 3 * N)]


def test_interleaved_warmup_fills_until_the_first_backward():
    """Python and C oracles: with M >= 2N micro-batches every device of the
    Interleaved 1F1B DAG satisfies the fill property (see
    _fill_violations).  Both oracles' warm-up lengths are pinned by it;
    the closed form (VM + N - 1)(f + b) does not separate a warm-up one
    step shorter or longer."""
    for N, V, M in _FILL_CASES:
        S = N * V
        _, fF, fB = _python_finish_arrays(S, M, 2, V, [1] * S, [1] * S)
        assert _fill_violations(fF, fB, N, V, M) == [], (N, V, M)
        _, cF, cB = coracle.finish_times(S, M, [1] * S, [1] * S, [0] * (S - 1), [0] * (S - 1), schedule=2, V=V)
        assert _fill_violations(cF, cB, N, V, M) == [], (N, V, M)
        assert (cF == fF).all() and (cB == fB).all()


def test_interleaved_one_group_runs_every_forward_first():
    """M = N micro-batches (one group): each device runs all V M forwards
    before any backward, the special case of the interleaved schedule's
    reference implementation (Megatron-LM), where no warm-up can fill the
    time of the first device.  Checked on the C oracle's finish times with
    unit weights; this case is structural, no closed form separates it."""
    for N in range(2, 7):
        for V in range(2, 4):
            S = N * V
            _, cF, cB = coracle.finish_times(S, N, [1] * S, [1] * S, [0] * (S - 1), [0] * (S - 1), schedule=2, V=V)
            for q in range(N):
                st = [j for j in range(S) if j % N == q]
                assert max(int(cF[j].max()) for j in st) < min(int(cB[j].min()) for j in st)


def _shifted_interleaved_order(delta):
    def order(N, V, M, p):
        q, total = p - 1, V * M
        w = total if M == N else max(0, min(2 * (N - q - 1) + (V - 1) * N + delta, total))
        mb = lambda k: (k // (N * V)) * N + k % N + 1                                    # noqa: E731
        fwd = lambda k: ("F", ((k % (N * V)) // N) * N + q + 1, mb(k))                     # noqa: E731
        bwd = lambda k: ("B", (V - 1 - (k % (N * V)) // N) * N + q + 1, mb(k))             # noqa: E731
        o = [fwd(k) for k in range(w)]
        for i in range(total - w):
            o += [fwd(w + i), bwd(i)]
        return o + [bwd(k) for k in range(total - w, total)]
    return order


@pytest.mark.parametrize("delta", [-1, 1])
def test_planted_interleaved_warmup_mistakes_fail_the_fill_pin(delta, monkeypatch, tmp_path):
    """A warm-up one forward shorter or longer, planted in the Python oracle
    and in a copy of the C oracle, fails the fill property on every case."""
    import ctypes
    import subprocess

    monkeypatch.setattr(dag, "interleaved_order", _shifted_interleaved_order(delta))
    monkeypatch.setattr(dag, "_DAG_CACHE", {})
    src = open(coracle.SRC).read()
    expr = "2 * (N - q - 1) + (V - 1) * N"
    assert src.count(expr) == 2
    mutated = src.replace(expr, f"(2 * (N - q - 1) + (V - 1) * N + ({delta}))")
    (tmp_path / "oracle.c").write_text(mutated)
    so = tmp_path / "libmut.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-shared", "-fPIC", "-pthread", str(tmp_path / "oracle.c"),
                    "-o", str(so)], check=True)
    mut = ctypes.CDLL(str(so))
    mut.oc_finish_times.restype = ctypes.c_int64
    mut.oc_finish_times.argtypes = [ctypes.c_int] * 4 + [ctypes.c_void_p] * 7
    for N, V, M in _FILL_CASES:
        S = N * V
        _, fF, fB = _python_finish_arrays(S, M, 2, V, [1] * S, [1] * S)
        assert _fill_violations(fF, fB, N, V, M), ("python", N, V, M)
        one = np.ones(S, dtype=np.uint64)
        zero = np.zeros(max(S - 1, 1), dtype=np.uint32)
        cF = np.zeros((S, M), dtype=np.uint64)
        cB = np.zeros((S, M), dtype=np.uint64)
        assert mut.oc_finish_times(S, M, 2, V, one.ctypes.data, one.ctypes.data, None, zero.ctypes.data,
                                   zero.ctypes.data, cF.ctypes.data, cB.ctypes.data) > 0
        assert _fill_violations(cF, cB, N, V, M), ("C", N, V, M)


# ------------------------------------------ Eq. 2's all-reduce term d_i

def test_eq2_is_exact_for_one_stage_with_allreduce():
    """S = 1: the stage runs its 2M nodes back to back and then its
    all-reduce node, so T = M (f_1 + b_1) + d_1, which is exactly g(S_1) of
    Eq. 2.  Python: eq2_bound equals that value and the DAG's T.  C: the
    early-stop pass prunes the candidate at bound T - 1 and keeps it at T,
    which fails if d_1 were dropped from either side (d_1 >= 1 here)."""
    rng = np.random.default_rng(44)
    for trial in range(40):
        L, M, T = int(rng.integers(1, 6)), int(rng.integers(1, 20)), int(rng.integers(1, 4))
        prob = W.random_problem(rng, L, 1, M, T, mem_hi=5, cap=1000)
        prob.allreduce = rng.integers(1, 5000, size=(T, L)).astype(np.uint32)
        for t in range(T):
            f, b, d = int(prob.fwd[t].sum()), int(prob.bwd[t].sum()), int(prob.allreduce[t].sum())
            exact = M * (f + b) + d
            assert dag.eq2_bound([f], [b], M, [d]) == exact
            assert dag.longest_path(dag.dag_for(1, M), [f], [b], [], [], [d]) == exact
            cands = W.Candidates(first=t, count=1)
            assert coracle.bounded(prob, cands, exact - 1)[1:3] == (0, 1)
            best, ev, pr, _ = coracle.bounded(prob, cands, exact)
            assert (ev, pr) == (1, 0) and best == (0, exact)


def test_eq2_is_exact_when_the_last_stage_dominates():
    """S = 2 with a weightless first stage and no transfer time: stage 2
    runs alone, so T = M (f_2 + b_2) + max(d_1, d_2) (B_{1,M} ends with
    B_{2,M}); Eq. 2's g(S_2) = M (f_2 + b_2) + max(b_1 + d_1, d_2) equals it."""
    rng = np.random.default_rng(45)
    for _ in range(60):
        M = int(rng.integers(1, 12))
        f2, b2 = int(rng.integers(1, 500)), int(rng.integers(1, 500))
        d = [int(rng.integers(0, 3000)), int(rng.integers(0, 3000))]
        exact = M * (f2 + b2) + max(d)
        assert dag.longest_path(dag.dag_for(2, M), [0, f2], [0, b2], [0], [0], d) == exact
        assert dag.eq2_bound([0, f2], [0, b2], M, d) == exact
        assert coracle.finish_times(2, M, [0, f2], [0, b2], [0], [0], d=d)[0] == exact
