"""Pins of the pruned-search oracle (Sec. 4.2, Theorems 1 and 2) on the CPU.

The search oracle (oracle/search.py, and its C twin in oracle/oracle.c) is
checked against brute force over every candidate, against the counts of
compositions, and against the paper's layer-level guarantee (Theorem 2) in
the setting it is proved for, where plausible wrong readings of "ridge-like"
lose the optimum.
"""
import itertools
import math

import numpy as np
import pytest

from oracle import coracle, dag
from oracle import search as SR
from paper_2609_06086_amd import workloads as W


def test_rank_composition_inverts_unrank_and_follows_itertools():
    for L in range(1, 11):
        for S in range(1, L + 1):
            for r, cuts in enumerate(itertools.combinations(range(1, L), S - 1)):
                assert SR.rank_composition(L, S, cuts) == r
                assert dag.unrank_composition(L, S, r) == cuts


def _no_valley(seq):
    """Independent form of 'first rises, then falls': no i < j < k with
    seq[i] > seq[j] < seq[k]."""
    n = len(seq)
    return not any(seq[i] > seq[j] < seq[k] for i in range(n) for j in range(i + 1, n) for k in range(j + 1, n))


def test_ridge_like_matches_the_no_valley_definition():
    for n in range(0, 7):
        for seq in itertools.product(range(1, 5), repeat=n):
            assert SR.ridge_like(seq) == _no_valley(seq), seq
    assert SR.ridge_like([1, 2, 2, 5, 3, 3, 1]) and not SR.ridge_like([3, 1, 2])


def _prefix_count(L, S):
    """Partial configurations of one row with no pruning: stage x < S can end
    at c_x <= L - (S - x), giving C(L - S + x, x) prefixes; C(L-1, S-1) leaves."""
    return sum(math.comb(L - S + x, x) for x in range(1, S)) + math.comb(L - 1, S - 1)


def test_unpruned_search_visits_every_prefix_and_finds_the_exhaustive_best():
    rng = np.random.default_rng(30)
    for _ in range(20):
        S = int(rng.integers(1, 5))
        L = S + int(rng.integers(0, 7))
        M = int(rng.integers(1, 6))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=5, cap=10 ** 6)
        res = SR.stage_search(prob, 2 ** 31, stage_pruning=False)
        assert res["visited"] == prob.A * _prefix_count(L, S)
        assert res["evaluated"] == prob.A * math.comb(L - 1, S - 1)
        assert res["pruned_memory"] == res["pruned_ridge"] == res["pruned_bound"] == 0
        # the winner is the first (row, rank) among the smallest makespans
        best = None
        T, f = dag.evaluate(prob, W.Candidates(first=0, count=prob.n_candidates))
        for a in range(prob.A):
            for r in range(math.comb(L - 1, S - 1)):
                t = int(T[r * prob.A + a])
                if best is None or t < best[0]:
                    best = (t, r * prob.A + a)
        assert res["best"] == (best[1], best[0])


def test_theorem1_stage_pruning_keeps_the_optimum():
    """Theorem 1: pruning prefixes with g(S_x) > T_min never loses the best."""
    rng = np.random.default_rng(31)
    for trial in range(40):
        S = int(rng.integers(1, 6))
        L = S + int(rng.integers(0, 7))
        M = int(rng.integers(1, 9))
        T = int(rng.integers(1, 3))
        prob = W.random_problem(rng, L, S, M, T, mem_hi=30, cap=int(rng.integers(30, 150)))
        prob.schedule = trial % 2
        if trial % 3 == 0:
            prob.allreduce = rng.integers(0, 400, size=(T, L)).astype(np.uint32)
        ex = SR.exhaustive_best(prob)
        for rpc in (0, 1, 2):
            res = SR.stage_search(prob, 2 ** 31, rows_per_chunk=rpc)
            assert res["best"] == ex
            if ex is not None:
                assert SR.stage_search(prob, ex[1], rows_per_chunk=rpc)["best"] == ex
                assert SR.stage_search(prob, ex[1] - 1, rows_per_chunk=rpc)["best"] is None
                assert res["visited"] <= SR.stage_search(prob, 2 ** 31, stage_pruning=False)["visited"]


def test_ridge_filter_is_the_exhaustive_best_over_ridge_like_candidates():
    rng = np.random.default_rng(32)
    for trial in range(30):
        S = int(rng.integers(2, 6))
        L = S + int(rng.integers(1, 7))
        M = int(rng.integers(1, 8))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=30, cap=int(rng.integers(40, 150)))
        best = None
        for a in range(prob.A):
            types = dag.assignment_row(prob, a)
            for r, cuts in enumerate(itertools.combinations(range(1, L), S - 1)):
                cnt = SR.layer_counts(L, cuts)
                if not all(_no_valley([cnt[s] for s in range(S) if types[s] == t]) for t in range(2)):
                    continue
                F, B, _, _, ok = dag.stage_weights(prob, cuts, types)
                if ok:
                    t = dag.longest_path(dag.dag_for(S, M), F, B, prob.comm_fwd, prob.comm_bwd)
                    if best is None or t < best[0]:
                        best = (t, r * prob.A + a)
        res = SR.stage_search(prob, 2 ** 31, ridge=True)
        assert res["best"] == (None if best is None else (best[1], best[0]))


def _theorem2_case(rng):
    """Theorem 2's setting: Eager 1F1B; identical layers per type with
    b = r f (Assumption 1, r = 2); transfers <= (r-1)/2 of a layer's forward
    time (Assumption 2); M >= 2S (Assumption 3); memory limits that grow
    along the pipeline (Lemma on memory limits), here from layers whose
    footprint falls with depth."""
    S = int(rng.integers(3, 6))
    L = S + int(rng.integers(3, 9))
    M = 2 * S + int(rng.integers(0, 3))
    f = [int(rng.integers(10, 40)) for _ in range(2)]
    prob = W.random_problem(rng, L, S, M, 2)
    prob.fwd = np.array([[f[t]] * L for t in range(2)], dtype=np.uint32)
    prob.bwd = 2 * prob.fwd
    c = [int(rng.integers(0, max(1, min(f) // 2))) for _ in range(S - 1)]
    prob.comm_fwd = np.array(c, dtype=np.uint32)
    prob.comm_bwd = np.array(c, dtype=np.uint32)
    prob.mem = np.array([round(100 * (1 + 2 * (L - 1 - k) / (L - 1))) for k in range(L)], dtype=np.uint32)
    prob.cap = np.array([int(rng.integers(250, 700))] * 2, dtype=np.uint32)
    prob.schedule = 1
    return prob


def test_theorem2_ridge_like_optimum_exists_and_wrong_readings_lose_it():
    """Under Theorem 2's assumptions the ridge-filtered search finds the
    exhaustive optimum.  Reading "ridge-like" as non-increasing only, or as
    falling-then-rising, loses it in some of these cases."""
    rng = np.random.default_rng(33)
    wrong = {"non-increasing": lambda q: all(q[i] >= q[i + 1] for i in range(len(q) - 1)),
             "valley": lambda q: SR.ridge_like([-x for x in q])}
    lost = {k: 0 for k in wrong}
    checked = 0
    while checked < 25:
        prob = _theorem2_case(rng)
        ex = SR.exhaustive_best(prob)
        if ex is None:
            continue
        checked += 1
        res = SR.stage_search(prob, 2 ** 31, ridge=True)
        assert res["best"] is not None and res["best"][1] == ex[1]
        S, L = prob.S, prob.L
        for name, pred in wrong.items():
            best = None
            for a in range(prob.A):
                types = dag.assignment_row(prob, a)
                for cuts in itertools.combinations(range(1, L), S - 1):
                    cnt = SR.layer_counts(L, cuts)
                    if not all(pred([cnt[s] for s in range(S) if types[s] == t]) for t in range(2)):
                        continue
                    F, B, _, _, ok = dag.stage_weights(prob, cuts, types)
                    if ok:
                        t = dag.longest_path(dag.dag_for(S, prob.M, 1), F, B, prob.comm_fwd, prob.comm_bwd)
                        best = t if best is None else min(best, t)
            lost[name] += best != ex[1]
    assert all(v > 0 for v in lost.values()), lost


def test_c_search_equals_python_search():
    rng = np.random.default_rng(34)
    for trial in range(25):
        S = int(rng.integers(1, 6))
        L = S + int(rng.integers(0, 8))
        M = int(rng.integers(1, 9))
        T = int(rng.integers(1, 4))
        prob = W.random_problem(rng, L, S, M, T, mem_hi=30, cap=int(rng.integers(30, 150)),
                                assign_rows=None if T ** S < 40 else 7)
        prob.schedule = trial % 2
        if trial % 4 == 1:
            prob.allreduce = rng.integers(0, 300, size=(T, L)).astype(np.uint32)
        ex = SR.exhaustive_best(prob)
        bound = 2 ** 31 if ex is None or trial % 2 else ex[1] + int(rng.integers(0, 50))
        for rpc in (0, 1, 3):
            for ridge in (False, True):
                a = SR.stage_search(prob, bound, rows_per_chunk=rpc, ridge=ridge)
                b = coracle.search(prob, bound, rows_per_chunk=rpc, ridge=ridge, nthreads=3)
                assert a == b


def test_ramp_chunks_cover_the_rows_once_in_doubling_sizes():
    for n in (0, 1, 2, 7, 64, 100):
        for rpc in (1, 3, 8, 1000):
            b = SR.chunk_bounds(n, rpc, True)
            assert [c0 for c0, _ in b] == ([0] + [c1 for _, c1 in b][:-1] if n else [])
            assert (b[-1][1] if b else 0) == n
            sizes = [c1 - c0 for c0, c1 in b]
            for k, sz in enumerate(sizes[:-1]):
                assert sz == min(2 ** k, rpc)
            assert SR.chunk_bounds(n, rpc, False) == [(c0, min(n, c0 + rpc)) for c0 in range(0, n, rpc)]


def test_ramp_search_is_the_chain_of_its_chunks():
    """R17 with growing chunks: the search equals one fixed-chunk search per
    chunk, each against min(bound, best of the chunks before), with the
    counters summed and the first strictly better result kept."""
    rng = np.random.default_rng(36)
    for trial in range(12):
        S = int(rng.integers(1, 5))
        L = S + int(rng.integers(0, 7))
        M = int(rng.integers(1, 9))
        T = int(rng.integers(2, 4))
        prob = W.random_problem(rng, L, S, M, T, mem_hi=30, cap=int(rng.integers(30, 150)),
                                assign_rows=13)
        prob.schedule = trial % 2
        bound = 2 ** 31 if trial % 3 == 0 else int(coracle.evaluate(
            prob, W.random_candidates(rng, prob, 30))[0].min())
        for rpc, ridge in ((4, False), (16, True), (0, False)):
            got = SR.stage_search(prob, bound, rows_per_chunk=rpc, ridge=ridge, ramp=True)
            want = dict(visited=0, evaluated=0, pruned_memory=0, pruned_ridge=0, pruned_bound=0)
            best = None
            size, c0 = 1, 0
            cap = rpc if rpc > 0 else prob.A
            while c0 < prob.A:
                n = min(size, cap, prob.A - c0)
                b = bound if best is None else min(bound, best[1])
                r = SR.stage_search(prob, b, first_row=c0, n_rows=n, ridge=ridge)
                for k in want:
                    want[k] += r[k]
                if r["best"] is not None and (best is None or r["best"][1] < best[1]):
                    best = r["best"]
                c0 += n
                size *= 2
            want["best"] = best
            assert got == want
            assert coracle.search(prob, bound, rows_per_chunk=rpc, ridge=ridge, ramp=True, nthreads=3) == got


def test_evaluated_candidates_are_those_within_eq2_of_the_bound():
    """With a fixed bound (one chunk) the search evaluates exactly the
    feasible candidates whose Eq. 2 bound max_x g(S_x) is <= b: every prefix
    test is g(S_x) <= b, and the candidate's own Eq. 2 bound is their max."""
    rng = np.random.default_rng(35)
    for trial in range(25):
        S = int(rng.integers(1, 6))
        L = S + int(rng.integers(0, 7))
        M = int(rng.integers(1, 9))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=30, cap=int(rng.integers(30, 150)))
        if trial % 2:
            prob.allreduce = rng.integers(0, 400, size=(2, L)).astype(np.uint32)
        ex = SR.exhaustive_best(prob)
        if ex is None:
            continue
        b = ex[1] + int(rng.integers(0, 3000))
        want = 0
        for a in range(prob.A):
            types = dag.assignment_row(prob, a)
            for cuts in itertools.combinations(range(1, L), S - 1):
                F, B, _, D, ok = dag.stage_weights(prob, cuts, types, prob.allreduce)
                want += ok and dag.eq2_bound(F, B, M, D if prob.allreduce is not None else None) <= b
        assert SR.stage_search(prob, b)["evaluated"] == want
