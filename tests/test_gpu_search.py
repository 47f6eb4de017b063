"""GPU parity of the pruned configuration search (poseidon_search) against
the C oracle (oracle/oracle.c, oc_search), which is pinned against brute
force and the paper's theorems in tests/test_search_pins.py.

Everything is integer: the best (joint index, makespan) and all five
counters must be identical for the same bound and chunking.
"""
import json
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import coracle  # noqa: E402
from paper_2609_06086_amd import poseidon as P  # noqa: E402
from paper_2609_06086_amd import workloads as W  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def check(prob, bound, dev, **kw):
    ctx = P.poseidon_load_costs(prob, 0)
    b, st = P.poseidon_search(ctx, bound, **kw)
    ctx.close()
    okw = dict(kw)
    ridge = okw.pop("ridge", False)
    sp = okw.pop("stage_pruning", True)
    o = coracle.search(prob, bound, ridge=ridge, stage_pruning=sp, **okw)
    got = (b.index, b.makespan) if b.index is not None else None
    assert got == o["best"], (got, o)
    assert (st.visited, st.evaluated, st.pruned_memory, st.pruned_ridge, st.pruned_bound) == \
        (o["visited"], o["evaluated"], o["pruned_memory"], o["pruned_ridge"], o["pruned_bound"]), (st, o)
    return b, st


def test_search_random_problems(dev):
    rng = np.random.default_rng(120)
    for trial in range(60):
        S = trial % 8 + 1
        L = S + int(rng.integers(0, 12))
        M = int(rng.integers(1, 3 * S + 8))
        T = int(rng.integers(1, 4))
        prob = W.random_problem(rng, L, S, M, T, cost_hi=400, mem_hi=30, cap=int(rng.integers(30, 200)),
                                assign_rows=None if T ** S < 300 else 9)
        prob.schedule = trial % 3 == 1
        if trial % 4 == 2:
            prob.allreduce = rng.integers(0, 2000, size=(T, L)).astype(np.uint32)
        bound = 2 ** 31 - 1 if trial % 5 == 0 else None
        if bound is None:
            To, fo = coracle.evaluate(prob, W.random_candidates(rng, prob, 200))
            bound = int(To[fo].min()) if fo.any() else 2 ** 31 - 1
        for kw in (dict(), dict(rows_per_chunk=1), dict(ridge=True, rows_per_chunk=3),
                   dict(stage_pruning=False), dict(ramp=True, rows_per_chunk=4)):
            check(prob, bound, dev, **kw)


def test_search_monotone_last_stage(dev):
    """Per-layer costs within 30 % of each other across types and M >= 2: every
    type pair satisfies the condition under which the last stage's outcomes
    are counted as ranges (ridge prefix in closed form, Eq. 2 prefix by
    binary search), with ridge on and off, stage pruning on and off, tight
    and loose bounds, 2..8 stages, and M = 1 where only same-type pairs do."""
    rng = np.random.default_rng(124)
    for trial in range(40):
        S = trial % 7 + 2
        L = S + int(rng.integers(1, 14))
        M = 1 if trial % 10 == 9 else int(rng.integers(2, 3 * S + 8))
        T = int(rng.integers(2, 4))
        prob = W.random_problem(rng, L, S, M, T, cost_lo=300, cost_hi=390, mem_hi=30,
                                cap=int(rng.integers(40, 250)), assign_rows=None if T ** S < 300 else 11)
        prob.schedule = trial % 3 == 2
        To, fo = coracle.evaluate(prob, W.random_candidates(rng, prob, 300))
        tight = int(np.sort(To[fo])[min(3, int(fo.sum()) - 1)]) if fo.any() else 2 ** 31 - 1
        for bound, kw in ((tight, dict()), (tight, dict(ridge=True, rows_per_chunk=2)),
                          (2 ** 31 - 1, dict(ridge=True)), (tight, dict(stage_pruning=False, ridge=True))):
            check(prob, bound, dev, **kw)


def test_search_long_models_unfused(dev):
    """L > 129 layers: one block's grandchildren could exceed a frontier piece,
    so the level before the last cut is expanded on its own (the fused
    expansion covers L <= 129 everywhere else)."""
    rng = np.random.default_rng(125)
    for S, rows in ((3, 4), (4, 3), (5, 2)):
        L = 140 + int(rng.integers(0, 20))
        prob = W.random_problem(rng, L, S, 2 * S + 3, 2, cost_lo=200, cost_hi=300, mem_hi=30,
                                cap=int(rng.integers(900, 1600)), assign_rows=rows)
        To, fo = coracle.evaluate(prob, W.random_candidates(rng, prob, 400))
        bound = int(np.sort(To[fo])[2]) if fo.sum() > 2 else 2 ** 31 - 1
        for kw in (dict(), dict(ridge=True, rows_per_chunk=1)):
            check(prob, bound, dev, **kw)


def test_search_deep_pipelines(dev):
    """S = 9..16 stages with few spare layers (every level of the frontier,
    the last-cut test at level S-2, wide composition ranks)."""
    rng = np.random.default_rng(123)
    for S in range(9, 17):
        L = S + int(rng.integers(1, 7))
        M = int(rng.integers(1, 2 * S + 4))
        prob = W.random_problem(rng, L, S, M, 2, cost_hi=300, mem_hi=30, cap=int(rng.integers(60, 200)),
                                assign_rows=int(rng.integers(1, 6)))
        prob.schedule = S % 2
        for kw in (dict(), dict(ridge=True, rows_per_chunk=2), dict(ramp=True, rows_per_chunk=2)):
            check(prob, 2 ** 31 - 1, dev, **kw)


def test_search_maximum_layer_and_type_counts(dev):
    """T = 8 with L = 256 (the largest tables: cut values up to 255, LDS stage
    and search tables for 8 types; above the fused-level limit) and with
    L = 120, S = 4 (fused), with and without all-reduce times, the ridge
    filter and growing chunks."""
    rng = np.random.default_rng(124)
    for trial in range(6):
        L, S = (256, 3) if trial < 4 else (120, 4)
        prob = W.random_problem(rng, L, S, 6, 8, cost_lo=50, cost_hi=400, mem_hi=20, cap=int(rng.integers(900, 3000)),
                                assign_rows=5)
        if trial % 2:
            prob.allreduce = rng.integers(0, 3000, size=(8, L)).astype(np.uint32)
        prob.schedule = (trial // 2) % 2
        To, fo = coracle.evaluate(prob, W.random_candidates(rng, prob, 300))
        bound = int(To[fo].min()) if fo.any() else 2 ** 31 - 1
        for kw in (dict(), dict(ridge=True, rows_per_chunk=2), dict(ramp=True, rows_per_chunk=2)):
            check(prob, bound, dev, **kw)


def test_search_row_ranges_and_no_result(dev):
    rng = np.random.default_rng(121)
    prob = W.random_problem(rng, 12, 4, 9, 3, mem_hi=30, cap=90)
    check(prob, 2 ** 31 - 1, dev, first_row=5, n_rows=40, rows_per_chunk=7)
    check(prob, 2 ** 31 - 1, dev, first_row=prob.A - 1, n_rows=1)
    b, st = check(prob, 1, dev)
    assert b.status == P.POSEIDON_NO_FEASIBLE and b.index is None


def test_search_frontier_pieces(dev):
    """Levels wider than one frontier piece (4 Mi nodes): 2000 rows of a
    5-stage, 40-layer problem with no pruning reach 16.9 M partial and
    1.6 x 10^8 complete configurations."""
    rng = np.random.default_rng(122)
    prob = W.random_problem(rng, 40, 5, 2, 2, mem_hi=10, cap=10 ** 6, assign_rows=2000)
    check(prob, 2 ** 31 - 1, dev, stage_pruning=False)


def test_search_workload4_rows(dev):
    """The 8-stage, 3-type workload: 48 assignment rows, bound from its 500
    warm-up samples, chunks of 16 rows, with and without the ridge filter, and
    in chunks growing from one row to 16."""
    wl = W.workload(4)
    c = wl.cands
    To, fo = coracle.evaluate(wl.problem, W.Candidates(comp_rank=c.comp_rank[:500].copy(),
                                                       assign_idx=c.assign_idx[:500].copy()))
    bound = int(To[fo].min())
    check(wl.problem, bound, dev, first_row=0, n_rows=48, rows_per_chunk=16)
    check(wl.problem, bound, dev, first_row=3000, n_rows=48, rows_per_chunk=16, ridge=True)
    check(wl.problem, bound, dev, first_row=100, n_rows=40, rows_per_chunk=16, ramp=True)


def test_search_workload6_eager_rows(dev):
    """All-reduce nodes and Eager 1F1B in the leaves' DAG."""
    wl = W.workload(6)
    prob = wl.problem
    prob.schedule = P.SCHEDULE_EAGER_1F1B
    c = wl.cands
    To, fo = coracle.evaluate(prob, W.Candidates(comp_rank=c.comp_rank[:500].copy(),
                                                 assign_idx=c.assign_idx[:500].copy()))
    check(prob, int(To[fo].min()), dev, first_row=100, n_rows=24, rows_per_chunk=8, ridge=True)


def test_search_workload4_full_golden(dev):
    """The whole 8-stage, 3-type search as the benchmark runs it (all 6561
    rows x C(79,7) compositions, warm-up bound, chunks growing to 512 rows),
    without and with the ridge filter, against the oracle's result and
    counters stored by tests/golden/make_golden.py."""
    gold = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "full_workloads.json")))["cfg4_search"]
    wl = W.workload(4)
    c = wl.cands
    To, fo = coracle.evaluate(wl.problem, W.Candidates(comp_rank=c.comp_rank[:gold["warmup"]].copy(),
                                                       assign_idx=c.assign_idx[:gold["warmup"]].copy()))
    assert int(To[fo].min()) == gold["bound"]
    ctx = P.poseidon_load_costs(wl.problem, 0)
    try:
        for name, ridge in (("plain", False), ("ridge", True)):
            b, st = P.poseidon_search(ctx, gold["bound"], rows_per_chunk=gold["rows_per_chunk"], ridge=ridge,
                                      ramp=gold["ramp"])
            g = gold[name]
            assert (b.index, b.makespan) == (g["best_index"], g["best_makespan"])
            assert (st.visited, st.evaluated, st.pruned_memory, st.pruned_ridge, st.pruned_bound) == \
                (g["visited"], g["evaluated"], g["pruned_memory"], g["pruned_ridge"], g["pruned_bound"])
    finally:
        ctx.close()
