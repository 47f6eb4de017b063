"""The allocation-free evaluation entry point against the allocating one.

poseidon_eval_candidates_noalloc runs the same kernels on the library's
fixed per-GPU scratch, in chunks sized to it.  Its makespans, feasibility
bits and argmin must equal poseidon_eval_candidates' bit for bit, on two
calls in a row (the second with a smaller input, so the scratch holds the
first call's leftovers), for every schedule, range and list mode, the
slot-table path and calls much longer than one scratch chunk.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2609_06086_amd import poseidon as P  # noqa: E402
from paper_2609_06086_amd import workloads as W  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def _args(cands, dev, lo, hi):
    if not cands.is_list:
        return dict(first=cands.first + lo, count=hi - lo)
    d = dict(comp_rank=torch.from_numpy(cands.comp_rank[lo:hi].view(np.int64)).to(dev))
    if cands.assign_idx is not None:
        d["assign_idx"] = torch.from_numpy(cands.assign_idx[lo:hi].view(np.int32)).to(dev)
    return d


def _run(fn, ctx, args, n, dev):
    T = torch.full((max(n, 1),), -7, dtype=torch.int32, device=dev)
    bits = torch.full((max((n + 31) // 32, 1),), -7, dtype=torch.int32, device=dev)
    best = fn(ctx, makespan_out=T, feasible_bits_out=bits, **args)
    return T.cpu().numpy()[:n], bits.cpu().numpy()[:(n + 31) // 32], (best.index, best.makespan, best.status)


def _compare(prob, cands, dev, spans):
    """Calls of the given [lo, hi) spans in a row, each through both entry
    points on one context; every output must agree exactly."""
    ctx = P.poseidon_load_costs(prob, 0)
    for lo, hi in spans:
        a = _args(cands, dev, lo, hi)
        T0, b0, r0 = _run(P.poseidon_eval_candidates, ctx, a, hi - lo, dev)
        T1, b1, r1 = _run(P.poseidon_eval_candidates_noalloc, ctx, a, hi - lo, dev)
        assert np.array_equal(T0, T1), f"makespans differ at {np.nonzero(T0 != T1)[0][:10]} (span {lo}, {hi})"
        assert np.array_equal(b0, b1), f"feasibility words differ (span {lo}, {hi})"
        assert r0 == r1, (r0, r1)
        assert P.poseidon_last_best(ctx).index == r1[0]
    ctx.close()


def test_noalloc_matches_on_the_16_stage_workload(dev):
    """2^21 + 5 candidates of the 16-stage workload (several scratch chunks,
    a ragged last one), then 300,001 of them."""
    wl = W.workload(5)
    _compare(wl.problem, wl.cands, dev, [(0, (1 << 21) + 5), (1000, 301_001)])


def test_noalloc_matches_with_assignments_and_schedules(dev):
    """The 8-stage, 3-type workload (assignment indices) under 1F1B and Eager
    1F1B, and the 16-stage workload as Interleaved 1F1B on 8 devices."""
    wl = W.workload(4)
    for sched in (P.SCHEDULE_1F1B, P.SCHEDULE_EAGER_1F1B):
        wl.problem.schedule = sched
        _compare(wl.problem, wl.cands, dev, [(0, 1_500_007), (77, 100_077)])
    ilv = W.interleaved_variant(W.workload(5), 2)
    _compare(ilv.problem, ilv.cands, dev, [(0, 900_001), (5, 70_005)])


def test_noalloc_matches_in_range_mode_and_on_the_table_path(dev):
    """Range mode with first > 0 (the joint index) on the 8-stage, 2-type
    exhaustive workload; a short pipeline (M < S, no cascade); an empty call."""
    wl = W.workload(3)
    _compare(wl.problem, wl.cands, dev, [(12_345, 1_212_345), (99, 64_099)])
    rng = np.random.default_rng(160)
    prob = W.random_problem(rng, 20, 12, 5, 2, mem_hi=30, cap=200, assign_rows=4)
    _compare(prob, W.random_candidates(rng, prob, 400_000), dev, [(0, 400_000), (3, 1_003)])
    ctx = P.poseidon_load_costs(wl.problem, 0)
    b = P.poseidon_eval_candidates_noalloc(ctx, first=0, count=0)
    assert b.status == P.POSEIDON_NO_FEASIBLE and b.index is None
    ctx.close()
