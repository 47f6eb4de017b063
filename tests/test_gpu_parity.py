"""GPU parity: the HIP path through the C-ABI against the CPU oracle.

Makespans, feasibility bits and the argmin must be bit-identical (all
arithmetic is exact integer arithmetic).  Small and mid-size cases compare
every output with the oracle; the full-size workloads compare SHA-256
digests of the full output arrays and the argmin with values the committed
script tests/golden/make_golden.py wrote from the oracle.
"""
import hashlib
import itertools
import json
import math
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import coracle, dag  # noqa: E402
from paper_2609_06086_amd import poseidon as P  # noqa: E402
from paper_2609_06086_amd import workloads as W  # noqa: E402

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden", "full_workloads.json")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def unpack_bits(words: np.ndarray, n: int) -> np.ndarray:
    """Feasibility of candidate i = bit i % 32 of uint32 word i / 32."""
    return np.unpackbits(words.astype("<u4").view(np.uint8), bitorder="little")[:n].astype(bool)


def pack_bits(f: np.ndarray) -> np.ndarray:
    """Bit i % 32 of uint32 word i / 32, as the library writes them."""
    pad = (-len(f)) % 32
    return np.packbits(np.concatenate([f.astype(bool), np.zeros(pad, bool)]), bitorder="little").view("<u4")


def to_dev(cands, dev):
    if not cands.is_list:
        return dict(first=cands.first, count=cands.count)
    d = dict(comp_rank=torch.from_numpy(cands.comp_rank.view(np.int64)).to(dev))
    if cands.assign_idx is not None:
        d["assign_idx"] = torch.from_numpy(cands.assign_idx.view(np.int32)).to(dev)
    return d


def gpu_eval(ctx, cands, dev, n=None):
    n = len(cands) if n is None else n
    T = torch.full((max(n, 1),), -1, dtype=torch.int32, device=dev)
    bits = torch.full((max((n + 31) // 32, 1),), -1, dtype=torch.int32, device=dev)
    best = P.poseidon_eval_candidates(ctx, makespan_out=T, feasible_bits_out=bits, **to_dev(cands, dev))
    Tg = T.cpu().numpy().view(np.uint32)[:n]
    fg = unpack_bits(bits.cpu().numpy().view(np.uint32), n)
    return Tg, fg, best


def check_against_oracle(prob, cands, dev, python_oracle=False):
    ctx = P.poseidon_load_costs(prob, 0)
    Tg, fg, best = gpu_eval(ctx, cands, dev)
    if python_oracle:
        To, fo = dag.evaluate(prob, cands)
        To = To.astype(np.uint32)
    else:
        To, fo = coracle.evaluate(prob, cands)
    assert np.array_equal(Tg, To), f"makespans differ at {np.nonzero(Tg != To)[0][:10]}"
    assert np.array_equal(fg, fo), "feasibility differs"
    ob = coracle.argmin(To, fo)
    if ob is None:
        assert best.status == P.POSEIDON_NO_FEASIBLE and best.index is None
    else:
        # range mode reports the joint index first + position, list mode the position
        assert (best.index, best.makespan) == (ob[0] + index_base(cands), ob[1])
    ctx.close()
    return Tg, fg, best


def index_base(cands):
    return 0 if cands.is_list else cands.first


# ------------------------------------------------------------ named workloads

def test_workload1_exhaustive_vs_python_oracle(dev):
    wl = W.workload(1)
    check_against_oracle(wl.problem, wl.cands, dev, python_oracle=True)


def test_workload2_exhaustive(dev):
    wl = W.workload(2)
    check_against_oracle(wl.problem, wl.cands, dev)


def test_workload3_subrange_ragged(dev):
    wl = W.workload(3)
    first, count = 12_345_679, 3_000_001
    check_against_oracle(wl.problem, W.Candidates(first=first, count=count), dev)


def test_workload4_list_prefix(dev):
    wl = W.workload(4)
    n = 1_000_003
    c = W.Candidates(comp_rank=wl.cands.comp_rank[:n].copy(), assign_idx=wl.cands.assign_idx[:n].copy())
    check_against_oracle(wl.problem, c, dev)


def test_workload5_list_prefix(dev):
    wl = W.workload(5)
    n = 300_001
    c = W.Candidates(comp_rank=wl.cands.comp_rank[:n].copy())
    check_against_oracle(wl.problem, c, dev)


# ------------------------------------------------------------- random shapes

def test_every_stage_count_fast_path(dev):
    """S = 1..16 with M >= S (register-stencil path), random tables."""
    rng = np.random.default_rng(100)
    for S in range(1, 17):
        for M in (S, S + 1, S + int(rng.integers(2, 40))):
            L = S + int(rng.integers(0, 12))
            T = int(rng.integers(1, 4))
            prob = W.random_problem(rng, L, S, M, T, cost_hi=500, mem_hi=40, cap=int(rng.integers(40, 200)),
                                    assign_rows=None if T ** S < 5000 else 6)
            cands = W.random_candidates(rng, prob, int(rng.integers(1, 700)))
            check_against_oracle(prob, cands, dev)


def test_list_decode_every_stage_count_and_column_length(dev):
    """List-mode unranking for S = 2..16 at every Pascal column length the
    kernels use (L up to 32, 64, 128 and 256: 5 to 8 levels, so every set of
    bucket tables and search lengths), with 32-bit or 64-bit ranks as the
    composition count requires (below 2^63 here): random ranks plus the first
    two and the last two, every makespan and mask bit against the oracle."""
    rng = np.random.default_rng(153)
    for S in range(2, 17):
        for lo, hi in ((S, 32), (33, 64), (65, 128), (129, 256)):
            Ls = [L for L in range(max(lo, S), hi + 1) if math.comb(L - 1, S - 1) < 2 ** 63]
            if not Ls:
                continue
            L = int(rng.choice(Ls))
            prob = W.random_problem(rng, L, S, S, 2, cost_hi=500, mem_hi=40, cap=10 ** 6, assign_rows=1)
            n_comp = prob.n_compositions
            edge = np.array([0, min(1, n_comp - 1), max(n_comp - 2, 0), n_comp - 1], dtype=np.uint64)
            ranks = np.concatenate([rng.integers(0, n_comp, size=1500, dtype=np.uint64), edge])
            check_against_oracle(prob, W.Candidates(comp_rank=np.ascontiguousarray(ranks)), dev)


def test_short_pipelines_table_path(dev):
    """M < S (slot-table path)."""
    rng = np.random.default_rng(101)
    for _ in range(40):
        S = int(rng.integers(2, 17))
        M = int(rng.integers(1, S))
        L = S + int(rng.integers(0, 10))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=30, cap=int(rng.integers(30, 200)), assign_rows=3)
        check_against_oracle(prob, W.random_candidates(rng, prob, int(rng.integers(1, 400))), dev)


def test_range_mode_with_assignments(dev):
    """Range mode over joint indices r * A + a with A > 1 (digits and table)."""
    rng = np.random.default_rng(102)
    for trial in range(12):
        S = int(rng.integers(1, 6))
        L = S + int(rng.integers(0, 8))
        M = int(rng.integers(1, 20))
        T = int(rng.integers(1, 4))
        prob = W.random_problem(rng, L, S, M, T, mem_hi=30, cap=int(rng.integers(30, 150)),
                                assign_rows=None if trial % 2 else int(rng.integers(1, 6)))
        n = prob.n_candidates
        first = int(rng.integers(0, n))
        count = int(rng.integers(1, n - first + 1))
        check_against_oracle(prob, W.Candidates(first=first, count=count), dev)
        check_against_oracle(prob, W.Candidates(first=0, count=n), dev)


def test_random_problems_python_oracle(dev):
    rng = np.random.default_rng(103)
    for _ in range(10):
        S = int(rng.integers(1, 5))
        L = S + int(rng.integers(0, 5))
        M = int(rng.integers(1, 7))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=30, cap=int(rng.integers(30, 120)))
        check_against_oracle(prob, W.Candidates(first=0, count=prob.n_candidates), dev, python_oracle=True)


def _lex_rank(L, cuts):
    """Lexicographic rank of a sorted cut tuple among all (S-1)-subsets of
    {1..L-1}: the tuples that share the first j-1 cuts and have a smaller
    j-th cut come first."""
    k, r, prev = len(cuts), 0, 0
    for j, c in enumerate(cuts, start=1):
        for v in range(prev + 1, c):
            r += math.comb(L - 1 - v, k - j)
        prev = c
    return r


def test_memory_cap_equality_is_feasible(dev):
    """A stage whose memory equals its type's cap fits; one MB less does not
    (Sec. 3.2; the comparison is inclusive), through the evaluation, the
    early-stop pass and the search.  Every layer takes 100 MB, so a stage of
    n layers takes 100 n MB."""
    rng = np.random.default_rng(115)
    for S, L in ((1, 4), (3, 9), (8, 20), (16, 30)):
        prob = W.random_problem(rng, L, S, 2 * S, 2, cost_hi=300, mem_lo=100, mem_hi=100, assign_rows=1)
        prob.assign = np.zeros((1, S), np.uint8)
        counts = np.array([len(c) for c in np.array_split(np.arange(L), S)])
        cuts = tuple(int(x) for x in np.cumsum(counts)[:-1])
        rank = _lex_rank(L, cuts)
        assert dag.unrank_composition(L, S, rank) == cuts
        cands = W.Candidates(comp_rank=np.array([rank], np.uint64), assign_idx=np.array([0], np.uint32))
        for cap, ok in ((100 * int(counts.max()), True), (100 * int(counts.max()) - 1, False)):
            prob.cap = np.array([cap, cap], np.uint32)
            _, fg, best = check_against_oracle(prob, cands, dev)
            assert bool(fg[0]) == ok and (best.index == 0) == ok
            b, st = bounded_vs_oracle(prob, cands, 2 ** 31 - 1, 0, dev)
            assert (st.evaluated, st.infeasible) == ((1, 0) if ok else (0, 1))
        if S > 1:
            # every composition of the single row, cap equal to the largest stage of the balanced one
            prob.cap = np.array([100 * int(counts.max())] * 2, np.uint32)
            ctx = P.poseidon_load_costs(prob, 0)
            b, st = P.poseidon_search(ctx, 2 ** 31 - 1)
            o = coracle.search(prob, 2 ** 31 - 1)
            ctx.close()
            assert (b.index, b.makespan) == o["best"] and st.pruned_memory == o["pruned_memory"] > 0


def test_duplicates_tie_to_smallest_index(dev):
    wl = W.workload(2)
    rng = np.random.default_rng(104)
    c = W.random_candidates(rng, wl.problem, 5000)
    To, fo = coracle.evaluate(wl.problem, c)
    b = coracle.argmin(To, fo)
    # copy the winner to several later positions and to one earlier position
    for j in (4999, 3000, 17):
        c.comp_rank[j] = c.comp_rank[b[0]]
        c.assign_idx[j] = c.assign_idx[b[0]]
    _, _, best = check_against_oracle(wl.problem, c, dev)
    assert best.index == min(17, b[0])


def test_no_feasible_candidate(dev):
    wl = W.workload(2)
    prob = wl.problem
    prob.cap = np.array([1000, 1000], np.uint32)     # below any stage's memory
    _, fg, best = check_against_oracle(prob, W.Candidates(first=0, count=5000), dev)
    assert not fg.any() and best.status == P.POSEIDON_NO_FEASIBLE


def test_empty_and_single(dev):
    wl = W.workload(2)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    b = P.poseidon_eval_candidates(ctx, first=0, count=0)
    assert b.status == P.POSEIDON_NO_FEASIBLE
    To, fo = coracle.evaluate(wl.problem, W.Candidates(first=71919, count=1))
    T = torch.zeros(1, dtype=torch.int32, device=dev)
    b = P.poseidon_eval_candidates(ctx, first=71919, count=1, makespan_out=T)
    assert int(T.cpu().numpy().view(np.uint32)[0]) == int(To[0])
    assert (b.index, b.makespan) == (71919, int(To[0]))
    ctx.close()


def test_range_mode_reports_the_joint_index(dev):
    """Range mode: best.index is the joint index rank * A + a of the winning
    candidate (not its position in the call), for the evaluation, the
    early-stop pass and poseidon_last_best.  The expected index comes from
    enumerating the candidates in the oracle's own order."""
    rng = np.random.default_rng(150)
    for trial in range(8):
        S = int(rng.integers(2, 5))
        L = S + int(rng.integers(1, 6))
        T = int(rng.integers(2, 4))
        prob = W.random_problem(rng, L, S, int(rng.integers(1, 12)), T, mem_hi=30, cap=int(rng.integers(60, 150)),
                                assign_rows=None if trial % 2 else 5)
        n = prob.n_candidates
        first = int(rng.integers(1, n // 2 + 1))
        count = n - first
        lst = dag.candidate_list(prob, W.Candidates(first=0, count=n))
        To, fo = dag.evaluate(prob, W.Candidates(first=0, count=n))
        win = min((int(To[i]), i) for i in range(first, n) if fo[i]) if fo[first:].any() else None
        ctx = P.poseidon_load_costs(prob, 0)
        b = P.poseidon_eval_candidates(ctx, first=first, count=count)
        lb = P.poseidon_last_best(ctx)
        bb, _ = P.poseidon_eval_candidates_bounded(ctx, 2 ** 31 - 1, chunk=3, first=first, count=count)
        ctx.close()
        if win is None:
            assert b.index is None and bb.index is None
            continue
        t, i = win
        cuts, types = lst[i][1], lst[i][2]
        rank = list(itertools.combinations(range(1, L), S - 1)).index(tuple(cuts))
        a = dag.all_assignments(prob).index(tuple(types))
        assert rank * prob.A + a == i
        assert (b.index, b.makespan) == (lb.index, lb.makespan) == (bb.index, bb.makespan) == (i, t)


def test_invalid_rank_in_list_reports_einval(dev):
    wl = W.workload(2)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    ranks = torch.tensor([0, 5, 4495, 7], dtype=torch.int64, device=dev)   # 4495 = C(31,3): out of range
    with pytest.raises(P.PoseidonError) as ei:
        P.poseidon_eval_candidates(ctx, comp_rank=ranks)
    assert ei.value.status == P.POSEIDON_E_INVAL
    # the context stays usable
    b = P.poseidon_eval_candidates(ctx, first=0, count=100)
    To, fo = coracle.evaluate(wl.problem, W.Candidates(first=0, count=100))
    assert (b.index, b.makespan) == coracle.argmin(To, fo)
    ctx.close()


def test_range_past_end_is_rejected(dev):
    wl = W.workload(2)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    with pytest.raises(P.PoseidonError) as ei:
        P.poseidon_eval_candidates(ctx, first=71000, count=921)
    assert ei.value.status == P.POSEIDON_E_INVAL
    ctx.close()


def test_context_reuse_across_sizes(dev):
    """One context, calls of growing and shrinking size (the straggler queues
    of the steady-state cascade are grown on demand and reused)."""
    wl = W.workload(4)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    for n in (1000, 200_003, 77, 1_000_001, 5000):
        c = W.Candidates(comp_rank=wl.cands.comp_rank[:n].copy(), assign_idx=wl.cands.assign_idx[:n].copy())
        Tg, fg, best = gpu_eval(ctx, c, dev)
        To, fo = coracle.evaluate(wl.problem, c)
        assert np.array_equal(Tg, To) and np.array_equal(fg, fo)
        assert (best.index, best.makespan) == coracle.argmin(To, fo)
    ctx.close()


def test_long_steady_part_small_stage_count(dev):
    """Many steady iterations for few stages (a deep cascade)."""
    rng = np.random.default_rng(107)
    for S, M in ((1, 300), (2, 200), (3, 150), (5, 400), (16, 600)):
        L = S + 10
        prob = W.random_problem(rng, L, S, M, 2, cost_hi=300, comm_hi=60, mem_hi=30, cap=300)
        check_against_oracle(prob, W.random_candidates(rng, prob, 3000), dev)


# --------------------------------------------------------- argmin, async

def test_argmin_entry_point(dev):
    rng = np.random.default_rng(105)
    wl = W.workload(2)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    n = 100_001
    Tn = rng.integers(1, 1000, n).astype(np.uint32)
    fn = rng.random(n) < 0.3
    words = pack_bits(fn)
    Td = torch.from_numpy(Tn.view(np.int32)).to(dev)
    Bd = torch.from_numpy(words.view(np.int32)).to(dev)
    b = P.poseidon_argmin(ctx, Td, Bd, index_base=1000)
    ob = coracle.argmin(Tn, fn)
    assert (b.index, b.makespan) == (ob[0] + 1000, ob[1])
    b = P.poseidon_argmin(ctx, Td)          # no bits: all feasible
    assert (b.index, b.makespan) == (int(np.argmin(Tn)), int(Tn.min()))
    ctx.close()


def test_async_then_last_best(dev):
    wl = W.workload(2)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    s = torch.cuda.current_stream()
    P.poseidon_eval_candidates(ctx, first=0, count=71920, want_best=False, stream=s)
    b = P.poseidon_last_best(ctx, stream=s)
    To, fo = coracle.evaluate(wl.problem, wl.cands)
    assert (b.index, b.makespan) == coracle.argmin(To, fo)
    # repeated calls give identical results
    for _ in range(3):
        b2 = P.poseidon_eval_candidates(ctx, first=0, count=71920)
        assert (b2.index, b2.makespan) == (b.index, b.makespan)
    ctx.close()


# ------------------------------------------------------------- early stop

def bounded_vs_oracle(prob, cands, bound, chunk, dev, ramp=False):
    ctx = P.poseidon_load_costs(prob, 0)
    b, st = P.poseidon_eval_candidates_bounded(ctx, bound, chunk=chunk, ramp=ramp, **to_dev(cands, dev))
    ob, ev, pr, inf = coracle.bounded(prob, cands, bound, chunk, ramp=ramp)
    got = (b.index, b.makespan) if b.index is not None else None
    assert got == (None if ob is None else (ob[0] + index_base(cands), ob[1]))
    assert (st.evaluated, st.pruned, st.infeasible) == (ev, pr, inf)
    ctx.close()
    return b, st


def test_bounded_largest_pascal_columns(dev):
    """S = 16 with L > 128 (256-row Pascal columns), 64-bit ranks and eight
    device types: with all-reduce times the prefix filter's columns, stage
    entries and screen buffer exceed a block's 64 KB of LDS (25,088 + 33,792
    + 8,320 bytes), so it reads the stage entries from global memory;
    without them everything fits.  Several chunk sizes."""
    rng = np.random.default_rng(141)
    for ar in (False, True):
        prob = W.random_problem(rng, 130, 16, 40, 8, cost_lo=50, cost_hi=400, mem_hi=20, cap=400, assign_rows=1)
        if ar:
            _with_allreduce(rng, prob, hi=3000)
        cands = W.random_candidates(rng, prob, 6000)
        assert int(cands.comp_rank.max()) > 2 ** 32
        To, fo = check_against_oracle(prob, cands, dev)[:2]
        bound = int(np.sort(To[fo])[40]) if fo.sum() > 40 else 2 ** 31 - 1
        for chunk in (0, 777, 4096):
            bounded_vs_oracle(prob, cands, bound, chunk, dev)


def test_bounded_random(dev):
    rng = np.random.default_rng(106)
    for trial in range(20):
        S = int(rng.integers(1, 9))
        L = S + int(rng.integers(1, 14))
        M = int(rng.integers(1, 30))
        prob = W.random_problem(rng, L, S, M, 3, mem_hi=30, cap=int(rng.integers(40, 200)))
        cands = W.random_candidates(rng, prob, int(rng.integers(1, 20000)))
        To, fo = coracle.evaluate(prob, cands)
        warm = coracle.argmin(To[:50], fo[:50])
        bound = warm[1] if warm else 2 ** 31
        for chunk, ramp in ((0, False), (4096, False), (777, False), (100, True)):
            b, _ = bounded_vs_oracle(prob, cands, bound, chunk, dev, ramp)
            ex = coracle.argmin(To, fo)
            if ex is not None and ex[1] <= bound:
                assert (b.index, b.makespan) == ex   # Theorem 1: same argmin as exhaustive


def test_bounded_workload4_prefix(dev):
    wl = W.workload(4)
    n = 1 << 20
    c = W.Candidates(comp_rank=wl.cands.comp_rank[:n].copy(), assign_idx=wl.cands.assign_idx[:n].copy())
    To, fo = coracle.evaluate(wl.problem, W.Candidates(comp_rank=c.comp_rank[:500], assign_idx=c.assign_idx[:500]))
    bound = coracle.argmin(To, fo)[1]
    for chunk, ramp in ((0, False), (1 << 16, False), (100_000, False), (1 << 12, True)):
        b, st = bounded_vs_oracle(wl.problem, c, bound, chunk, dev, ramp)
        assert st.pruned > 0


def test_bounded_stage1_screen(dev):
    """Early stop where the prefix filter decides stage 1 from the
    composition rank before decoding any cut (S >= 10, or all-reduce times):
    base-T digit, table and fixed assignments, list and range mode, pieces
    of 1, 255, 257 and several thousand candidates (a screened tile holds
    256), three chunkings, caps and bounds under which many candidates fail
    stage 1 on memory and many on Eq. 2.  Counts and argmin equal the
    oracle's."""
    rng = np.random.default_rng(151)
    seen_mem = seen_bound = 0
    for S, T, rows, ar in ((10, 2, None, False), (12, 3, None, False), (16, 2, None, False), (11, 3, 6, False),
                           (16, 4, 1, False), (5, 3, None, True), (8, 2, 4, True)):
        L = S + int(rng.integers(2, 50))
        M = int(rng.integers(S, 3 * S + 1))
        cap = int(40 * L / S * 0.9)   # stages well above the mean length exceed it
        prob = W.random_problem(rng, L, S, M, T, cost_lo=20, cost_hi=400, mem_hi=40, cap=cap, assign_rows=rows)
        if ar:
            _with_allreduce(rng, prob, hi=2000)
        total = prob.n_compositions * prob.A
        sets = [W.random_candidates(rng, prob, n) for n in (1, 255, 257, 6000)]
        n = min(5000, total)
        sets.append(W.Candidates(first=int(rng.integers(0, total - n + 1)), count=n))
        for cands in sets:
            To, fo = coracle.evaluate(prob, cands)
            ok = np.sort(To[fo])
            bound = int(ok[len(ok) // 10]) if len(ok) else 2 ** 31 - 1
            for chunk, ramp in ((0, False), (777, False), (64, True)):
                _, st = bounded_vs_oracle(prob, cands, bound, chunk, dev, ramp)
                seen_mem += st.infeasible
                seen_bound += st.pruned
    assert seen_mem > 0 and seen_bound > 0


def test_bounded_stage1_screen_invalid_rank(dev):
    """An out-of-range rank reaches the screened prefix filter's error flag
    (it is kept for the decode, which reports it) and the context stays
    usable."""
    rng = np.random.default_rng(152)
    prob = W.random_problem(rng, 30, 12, 20, 2, mem_hi=20)
    cands = W.random_candidates(rng, prob, 1000)
    bad = cands.comp_rank.copy()
    bad[600] = prob.n_compositions
    ctx = P.poseidon_load_costs(prob, 0)
    d = to_dev(W.Candidates(comp_rank=bad, assign_idx=cands.assign_idx), dev)
    with pytest.raises(P.PoseidonError) as ei:
        P.poseidon_eval_candidates_bounded(ctx, 2 ** 31 - 1, **d)
    assert ei.value.status == P.POSEIDON_E_INVAL
    ctx.close()
    bounded_vs_oracle(prob, cands, 2 ** 31 - 1, 0, dev)


def test_bounded_bound_below_optimum(dev):
    wl = W.workload(2)
    To, fo = coracle.evaluate(wl.problem, wl.cands)
    opt = coracle.argmin(To, fo)[1]
    b, st = bounded_vs_oracle(wl.problem, wl.cands, opt - 1, 0, dev)
    assert b.status == P.POSEIDON_NO_FEASIBLE
    b, st = bounded_vs_oracle(wl.problem, wl.cands, opt, 0, dev)
    assert b.makespan == opt


# ---------------------------------------------------------- full sizes

def _golden():
    if not os.path.exists(GOLD):
        pytest.skip("golden file missing")
    return json.load(open(GOLD))


@pytest.mark.parametrize("cfg", [3, 4, 5])
def test_full_workload_matches_golden(cfg, dev):
    g = _golden()[f"cfg{cfg}"]
    wl = W.workload(cfg)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    Tg, fg, best = gpu_eval(ctx, wl.cands, dev)
    assert len(Tg) == g["n"]
    words = pack_bits(fg)
    assert int(fg.sum()) == g["n_feasible"]
    assert (best.index, best.makespan) == (g["best_index"], g["best_makespan"])
    assert int(Tg.min()) == g["makespan_min"] and int(Tg.max()) == g["makespan_max"]
    assert hashlib.sha256(Tg.astype("<u4").tobytes()).hexdigest() == g["makespan_sha256"]
    assert hashlib.sha256(words.astype("<u4").tobytes()).hexdigest() == g["feasible_bits_sha256"]
    # sampled entries recomputed by the oracle one by one
    rng = np.random.default_rng(cfg)
    pick = rng.choice(len(Tg), 2000, replace=False)
    if wl.cands.is_list:
        sub = W.Candidates(comp_rank=wl.cands.comp_rank[pick],
                           assign_idx=None if wl.cands.assign_idx is None else wl.cands.assign_idx[pick])
        To, fo = coracle.evaluate(wl.problem, sub)
        assert np.array_equal(Tg[pick], To) and np.array_equal(fg[pick], fo)
    ctx.close()


def test_full_workload4_bounded_matches_golden(dev):
    g = _golden()["cfg4"]
    wl = W.workload(4)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    d = to_dev(wl.cands, dev)
    # warm-up: exact evaluation of the first 500 entries sets the bound
    wb = P.poseidon_eval_candidates(ctx, comp_rank=d["comp_rank"][:g["warmup"]],
                                    assign_idx=d["assign_idx"][:g["warmup"]])
    assert wb.makespan == g["warmup_bound"]
    for chunk, exp in g["bounded"].items():
        b, st = P.poseidon_eval_candidates_bounded(ctx, wb.makespan, chunk=int(chunk), **d)
        assert (b.index, b.makespan) == (exp["best_index"], exp["best_makespan"])
        assert (st.evaluated, st.pruned, st.infeasible) == (exp["evaluated"], exp["pruned"], exp["infeasible"])
        # Theorem 1: the early-stop pass finds the exhaustive argmin
        assert (b.index, b.makespan) == (g["best_index"], g["best_makespan"])
    ctx.close()


def test_call_longer_than_one_chunk(dev):
    """2^26 + 5,000 candidates: the library works in chunks of 2^26, so the
    argmin is folded across chunks and the early-stop pass decodes in pieces."""
    g = _golden()["cfg4"]
    wl = W.workload(4)
    rng = np.random.default_rng(108)
    extra = W.random_candidates(rng, wl.problem, 5000)
    c = W.Candidates(comp_rank=np.concatenate([wl.cands.comp_rank, extra.comp_rank]),
                     assign_idx=np.concatenate([wl.cands.assign_idx, extra.assign_idx]))
    n0 = len(wl.cands)
    Te, fe = coracle.evaluate(wl.problem, extra)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    Tg, fg, best = gpu_eval(ctx, c, dev)
    assert np.array_equal(Tg[n0:], Te) and np.array_equal(fg[n0:], fe)
    assert hashlib.sha256(Tg[:n0].astype("<u4").tobytes()).hexdigest() == g["makespan_sha256"]
    be = coracle.argmin(Te, fe)
    exp = min((g["best_makespan"], g["best_index"]), (be[1], be[0] + n0))
    assert (best.makespan, best.index) == exp
    d = to_dev(c, dev)
    b, st = P.poseidon_eval_candidates_bounded(ctx, g["warmup_bound"], chunk=0, **d)
    assert (b.makespan, b.index) == exp
    # one chunk: every candidate against the warm-up bound, so the counts are
    # those of the full list plus those of the extra entries
    _, ev, pr, inf = coracle.bounded(wl.problem, extra, g["warmup_bound"], 0)
    e0 = g["bounded"]["0"]
    assert (st.evaluated, st.pruned, st.infeasible) == (e0["evaluated"] + ev, e0["pruned"] + pr,
                                                        e0["infeasible"] + inf)
    ctx.close()


def test_range_mode_consecutive_ranks_across_chunks(dev):
    """Range mode with one assignment decodes four consecutive ranks per lane
    (the first unranked, the next three by the lexicographic successor): a
    range of 2^26 + 3,001 compositions from an odd offset spans two chunks,
    and ranges that end at the last composition put the successor step past
    it on lanes beyond the call only."""
    rng = np.random.default_rng(120)
    prob = W.random_problem(rng, 60, 8, 12, 2, cost_hi=400, comm_hi=50, mem_hi=30, cap=300, assign_rows=1)
    n_comp = math.comb(59, 7)
    for first, count in ((123457, (1 << 26) + 3001), (n_comp - 5001, 5001), (n_comp - 3, 3), (0, 1)):
        check_against_oracle(prob, W.Candidates(first=first, count=count), dev)


def test_range_mode_consecutive_ranks_every_stage_count(dev):
    """The range-mode successor decode for S = 1..16 and for L up to 256 (64-bit
    ranks, the Pascal table's full column): ragged ranges from random
    offsets, the first ranks and the last ones."""
    rng = np.random.default_rng(121)
    for S in range(1, 17):
        # the longest model up to 256 layers whose compositions are counted below 2^63
        L_max = max(L for L in range(S, 257) if math.comb(L - 1, S - 1) < 2 ** 63)
        for L in (S, S + int(rng.integers(1, 30)), L_max):
            M = S + int(rng.integers(0, 20))
            prob = W.random_problem(rng, L, S, M, 2, cost_hi=400, comm_hi=50, mem_hi=30,
                                    cap=int(rng.integers(60, 3000)), assign_rows=1)
            n_comp = math.comb(L - 1, S - 1)
            count = int(min(n_comp, rng.integers(1, 9000)))
            for first in {0, int(rng.integers(0, n_comp - count + 1)), n_comp - count}:
                check_against_oracle(prob, W.Candidates(first=first, count=count), dev)


# ------------------------------------------------------ DP all-reduce

def _with_allreduce(rng, prob, hi=3000):
    prob.allreduce = rng.integers(0, hi, size=(prob.T, prob.L)).astype(np.uint32)
    return prob


def test_allreduce_random_problems(dev):
    """R_s nodes: T = max_s(finish(B_{s,M}) + R_s), both DP paths and the cascade."""
    rng = np.random.default_rng(109)
    for trial in range(30):
        S = int(rng.integers(1, 17))
        M = int(rng.integers(1, 3 * S + 20))
        L = S + int(rng.integers(0, 10))
        T = int(rng.integers(1, 4))
        prob = W.random_problem(rng, L, S, M, T, cost_hi=400, mem_hi=30, cap=int(rng.integers(30, 200)),
                                assign_rows=None if T ** S < 5000 else 5)
        # all-reduce large enough to decide the makespan in some candidates
        _with_allreduce(rng, prob, hi=int(rng.integers(1, 400)) * max(M, 1))
        check_against_oracle(prob, W.random_candidates(rng, prob, int(rng.integers(1, 2000))), dev)


def test_allreduce_python_oracle_and_bounded(dev):
    rng = np.random.default_rng(110)
    for _ in range(6):
        S = int(rng.integers(1, 5))
        L = S + int(rng.integers(0, 5))
        M = int(rng.integers(1, 7))
        prob = _with_allreduce(rng, W.random_problem(rng, L, S, M, 2, mem_hi=30, cap=int(rng.integers(30, 120))),
                               hi=2000)
        full = W.Candidates(first=0, count=prob.n_candidates)
        check_against_oracle(prob, full, dev, python_oracle=True)
        To, fo = coracle.evaluate(prob, full)
        ex = coracle.argmin(To, fo)
        if ex is not None:
            for chunk in (0, 5):
                b, _ = bounded_vs_oracle(prob, full, int(To[fo].max()), chunk, dev)
                assert (b.index, b.makespan) == ex


def test_workload6_prefix_exhaustive_and_bounded(dev):
    wl = W.workload(6)
    n = 500_003
    c = W.Candidates(comp_rank=wl.cands.comp_rank[:n].copy(), assign_idx=wl.cands.assign_idx[:n].copy())
    check_against_oracle(wl.problem, c, dev)
    To, fo = coracle.evaluate(wl.problem, W.Candidates(comp_rank=c.comp_rank[:500], assign_idx=c.assign_idx[:500]))
    bound = coracle.argmin(To, fo)[1]
    for chunk in (0, 100_000):
        bounded_vs_oracle(wl.problem, c, bound, chunk, dev)


def test_full_workload6_matches_golden(dev):
    gall = _golden()
    if "cfg6" not in gall:
        pytest.skip("no golden for workload 6")
    g = gall["cfg6"]
    wl = W.workload(6)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    Tg, fg, best = gpu_eval(ctx, wl.cands, dev)
    assert hashlib.sha256(Tg.astype("<u4").tobytes()).hexdigest() == g["makespan_sha256"]
    assert hashlib.sha256(pack_bits(fg).astype("<u4").tobytes()).hexdigest() == g["feasible_bits_sha256"]
    assert (best.index, best.makespan) == (g["best_index"], g["best_makespan"])
    d = to_dev(wl.cands, dev)
    for chunk, exp in g["bounded"].items():
        b, st = P.poseidon_eval_candidates_bounded(ctx, g["warmup_bound"], chunk=int(chunk), **d)
        assert (b.index, b.makespan) == (exp["best_index"], exp["best_makespan"])
        assert (st.evaluated, st.pruned, st.infeasible) == (exp["evaluated"], exp["pruned"], exp["infeasible"])
    ctx.close()


# ---------------------------------------------------------- Eager 1F1B

def test_eager_random_problems(dev):
    """Schedule-table DP (newest / previous forward, newest backward per
    stage) against the oracle's Eager 1F1B DAG, S = 1..16, any M."""
    rng = np.random.default_rng(111)
    for trial in range(48):
        S = trial % 16 + 1
        M = int(rng.integers(1, 3 * S + 24))
        L = S + int(rng.integers(0, 10))
        T = int(rng.integers(1, 4))
        prob = W.random_problem(rng, L, S, M, T, cost_hi=400, mem_hi=30, cap=int(rng.integers(30, 200)),
                                assign_rows=None if T ** S < 5000 else 5)
        prob.schedule = P.SCHEDULE_EAGER_1F1B
        if trial % 3 == 0:
            _with_allreduce(rng, prob, hi=int(rng.integers(1, 400)) * M)
        check_against_oracle(prob, W.random_candidates(rng, prob, int(rng.integers(1, 1500))), dev)


def test_eager_closed_form_edges(dev):
    """Closed form at its smallest M = 2S-1 (no steady pair for stage 1),
    odd and even steady pair counts, long steady parts."""
    rng = np.random.default_rng(113)
    for S, M in [(1, 1), (1, 2), (2, 3), (2, 4), (5, 9), (5, 10), (8, 15), (8, 16), (16, 31), (16, 32),
                 (16, 33), (3, 200), (3, 201), (12, 129)]:
        L = S + int(rng.integers(0, 8))
        prob = W.random_problem(rng, L, S, M, 2, cost_hi=300, mem_hi=30, cap=int(rng.integers(30, 200)),
                                assign_rows=None if 2 ** S < 5000 else 5)
        prob.schedule = P.SCHEDULE_EAGER_1F1B
        check_against_oracle(prob, W.random_candidates(rng, prob, int(rng.integers(100, 1200))), dev)


def test_long_pipelines_both_schedules(dev):
    """S * M well above 4096 under 1F1B and Eager 1F1B (the closed forms'
    host check simulates every M), with and without all-reduce times."""
    rng = np.random.default_rng(114)
    for schedule in (P.SCHEDULE_1F1B, P.SCHEDULE_EAGER_1F1B):
        for S, M in ((16, 300), (8, 700), (12, 1001)):
            prob = W.random_problem(rng, S + 9, S, M, 2, cost_hi=300, comm_hi=60, mem_hi=30, cap=300,
                                    assign_rows=None if 2 ** S < 5000 else 6)
            prob.schedule = schedule
            if M == 700:
                _with_allreduce(rng, prob, hi=400 * M)
            check_against_oracle(prob, W.random_candidates(rng, prob, 2500), dev)


def test_eager_python_oracle_and_bounded(dev):
    rng = np.random.default_rng(112)
    for trial in range(8):
        S = int(rng.integers(1, 5))
        L = S + int(rng.integers(0, 5))
        M = int(rng.integers(1, 9))
        prob = W.random_problem(rng, L, S, M, 2, mem_hi=30, cap=int(rng.integers(30, 120)))
        prob.schedule = P.SCHEDULE_EAGER_1F1B
        if trial % 2:
            _with_allreduce(rng, prob, hi=1500)
        full = W.Candidates(first=0, count=prob.n_candidates)
        check_against_oracle(prob, full, dev, python_oracle=True)
        To, fo = coracle.evaluate(prob, full)
        ex = coracle.argmin(To, fo)
        if ex is not None:
            for chunk in (0, 7):
                b, _ = bounded_vs_oracle(prob, full, int(To[fo].max()), chunk, dev)
                assert (b.index, b.makespan) == ex


def test_eager_workload4_prefix_and_bounded(dev):
    """The 8-stage, 64-micro-batch, 3-type workload under Eager 1F1B."""
    wl = W.workload(4)
    prob = wl.problem
    prob.schedule = P.SCHEDULE_EAGER_1F1B
    n = 400_003
    c = W.Candidates(comp_rank=wl.cands.comp_rank[:n].copy(), assign_idx=wl.cands.assign_idx[:n].copy())
    check_against_oracle(prob, c, dev)
    To, fo = coracle.evaluate(prob, W.Candidates(comp_rank=c.comp_rank[:500], assign_idx=c.assign_idx[:500]))
    bound = coracle.argmin(To, fo)[1]
    for chunk in (0, 100_000):
        b, st = bounded_vs_oracle(prob, c, bound, chunk, dev)
        assert st.pruned > 0


def test_eager_differs_from_1f1b(dev):
    """The schedule field reaches the kernels: same candidates, other makespans."""
    wl = W.workload(2)
    prob = wl.problem
    c0 = P.poseidon_load_costs(prob, 0)
    T0, _, _ = gpu_eval(c0, wl.cands, dev)
    prob.schedule = P.SCHEDULE_EAGER_1F1B
    c1 = P.poseidon_load_costs(prob, 0)
    T1, _, _ = gpu_eval(c1, wl.cands, dev)
    assert (T0 != T1).any()
    To, _ = coracle.evaluate(prob, wl.cands)
    assert np.array_equal(T1, To)
    c0.close()
    c1.close()


@pytest.mark.parametrize("cfg", [4, 5])
def test_full_workload_eager_matches_golden(cfg, dev):
    """Full-size workloads under Eager 1F1B: closed form, steady-state
    cascade and early stop against digests the oracle wrote."""
    gall = _golden()
    key = f"cfg{cfg}_eager"
    if key not in gall:
        pytest.skip(f"no golden for {key}")
    g = gall[key]
    wl = W.workload(cfg)
    wl.problem.schedule = P.SCHEDULE_EAGER_1F1B
    ctx = P.poseidon_load_costs(wl.problem, 0)
    Tg, fg, best = gpu_eval(ctx, wl.cands, dev)
    assert hashlib.sha256(Tg.astype("<u4").tobytes()).hexdigest() == g["makespan_sha256"]
    assert hashlib.sha256(pack_bits(fg).astype("<u4").tobytes()).hexdigest() == g["feasible_bits_sha256"]
    assert (best.index, best.makespan) == (g["best_index"], g["best_makespan"])
    d = to_dev(wl.cands, dev)
    for chunk, exp in g["bounded"].items():
        b, st = P.poseidon_eval_candidates_bounded(ctx, g["warmup_bound"], chunk=int(chunk), **d)
        assert (b.index, b.makespan) == (exp["best_index"], exp["best_makespan"])
        assert (st.evaluated, st.pruned, st.infeasible) == (exp["evaluated"], exp["pruned"], exp["infeasible"])
    ctx.close()


def test_maximum_layer_and_type_counts(dev):
    """L = 256 (the Pascal table's full column, cut values up to 255) with
    T = 8 device types, all-reduce nodes, 1F1B and Eager 1F1B, list mode with
    random and extreme ranks; and T = 8 with all 8^8 assignment digits.  (Both
    at once would overflow the 64-bit joint index, which the library refuses.)"""
    rng = np.random.default_rng(140)
    for schedule in (P.SCHEDULE_1F1B, P.SCHEDULE_EAGER_1F1B):
        prob = W.random_problem(rng, 256, 8, 40, 8, cost_lo=50, cost_hi=400, mem_hi=20, cap=2000, assign_rows=97)
        prob.schedule = schedule
        _with_allreduce(rng, prob, hi=3000)
        cands = W.random_candidates(rng, prob, 5000)
        assert int(cands.comp_rank.max()) > 2 ** 32    # wide ranks (u64 Pascal table)
        check_against_oracle(prob, cands, dev)
        n_comp = prob.n_compositions
        edge = W.Candidates(comp_rank=np.array([0, 1, n_comp - 2, n_comp - 1], dtype=np.uint64),
                            assign_idx=np.array([0, prob.A - 1, 50, prob.A - 2], dtype=np.uint32))
        check_against_oracle(prob, edge, dev)
        digits = W.random_problem(rng, 40, 8, 24, 8, mem_hi=20, cap=400)
        digits.schedule = schedule
        assert digits.A == 8 ** 8
        check_against_oracle(digits, W.random_candidates(rng, digits, 5000), dev)
