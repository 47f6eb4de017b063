"""GPU parity of Interleaved 1F1B (Sec. 4.1.4) against the C oracle, which
is pinned in tests/test_oracle_pins.py (the paper's node and edge counts,
the uniform closed form, an event simulation).  Bit-exact makespans,
feasibility bits and argmin."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import coracle, dag  # noqa: E402
from paper_2609_06086_amd import poseidon as P  # noqa: E402
from paper_2609_06086_amd import workloads as W  # noqa: E402

from test_gpu_parity import check_against_oracle  # noqa: E402

pytestmark = pytest.mark.gpu

PAIRS = [(4, 2), (6, 2), (6, 3), (8, 2), (8, 4), (9, 3), (10, 2), (10, 5), (12, 2), (12, 3), (12, 4), (12, 6),
         (14, 2), (14, 7), (15, 3), (15, 5), (16, 2), (16, 4), (16, 8)]


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def _problem(rng, S, N, M, T, ar=False, table=False):
    V = S // N
    L = S + int(rng.integers(0, 10))
    prob = W.random_problem(rng, L, S, M, T, cost_hi=400, mem_hi=30, cap=int(rng.integers(60, 400)))
    prob.schedule, prob.V = P.SCHEDULE_INTERLEAVED_1F1B, V
    if table or T ** N > 5000:
        prob.assign = rng.integers(0, T, size=(int(rng.integers(1, 7)), N)).astype(np.uint8)
    if ar:
        prob.allreduce = rng.integers(0, 3000, size=(T, L)).astype(np.uint32)
    return prob


def test_interleaved_every_stage_device_pair(dev):
    rng = np.random.default_rng(130)
    for k, (S, N) in enumerate(PAIRS):
        for M in (N, 2 * N, N * int(rng.integers(3, 9))):
            prob = _problem(rng, S, N, M, int(rng.integers(1, 4)), ar=k % 3 == 1, table=k % 4 == 2)
            check_against_oracle(prob, W.random_candidates(rng, prob, int(rng.integers(1, 900))), dev)


def test_interleaved_cascade_long_pipelines(dev):
    """Many steady periods for every (S, N) pair: lanes whose live registers
    settle at the first checkpoint jump to the end of the periods, the others
    are queued and resumed level by level (checkpoints at 2, 4, 8, 16
    periods); single-layer stages with close compute times settle late."""
    rng = np.random.default_rng(134)
    for k, (S, N) in enumerate(PAIRS):
        M = N * int(rng.integers(10, 34))
        prob = _problem(rng, S, N, M, int(rng.integers(1, 4)), ar=k % 2 == 0, table=k % 3 == 1)
        check_against_oracle(prob, W.random_candidates(rng, prob, int(rng.integers(200, 700))), dev)


def test_interleaved_cascade_uniform_and_tied_stages(dev):
    """Stages with equal compute times (ties between critical cycles) and no
    transfers: the steady state settles at once or never within the run;
    both must give the oracle's values, and the uniform closed form
    T = (VM + N - 1)(f + b) when every stage has one layer."""
    rng = np.random.default_rng(135)
    for S, N in ((8, 4), (12, 6), (16, 8), (16, 4)):
        M = 24 * N
        prob = _problem(rng, S, N, M, 2)
        prob.L = S + 4
        prob.fwd = np.full((2, prob.L), 5, np.uint32)
        prob.fwd[1] = 9
        prob.bwd = 2 * prob.fwd
        prob.mem = np.ones(prob.L, np.uint32)
        prob.comm_fwd = rng.integers(0, 2, size=S - 1).astype(np.uint32)
        prob.comm_bwd = prob.comm_fwd.copy()
        prob.allreduce = None
        check_against_oracle(prob, W.random_candidates(rng, prob, 400), dev)
        one = W.Candidates(first=0, count=1)
        prob.L = S
        prob.fwd, prob.bwd = prob.fwd[:, :S].copy(), prob.bwd[:, :S].copy()
        prob.mem = prob.mem[:S].copy()
        prob.comm_fwd = np.zeros(S - 1, np.uint32)
        prob.comm_bwd = np.zeros(S - 1, np.uint32)
        prob.assign = np.zeros((1, N), np.uint8)
        ctx = P.poseidon_load_costs(prob, 0)
        T = torch.empty(1, dtype=torch.int32, device=dev)
        P.poseidon_eval_candidates(ctx, first=one.first, count=one.count, makespan_out=T)
        assert int(T.cpu()[0]) == (S // N * M + N - 1) * 15
        ctx.close()


def test_interleaved_python_oracle_exhaustive(dev):
    rng = np.random.default_rng(131)
    for S, N in ((4, 2), (6, 3), (6, 2)):
        prob = _problem(rng, S, N, N * 2, 2, ar=S == 6)
        prob.L = S + 2
        prob.fwd, prob.bwd = prob.fwd[:, :prob.L].copy(), prob.bwd[:, :prob.L].copy()
        prob.mem = prob.mem[:prob.L].copy()
        if prob.allreduce is not None:
            prob.allreduce = prob.allreduce[:, :prob.L].copy()
        check_against_oracle(prob, W.Candidates(first=0, count=prob.n_candidates), dev, python_oracle=True)


def test_interleaved_uniform_closed_form(dev):
    """Equal per-layer costs, one layer per virtual stage, no transfers:
    T = (VM + N - 1)(f + b) for every candidate."""
    rng = np.random.default_rng(132)
    for S, N in ((8, 4), (12, 3), (16, 8)):
        M = 4 * N
        prob = _problem(rng, S, N, M, 1)
        prob.L = S
        prob.fwd = np.full((1, S), 7, np.uint32)
        prob.bwd = np.full((1, S), 11, np.uint32)
        prob.mem = np.ones(S, np.uint32)
        prob.comm_fwd = np.zeros(S - 1, np.uint32)
        prob.comm_bwd = np.zeros(S - 1, np.uint32)
        prob.assign = None
        ctx = P.poseidon_load_costs(prob, 0)
        T = torch.empty(1, dtype=torch.int32, device=dev)
        P.poseidon_eval_candidates(ctx, first=0, count=1, makespan_out=T)
        assert int(T.cpu()[0]) == (S // N * M + N - 1) * 18
        ctx.close()


def test_interleaved_rejected_by_bound_and_search(dev):
    rng = np.random.default_rng(133)
    prob = _problem(rng, 8, 4, 8, 2)
    ctx = P.poseidon_load_costs(prob, 0)
    with pytest.raises(P.PoseidonError):
        P.poseidon_eval_candidates_bounded(ctx, 10 ** 6, first=0, count=10)
    with pytest.raises(P.PoseidonError):
        P.poseidon_search(ctx, 10 ** 6)
    ctx.close()


def test_full_workload5_interleaved_matches_golden(dev):
    """The 16-stage workload as 16 virtual stages on 8 devices (V = 2), all
    2^24 candidates, against digests the oracle wrote."""
    import hashlib
    import json
    import os
    from test_gpu_parity import GOLD, gpu_eval, pack_bits
    if not os.path.exists(GOLD):
        pytest.skip("golden file missing")
    g = json.load(open(GOLD)).get("cfg5_interleaved")
    if g is None:
        pytest.skip("no golden for the interleaved workload")
    wl = W.interleaved_variant(W.workload(5), 2)
    ctx = P.poseidon_load_costs(wl.problem, 0)
    Tg, fg, best = gpu_eval(ctx, wl.cands, dev)
    assert hashlib.sha256(Tg.astype("<u4").tobytes()).hexdigest() == g["makespan_sha256"]
    assert hashlib.sha256(pack_bits(fg).astype("<u4").tobytes()).hexdigest() == g["feasible_bits_sha256"]
    assert (best.index, best.makespan) == (g["best_index"], g["best_makespan"])
    ctx.close()
