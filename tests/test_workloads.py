"""The seeded synthetic workloads: reproducible, in range, right shapes."""
import math

import numpy as np

from paper_2609_06086_amd import workloads as W


def test_reproducible_and_shaped():
    for cfg in W.WORKLOAD_IDS:
        a = W.workload(cfg, n_samples=1000 if cfg >= 4 else None)
        b = W.workload(cfg, n_samples=1000 if cfg >= 4 else None)
        p, q = a.problem, b.problem
        for name in ("fwd", "bwd", "comm_fwd", "comm_bwd", "mem", "cap"):
            assert np.array_equal(getattr(p, name), getattr(q, name))
            assert getattr(p, name).dtype == np.uint32
        assert p.fwd.shape == (p.T, p.L) and p.mem.shape == (p.L,) and p.cap.shape == (p.T,)
        assert p.comm_fwd.shape == (p.S - 1,)
        assert np.array_equal(p.bwd, 2 * p.fwd)
        assert np.array_equal(p.comm_fwd, p.comm_bwd)
        assert ((p.mem >= 1024) & (p.mem <= 2048)).all()
        if a.cands.is_list:
            assert np.array_equal(a.cands.comp_rank, b.cands.comp_rank)
            assert int(a.cands.comp_rank.max()) < p.n_compositions


def test_shapes_of_the_five_workloads():
    expect = {1: (8, 2, 4, 2, 4), 2: (32, 4, 16, 2, 16), 3: (48, 8, 32, 2, 1),
              4: (80, 8, 64, 3, 6561), 5: (126, 16, 128, 4, 1)}
    for cfg, (L, S, M, T, A) in expect.items():
        p = W.workload(cfg, n_samples=10).problem
        assert (p.L, p.S, p.M, p.T, p.A) == (L, S, M, T, A)
    p5 = W.workload(5, n_samples=10).problem
    assert sorted(p5.assign[0].tolist()) == [0] * 4 + [1] * 4 + [2] * 4 + [3] * 4
    assert W.workload(3).problem.assign[0].tolist() == [0, 0, 0, 0, 1, 1, 1, 1]
    assert math.comb(125, 15) == W.workload(5, n_samples=10).problem.n_compositions


def test_speed_scaling_rounds_half_up():
    p = W.workload(2).problem
    assert np.array_equal(p.fwd[1], (32 * p.fwd[0].astype(np.int64) + 10) // 20)
    p4 = W.workload(4, n_samples=10).problem
    base = p4.fwd[0].astype(np.int64)
    assert np.array_equal(p4.fwd[1], (20 * base + 17) // 34)
    assert np.array_equal(p4.fwd[2], (20 * base + 26) // 52)
