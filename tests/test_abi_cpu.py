"""The C-ABI library on the CPU: it loads, exports every declared entry
point, and rejects invalid problems before touching the GPU."""
import math
import os
import re
import subprocess
import sys

import numpy as np
import pytest

from paper_2609_06086_amd import poseidon as P
from paper_2609_06086_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "poseidon.h")


def declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(poseidon_[a-z_]+)\s*\(", txt)))


def test_library_exports_every_declared_symbol():
    syms = declared()
    assert "poseidon_load_costs" in syms and "poseidon_eval_candidates" in syms
    out = subprocess.run(["nm", "-D", "--defined-only", P.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = set(re.findall(r"\bT (poseidon_[a-z_]+)", out))
    assert set(syms) <= exported, set(syms) - exported
    assert set(P.EXPORTS) == set(syms)
    lib = P.lib()
    for s in syms:
        assert hasattr(lib, s)


def test_strerror():
    assert P.strerror(0) == "ok"
    assert "invalid" in P.strerror(P.POSEIDON_E_INVAL)
    assert P.strerror(12345) == "unknown status"


def test_validate_counts_candidates():
    assert P.poseidon_validate(W.workload(1).problem) == 28
    assert P.poseidon_validate(W.workload(2).problem) == 71920
    assert P.poseidon_validate(W.workload(3).problem) == 62891499
    assert P.poseidon_validate(W.workload(4, n_samples=4).problem) == 2898753715 * 6561
    assert P.poseidon_validate(W.workload(5, n_samples=4).problem) == 9064807833193439800


def _small():
    rng = np.random.default_rng(0)
    return W.random_problem(rng, 10, 3, 4, 2)


def _status(prob):
    with pytest.raises(P.PoseidonError) as ei:
        P.poseidon_validate(prob)
    return ei.value.status


def test_validation_errors():
    p = _small()
    p.S = 11                              # S > L
    assert _status(p) == P.POSEIDON_E_INVAL
    p = _small(); p.S = 0
    assert _status(p) == P.POSEIDON_E_INVAL
    p = _small(); p.T = 0
    assert _status(p) == P.POSEIDON_E_INVAL
    p = _small(); p.M = 0
    assert _status(p) == P.POSEIDON_E_INVAL
    p = _small(); p.fwd = None
    assert _status(p) == P.POSEIDON_E_INVAL
    p = _small(); p.comm_fwd = None
    assert _status(p) == P.POSEIDON_E_INVAL
    p = _small(); p.assign = np.array([[0, 1, 2]], np.uint8)   # type id 2 >= T = 2
    assert _status(p) == P.POSEIDON_E_INVAL
    # S above the compiled maximum
    rng = np.random.default_rng(1)
    p = W.random_problem(rng, 40, 17, 4, 1)
    assert _status(p) == P.POSEIDON_E_INVAL
    # L above the maximum
    p = W.random_problem(rng, 300, 4, 4, 1)
    assert _status(p) == P.POSEIDON_E_INVAL
    # unknown schedule
    p = _small(); p.schedule = 2
    assert _status(p) == P.POSEIDON_E_INVAL
    p = _small(); p.schedule = P.SCHEDULE_EAGER_1F1B
    assert P.poseidon_validate(p) > 0


def test_overflow_guard():
    """A makespan that could reach 2^31 is refused (E_RANGE)."""
    rng = np.random.default_rng(2)
    p = W.random_problem(rng, 16, 4, 1000, 2, cost_lo=1000, cost_hi=1000)
    # every path is at most M * (sum of slowest fwd+bwd + comm) = 1000*(16*2000 + comm) < 2^31
    assert P.poseidon_validate(p) > 0
    p.M = 100000
    assert _status(p) == P.POSEIDON_E_RANGE


def test_too_many_assignments():
    rng = np.random.default_rng(3)
    p = W.random_problem(rng, 40, 16, 4, 8)   # 8^16 assignments > 2^32
    assert _status(p) == P.POSEIDON_E_RANGE


def test_load_costs_rejects_before_device():
    p = _small()
    p.S = 11
    with pytest.raises(P.PoseidonError) as ei:
        P.poseidon_load_costs(p, 0)
    assert ei.value.status == P.POSEIDON_E_INVAL


def test_closed_form_schedules_pass_the_host_self_check():
    """poseidon_load_costs simulates the slot schedule and compares it with
    the closed forms the kernels hard-code (1F1B for M >= S, Eager 1F1B for
    M >= 2S-1, including which forwards read the upstream's previous
    forward); a mismatch returns E_INVAL before any device call.  Without a
    GPU a passing check ends at the device step (E_DEVICE)."""
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("needs a host without a GPU")
    rng = np.random.default_rng(4)
    for sched in (P.SCHEDULE_1F1B, P.SCHEDULE_EAGER_1F1B):
        for S in range(1, 17):
            Ms = list(range(1, 2 * S + 6)) + [64, 255, 256, 600, 2048]
            if S in (8, 15, 16):
                Ms += [4097, 65537, P.M_MAX]
            for M in Ms:
                p = W.random_problem(rng, S + 2, S, M, 1, cost_lo=0, cost_hi=0 if M > 60000 else 1000,
                                     comm_hi=0 if M > 60000 else 100)
                p.schedule = sched
                with pytest.raises(P.PoseidonError) as ei:
                    P.poseidon_load_costs(p, 0)
                assert ei.value.status == P.POSEIDON_E_DEVICE, (sched, S, M)


def test_micro_batch_limit():
    """M above POSEIDON_M_MAX (2^20) is refused before any device call."""
    p = W.random_problem(np.random.default_rng(9), 20, 16, P.M_MAX, 2, cost_lo=0, cost_hi=0, comm_hi=0)
    assert P.poseidon_validate(p) > 0
    p.M = P.M_MAX + 1
    assert _status(p) == P.POSEIDON_E_INVAL


def test_search_rejects_bad_arguments_before_device():
    b, st = P._Best(), P._SearchStats()
    assert P.lib().poseidon_search(None, 0, 1, 100, 0, 0, P.C.byref(b), P.C.byref(st), None) == P.POSEIDON_E_INVAL


def test_interleaved_validation():
    rng = np.random.default_rng(6)
    p = W.random_problem(rng, 12, 8, 8, 2)
    p.schedule, p.V = P.SCHEDULE_INTERLEAVED_1F1B, 2     # 4 devices, M = 8 a multiple of 4
    assert P.poseidon_validate(p) == math.comb(11, 7) * 2 ** 4
    for V, M in ((1, 8), (3, 8), (2, 6), (8, 8)):        # V < 2, S % V, M % N, one device
        q = W.random_problem(rng, 12, 8, M, 2)
        q.schedule, q.V = P.SCHEDULE_INTERLEAVED_1F1B, V
        assert _status(q) == P.POSEIDON_E_INVAL, (V, M)
    p.assign = np.array([[0, 1, 1, 0], [1, 1, 0, 0]], dtype=np.uint8)   # rows per device
    assert P.poseidon_validate(p) == math.comb(11, 7) * 2
    p.assign = np.array([[0, 1, 2, 0]], dtype=np.uint8)
    assert _status(p) == P.POSEIDON_E_INVAL


def test_interleaved_schedules_pass_the_host_checks():
    """For every (virtual stages, devices) pair the library supports and a
    range of M, the host's simulation of the Interleaved 1F1B schedule keeps
    one node per device per slot and input depths the stencil holds (else
    E_INVAL before any device call; without a GPU a pass ends at E_DEVICE)."""
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("needs a host without a GPU")
    rng = np.random.default_rng(7)
    pairs = [(4, 2), (6, 2), (6, 3), (8, 2), (8, 4), (9, 3), (10, 2), (10, 5), (12, 2), (12, 3), (12, 4), (12, 6),
             (14, 2), (14, 7), (15, 3), (15, 5), (16, 2), (16, 4), (16, 8)]
    for S, N in pairs:
        for k in (1, 2, 3, 5, 8, 13, 40):
            p = W.random_problem(rng, S + 3, S, N * k, 1)
            p.schedule, p.V = P.SCHEDULE_INTERLEAVED_1F1B, S // N
            with pytest.raises(P.PoseidonError) as ei:
                P.poseidon_load_costs(p, 0)
            assert ei.value.status == P.POSEIDON_E_DEVICE, (S, N, N * k)


def test_joint_index_overflow_is_refused():
    """C(255, 7) compositions x 8^8 assignment digits exceed the 64-bit joint
    index rank * A + a."""
    p = W.random_problem(np.random.default_rng(8), 256, 8, 4, 8)
    assert _status(p) == P.POSEIDON_E_RANGE


def test_bench_refuses_more_than_one_gpu():
    """The benchmark measures one GPU: --gpus N > 1 exits with status 2 and a
    message, before it imports torch or touches a device."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=root)
    assert r.returncode == 2
    assert "measures one GPU" in r.stderr and r.stdout == ""
