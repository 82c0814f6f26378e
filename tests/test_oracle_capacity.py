"""Pins of the oracle's effective capacity (Sec. 3.4, Eq. 12):
C_eff = C - gamma * sum over pending jobs of each job's componentwise
smallest demand vector over its allowed family."""
import numpy as np
import pytest

import oracle
import workloads
from tests._helpers import brute_effective_capacity, queue_instance, read_golden


def _hand():
    g = read_golden("hand_ceff.txt")
    inst = queue_instance(g["offsets"], g["demand"], g["feasible"], g["capacity"])
    return g, inst


def test_hand_worked_example():
    """Hand-derived values: componentwise minima taken from different
    configurations, a masked configuration ignored, pending-job mask."""
    g, inst = _hand()
    o = oracle.Oracle(inst)
    for gamma, queued, want in g["cases"]:
        got = o.effective_capacity(0, g["capacity"], gamma[0], np.array(queued, np.uint8))
        assert np.array_equal(got, np.array(want)), (gamma, queued, got)


def test_brute_force_exact_rationals():
    """Random ragged families with a feasibility mask and a pending mask,
    values spread over many binades: equal to the exact-rational
    computation rounded once."""
    for seed in range(6):
        rng = np.random.default_rng(seed)
        N, R = 40, 5
        sizes = rng.integers(1, 7, N)
        off = np.concatenate([[0], np.cumsum(sizes)])
        nnz = int(off[-1])
        dem = (rng.random((nnz, R)) * np.exp2(rng.integers(-30, 30, (nnz, R)))).astype(np.float32)
        dem[rng.random((nnz, R)) < 0.1] = 0.0
        feas = (rng.random(nnz) < 0.8).astype(np.uint8)
        for j in range(N):
            feas[off[j] + rng.integers(0, sizes[j])] = 1
        cap = rng.normal(0, 1e6, R)
        inst = queue_instance(off, dem, feas, cap)
        queued = (rng.random(N) < 0.7).astype(np.uint8)
        o = oracle.Oracle(inst)
        for gamma in (0.0, 0.3, 0.5, 1.0, float(rng.random())):
            for q in (None, queued):
                got = o.effective_capacity(0, cap, gamma, q)
                want = brute_effective_capacity(inst, 0, cap, gamma, q)
                assert np.array_equal(got, want), (seed, gamma)


def test_tiny_closed_form():
    """Tiny: every job has a 1-GPU configuration with 16 GB of host memory
    per GPU, so the GPU and host-memory minima are 1 and 16 for every job:
    C_eff = (64 - 64 gamma, ., ., 32768 - 1024 gamma)."""
    inst = workloads.make("tiny")
    o = oracle.Oracle(inst)
    for gamma in (0.0, 0.25, 0.5, 1.0):
        got = o.effective_capacity(0, inst.capacity[0], gamma)
        assert got[0] == 64.0 - 64.0 * gamma
        assert got[3] == 32768.0 - 1024.0 * gamma


def test_gamma_zero_and_empty_queue_keep_capacity():
    inst = workloads.make("small", n_jobs=300)
    o = oracle.Oracle(inst)
    cap = inst.capacity[0]
    assert np.array_equal(o.effective_capacity(0, cap, 0.0), cap)
    assert np.array_equal(o.effective_capacity(0, cap, 1.0, np.zeros(inst.N, np.uint8)), cap)


def test_monotone_in_gamma_and_queue():
    """More reservation never raises the capacity: C_eff is non-increasing in
    gamma and in the set of pending jobs (demands are non-negative)."""
    inst = workloads.make("ragged", n_jobs=2000)
    o = oracle.Oracle(inst)
    cap = inst.capacity[0]
    prev = cap.copy()
    for gamma in np.linspace(0, 1, 9):
        cur = o.effective_capacity(0, cap, gamma)
        assert np.all(cur <= prev)
        prev = cur
    rng = np.random.default_rng(1)
    q1 = (rng.random(inst.N) < 0.3).astype(np.uint8)
    q2 = q1 | (rng.random(inst.N) < 0.3).astype(np.uint8)
    assert np.all(o.effective_capacity(0, cap, 0.7, q2) <= o.effective_capacity(0, cap, 0.7, q1))


def test_single_config_families_subtract_their_demand():
    """K_j = 1: the minimum is the configuration itself, so with gamma = 1
    C_eff = C - exact sum of the demands (integers here: exact)."""
    rng = np.random.default_rng(2)
    N, R = 500, 4
    dem = rng.integers(0, 1000, (N, R)).astype(np.float32)
    cap = np.full(R, 1e7)
    inst = queue_instance(np.arange(N + 1), dem, None, cap)
    got = oracle.Oracle(inst).effective_capacity(0, cap, 1.0)
    assert np.array_equal(got, cap - dem.astype(np.float64).sum(axis=0))


def test_no_allowed_configuration_is_an_error():
    inst = queue_instance([0, 2], [[1.0], [2.0]], [0, 0], [5.0])
    with pytest.raises(ValueError):
        oracle.Oracle(inst).effective_capacity(0, [5.0], 0.5)


def test_warm_start_converges_faster_on_epoch_market():
    """On the unit-share epoch market, prices carried over from the previous
    epoch reach the stop tolerance in far fewer iterations than a cold start
    (the behaviour the paper reports for warm starts)."""
    act, que = workloads.epoch_market(4000)
    pend = workloads.epoch_pending(que.N, 3)
    qo = oracle.Oracle(que)
    lam = None
    for e in range(3):
        act.capacity = qo.effective_capacity(0, np.full(act.R, 4000.0), 0.5, pend[e])[None]
        o = oracle.Oracle(act)
        cold = o.solve(iters=1000, tol=1e-3, trace=False)
        warm = o.solve(lam0=cold["lam"] if lam is None else lam, iters=1000, tol=1e-3, trace=False)
        lam = warm["lam"].copy()
        assert cold["iters_done"][0] < 1000
        if e > 0:
            assert warm["iters_done"][0] * 3 < cold["iters_done"][0], (e, warm["iters_done"], cold["iters_done"])
