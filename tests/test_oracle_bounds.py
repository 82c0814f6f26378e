"""Oracle pins from the mathematics of the Lagrangian dual (Sec. 3.2.2, Eq. 6)
and the projected-subgradient update (Eq. 8), checked against brute force,
an LP solver and exact rational arithmetic on tiny instances."""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads
from tests._helpers import brute_force_optimum, exact_score, lp_optimum

TINY_SEEDS = list(range(8))


def _eps(inst, lam, b=0):
    scale = float(np.abs(inst.utility[b]).sum()) + float(np.abs(lam) @ np.abs(inst.capacity[b]))
    return 1e-9 * (1.0 + scale)


def _lams(res, inst, b=0):
    """lambda^t for t = 1..T (lambda^1 = lam0)."""
    return np.concatenate([inst.lam0[b][None], res["tr_lam"][:-1, b]], axis=0)


@pytest.mark.parametrize("seed", TINY_SEEDS)
def test_weak_duality_and_lp_sandwich(seed):
    """g(lambda) >= LP* >= P* for every lambda >= 0 (weak duality of the
    relaxation of Eq. 3); min_t g(lambda^t) approaches LP* as T grows with
    eta0/sqrt(t) steps (textbook subgradient-method convergence)."""
    inst = workloads.random_small(seed, 6, 5, 3, dyadic=(seed % 2 == 0), iters=400, eta0=0.1)
    P, _ = brute_force_optimum(inst)
    LP = lp_optimum(inst)
    res = oracle.Oracle(inst).solve()
    lams = _lams(res, inst)
    duals = res["tr_dual"][:, 0]
    assert P is not None
    assert float(P) <= LP + 1e-9 * (1 + abs(LP))
    for t in range(inst.iters):
        assert duals[t] >= LP - _eps(inst, lams[t]), (t, duals[t], LP)
    gap_early = duals[:20].min() - LP
    gap_late = duals.min() - LP
    assert gap_late <= max(0.5 * gap_early, 1e-6 * (1 + abs(LP)))


@pytest.mark.parametrize("seed", TINY_SEEDS)
def test_dual_value_is_the_max_of_the_lagrangian(seed):
    """g(lambda^t) computed at the oracle's selection equals the brute-force
    maximum of the Lagrangian (Eq. 6) over all selections, exactly."""
    inst = workloads.random_small(100 + seed, 5, 4, 2, dyadic=True, iters=30, eta0=0.125,
                                  rule=workloads.STEP_CONST)
    res = oracle.Oracle(inst).solve(trace_choice=True)
    lams = _lams(res, inst)
    off = inst.offsets
    for t in (0, 5, 29):
        lam = lams[t]
        best = Fraction(0)
        for j in range(inst.N):
            best += max(exact_score(inst, 0, e, lam) for e in range(off[j], off[j + 1]))
        best += sum(Fraction(float(lam[r])) * Fraction(float(inst.capacity[0, r]))
                    for r in range(inst.R))
        assert abs(float(best) - res["tr_dual"][t, 0]) <= _eps(inst, lam)


@pytest.mark.parametrize("seed", TINY_SEEDS)
def test_per_job_choice_is_exact_argmax(seed):
    """Each job's choice maximises its exact (rational) reduced utility up to
    a 2^-40 relative band, and is the lowest index among configurations whose
    exact score equals the best (Sec. 3.2.2 subproblem, lowest-index ties)."""
    inst = workloads.random_small(200 + seed, 20, 8, 4, iters=60, eta0=0.05)
    res = oracle.Oracle(inst).solve(trace_choice=True)
    lams = _lams(res, inst)
    off = inst.offsets
    for t in (0, 1, 7, 59):
        lam = lams[t]
        for j in range(inst.N):
            scores = [exact_score(inst, 0, e, lam) for e in range(off[j], off[j + 1])]
            c = int(res["tr_choice"][t, 0, j])
            best = max(scores)
            mag = abs(Fraction(float(inst.utility[0, off[j] + c]))) + sum(
                Fraction(float(lam[r])) * Fraction(float(inst.demand[0, off[j] + c, r]))
                for r in range(inst.R))
            assert best - scores[c] <= mag * Fraction(1, 2 ** 40)
            if scores[c] == best:
                assert c == scores.index(best)


@pytest.mark.parametrize("seed", TINY_SEEDS)
def test_ergodic_feasibility_identity(seed):
    """Summing Eq. 8 over t: sum_t eta_t (U^t - C) <= lambda^{T+1} - lambda^1,
    with equality for a resource that was never clamped at zero."""
    inst = workloads.random_small(300 + seed, 15, 6, 3, iters=200, eta0=0.05)
    res = oracle.Oracle(inst).solve()
    lams = _lams(res, inst)
    T = inst.iters
    etas = np.array([oracle.eta(inst.rule, inst.eta0[0], t) for t in range(1, T + 1)])
    for r in range(inst.R):
        lhs = math.fsum(etas[t] * (res["tr_U"][t, 0, r] - inst.capacity[0, r]) for t in range(T))
        rhs = res["lam"][0, r] - inst.lam0[0, r]
        tol = 1e-12 * (T + 1) * (1 + abs(rhs) + math.fsum(abs(etas * (res["tr_U"][:, 0, r] - inst.capacity[0, r]))))
        assert lhs <= rhs + tol
        raw = lams + etas[:, None] * (res["tr_U"][:, 0] - inst.capacity[0])
        if (raw[:, r] > 0).all():
            assert abs(lhs - rhs) <= tol


def test_tiny_config_complementary_slackness():
    """Tiny workload (64 jobs on 64 GPUs): GPU demands are integers and the
    only feasible selections put every job on one GPU.  Once that happens,
    U_gpu = C_gpu exactly and the GPU price stops moving bitwise (Eq. 8 with
    zero excess).  The integer optimum is then sum_j max over one-GPU configs,
    valid because the other resources are slack there; every dual value bounds
    it from above."""
    inst = workloads.make("tiny")
    res = oracle.Oracle(inst).solve(trace_choice=True)
    off, K = inst.offsets, 8
    g1 = [k for k in range(K) if inst.demand[0, k, 0] == 1.0]
    assert g1 == [0, 4]
    # the closed-form optimum over one-GPU configurations
    sel = [off[j] + max(g1, key=lambda k: (inst.utility[0, off[j] + k], -k)) for j in range(inst.N)]
    use = inst.demand[0, sel].astype(np.float64).sum(axis=0)
    assert use[0] == 64.0 and (use[1:] <= inst.capacity[0, 1:]).all()
    P = math.fsum(float(inst.utility[0, e]) for e in sel)
    assert (res["tr_dual"][:, 0] >= P - 1e-9 * P).all()
    on_g1 = [t for t in range(inst.iters) if res["tr_U"][t, 0, 0] == 64.0]
    assert on_g1, "the GPU resource never became exactly tight"
    lams = _lams(res, inst)
    for t in on_g1:
        assert res["tr_lam"][t, 0, 0] == lams[t][0]


@pytest.mark.parametrize("name", ["large", "batched"])
def test_infeasible_resources_price_grows(name):
    """Capacities below the all-minimum demand (Large: 60% of it; Batched:
    16,384 jobs on <= 1024 GPUs): every price rises by at least
    eta_t (sum_j min_k d_jkr - C_r) > 0 at every iteration (Eq. 8)."""
    inst = workloads.make(name, n_jobs=512) if name == "large" else \
        workloads.make(name, n_jobs=512, n_clusters=2)
    res = oracle.Oracle(inst).solve(iters=25)
    K = inst.dense_k
    for b in range(inst.B):
        d = inst.demand[b].reshape(inst.N, K, inst.R).astype(np.float64)
        smin = np.array([math.fsum(d[:, :, r].min(axis=1)) for r in range(inst.R)])
        lams = _lams(res, inst, b)
        for t in range(25):
            eta = oracle.eta(inst.rule, inst.eta0[b], t + 1)
            if name == "large":
                assert (smin > inst.capacity[b]).all()
            inc = res["tr_lam"][t, b] - lams[t]
            over = smin > inst.capacity[b]
            assert (inc[over] >= eta * (smin - inst.capacity[b])[over] * (1 - 1e-12)).all()
            assert (inc[over] > 0).all()
