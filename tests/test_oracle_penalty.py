"""Oracle pins for the penalty Gamma of the ESP score (Eq. 7, Sec. 3.2.3):
a switching cost for leaving the current configuration and a per-
configuration interference penalty, both subtracted after the rent."""
import numpy as np
import pytest

import oracle
import workloads
from tests._helpers import brute_force_optimum, exact_score, golden_instance, lp_optimum, read_golden


def _run(inst, **kw):
    return oracle.Oracle(inst).solve(trace_choice=True, **kw)


def test_hand_trace_primal_values():
    g = read_golden("hand_penalty.txt")
    inst = golden_instance(g)
    o = oracle.Oracle(inst)
    assert o.primal_value(0, [0]) == g["primal"][0]
    assert o.primal_value(0, [1]) == g["primal"][1]


def test_zero_penalty_is_the_plain_method():
    """Gamma = 0 (zero switching cost, zero penalties, or no current
    configuration) leaves the trajectory bitwise unchanged."""
    base = workloads.random_small(61, 30, 8, 3, iters=60)
    ref = _run(base)
    for variant in range(3):
        p = workloads.random_small(61, 30, 8, 3, iters=60)
        workloads.with_penalties(p, 61)
        if variant == 0:
            p.switch_cost[:] = 0.0
            p.penalty[:] = 0.0
        elif variant == 1:
            p.current[:] = -1
            p.penalty[:] = 0.0
        else:
            p.switch_cost[:] = 0.0
            p.penalty = None
        r = _run(p)
        assert np.array_equal(r["tr_choice"], ref["tr_choice"])
        assert np.array_equal(r["tr_lam"], ref["tr_lam"])


def test_dyadic_penalty_equals_utility_shift():
    """With dyadic values the subtraction is exact in either order, so a
    penalty p_jk gives the same trajectory as the utility u_jk - p_jk."""
    a = workloads.random_small(62, 40, 8, 3, dyadic=True, iters=80, rule=workloads.STEP_CONST, eta0=0.125)
    workloads.with_penalties(a, 62, switch_cost=0.0, dyadic=True)
    a.current[:] = -1
    b = workloads.random_small(62, 40, 8, 3, dyadic=True, iters=80, rule=workloads.STEP_CONST, eta0=0.125)
    shifted = a.utility.astype(np.float64) - a.penalty.astype(np.float64)
    assert np.array_equal(shifted.astype(np.float32).astype(np.float64), shifted)
    b.utility = shifted.astype(np.float32)
    ra, rb = _run(a), _run(b)
    assert np.array_equal(ra["tr_choice"], rb["tr_choice"])
    assert np.array_equal(ra["tr_lam"], rb["tr_lam"])


def test_prohibitive_switching_cost_keeps_current_configs():
    """gamma_0 far above any utility or rent difference: every job with a
    current configuration keeps it, so U is constant and lambda follows the
    K = 1 recursion of Eq. 8."""
    inst = workloads.random_small(63, 50, 10, 4, iters=40)
    workloads.with_penalties(inst, 63, switch_cost=1e12, frac_current=1.0)
    r = _run(inst)
    assert (r["tr_choice"][:, 0] == inst.current[0]).all()
    assert (r["tr_U"][:, 0] == r["tr_U"][0, 0]).all()


@pytest.mark.parametrize("seed", range(5))
def test_penalized_bounds_and_optimality(seed):
    """Weak duality and per-job exact optimality with the penalised objective."""
    inst = workloads.random_small(700 + seed, 6, 5, 3, iters=150, eta0=0.1)
    workloads.with_penalties(inst, 700 + seed, switch_cost=0.3, penalty_scale=0.5)
    P, _ = brute_force_optimum(inst)
    LP = lp_optimum(inst)
    res = _run(inst)
    lams = np.concatenate([inst.lam0, res["tr_lam"][:-1, 0]], axis=0)
    assert P is None or float(P) <= LP + 1e-9
    for t in range(inst.iters):
        assert res["tr_dual"][t, 0] >= LP - 1e-9 * (1 + abs(LP) + np.abs(lams[t]).sum() * 10)
    off = inst.offsets
    for t in (0, 10, 149):
        for j in range(inst.N):
            sc = [exact_score(inst, 0, e, lams[t], j) for e in range(off[j], off[j + 1])]
            c = int(res["tr_choice"][t, 0, j])
            assert sc[c] == max(sc) and c == sc.index(max(sc))
