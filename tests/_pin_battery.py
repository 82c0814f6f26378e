"""Run a compact battery of oracle pins against one oracle library build.

Usage: python -m tests._pin_battery <path-to-liboracle.so>
Exit status 0 when every pin passes, 1 when any fails.  Used to show that
plausible mistakes planted in a copy of the oracle are caught."""
import math
import sys
import traceback
from fractions import Fraction

import numpy as np

import oracle
import workloads
from tests._helpers import (brute_effective_capacity, check_first_fit, exact_score, exact_sq_dist, golden_instance,
                           lp_optimum, queue_instance, read_golden, schedule_fixture, store_instance)


def battery(L) -> None:
    # hand-derived traces (Sec. 3.2.2 argmax, Eq. 8 update)
    for name in ("hand_r1_tie.txt", "hand_r2.txt", "hand_projection.txt", "hand_penalty.txt"):
        g = read_golden(name)
        res = oracle.Oracle(golden_instance(g), L).solve(trace_choice=True)
        for i, row in enumerate(g["trace"]):
            assert list(res["tr_choice"][i, 0]) == [int(x) for x in row[2]]
            assert np.array_equal(res["tr_U"][i, 0], np.array(row[3]))
            assert np.array_equal(res["tr_lam"][i, 0], np.array(row[4]))
            assert res["tr_dual"][i, 0] == row[5][0]
        assert list(res["choice"][0]) == [int(x) for x in g["final_choice"]]
        for x in res["tr_lam"].ravel():
            assert math.copysign(1.0, x) > 0
    # early stop (hand_tol.txt): where a tolerance stops the loop
    g = read_golden("hand_tol.txt")
    o = oracle.Oracle(golden_instance(g), L)
    res = o.solve(tol=g["tol"][0], trace_choice=True)
    assert int(res["iters_done"][0]) == int(g["iters_done"][0])
    for i, row in enumerate(g["trace"]):
        assert np.array_equal(res["tr_lam"][i, 0], np.array(row[4]))
    assert np.array_equal(res["lam"][0], np.array(g["final_lam"]))
    for tol, n, lam in g["cases"]:
        r = o.solve(tol=tol[0])
        assert int(r["iters_done"][0]) == int(n[0]) and np.array_equal(r["lam"][0], np.array(lam))
    # step sizes
    assert oracle.eta(1, 0.01, 1, L) == 0.01 and oracle.eta(1, 1.0, 4, L) == 0.5
    assert oracle.eta(0, 0.3, 7, L) == 0.3
    # exact sums against math.fsum
    rng = np.random.default_rng(5)
    for _ in range(10):
        v = (rng.random(500) * np.exp2(rng.integers(-140, 120, 500))).astype(np.float32)
        assert oracle.exact_sum_f32(v, L) == math.fsum(float(x) for x in v)
    assert oracle.exact_sum_f32(np.array([2.0 ** 53, 1.0], np.float32), L) == 2.0 ** 53
    assert oracle.exact_sum_f32(np.array([2.0 ** 53, 2.0, 1.0], np.float32), L) == 2.0 ** 53 + 4
    # exact per-job optimality and LP weak duality on random instances,
    # without and with the penalty of Eq. 7
    for seed in (3, 4, 5):
        inst = workloads.random_small(seed, 6, 5, 3, iters=40, eta0=0.1)
        if seed == 5:
            workloads.with_penalties(inst, seed)
        res = oracle.Oracle(inst, L).solve(trace_choice=True)
        lams = np.concatenate([inst.lam0, res["tr_lam"][:-1, 0]], axis=0)
        LP = lp_optimum(inst)
        off = inst.offsets
        for t in (0, 3, 39):
            assert res["tr_dual"][t, 0] >= LP - 1e-7
            for j in range(inst.N):
                sc = [exact_score(inst, 0, e, lams[t]) for e in range(off[j], off[j + 1])]
                c = int(res["tr_choice"][t, 0, j])
                assert sc[c] == max(sc) and c == sc.index(max(sc))
            U = res["tr_U"][t, 0]
            for r in range(inst.R):
                vals = [float(inst.demand[0, off[j] + res["tr_choice"][t, 0, j], r]) for j in range(inst.N)]
                assert U[r] == math.fsum(vals)
    # effective capacity (Eq. 12): hand example and exact rationals
    g = read_golden("hand_ceff.txt")
    q = queue_instance(g["offsets"], g["demand"], g["feasible"], g["capacity"])
    for gamma, queued, want in g["cases"]:
        got = oracle.Oracle(q, L).effective_capacity(0, g["capacity"], gamma[0], np.array(queued, np.uint8))
        assert np.array_equal(got, np.array(want))
    rng = np.random.default_rng(9)
    sizes = rng.integers(1, 6, 30)
    off = np.concatenate([[0], np.cumsum(sizes)])
    dem = (rng.random((int(off[-1]), 3)) * np.exp2(rng.integers(-20, 20, (int(off[-1]), 3)))).astype(np.float32)
    q = queue_instance(off, dem, None, [1e3, -5.0, 0.0])
    pend = (rng.random(30) < 0.6).astype(np.uint8)
    got = oracle.Oracle(q, L).effective_capacity(0, q.capacity[0], 0.3, pend)
    assert np.array_equal(got, brute_effective_capacity(q, 0, q.capacity[0], 0.3, pend))
    # nearest-profile fallback: hand example (with and without a masked entry)
    # and exact-rational optimality on a random store
    g = read_golden("hand_nearest.txt")
    for mask, key in ((None, "querys"), (g["masked"], "masked_querys")):
        o = oracle.Oracle(store_instance(g["offsets"], g["utility"], g["demand"], mask), L)
        for fam, qv, k, est in g[key]:
            kk, ee = o.nearest_batch(0, [int(fam[0])], [qv])
            assert kk[0] == int(k[0])
            assert (math.isnan(ee[0]) and math.isnan(est[0])) or ee[0] == est[0]
    rng = np.random.default_rng(11)
    sizes = rng.integers(1, 12, 25)
    off = np.concatenate([[0], np.cumsum(sizes)])
    dem = (rng.random((int(off[-1]), 4)) * np.exp2(rng.integers(-8, 8, 4))).astype(np.float32)
    o = oracle.Oracle(store_instance(off, rng.random(int(off[-1])), dem), L)
    for _ in range(100):
        f = int(rng.integers(0, 25))
        qv = (rng.random(4) * np.exp2(rng.integers(-8, 8, 4))).astype(np.float32)
        k = o.nearest(0, f, qv)[0]
        ex = [exact_sq_dist(qv, dem[e]) for e in range(off[f], off[f + 1])]
        assert ex[k] <= min(ex) * (1 + 2.0 ** -40)
    # outer rounds of Alg. 1: hand example, first fit, pairs and penalties
    inst, m, results = schedule_fixture()
    inst.penalty = np.array([[0.5, 2.0, 1.0, 0.25]], np.float32)      # reset by Alg. 1's first step
    o = oracle.Oracle(inst, L)
    for M, nr, V, ch, g0, g1, pen in results:
        r = o.schedule(0, m, int(M[0]), inst.iters)
        assert r["rounds"] == int(nr[0]) and r["violations"] == int(V[0])
        assert list(r["choice"]) == [int(x) for x in ch]
        assert list(r["occ"][0]) == [int(x) for x in g0] and list(r["occ"][1]) == [int(x) for x in g1]
        assert list(r["penalty"]) == pen
    inst = workloads.make("small", n_jobs=600)
    m = workloads.iac_model(inst)
    o = oracle.Oracle(inst, L)
    ch = o.select(0, np.full(inst.R, 0.05))
    occ, _ = o.binpack(0, m, ch)
    check_first_fit(inst, 0, m, ch, occ)
    from tests.test_oracle_schedule import _exact_pairs
    r1 = o.schedule(0, m, 1, 40)
    ch, occ = r1["choice"], r1["occ"]
    check_first_fit(inst, 0, m, ch, occ)
    V, inc = o.iac_eval(0, m, ch, occ)
    Vx, incx = _exact_pairs(inst, 0, m, ch, occ)
    assert V == Vx and V > 0
    for j in range(inst.N):
        assert abs(inc[j] - float(incx.get(j, 0))) <= 1e-14
    r2 = o.schedule(0, m, 2, 40)
    assert r1["violations"] == V
    if r1["violations"]:
        V1, inc1 = o.iac_eval(0, m, r1["choice"], r1["occ"])
        for j in range(inst.N):
            e = inst.offsets[j] + r1["choice"][j]
            want = np.float32(m.kappa * inc1[j]) if inc1[j] > 0 else np.float32(0)
            assert r1["penalty"][e] == want
        assert r2["rounds"] == 2


def main(path: str) -> int:
    try:
        battery(oracle.bind(path))
    except Exception:                       # any failed pin
        traceback.print_exc(limit=2)
        return 1
    return 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1]))
