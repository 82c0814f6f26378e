"""Pins of the oracle's outer ESP-IAC rounds (Sec. 3.4, Alg. 1; Eq. 11):
first-fit BinPack, co-located pairs against the adaptive thresholds, penalty
updates for the offending configurations, and the round loop."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads
from tests._helpers import check_first_fit, schedule_fixture


def test_hand_worked_example():
    inst, m, results = schedule_fixture()
    o = oracle.Oracle(inst)
    for M, nr, V, ch, g0, g1, pen in results:
        r = o.schedule(0, m, int(M[0]), inst.iters)
        assert r["rounds"] == int(nr[0]) and r["violations"] == int(V[0])
        assert list(r["choice"]) == [int(x) for x in ch]
        assert list(r["occ"][0]) == [int(x) for x in g0] and list(r["occ"][1]) == [int(x) for x in g1]
        assert list(r["penalty"]) == pen
        assert np.array_equal(r["lam"], np.zeros(3))


def test_gamma_starts_from_zero():
    """Alg. 1 resets the interference penalties before its first round: a
    schedule started from any penalties equals one started from none."""
    inst, m, results = schedule_fixture()
    inst.penalty = np.array([[0.5, 2.0, 1.0, 0.25]], np.float32)
    o = oracle.Oracle(inst)
    for M, nr, V, ch, g0, g1, pen in results:
        r = o.schedule(0, m, int(M[0]), inst.iters)
        assert r["rounds"] == int(nr[0]) and list(r["penalty"]) == pen


def _instances():
    yield workloads.make("tiny"), 0
    yield workloads.make("small", n_jobs=600), 0
    b = workloads.make("batched", n_jobs=600, n_clusters=2)
    yield b, 0
    yield b, 1


def test_binpack_is_first_fit():
    for inst, b in _instances():
        m = workloads.iac_model(inst)
        o = oracle.Oracle(inst)
        for lam in (np.zeros(inst.R), np.full(inst.R, 1e-3), np.full(inst.R, 0.05)):
            ch = o.select(b, lam)
            occ, placed = o.binpack(b, m, ch)
            check_first_fit(inst, b, m, ch, occ)
            assert placed == sum(int(inst.demand[b, inst.offsets[j] + ch[j], 0]) for j in set(occ[occ >= 0].tolist()))


def _exact_pairs(inst, b, m, ch, occ):
    """Violating pairs and the largest excess per job, in exact rationals."""
    G = int(m.gpus[b])
    used = sum(1 for h in range(G) if occ[h][0] >= 0)
    add = Fraction(m.beta) * (Fraction(used, G) / Fraction(m.u_target) - 1)
    add = min(add, Fraction(m.beta_max))
    V, inc = 0, {}
    for h in range(G):
        js = [int(j) for j in occ[h] if j >= 0]
        for x in range(len(js)):
            for y in range(x + 1, len(js)):
                jx, jy = js[x], js[y]
                ex, ey = inst.offsets[jx] + ch[jx], inst.offsets[jy] + ch[jy]
                sxy = 1 + Fraction(float(m.sensitivity[b, ex])) * Fraction(float(m.pressure[b, ey]))
                syx = 1 + Fraction(float(m.sensitivity[b, ey])) * Fraction(float(m.pressure[b, ex]))
                ox = sxy - (Fraction(float(m.tau_base[b, jx])) + add)
                oy = syx - (Fraction(float(m.tau_base[b, jy])) + add)
                if ox > 0:
                    inc[jx] = max(inc.get(jx, 0), ox)
                if oy > 0:
                    inc[jy] = max(inc.get(jy, 0), oy)
                V += (ox > 0 or oy > 0)
    return V, inc


def test_iac_pairs_match_exact_rationals():
    """Violations and excesses against exact-rational recomputation (the
    binary64 values differ from the exact ones by a few ulps; no excess in
    these inputs lies within 1e-12 of zero)."""
    total = 0
    for inst, b in _instances():
        m = workloads.iac_model(inst)
        o = oracle.Oracle(inst)
        r = o.schedule(b, m, 1, 40)                  # the first round's selection and packing
        ch, occ = r["choice"], r["occ"]
        V, inc = o.iac_eval(b, m, ch, occ)
        Vx, incx = _exact_pairs(inst, b, m, ch, occ)
        assert V == Vx == r["violations"]
        total += V
        for j in range(inst.N):
            want = float(incx.get(j, 0))
            assert abs(inc[j] - want) <= 1e-14 * max(1.0, abs(want)), j
    assert total > 0


def test_no_sensitivity_means_one_round():
    """a = 0: no pair can exceed a threshold >= 1, so Alg. 1 stops after one
    round with no penalty, at the plain tatonnement's prices and choice."""
    inst = workloads.make("small", n_jobs=500)
    m = workloads.iac_model(inst)
    m.sensitivity = np.zeros_like(m.sensitivity)
    o = oracle.Oracle(inst)
    r = o.schedule(0, m, 3, 60)
    plain = o.solve(iters=60, trace=False)
    assert r["rounds"] == 1 and r["violations"] == 0 and not r["penalty"].any()
    assert np.array_equal(r["lam"], plain["lam"][0]) and np.array_equal(r["choice"], plain["choice"][0])


def test_whole_gpu_configurations_never_share():
    """Every configuration uses a whole GPU's compute: no GPU holds two
    jobs, so there is no pair and no violation."""
    inst = workloads.make("tiny")
    inst.demand = inst.demand.copy()
    inst.demand[0, :, 2] = inst.demand[0, :, 0]              # compute share g * 1
    m = workloads.iac_model(inst)
    r = oracle.Oracle(inst).schedule(0, m, 3, 50)
    assert r["rounds"] == 1 and r["violations"] == 0
    assert (r["occ"][:, 1] == -1).all()


def test_penalties_grow_only_on_offending_choices():
    """Per round, Gamma rises exactly at the chosen configurations of jobs
    with a positive excess (by kappa * excess, rounded to fp32) and nowhere
    else; the loop ends at the first round without violations."""
    inst = workloads.make("small", n_jobs=600)
    m = workloads.iac_model(inst)
    o = oracle.Oracle(inst)
    prev = np.zeros(inst.nnz, np.float32)
    for M in (1, 2, 3):
        r = o.schedule(0, m, M, 80)
        if r["rounds"] < M:
            assert r["violations"] == 0
            break
        diff = np.nonzero(r["penalty"] != prev)[0]
        # replay the last round's evaluation
        occ, ch = r["occ"], r["choice"]
        V, inc = o.iac_eval(0, m, ch, occ)
        assert V == r["violations"]
        want = {int(inst.offsets[j] + ch[j]) for j in range(inst.N) if inc[j] > 0}
        assert set(diff.tolist()) == want
        for e in want:
            j = int(np.searchsorted(inst.offsets, e, side="right") - 1)
            assert r["penalty"][e] == np.float32(float(prev[e]) + m.kappa * inc[j])
        assert (r["penalty"] >= prev).all()
        prev = r["penalty"]
