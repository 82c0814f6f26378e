"""Oracle pins against hand-derived traces, closed forms and library routines.

Each fixture under tests/golden/ was derived by hand from Sec. 3.2.2 (per-job
argmax) and Eq. 8 (Sec. 3.2.3); its header gives the derivation.
"""
import math
import struct

import numpy as np
import pytest

import oracle
import workloads
from tests._helpers import brute_force_optimum, golden_instance, read_golden


def _bits(x: float) -> int:
    return struct.unpack("<Q", struct.pack("<d", x))[0]


@pytest.mark.parametrize("name", ["hand_r1_tie.txt", "hand_r2.txt", "hand_projection.txt", "hand_penalty.txt"])
def test_hand_trace(name):
    g = read_golden(name)
    inst = golden_instance(g)
    o = oracle.Oracle(inst)
    res = o.solve(trace_choice=True)
    R = inst.R
    lam = np.array(inst.lam0[0])
    for i, row in enumerate(g["trace"]):
        t, lam_t, ch, U, lam_next, dual = row
        assert int(t[0]) == i + 1
        assert np.array_equal(lam, np.array(lam_t)), (i, lam, lam_t)
        assert list(res["tr_choice"][i, 0]) == [int(x) for x in ch], (i, res["tr_choice"][i, 0], ch)
        assert np.array_equal(res["tr_U"][i, 0], np.array(U)), (i, res["tr_U"][i, 0], U)
        assert np.array_equal(res["tr_lam"][i, 0], np.array(lam_next)), (i, res["tr_lam"][i, 0])
        assert res["tr_dual"][i, 0] == dual[0], (i, res["tr_dual"][i, 0], dual)
        lam = res["tr_lam"][i, 0]
    assert list(res["choice"][0]) == [int(x) for x in g["final_choice"]]
    assert np.array_equal(res["U"][0], np.array(g["final_U"]))
    assert np.array_equal(res["lam"][0], np.array(g["final_lam"]))
    # a stored price is never -0.0 (projection onto lambda >= 0 of Eq. 8)
    for x in list(res["tr_lam"].ravel()) + list(res["lam"].ravel()):
        assert _bits(x) >> 63 == 0
    assert R == len(g["final_lam"])


def test_hand_trace_steps_match_single_step_api():
    """The loop equals repeated select/demand/update (Sec. 3.2.3)."""
    g = read_golden("hand_r2.txt")
    inst = golden_instance(g)
    o = oracle.Oracle(inst)
    lam = inst.lam0[0].copy()
    for t, row in enumerate(g["trace"], start=1):
        ch, U, lam = o.step(0, lam, t)
        assert list(ch) == [int(x) for x in row[2]]
        assert np.array_equal(lam, np.array(row[4]))


def test_eta_rules_closed_forms():
    """Eq. 8 step sizes: eta0 fixed, or eta0/sqrt(t) with t = 1, 2, ..."""
    assert oracle.eta(workloads.STEP_CONST, 0.3, 1) == 0.3
    assert oracle.eta(workloads.STEP_CONST, 0.3, 999) == 0.3
    assert oracle.eta(workloads.STEP_INV_SQRT, 0.01, 1) == 0.01      # t is 1-based
    assert oracle.eta(workloads.STEP_INV_SQRT, 1.0, 4) == 0.5
    assert oracle.eta(workloads.STEP_INV_SQRT, 3.0, 9) == 1.0
    assert oracle.eta(workloads.STEP_INV_SQRT, 1.0, 1 << 40) == 2.0 ** -20
    # correctly rounded IEEE division and square root (Python floats are binary64)
    for t in (2, 3, 5, 7, 10, 1000, 123457):
        assert oracle.eta(workloads.STEP_INV_SQRT, 0.01, t) == 0.01 / math.sqrt(t)


def test_single_config_closed_form_inv_sqrt():
    """K_j = 1 for every job: the selection never changes, U is constant and
    lambda^{T+1} = lambda^1 + (U - C) sum_t eta0/sqrt(t) while U > C (Eq. 8)."""
    N, R, T = 5, 3, 50
    u = np.ones((1, N), np.float32)
    d = np.tile(np.array([1.0, 2.0, 0.5], np.float32), (N, 1))[None]
    cap = np.array([[4.0, 9.0, 1.0]])
    inst = workloads.Instance("k1", 0, workloads.uniform_offsets(N, 1), u, d, cap, np.array([1.0]),
                              workloads.STEP_INV_SQRT, np.zeros((1, R)), T)
    res = oracle.Oracle(inst).solve()
    assert (res["choice"] == 0).all()
    U = np.array([5.0, 10.0, 2.5])
    assert np.array_equal(res["tr_U"][:, 0], np.tile(U, (T, 1)))
    # first step uses eta_1 = eta0 exactly
    assert np.array_equal(res["tr_lam"][0, 0], U - cap[0])
    s = math.fsum(1.0 / math.sqrt(t) for t in range(1, T + 1))
    expect = (U - cap[0]) * s
    assert np.allclose(res["lam"][0], expect, rtol=T * 2.0 ** -52, atol=0)


def test_zero_price_fixed_point():
    """lambda^1 = 0 and the utility-maximising selection fits: prices stay
    +0.0 bitwise and every job keeps argmax_k u_jk (lowest index on ties)."""
    inst = workloads.random_small(7, 12, 6, 3)
    best = np.array([int(np.argmax(inst.utility[0, inst.offsets[j]:inst.offsets[j + 1]]))
                     for j in range(inst.N)])
    used = np.array([inst.demand[0, inst.offsets[j] + best[j]] for j in range(inst.N)],
                    dtype=np.float64).sum(axis=0)
    inst.capacity = (used + 1.0)[None]
    res = oracle.Oracle(inst).solve(iters=20, trace_choice=True)
    assert (res["tr_choice"][:, 0] == best).all()
    for x in res["tr_lam"].ravel():
        assert _bits(x) == 0
    assert np.array_equal(res["choice"][0], best)


def test_exact_sum_matches_fsum():
    """Aggregate demand is the exact sum rounded once; Python's math.fsum is a
    correctly rounded float sum, so the two agree on every input."""
    rng = np.random.default_rng(123)
    cases = [
        rng.random(1000).astype(np.float32),
        (rng.random(4000) * np.exp2(rng.integers(-149, 127, 4000))).astype(np.float32),
        np.full(777, 0.1, np.float32),
        np.array([2.0 ** 100, 2.0 ** -100, 1.0, 2.0 ** -149], np.float32),
        np.array([3.4028235e38] * 64, np.float32),
        np.array([1.0, 2.0 ** -24, 2.0 ** -24], np.float32),             # tie cases
        np.array([1.0] + [2.0 ** -54] * 3, np.float32),
        np.array([2.0 ** 53, 1.0], np.float32),
        np.array([2.0 ** 53, 1.0, 2.0 ** -60], np.float32),
        np.array([], np.float32),
        np.array([0.0, -0.0], np.float32),
        (rng.integers(1, 9, 100000)).astype(np.float32),
    ]
    for _ in range(20):
        n = int(rng.integers(1, 3000))
        lo, hi = sorted(rng.integers(-149, 128, 2))
        cases.append((rng.random(n) * np.exp2(rng.integers(lo, hi + 1, n))).astype(np.float32))
    for v in cases:
        assert oracle.exact_sum_f32(v) == math.fsum(float(x) for x in v)
    # closed forms
    assert oracle.exact_sum_f32(np.full(3, 2.0 ** -149, np.float32)) == 3 * 2.0 ** -149
    assert oracle.exact_sum_f32(np.array([2.0 ** 53, 1.0], np.float32)) == 2.0 ** 53      # tie to even
    assert oracle.exact_sum_f32(np.array([2.0 ** 53, 1.0, 2.0 ** -60], np.float32)) == 2.0 ** 53 + 2
    assert oracle.exact_sum_f32(np.array([2.0 ** 53, 2.0, 1.0], np.float32)) == 2.0 ** 53 + 4


def test_case1_reshaping_selection():
    """Paper Sec. 5.3 Case 1: the price on GPU memory steers BERT to
    checkpointing (24 GB) and ResNet-50 to AMP (14 GB), 38 GB of 40 GB.
    Utilities are assumed (the paper gives none)."""
    g = read_golden("case1_bert_resnet.txt")
    u = np.array([g["assumed_bert_utility"] + g["assumed_resnet_utility"]], np.float32)
    d = np.array(g["bert_gb"] + g["resnet_gb"], np.float32).reshape(1, 4, 1)
    cap = np.array([g["capacity_gb"]])
    inst = workloads.Instance("case1", 0, np.array([0, 2, 4]), u, d, cap, np.array([5e-4]),
                              workloads.STEP_CONST, np.zeros((1, 1)), 30)
    best, arg = brute_force_optimum(inst)
    assert arg == (1, 1)
    res = oracle.Oracle(inst).solve(trace_choice=True)
    feas = [i for i in range(inst.iters) if res["tr_U"][i, 0, 0] <= cap[0]]
    assert feas, "ESP never reached a feasible selection"
    first = feas[0]
    assert list(res["tr_choice"][first, 0]) == [1, 1]
    assert res["tr_U"][first, 0, 0] == g["fit_gb"][0]
    assert res["tr_primal"][first, 0] == float(best)


def test_case2_memory_price_rises_under_overload():
    """Paper Sec. 5.3 Case 2: under GPU-memory overload the memory price rises
    (Eq. 8) until the jobs move to lower-memory configurations.  Memory
    footprints follow the ranges of Table 2 (ResNet-50 12-24, BERT 24-36,
    PPO 8-24, NCF 4-16 GB) on two 40 GB GPUs; utilities are assumed."""
    mem = [[24, 18, 12], [36, 30, 24], [24, 16, 8], [16, 10, 4]]
    u = np.array([[1.0, 0.9, 0.8] * 4], np.float32)
    d = np.array(mem, np.float32).reshape(1, 12, 1)
    inst = workloads.Instance("case2", 0, workloads.uniform_offsets(4, 3), u, d, np.array([[80.0]]),
                              np.array([2e-3]), workloads.STEP_CONST, np.zeros((1, 1)), 40)
    res = oracle.Oracle(inst).solve(trace_choice=True)
    lam = np.concatenate([[0.0], res["tr_lam"][:, 0, 0]])
    U = res["tr_U"][:, 0, 0]
    over = U > 80.0
    assert over[0]
    for i in range(inst.iters):
        if over[i]:
            assert lam[i + 1] > lam[i]
        else:
            assert lam[i + 1] <= lam[i]
    first_fit = int(np.argmax(~over))
    assert not over[first_fit]
    assert (res["tr_choice"][first_fit, 0] > 0).any()      # some job moved off its peak config


def test_hand_tol_stop_rule():
    """The early-stop reading (hand_tol.txt): the oracle stops after the
    first update where every resource's price change is within tol times
    max(1, the pre-update price), reports that many updates, re-selects at
    the prices reached, and leaves the later trace rows untouched."""
    g = read_golden("hand_tol.txt")
    inst = golden_instance(g)
    o = oracle.Oracle(inst)
    res = o.solve(tol=g["tol"][0], trace_choice=True)
    done = int(g["iters_done"][0])
    assert int(res["iters_done"][0]) == done
    for i, row in enumerate(g["trace"]):
        t, lam_t, ch, U, lam_next, dual, flags = row
        assert np.array_equal(res["tr_U"][i, 0], np.array(U)), i
        assert np.array_equal(res["tr_lam"][i, 0], np.array(lam_next)), i
        assert res["tr_dual"][i, 0] == dual[0], i
        # the stop test of the reading, from the fixture's own prices
        ok = [abs(b - a) <= g["tol"][0] * max(1.0, a) for a, b in zip(lam_t, lam_next)]
        assert ok == [bool(x) for x in flags], i
    assert np.isnan(res["tr_lam"][done:]).all() and np.isnan(res["tr_U"][done:]).all()
    assert list(res["choice"][0]) == [int(x) for x in g["final_choice"]]
    assert np.array_equal(res["U"][0], np.array(g["final_U"]))
    assert np.array_equal(res["lam"][0], np.array(g["final_lam"]))
    for tol, n, lam in g["cases"]:
        r = o.solve(tol=tol[0])
        assert int(r["iters_done"][0]) == int(n[0]), tol
        assert np.array_equal(r["lam"][0], np.array(lam)), tol
    # tol = 0 runs every iteration
    assert int(o.solve(tol=0.0)["iters_done"][0]) == inst.iters
