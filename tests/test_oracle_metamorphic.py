"""Exact metamorphic relations of the oracle (Sec. 3.2.2-3.2.3).

Scaling by powers of two commutes with binary64 rounding (no overflow or
subnormals here), the exact demand sum does not depend on job order, and a
duplicate configuration at a higher index can never win a tie.  Each relation
is checked bitwise on whole traces."""
import numpy as np
import pytest

import oracle
import workloads


def _inst(seed, **kw):
    kw.setdefault("iters", 40)
    return workloads.random_small(seed, 24, 7, 4, **kw)


def _run(inst, **kw):
    return oracle.Oracle(inst).solve(trace_choice=True, **kw)


@pytest.mark.parametrize("a", [-3, 5])
def test_scale_utility_prices_step(a):
    """u * 2^a, eta0 * 2^a, lambda^1 * 2^a: identical choices, prices * 2^a."""
    base = _inst(11)
    base.lam0 = np.full((1, base.R), 0.25)
    s = 2.0 ** a
    sc = _inst(11)
    sc.utility = (base.utility * np.float32(s)).astype(np.float32)
    sc.eta0 = base.eta0 * s
    sc.lam0 = base.lam0 * s
    r0, r1 = _run(base), _run(sc)
    assert np.array_equal(r0["tr_choice"], r1["tr_choice"])
    assert np.array_equal(r0["tr_lam"] * s, r1["tr_lam"])
    assert np.array_equal(r0["tr_U"], r1["tr_U"])


@pytest.mark.parametrize("bexp", [-2, 3])
def test_scale_demand_capacity(bexp):
    """d * 2^b, C * 2^b, lambda^1 * 2^-b, eta0 * 2^-2b: identical choices,
    prices * 2^-b, demand sums * 2^b."""
    base = _inst(12)
    base.lam0 = np.full((1, base.R), 0.5)
    s = 2.0 ** bexp
    sc = _inst(12)
    sc.demand = (base.demand * np.float32(s)).astype(np.float32)
    sc.capacity = base.capacity * s
    sc.lam0 = base.lam0 / s
    sc.eta0 = base.eta0 / (s * s)
    r0, r1 = _run(base), _run(sc)
    assert np.array_equal(r0["tr_choice"], r1["tr_choice"])
    assert np.array_equal(r0["tr_lam"] / s, r1["tr_lam"])
    assert np.array_equal(r0["tr_U"] * s, r1["tr_U"])


def test_job_permutation():
    """Permuting jobs permutes choices; demand sums and prices are bitwise
    unchanged (the aggregate demand is an exact sum)."""
    base = _inst(13)
    rng = np.random.default_rng(0)
    perm = rng.permutation(base.N)
    off = base.offsets
    ent = np.concatenate([np.arange(off[j], off[j + 1]) for j in perm])
    sizes = (off[1:] - off[:-1])[perm]
    p = _inst(13)
    p.offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    p.utility = base.utility[:, ent]
    p.demand = base.demand[:, ent]
    r0, r1 = _run(base), _run(p)
    assert np.array_equal(r0["tr_choice"][:, :, perm], r1["tr_choice"])
    assert np.array_equal(r0["tr_lam"], r1["tr_lam"])
    assert np.array_equal(r0["tr_U"], r1["tr_U"])


def test_duplicate_configs_never_win():
    """Appending a copy of every configuration after the family changes
    nothing: a copy ties its original and the lower index wins."""
    base = _inst(14)
    off = base.offsets
    ent = np.concatenate([np.concatenate([np.arange(off[j], off[j + 1])] * 2) for j in range(base.N)])
    d = _inst(14)
    d.offsets = off * 2
    d.utility = base.utility[:, ent]
    d.demand = base.demand[:, ent]
    r0, r1 = _run(base), _run(d)
    assert np.array_equal(r0["tr_choice"], r1["tr_choice"])
    assert np.array_equal(r0["tr_lam"], r1["tr_lam"])


def test_identical_jobs_choose_alike():
    inst = _inst(15, dense=True)
    inst.utility[0] = np.tile(inst.utility[0, :7], inst.N)
    inst.demand[0] = np.tile(inst.demand[0, :7], (inst.N, 1))
    r = _run(inst)
    assert (r["tr_choice"][:, 0] == r["tr_choice"][:, 0, :1]).all()


def test_feasibility_mask_equals_removal():
    """Eq. 4: a configuration with T_j(c) < L_j is never selected.  Masking it
    gives the same trajectory as deleting it (choices mapped back to the
    original family index)."""
    base = _inst(16)
    rng = np.random.default_rng(1)
    off = base.offsets
    mask = (rng.random(base.nnz) < 0.7).astype(np.uint8)
    for j in range(base.N):
        if not mask[off[j]:off[j + 1]].any():
            mask[off[j] + rng.integers(0, off[j + 1] - off[j])] = 1
    masked = _inst(16)
    masked.feasible = mask[None]
    keep = np.flatnonzero(mask)
    sizes = np.array([mask[off[j]:off[j + 1]].sum() for j in range(base.N)])
    rem = _inst(16)
    rem.offsets = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    rem.utility = base.utility[:, keep]
    rem.demand = base.demand[:, keep]
    r_m, r_r = _run(masked), _run(rem)
    assert np.array_equal(r_m["tr_lam"], r_r["tr_lam"])
    for j in range(base.N):
        orig = np.flatnonzero(mask[off[j]:off[j + 1]])
        assert np.array_equal(orig[r_r["tr_choice"][:, 0, j]], r_m["tr_choice"][:, 0, j])
    # an empty family is an error
    masked.feasible = masked.feasible.copy()
    masked.feasible[0, off[3]:off[4]] = 0
    with pytest.raises(ValueError):
        oracle.Oracle(masked).solve(iters=2)


def test_warm_start_equals_one_run():
    """Checkpoint/resume of prices: T iterations equal T1 iterations followed
    by T - T1 more started at t = T1 + 1 from the saved prices, bitwise."""
    inst = _inst(17, iters=60)
    full = _run(inst)
    a = oracle.Oracle(inst).solve(iters=25, trace_choice=True)
    b = oracle.Oracle(inst).solve(lam0=a["lam"], iters=35, t_start=26, trace_choice=True)
    assert np.array_equal(np.concatenate([a["tr_lam"], b["tr_lam"]]), full["tr_lam"])
    assert np.array_equal(np.concatenate([a["tr_choice"], b["tr_choice"]]), full["tr_choice"])
    assert np.array_equal(b["choice"], full["choice"])


def test_early_stop_rule():
    """With tol > 0 the loop stops after the first update whose price change
    is within tol * max(1, lambda) on every resource."""
    inst = workloads.random_small(18, 10, 5, 2, iters=500, eta0=0.02)
    tol = 1e-3
    full = oracle.Oracle(inst).solve()
    st = oracle.Oracle(inst).solve(tol=tol)
    n = int(st["iters_done"][0])
    lams = np.concatenate([inst.lam0, full["tr_lam"][:, 0]], axis=0)
    conv = [bool(np.all(np.abs(lams[t + 1] - lams[t]) <= tol * np.maximum(1.0, lams[t])))
            for t in range(inst.iters)]
    assert n == (conv.index(True) + 1 if True in conv else inst.iters)
    assert np.array_equal(st["lam"][0], lams[n])
    assert np.array_equal(st["tr_lam"][:n], full["tr_lam"][:n])


def test_clusters_are_independent():
    """B clusters solve as B separate problems (per-cluster prices, capacity
    and step size)."""
    both = workloads.random_small(19, 9, 5, 3, n_clusters=3, iters=30)
    both.eta0 = np.array([0.01, 0.05, 0.1])
    rb = _run(both)
    for b in range(3):
        one = workloads.random_small(19, 9, 5, 3, iters=30)
        one.utility = both.utility[b:b + 1]
        one.demand = both.demand[b:b + 1]
        one.capacity = both.capacity[b:b + 1]
        one.eta0 = both.eta0[b:b + 1]
        r1 = _run(one)
        assert np.array_equal(r1["tr_lam"][:, 0], rb["tr_lam"][:, b])
        assert np.array_equal(r1["tr_choice"][:, 0], rb["tr_choice"][:, b])
