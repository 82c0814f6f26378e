"""Pins of the oracle's nearest-profile fallback (RST, Sec. 3.1.2 and
Sec. 4.1): within the query's job-type family, the allowed entry closest in
l2 distance, lowest index among equal distances, and its throughput."""
import math

import numpy as np
import pytest

import oracle
import workloads
from tests._helpers import exact_sq_dist, read_golden, store_instance


def _hand(masked=False):
    g = read_golden("hand_nearest.txt")
    inst = store_instance(g["offsets"], g["utility"], g["demand"], g["masked"] if masked else None)
    return g, oracle.Oracle(inst)


def test_hand_worked_example():
    g, o = _hand()
    for fam, q, k, est in g["querys"]:
        got_k, _ = o.nearest(0, int(fam[0]), q)
        assert got_k == int(k[0]), (fam, q)
        kk, ee = o.nearest_batch(0, [int(fam[0])], [q])
        assert kk[0] == int(k[0])
        assert (math.isnan(ee[0]) and math.isnan(est[0])) or ee[0] == est[0]


def test_hand_masked_entry_is_not_a_candidate():
    g, o = _hand(masked=True)
    for fam, q, k, est in g["masked_querys"]:
        kk, ee = o.nearest_batch(0, [int(fam[0])], [q])
        assert kk[0] == int(k[0]) and ee[0] == est[0]


def _random_store(seed, n_fam=60, max_k=20, R=5, spread=30):
    rng = np.random.default_rng(seed)
    sizes = rng.integers(1, max_k + 1, n_fam)
    off = np.concatenate([[0], np.cumsum(sizes)])
    nnz = int(off[-1])
    scale = np.exp2(rng.integers(-spread, spread, R))
    dem = (rng.random((nnz, R)) * scale).astype(np.float32)
    util = rng.random(nnz).astype(np.float32)
    return store_instance(off, util, dem), rng, scale


def test_exact_rational_optimality():
    """The chosen entry's exact squared distance is the exact minimum up to
    a 2^-40 relative band (where binary64 rounding may reorder near-equal
    distances); outside any such band it is the unique exact minimiser."""
    for seed in range(5):
        inst, rng, scale = _random_store(seed)
        o = oracle.Oracle(inst)
        off = inst.offsets
        for _ in range(150):
            f = int(rng.integers(0, inst.N))
            q = (rng.random(inst.R) * scale).astype(np.float32)
            k, _ = o.nearest(0, f, q)
            ex = [exact_sq_dist(q, inst.demand[0, e]) for e in range(off[f], off[f + 1])]
            m = min(ex)
            assert ex[k] <= m * (1 + 2.0 ** -40) + 0, (seed, f)
            if sum(1 for x in ex if x <= m * (1 + 2.0 ** -40)) == 1:
                assert ex[k] == m


def test_query_equal_to_an_entry_finds_its_first_duplicate():
    inst, rng, _ = _random_store(7)
    o = oracle.Oracle(inst)
    off = inst.offsets
    for f in range(inst.N):
        e = int(rng.integers(off[f], off[f + 1]))
        q = inst.demand[0, e]
        k, d2 = o.nearest(0, f, q)
        first = next(i for i in range(off[f], off[f + 1]) if np.array_equal(inst.demand[0, i], q))
        assert d2 == 0.0 and k == first - off[f]


def test_one_dimension_matches_sorted_search():
    """R = 1 with integer values: the nearest entry of a sorted family is one
    of the two bracketing values found by bisection (ties to the lower
    value, which has the lower index)."""
    rng = np.random.default_rng(3)
    vals = np.sort(rng.choice(10000, 200, replace=False)).astype(np.float32)
    inst = store_instance([0, 200], np.arange(200), vals.reshape(200, 1))
    o = oracle.Oracle(inst)
    for qv in rng.integers(-50, 10050, 500):
        i = int(np.searchsorted(vals, qv))
        cands = [c for c in (i - 1, i) if 0 <= c < 200]
        want = min(cands, key=lambda c: (abs(float(vals[c]) - qv), c))
        assert o.nearest(0, 0, [qv])[0] == want


def test_metamorphic_translation_scaling_permutation():
    """Integer data: translating every vector and the query by the same
    integer vector, scaling all by a power of two, or permuting the
    resources leaves every answer unchanged (all exact)."""
    rng = np.random.default_rng(4)
    sizes = rng.integers(1, 15, 40)
    off = np.concatenate([[0], np.cumsum(sizes)])
    nnz = int(off[-1])
    dem = rng.integers(0, 64, (nnz, 4)).astype(np.float32)
    util = rng.random(nnz).astype(np.float32)
    qs = rng.integers(0, 64, (300, 4)).astype(np.float32)
    fam = rng.integers(0, 40, 300).astype(np.int32)
    base = oracle.Oracle(store_instance(off, util, dem)).nearest_batch(0, fam, qs)[0]
    shift = np.array([7, 100, 3, 55], np.float32)
    perm = np.array([2, 0, 3, 1])
    for d2, q2 in ((dem + shift, qs + shift), (dem * 8, qs * 8), (dem[:, perm], qs[:, perm])):
        got = oracle.Oracle(store_instance(off, util, d2)).nearest_batch(0, fam, q2)[0]
        assert np.array_equal(got, base)


def test_family_out_of_range():
    g, o = _hand()
    k, est = o.nearest_batch(0, [-1, 2, 99], np.zeros((3, 2)))
    assert list(k) == [-1, -1, -1] and np.isnan(est).all()
