"""GPU parity of RST's nearest-profile fallback (Sec. 3.1.2, Sec. 4.1)
through the C-ABI against the oracle: the nearest index is an integer
decided by binary64 distances computed in the same order on both sides, so
indices and estimates must be bit-exact.  Every case runs on both layouts of
the store: the structure-of-arrays columns and the entry-major copy
(ESP_OPT_PROFILE_STORE)."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads
from tests._helpers import read_golden, store_instance

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _run(store_solver, fam, q):
    n, e = store_solver.nearest_profile(torch.from_numpy(np.ascontiguousarray(fam)).cuda(),
                                        torch.from_numpy(np.ascontiguousarray(q)).cuda())
    torch.cuda.synchronize()
    return n.cpu().numpy(), e.cpu().numpy()


LAYOUTS = {"soa": 0, "aos": esp.ESP_OPT_PROFILE_STORE}


def _check(store, fam, q):
    o = oracle.Oracle(store)
    want = [o.nearest_batch(b, fam[b], q[b]) for b in range(store.B)]
    for name, flags in LAYOUTS.items():
        s = esp.Solver(store, flags=flags)
        n, e = _run(s, fam, q)
        for b, (k, est) in enumerate(want):
            assert np.array_equal(n[b], k), (name, b)
            assert np.array_equal(e[b].view(np.uint32), est.view(np.uint32)), (name, b)
        assert s.device_status() == 0
        s.close()


def test_hand_example_on_gpu():
    g = read_golden("hand_nearest.txt")
    _say("nearest hand example")
    for mask, key in ((None, "querys"), (g["masked"], "masked_querys")):
        store = store_instance(g["offsets"], g["utility"], g["demand"], mask)
        rows = [r for r in g[key] if 0 <= int(r[0][0]) < store.N]
        fam = np.array([[int(r[0][0]) for r in rows]], np.int32)
        q = np.array([[r[1] for r in rows]], np.float32)
        for flags in LAYOUTS.values():
            s = esp.Solver(store, flags=flags)
            n, e = _run(s, fam, q)
            assert list(n[0]) == [int(r[2][0]) for r in rows]
            assert list(e[0]) == [r[3][0] for r in rows]
            s.close()


STORES = {
    "csr_r6_ragged": lambda: workloads.make("ragged", n_jobs=3000),
    "csr_r3_masked": lambda: _masked(workloads.random_small(21, 900, 30, 3), 1),
    "csr_r8_batched": lambda: workloads.random_small(22, 400, 70, 8, n_clusters=3),
    "dense_k4_r1": lambda: workloads.random_small(23, 700, 4, 1, dense=True),
    "dense_k16_r5": lambda: workloads.random_small(24, 500, 16, 5, dense=True, n_clusters=2),
    "dense_k64_r8": lambda: _masked(workloads.random_small(25, 200, 64, 8, dense=True), 2),
    "tiny": lambda: workloads.make("tiny"),
    "csr_r8_long_families": lambda: _long_families(27, 8),
    "csr_r2_long_families": lambda: _long_families(28, 2),
}


def _long_families(seed, R):
    """Families from 1 to 256 configurations (the longest runs of the
    entry-major copy: 72 lines at R = 8), sizes that fill whole lines, more
    job types than one directory record holds."""
    rng = np.random.default_rng(seed)
    sizes = rng.choice([1, 2, 31, 32, 33, 64, 127, 128, 255, 256], 185)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    nnz = int(off[-1])
    return store_instance(off, rng.random(nnz), rng.random((nnz, R)).astype(np.float32))


def _masked(inst, seed):
    rng = np.random.default_rng(seed)
    f = (rng.random((inst.B, inst.nnz)) >= 0.3).astype(np.uint8)
    off = inst.offsets
    for b in range(inst.B):
        for j in range(inst.N):
            if not f[b, off[j]:off[j + 1]].any():
                f[b, off[j]] = 1
    inst.feasible = f
    return inst


@pytest.mark.parametrize("name", sorted(STORES))
def test_nearest_matches_oracle(name):
    store = STORES[name]()
    _say(f"nearest {name}: B={store.B} N={store.N} R={store.R} nnz={store.nnz}")
    fam, q = workloads.nn_queries(store, 5000, seed=7)
    _check(store, fam, q)


def test_small_integer_grid_has_many_ties():
    """Integer vectors on a coarse grid: many exactly equal distances, so
    the lowest-index rule decides most queries."""
    rng = np.random.default_rng(5)
    sizes = rng.integers(1, 200, 50)
    off = np.concatenate([[0], np.cumsum(sizes)])
    dem = rng.integers(0, 4, (int(off[-1]), 3)).astype(np.float32)
    store = store_instance(off, rng.random(int(off[-1])), dem)
    fam = rng.integers(0, 50, (1, 4000)).astype(np.int32)
    q = rng.integers(0, 4, (1, 4000, 3)).astype(np.float32) + 0.5 * rng.integers(0, 2, (1, 4000, 3))
    _say("nearest integer grid ties")
    _check(store, fam, q.astype(np.float32))


@pytest.mark.parametrize("layout", sorted(LAYOUTS))
def test_bad_queries_are_reported(layout):
    store = workloads.random_small(26, 100, 8, 3)
    s = esp.Solver(store, flags=LAYOUTS[layout])
    fam = np.array([[0, -1, 100, 5, 7]], np.int32)
    q = np.ones((1, 5, 3), np.float32)
    q[0, 3, 1] = np.nan
    q[0, 4, 2] = np.inf
    _say(f"nearest bad queries ({layout})")
    n, e = _run(s, fam, q)
    assert list(n[0, 1:]) == [-1, -1, -1, -1] and np.isnan(e[0, 1:]).all()
    assert n[0, 0] == oracle.Oracle(store).nearest(0, 0, q[0, 0])[0]
    assert s.device_status() != 0
    assert s.device_status() == 0                       # cleared by the read
    assert esp.lib().esp_nearest_profile(s.ctx, -1, None, None, None, None, None) == esp.ESP_ERR_INVALID_ARG
    assert esp.lib().esp_nearest_profile(s.ctx, 0, None, None, None, None, None) == esp.ESP_OK


def test_fullsize_ragged_store():
    """The Ragged table (1,048,576 job types, Geometric(0.08) families,
    R = 6) as the profile store, 1,048,576 queries in the launch
    configuration bench.py times: every answer equal to the oracle's."""
    store = workloads.make("ragged")
    fam, q = workloads.nn_queries(store, 1 << 20, seed=9)
    _say("nearest full-size ragged store, 1M queries")
    _check(store, fam, q)
