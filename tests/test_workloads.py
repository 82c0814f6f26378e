"""Seeded synthetic instances: determinism, shapes and the stated structure."""
import numpy as np
import pytest

import workloads
from workloads import _uniform


def test_counter_rng_is_random_access():
    idx = np.arange(1000, dtype=np.int64)
    full = _uniform(7, 3, idx)
    assert np.array_equal(full[[5, 999, 0]], _uniform(7, 3, np.array([5, 999, 0])))
    assert not np.array_equal(full, _uniform(8, 3, idx))
    assert ((full >= 0) & (full < 1)).all()
    assert abs(full.mean() - 0.5) < 0.05


@pytest.mark.parametrize("name,kw,shape", [
    ("tiny", {}, (1, 64, 8, 4)),
    ("small", {}, (1, 4096, 32, 4)),
    ("large", {"n_jobs": 1024}, (1, 1024, 64, 8)),
    ("batched", {"n_jobs": 256, "n_clusters": 3}, (3, 256, 64, 6)),
])
def test_dense_shapes_and_determinism(name, kw, shape):
    a, b = workloads.make(name, **kw), workloads.make(name, **kw)
    assert a.fingerprint() == b.fingerprint()
    B, N, K, R = shape
    assert (a.B, a.N, a.R, a.dense_k) == (B, N, R, K)
    assert a.utility.dtype == np.float32 and a.demand.dtype == np.float32
    assert a.utility.shape == (B, N * K) and a.demand.shape == (B, N * K, R)
    assert np.isfinite(a.utility).all() and np.isfinite(a.demand).all()
    assert (a.demand >= 0).all()
    assert a.capacity.shape == (B, R) and a.eta0.shape == (B,)
    assert (a.lam0 == 0).all()


def test_tiny_structure():
    t = workloads.make("tiny")
    d = t.demand[0].reshape(64, 8, 4)
    assert (d[:, :, 0] == np.array([1, 2, 4, 8, 1, 2, 4, 8])).all()
    assert (d[:, :, 3] == 16 * d[:, :, 0]).all()
    assert set(np.unique(d[:, :, 2] / d[:, :, 0])) <= {0.5, 1.0}
    assert np.array_equal(t.capacity[0], [64, 5120, 64, 32768])
    assert t.iters == 200 and t.rule == workloads.STEP_INV_SQRT and t.eta0[0] == 0.01


def test_large_capacity_is_sixty_percent_of_min_demand():
    L = workloads.make("large", n_jobs=2048)
    d = L.demand[0].reshape(2048, 64, 8).astype(np.float64)
    assert np.allclose(L.capacity[0], 0.6 * d.min(axis=1).sum(axis=0), rtol=1e-12)
    assert L.iters == 1000


def test_ragged_family_sizes():
    r = workloads.make("ragged", n_jobs=200000)
    K = np.diff(r.offsets)
    assert K.min() >= 1 and K.max() <= 256
    assert abs(K.mean() - 12.5) < 0.2                      # Geometric(p = 0.08) mean
    dd = r.demand[0].astype(np.float64)
    smin = np.minimum.reduceat(dd, r.offsets[:-1], axis=0).sum(axis=0)
    smax = np.maximum.reduceat(dd, r.offsets[:-1], axis=0).sum(axis=0)
    assert (r.capacity[0] >= smin).all() and (r.capacity[0] <= smax).all()
    assert r.R == 6 and r.iters == 300


def test_batched_cluster_parameters():
    b = workloads.make("batched", n_jobs=128, n_clusters=16)
    G = b.capacity[:, 0]
    assert ((G >= 256) & (G <= 1024)).all() and np.array_equal(G, np.floor(G))
    assert set(b.eta0) <= {0.005, 0.01, 0.02}
    assert np.array_equal(b.capacity[:, 1], 80 * G)
