"""Parity at the full workload sizes, in the launch configuration bench.py
times (default options), on sampled iterations the oracle recomputes one by
one, plus properties of the whole GPU trajectory that hold at any size.

For a sampled iteration t the oracle starts from the GPU's own prices
lambda^t and recomputes the selection, the exact demand and lambda^{t+1};
choices must match bit for bit, U and lambda within 1e-9 relative (they are
bitwise equal)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _close(gpu, ref, rel=1e-9):
    gpu, ref = np.asarray(gpu), np.asarray(ref)
    return bool(np.all(np.abs(gpu - ref) <= rel * np.maximum(np.abs(gpu), np.abs(ref))))


def _update_identity(inst, lams, U, lam_next, b):
    """Eq. 8 recomputed in numpy (binary64, same operation order) from the
    GPU's own trace, for every iteration."""
    T = U.shape[0]
    for t in range(T):
        eta = oracle.eta(inst.rule, float(inst.eta0[b]), t + 1)
        x = lams[t] + eta * (U[t] - inst.capacity[b])
        assert np.array_equal(np.where(x > 0.0, x, 0.0), lam_next[t]), t


def _run(inst, trace_choice):
    s = esp.Solver(inst)                       # bench.py's launch configuration
    lam = s.prices(inst.lam0)
    g = s.solve(lam, inst.iters, trace=True, trace_choice=trace_choice)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    return s, g


@pytest.mark.parametrize("name", ["large", "ragged"])
def test_fullsize_single_cluster(name):
    inst = workloads.make(name)
    T = inst.iters
    _say(f"full-size {name}: N={inst.N} nnz={inst.nnz} R={inst.R} T={T}")
    s, g = _run(inst, trace_choice=True)
    tr_lam = g["tr_lam"][:, 0].cpu().numpy()
    tr_U = g["tr_U"][:, 0].cpu().numpy()
    lams = np.concatenate([inst.lam0[:1], tr_lam[:-1]], axis=0)
    _update_identity(inst, lams, tr_U, tr_lam, 0)
    o = oracle.Oracle(inst)
    for t in sorted({1, 2, 3, T // 2, T - 1, T}):
        ch, U, lam_next = o.step(0, lams[t - 1], t)
        assert np.array_equal(g["tr_choice"][t - 1, 0].cpu().numpy(), ch), t
        assert _close(tr_U[t - 1], U) and np.array_equal(tr_U[t - 1], U), t
        assert _close(tr_lam[t - 1], lam_next) and np.array_equal(tr_lam[t - 1], lam_next), t
    final = g["lam"][0].cpu().numpy()
    ch = o.select(0, final)
    assert np.array_equal(g["choice"][0].cpu().numpy(), ch)
    assert np.array_equal(g["U"][0].cpu().numpy(), o.demand_sum(0, ch))
    assert (g["iters_done"].cpu().numpy() == T).all()


def test_fullsize_batched():
    inst = workloads.make("batched")
    T = inst.iters
    _say(f"full-size batched: B={inst.B} N={inst.N} R={inst.R} T={T}")
    s, g = _run(inst, trace_choice=False)
    tr_lam = g["tr_lam"].cpu().numpy()
    tr_U = g["tr_U"].cpu().numpy()
    o = oracle.Oracle(inst)
    for b in (0, 1, 97, inst.B - 1):
        lams = np.concatenate([inst.lam0[b][None], tr_lam[:-1, b]], axis=0)
        _update_identity(inst, lams, tr_U[:, b], tr_lam[:, b], b)
        for t in (1, 2, T // 2, T):
            ch, U, lam_next = o.step(b, lams[t - 1], t)
            assert np.array_equal(tr_U[t - 1, b], U), (b, t)
            assert np.array_equal(tr_lam[t - 1, b], lam_next), (b, t)
        final = g["lam"][b].cpu().numpy()
        ch = o.select(b, final)
        assert np.array_equal(g["choice"][b].cpu().numpy(), ch), b
        assert np.array_equal(g["U"][b].cpu().numpy(), o.demand_sum(b, ch)), b


def test_fullsize_tiny_small_exhaustive():
    """The two small workloads at full size, every iterate against the
    free-running oracle."""
    for name in ("tiny", "small"):
        inst = workloads.make(name)
        _say(f"full-size {name} exhaustive")
        s, g = _run(inst, trace_choice=True)
        ref = oracle.Oracle(inst).solve(trace_choice=True)
        assert np.array_equal(g["tr_choice"].cpu().numpy(), ref["tr_choice"])
        assert np.array_equal(g["tr_U"].cpu().numpy(), ref["tr_U"])
        assert np.array_equal(g["tr_lam"].cpu().numpy(), ref["tr_lam"])
        assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
