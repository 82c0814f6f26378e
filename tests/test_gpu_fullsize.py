"""Parity at the full workload sizes, every iterate, in the launch
configuration bench.py times (default options), and every loop driver at
the full sizes.

The oracle runs free from lambda^1 (its own prices, never the GPU's) in
chunks of CHUNK iterations: a chunk continues the previous chunk's final
prices with the step index advanced, which reproduces the single long solve
(the continuation is one of the oracle's metamorphic pins).  Every iterate t
compares c^t bit for bit and U^t, lambda^{t+1} within 1e-9 relative; the
exact demand sum makes them bitwise equal, so equality is asserted too
(paper Sec. 3.2.3, Eq. 8 and the definition of U_r under it).

Each test prints a progress line per chunk, so a slow oracle is never taken
for a hang; the oracle runs in the test process itself, sequentially."""
import functools

import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads

pytestmark = pytest.mark.gpu

CHUNK = 100
REL = 1e-9


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _close(gpu, ref, rel=REL):
    gpu, ref = np.asarray(gpu), np.asarray(ref)
    return bool(np.all(np.abs(gpu - ref) <= rel * np.maximum(np.abs(gpu), np.abs(ref))))


@functools.lru_cache(maxsize=1)
def _instance(name):
    return workloads.make(name)


def _sub_instance(inst, clusters):
    """The clusters `clusters` of a batched instance as an instance of their
    own (clusters are independent problems)."""
    idx = np.asarray(clusters)
    return workloads.Instance(f"{inst.name}[{','.join(map(str, clusters))}]", inst.seed, inst.offsets,
                              inst.utility[idx], inst.demand[idx], inst.capacity[idx], inst.eta0[idx],
                              inst.rule, inst.lam0[idx], inst.iters, dense_k=inst.dense_k)


def _oracle_chunks(inst, T):
    """Free-running oracle: yields (i0, ref) where ref holds iterations
    i0 + 1 .. i0 + n (1-based t) and, for the last chunk, the re-selection
    at the final prices."""
    o = oracle.Oracle(inst)
    lam = np.array(inst.lam0, dtype=np.float64)
    for i0 in range(0, T, CHUNK):
        n = min(CHUNK, T - i0)
        ref = o.solve(lam0=lam, iters=n, t_start=i0 + 1, trace=True, trace_choice=True, duals=False)
        yield i0, ref
        lam = ref["lam"]


def _gpu_solve(inst, mode=esp.ESP_MODE_AUTO, trace_choice=True):
    s = esp.Solver(inst, mode=mode)
    g = s.solve(s.prices(inst.lam0), inst.iters, trace=True, trace_choice=trace_choice)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    return s, g


def _compare_every_iterate(name, g, inst, T, clusters=None):
    """g: GPU solve outputs (device); clusters: which of g's clusters make up
    `inst` (None: all, in order)."""
    sel = slice(None) if clusters is None else torch.as_tensor(clusters, device=g["tr_U"].device)
    tr_U = g["tr_U"][:, sel].cpu().numpy()
    tr_lam = g["tr_lam"][:, sel].cpu().numpy()
    ref = None
    for i0, ref in _oracle_chunks(inst, T):
        n = ref["tr_U"].shape[0]
        ch = g["tr_choice"][i0:i0 + n][:, sel].cpu().numpy()
        for i in range(n):
            t = i0 + i + 1
            assert np.array_equal(ch[i], ref["tr_choice"][i]), f"{name}: choices differ at t={t}"
            assert _close(tr_U[i0 + i], ref["tr_U"][i]), f"{name}: U differs at t={t}"
            assert _close(tr_lam[i0 + i], ref["tr_lam"][i]), f"{name}: lambda differs at t={t}"
        assert np.array_equal(tr_U[i0:i0 + n], ref["tr_U"]), name
        assert np.array_equal(tr_lam[i0:i0 + n], ref["tr_lam"]), name
        _say(f"{name}: iterations {i0 + 1}..{i0 + n} of {T} equal to the oracle")
    # re-selection at the final prices (Alg. 1)
    assert np.array_equal(g["choice"][sel].cpu().numpy(), ref["choice"]), name
    assert np.array_equal(g["U"][sel].cpu().numpy(), ref["U"]), name
    assert np.array_equal(g["lam"][sel].cpu().numpy(), ref["lam"]), name


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["large", "ragged"])
def test_fullsize_every_iterate(name):
    inst = _instance(name)
    T = inst.iters
    _say(f"full-size {name} every iterate: N={inst.N} nnz={inst.nnz} R={inst.R} T={T}")
    s, g = _gpu_solve(inst)
    assert s.loop_driver() == esp.ESP_MODE_STREAM           # bench.py's driver at this size
    assert (g["iters_done"].cpu().numpy() == T).all()
    _compare_every_iterate(name, g, inst, T)
    s.close()


def _graph_solve(s, inst, T):
    """esp_solve captured in a HIP graph (one launch per iteration), replayed
    twice with eager work between the replays; returns the second replay's
    outputs after checking that both replays agree."""
    lam0 = s.prices(inst.lam0)
    lam = lam0.clone()
    out = {
        "choice": torch.empty((s.B, s.N), dtype=torch.int32, device="cuda"),
        "U": torch.empty((s.B, s.R), dtype=torch.float64, device="cuda"),
        "tr_lam": torch.empty((T, s.B, s.R), dtype=torch.float64, device="cuda"),
        "tr_U": torch.empty((T, s.B, s.R), dtype=torch.float64, device="cuda"),
        "tr_choice": torch.empty((T, s.B, s.N), dtype=torch.int32, device="cuda"),
    }
    tr = esp.esp_trace(out["tr_lam"].data_ptr(), out["tr_U"].data_ptr(), out["tr_choice"].data_ptr())
    graph = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=stream):
        lam.copy_(lam0)
        esp.esp_solve(s.ctx, lam, T, 1, 0.0, out["choice"], out["U"], tr, None, torch.cuda.current_stream())
    first = None
    for rep in range(2):
        lam.fill_(7.0)                                      # eager work between the replays
        for v in out.values():
            v.fill_(-1)
        s.solve(s.prices(np.full((s.B, s.R), 0.05)), 3)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        if first is None:
            first = {k: v.clone() for k, v in out.items()}
            first["lam"] = lam.clone()
    for k, v in first.items():
        assert torch.equal(v, lam if k == "lam" else out[k]), f"graph replays differ in {k}"
    out["lam"] = lam
    return out


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name", ["large", "ragged"])
def test_fullsize_drivers_bitwise(name):
    """The persistent driver (cooperative launches of up to 1024 iterations)
    and graph replays of the per-iteration launches reproduce the stream
    driver's whole trajectory bit for bit at full size (the stream
    trajectory is the one checked against the oracle above)."""
    inst = _instance(name)
    T = inst.iters
    _say(f"full-size {name} drivers: stream")
    s, ref = _gpu_solve(inst, mode=esp.ESP_MODE_STREAM)
    keys = ("tr_choice", "tr_U", "tr_lam", "choice", "U", "lam")
    _say(f"full-size {name} drivers: persistent")
    p, g = _gpu_solve(inst, mode=esp.ESP_MODE_PERSISTENT)
    assert p.loop_driver() == esp.ESP_MODE_PERSISTENT
    for k in keys:
        assert torch.equal(g[k], ref[k]), f"{name}: persistent driver differs in {k}"
    assert (g["iters_done"].cpu().numpy() == T).all()
    del g
    p.close()
    _say(f"full-size {name} drivers: graph replay")
    g = _graph_solve(s, inst, T)
    for k in keys:
        assert torch.equal(g[k], ref[k]), f"{name}: graph replay differs in {k}"
    assert s.device_status() == 0
    s.close()


BATCHED_CLUSTERS = (0, 1, 37, 97, 128, 171, 200, 255)


@pytest.mark.timeout(900)
def test_fullsize_batched_every_iterate():
    """All 256 clusters solved in one launch per iteration (bench.py's
    configuration); every iterate of 8 clusters spread over the batch against
    the free-running oracle, and the Eq. 8 update of every cluster at every
    iterate recomputed from the GPU's own demand sums."""
    inst = _instance("batched")
    T = inst.iters
    _say(f"full-size batched: B={inst.B} N={inst.N} R={inst.R} T={T}")
    s, g = _gpu_solve(inst)
    assert (g["iters_done"].cpu().numpy() == T).all()
    sub = _sub_instance(inst, BATCHED_CLUSTERS)
    _compare_every_iterate("batched", g, sub, T, clusters=list(BATCHED_CLUSTERS))
    # the remaining clusters: Eq. 8 from the GPU's U^t, every iterate
    tr_lam = g["tr_lam"].cpu().numpy()
    tr_U = g["tr_U"].cpu().numpy()
    lam_prev = np.concatenate([inst.lam0[None], tr_lam[:-1]], axis=0)
    for t in range(1, T + 1):
        eta = np.array([oracle.eta(inst.rule, float(e), t) for e in inst.eta0])
        x = lam_prev[t - 1] + eta[:, None] * (tr_U[t - 1] - inst.capacity)
        assert np.array_equal(np.where(x > 0.0, x, 0.0), tr_lam[t - 1]), t
    s.close()


@pytest.mark.timeout(600)
def test_fullsize_batched_persistent_bitwise():
    """The persistent driver on all 256 clusters reproduces the stream
    driver's trajectory bit for bit."""
    inst = _instance("batched")
    _say("full-size batched drivers: stream vs persistent")
    s, ref = _gpu_solve(inst, mode=esp.ESP_MODE_STREAM, trace_choice=False)
    s.close()
    p, g = _gpu_solve(inst, mode=esp.ESP_MODE_PERSISTENT, trace_choice=False)
    for k in ("tr_U", "tr_lam", "choice", "U", "lam"):
        assert torch.equal(g[k], ref[k]), f"batched: persistent driver differs in {k}"
    p.close()


def test_fullsize_tiny_small_exhaustive():
    """The two small workloads at full size, every iterate against the
    free-running oracle."""
    for name in ("tiny", "small"):
        inst = workloads.make(name)
        _say(f"full-size {name} exhaustive")
        s, g = _gpu_solve(inst)
        ref = oracle.Oracle(inst).solve(trace_choice=True)
        assert np.array_equal(g["tr_choice"].cpu().numpy(), ref["tr_choice"])
        assert np.array_equal(g["tr_U"].cpu().numpy(), ref["tr_U"])
        assert np.array_equal(g["tr_lam"].cpu().numpy(), ref["tr_lam"])
        assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
        s.close()
