"""GPU parity of the resident driver (ESP_MODE_RESIDENT): tiles held in
registers for the whole launch, every iteration completed inside the launch;
with several workgroups per cluster their exact sums travel as tagged
48-bit limbs.  Every iterate against the free-running oracle (bitwise), over
one and many workgroups, dense and CSR tables, one to three limbs, several
clusters, penalties, staggered stops, and solves longer than one launch."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _wide(inst, seed, span):
    rng = np.random.default_rng(seed)
    inst.demand = (inst.demand.astype(np.float64) *
                   np.exp2(rng.integers(-span, span + 1, inst.demand.shape))).astype(np.float32)
    inst.eta0 = np.full(inst.B, 1e-12)
    return inst


CASES = {
    # name: (instance, blocks_per_cluster (0 = library default), T)
    "tiny_1wg": (lambda: workloads.make("tiny"), 0, 200),
    "small_128wg": (lambda: workloads.make("small"), 0, 500),
    "small_64wg_2tiles": (lambda: workloads.make("small"), 64, 120),
    "small_3wg_ragged_tail": (lambda: workloads.make("small", n_jobs=190), 3, 80),   # 24 tiles, last partial
    "ragged_3000_csr": (lambda: workloads.make("ragged", n_jobs=3000), 0, 120),
    "ragged_150_csr_1wg": (lambda: workloads.make("ragged", n_jobs=150), 1, 60),
    "batched_3x515": (lambda: workloads.make("batched", n_jobs=515, n_clusters=3), 0, 100),
    "k64_r8_dyadic": (lambda: workloads.random_small(7, 130, 64, 8, dense=True, dyadic=True, iters=80,
                                                     rule=workloads.STEP_CONST), 0, 80),
    "r1_k4": (lambda: workloads.random_small(5, 301, 4, 1, dense=True, iters=80), 0, 80),
    "wide_2limbs_k16": (lambda: _wide(workloads.random_small(90, 3000, 16, 5, dense=True, iters=60), 5, 12), 0, 60),
    "wide_3limbs_k16": (lambda: _wide(workloads.random_small(90, 3000, 16, 5, dense=True, iters=60), 5, 36), 0, 60),
    "wide_3limbs_csr_r8": (lambda: _wide(workloads.random_small(94, 1200, 40, 8, iters=60), 5, 36), 0, 60),
    "penalties_small": (lambda: workloads.with_penalties(workloads.make("small", n_jobs=2000), 9), 0, 100),
    "penalties_csr": (lambda: workloads.with_penalties(workloads.make("ragged", n_jobs=2500), 8), 0, 100),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_resident_every_iterate_matches_oracle(name):
    make, blocks, T = CASES[name]
    inst = make()
    _say(f"resident {name} B={inst.B} N={inst.N} R={inst.R} T={T} blocks={blocks}")
    s = esp.Solver(inst, mode=esp.ESP_MODE_RESIDENT, blocks_per_cluster=blocks)
    assert s.loop_driver() == esp.ESP_MODE_RESIDENT
    g = s.solve(s.prices(inst.lam0), T, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    ref = oracle.Oracle(inst).solve(iters=T, trace_choice=True)
    for t in range(T):
        assert np.array_equal(g["tr_choice"][t].cpu().numpy(), ref["tr_choice"][t]), f"choices at t={t + 1}"
    assert np.array_equal(g["tr_U"].cpu().numpy(), ref["tr_U"])
    assert np.array_equal(g["tr_lam"].cpu().numpy(), ref["tr_lam"])
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    assert np.array_equal(g["U"].cpu().numpy(), ref["U"])
    assert np.array_equal(g["lam"].cpu().numpy(), ref["lam"])
    assert (g["iters_done"].cpu().numpy() == T).all()
    s.close()


def test_auto_takes_the_resident_driver_for_small_tables():
    for name in ("tiny", "small"):
        inst = workloads.make(name)
        s = esp.Solver(inst)
        assert s.loop_driver() == esp.ESP_MODE_RESIDENT, name
        s.close()
    s = esp.Solver(workloads.make("large", n_jobs=20000))          # 46 MB, 5,000 tiles
    assert s.loop_driver() == esp.ESP_MODE_PERSISTENT
    s.close()


def _staggered():
    """Four clusters (94 tiles each) stopping after 1, 3, 108 and all 120
    updates under tol = 1e-3."""
    inst = workloads.random_small(31, 1500, 16, 3, dense=True, n_clusters=4, iters=120, eta0=0.02)
    inst.eta0 = np.array([1e-5, 4e-5, 1e-3, 0.05], dtype=np.float64)
    return inst


def _tiny_tol():
    inst = workloads.make("tiny")
    inst.eta0 = np.array([0.05])
    return inst


@pytest.mark.parametrize("case,blocks", [("staggered", 12), ("staggered", 24), ("tiny", 1)])
def test_resident_stops_under_tol(case, blocks):
    inst = _staggered() if case == "staggered" else _tiny_tol()
    ref = oracle.Oracle(inst).solve(tol=1e-3, trace=True)
    n = [int(x) for x in ref["iters_done"]]
    if case == "staggered":
        assert n == [1, 3, 108, 120]
    _say(f"resident stops under tol: {case} blocks={blocks} stops={n}")
    s = esp.Solver(inst, mode=esp.ESP_MODE_RESIDENT, blocks_per_cluster=blocks)
    g = s.solve(s.prices(inst.lam0), inst.iters, tol=1e-3, trace=True)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    tl, tu = g["tr_lam"].cpu().numpy(), g["tr_U"].cpu().numpy()
    for b, k in enumerate(n):
        assert np.array_equal(tl[:k, b], ref["tr_lam"][:k, b]), b
        assert np.array_equal(tu[:k, b], ref["tr_U"][:k, b]), b
        assert np.isnan(tl[k:, b]).all(), b
    assert np.array_equal(g["iters_done"].cpu().numpy(), ref["iters_done"])
    assert np.array_equal(g["lam"].cpu().numpy(), ref["lam"])
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    s.close()


def test_resident_solve_longer_than_one_launch_and_warm_start():
    """1,100 iterations on Small: two resident launches (1,024 + 76), the
    second starting from the prices the first wrote; and the same solve split
    in two esp_solve calls (t_start)."""
    inst = workloads.make("small")
    T = 1100
    _say(f"resident T={T} small, and split at 600")
    ref = oracle.Oracle(inst).solve(iters=T, trace=True)
    s = esp.Solver(inst, mode=esp.ESP_MODE_RESIDENT)
    g = s.solve(s.prices(inst.lam0), T, trace=True)
    torch.cuda.synchronize()
    assert np.array_equal(g["tr_lam"].cpu().numpy(), ref["tr_lam"])
    assert np.array_equal(g["tr_U"].cpu().numpy(), ref["tr_U"])
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    lam = s.prices(inst.lam0)
    a = s.solve(lam, 600, trace=True)
    b = s.solve(lam, 500, t_start=601, trace=True)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a["tr_lam"], b["tr_lam"]]), g["tr_lam"])
    assert torch.equal(b["choice"], g["choice"])
    assert s.device_status() == 0
    s.close()


def test_resident_under_capture_is_refused():
    inst = workloads.make("tiny")
    s = esp.Solver(inst, mode=esp.ESP_MODE_RESIDENT)
    lam = s.prices(inst.lam0)
    graph = torch.cuda.CUDAGraph()
    codes = []
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=torch.cuda.Stream()):
        lam.mul_(1.0)
        try:
            esp.esp_solve(s.ctx, lam, 10, 1, 0.0, None, None, None, None, torch.cuda.current_stream())
        except esp.EspError as e:
            codes.append(e.code)
    assert codes == [esp.ESP_ERR_INVALID_ARG]
    s.close()
