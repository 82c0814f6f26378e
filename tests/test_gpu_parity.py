"""GPU parity: the HIP path through the C-ABI against the CPU oracle.

Choices must be bit-exact; demand sums and prices must agree within 1e-9
relative (they are in fact bitwise equal: both sides round the exact demand
sum once).  Every case prints its name before touching the GPU."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads

pytestmark = pytest.mark.gpu

REL = 1e-9


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _close(gpu, ref, floor=0.0):
    gpu, ref = np.asarray(gpu), np.asarray(ref)
    tol = REL * np.maximum(np.maximum(np.abs(gpu), np.abs(ref)), floor)
    return bool(np.all(np.abs(gpu - ref) <= tol))


def _check_trace(g, ref, n_iters):
    ch = g["tr_choice"].cpu().numpy()[:n_iters]
    assert np.array_equal(ch, ref["tr_choice"][:n_iters]), "per-iterate choices differ"
    U, lam = g["tr_U"].cpu().numpy()[:n_iters], g["tr_lam"].cpu().numpy()[:n_iters]
    assert _close(U, ref["tr_U"][:n_iters]) and _close(lam, ref["tr_lam"][:n_iters])
    # the exact demand sum makes them bitwise equal
    assert np.array_equal(U, ref["tr_U"][:n_iters])
    assert np.array_equal(lam, ref["tr_lam"][:n_iters])
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    assert np.array_equal(g["U"].cpu().numpy(), ref["U"])
    assert np.array_equal(g["lam"].cpu().numpy(), ref["lam"])


DENSE_CASES = {
    "tiny": lambda: workloads.make("tiny"),
    "small": lambda: workloads.make("small"),
    "large_4099": lambda: workloads.make("large", n_jobs=4099),                 # ragged tail tile
    "batched_3x515": lambda: workloads.make("batched", n_jobs=515, n_clusters=3),
    "k4_r1": lambda: workloads.random_small(5, 301, 4, 1, dense=True, iters=80),
    "k16_r3": lambda: workloads.random_small(6, 777, 16, 3, dense=True, iters=80),
    "k64_r8_dyadic": lambda: workloads.random_small(7, 130, 64, 8, dense=True, dyadic=True, iters=80,
                                                    rule=workloads.STEP_CONST),
}


MODES = {"stream": esp.ESP_MODE_STREAM, "persistent": esp.ESP_MODE_PERSISTENT}


@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("name", sorted(DENSE_CASES))
def test_free_running_trace_matches_oracle(name, mode):
    inst = DENSE_CASES[name]()
    T = min(inst.iters, 120)
    _say(f"free-running {name} mode={mode} B={inst.B} N={inst.N} K={inst.dense_k} R={inst.R} T={T}")
    s = esp.Solver(inst, mode=MODES[mode])
    g = s.solve(s.prices(inst.lam0), T, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    ref = oracle.Oracle(inst).solve(iters=T, trace_choice=True)
    _check_trace(g, ref, T)
    assert (g["iters_done"].cpu().numpy() == T).all()
    assert s.device_status() == 0


@pytest.mark.parametrize("name", ["tiny", "small", "large_4099", "batched_3x515"])
def test_teacher_forced_select(name):
    """esp_score_select at the oracle's own prices lambda^t returns the
    oracle's choices bitwise, for every sampled t."""
    inst = DENSE_CASES[name]()
    T = min(inst.iters, 60)
    _say(f"teacher-forced {name}")
    ref = oracle.Oracle(inst).solve(iters=T, trace_choice=True)
    lams = np.concatenate([inst.lam0[None], ref["tr_lam"][:-1]], axis=0)
    s = esp.Solver(inst)
    for t in sorted({0, 1, 2, T // 2, T - 1}):
        ch = s.score_select(s.prices(lams[t])).cpu().numpy()
        assert np.array_equal(ch, ref["tr_choice"][t]), t


@pytest.mark.parametrize("name", ["tiny", "batched_3x515", "k16_r3"])
def test_granular_equals_fused(name):
    """score_select -> reduce_demand -> update_prices, driven from the host,
    reproduces esp_solve's trace bitwise."""
    inst = DENSE_CASES[name]()
    T = 25
    _say(f"granular {name}")
    s = esp.Solver(inst)
    g = s.solve(s.prices(inst.lam0), T, trace=True, trace_choice=True)
    lam = s.prices(inst.lam0)
    for i in range(T):
        ch = s.score_select(lam)
        U = s.reduce_demand(ch)
        s.update_prices(U, i + 1, lam)
        torch.cuda.synchronize()
        assert torch.equal(ch, g["tr_choice"][i])
        assert torch.equal(U, g["tr_U"][i])
        assert torch.equal(lam, g["tr_lam"][i])
    assert s.device_status() == 0


def test_run_to_run_and_geometry_determinism():
    """Same inputs, different workgroup counts and loop drivers: bitwise
    identical results (integer demand sums do not depend on the tree)."""
    inst = workloads.make("large", n_jobs=6000)
    T = 40
    _say("determinism large_6000")
    outs = []
    for nb, mode in ((0, 1), (0, 1), (1, 1), (3, 1), (64, 1), (0, 2), (1, 2), (3, 2), (64, 2), (0, 2)):
        s = esp.Solver(inst, blocks_per_cluster=nb, mode=mode)
        g = s.solve(s.prices(inst.lam0), T, trace=True)
        torch.cuda.synchronize()
        outs.append((g["tr_lam"].cpu().numpy(), g["tr_U"].cpu().numpy(), g["choice"].cpu().numpy()))
        s.close()
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert np.array_equal(a, b)


def test_auto_driver_follows_table_size():
    """AUTO runs the resident driver for tables whose tiles fit the grid's
    registers, the persistent driver for other short passes and one launch
    per pass for large tables; explicit modes are kept."""
    _say("auto driver tiny/small/large")
    for name, kw, want in (("tiny", {}, esp.ESP_MODE_RESIDENT), ("small", {}, esp.ESP_MODE_RESIDENT),
                           ("large", {"n_jobs": 20000}, esp.ESP_MODE_PERSISTENT),
                           ("large", {}, esp.ESP_MODE_STREAM)):
        s = esp.Solver(workloads.make(name, **kw))
        assert s.loop_driver() == want, name
        s.close()
    s = esp.Solver(workloads.make("tiny"), mode=esp.ESP_MODE_STREAM)
    assert s.loop_driver() == esp.ESP_MODE_STREAM
    s.close()


@pytest.mark.parametrize("mode", sorted(MODES))
def test_warm_start_continues_bitwise(mode):
    inst = workloads.make("small")
    _say(f"warm start small {mode}")
    s = esp.Solver(inst, mode=MODES[mode])
    full = s.solve(s.prices(inst.lam0), 90, trace=True)
    lam = s.prices(inst.lam0)
    a = s.solve(lam, 40, trace=True)
    b = s.solve(lam, 50, t_start=41, trace=True)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a["tr_lam"], b["tr_lam"]]), full["tr_lam"])
    assert torch.equal(b["choice"], full["choice"])


@pytest.mark.parametrize("mode", sorted(MODES))
def test_early_stop_matches_oracle(mode):
    inst = workloads.random_small(18, 10, 4, 2, dense=True, iters=500, eta0=0.02)
    _say(f"early stop {mode}")
    tol = 1e-3
    ref = oracle.Oracle(inst).solve(tol=tol, trace_choice=True)
    s = esp.Solver(inst, mode=MODES[mode])
    g = s.solve(s.prices(inst.lam0), inst.iters, tol=tol, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    n = int(ref["iters_done"][0])
    assert n < inst.iters
    assert int(g["iters_done"].cpu()[0]) == n
    _check_trace(g, ref, n)


def test_mask_never_selected():
    inst = workloads.random_small(21, 200, 8, 3, dense=True, iters=60)
    rng = np.random.default_rng(3)
    mask = (rng.random((1, inst.nnz)) < 0.6).astype(np.uint8)
    mask.reshape(200, 8)[:, 5] = 1
    inst.feasible = mask
    _say("feasibility mask")
    ref = oracle.Oracle(inst).solve(trace_choice=True)
    s = esp.Solver(inst)
    g = s.solve(s.prices(inst.lam0), inst.iters, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    _check_trace(g, ref, inst.iters)


def test_device_errors_are_reported():
    inst = workloads.make("tiny")
    _say("device errors")
    s = esp.Solver(inst)
    bad = s.prices(np.full((1, 4), np.nan))
    s.solve(bad, 5)
    assert s.device_status() == esp.ESP_ERR_NONFINITE
    assert s.device_status() == 0                      # cleared
    neg = s.prices(np.array([[0.1, -1.0, 0.0, 0.0]]))
    s.score_select(neg)
    assert s.device_status() == esp.ESP_ERR_NONFINITE
    ch = torch.zeros((1, inst.N), dtype=torch.int32, device="cuda")
    ch[0, 7] = 8                                       # outside the family of 8
    U = s.reduce_demand(ch)
    assert s.device_status() == esp.ESP_ERR_INVALID_ARG
    assert torch.isnan(U).all()
    ch[0, 7] = 3
    U = s.reduce_demand(ch)
    torch.cuda.synchronize()
    assert not torch.isnan(U).any()
    ref = oracle.Oracle(inst).demand_sum(0, ch.cpu().numpy()[0])
    assert np.array_equal(U.cpu().numpy()[0], ref)


# ---------------------------------------------------------------------------
# CSR (ragged) families
# ---------------------------------------------------------------------------

def _extreme_families():
    """Families of 1 and 256 configurations (a full tile) mixed with others."""
    inst = workloads.random_small(31, 300, 9, 5, iters=60)
    rng = np.random.default_rng(31)
    K = rng.integers(1, 40, 300)
    K[[0, 7, 8, 9, 150]] = 256
    K[10:60] = 1
    off = np.concatenate([[0], np.cumsum(K)]).astype(np.int64)
    nnz = int(off[-1])
    inst.offsets = off
    inst.utility = (rng.random((1, nnz)) * 2).astype(np.float32)
    inst.demand = (rng.random((1, nnz, 5)) * 4).astype(np.float32)
    dd = inst.demand[0].astype(np.float64)
    smin = np.minimum.reduceat(dd, off[:-1], axis=0).sum(axis=0)
    smax = np.maximum.reduceat(dd, off[:-1], axis=0).sum(axis=0)
    inst.capacity = (smin + 0.5 * (smax - smin))[None]
    return inst


CSR_CASES = {
    "ragged_20000": lambda: workloads.make("ragged", n_jobs=20000),
    "random_r1": lambda: workloads.random_small(41, 2000, 30, 1, iters=80),
    "random_r8": lambda: workloads.random_small(42, 1500, 70, 8, iters=80),
    "random_k3_dense_layout": lambda: workloads.random_small(43, 999, 3, 4, dense=True, iters=80),
    "random_clusters_3": lambda: workloads.random_small(44, 700, 20, 3, n_clusters=3, iters=60),
    "extreme_families": _extreme_families,
    "ties_dyadic": lambda: workloads.random_small(45, 800, 12, 2, dyadic=True, iters=80,
                                                  rule=workloads.STEP_CONST, eta0=0.125),
}


@pytest.mark.parametrize("name", sorted(CSR_CASES))
def test_csr_free_running_trace_matches_oracle(name):
    inst = CSR_CASES[name]()
    T = min(inst.iters, 120)
    _say(f"csr free-running {name} B={inst.B} N={inst.N} nnz={inst.nnz} R={inst.R} T={T}")
    s = esp.Solver(inst)
    g = s.solve(s.prices(inst.lam0), T, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    ref = oracle.Oracle(inst).solve(iters=T, trace_choice=True)
    _check_trace(g, ref, T)
    assert s.device_status() == 0


@pytest.mark.parametrize("name", ["hand_r1_tie.txt", "hand_r2.txt", "hand_projection.txt"])
def test_hand_traces_on_gpu(name):
    """The hand-derived worked examples (ties, projection to +0.0) on the GPU."""
    from tests._helpers import golden_instance, read_golden
    g = read_golden(name)
    inst = golden_instance(g)
    _say(f"hand trace {name}")
    s = esp.Solver(inst)
    out = s.solve(s.prices(inst.lam0), inst.iters, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    for i, row in enumerate(g["trace"]):
        assert list(out["tr_choice"][i, 0].cpu().numpy()) == [int(x) for x in row[2]]
        assert np.array_equal(out["tr_U"][i, 0].cpu().numpy(), np.array(row[3]))
        assert np.array_equal(out["tr_lam"][i, 0].cpu().numpy(), np.array(row[4]))
    assert list(out["choice"][0].cpu().numpy()) == [int(x) for x in g["final_choice"]]
    assert np.array_equal(out["lam"][0].cpu().numpy(), np.array(g["final_lam"]))
    assert not np.signbit(out["tr_lam"].cpu().numpy()).any()


def test_csr_teacher_forced_and_granular():
    inst = workloads.make("ragged", n_jobs=30000)
    T = 30
    _say("csr teacher-forced + granular ragged_30000")
    ref = oracle.Oracle(inst).solve(iters=T, trace_choice=True)
    lams = np.concatenate([inst.lam0[None], ref["tr_lam"][:-1]], axis=0)
    s = esp.Solver(inst)
    for t in (0, 1, 15, T - 1):
        ch = s.score_select(s.prices(lams[t]))
        assert np.array_equal(ch.cpu().numpy(), ref["tr_choice"][t]), t
        U = s.reduce_demand(ch)
        assert np.array_equal(U.cpu().numpy(), ref["tr_U"][t])
    lam = s.prices(lams[4])
    s.update_prices(s.prices(ref["tr_U"][4]), 5, lam)
    assert np.array_equal(lam.cpu().numpy(), ref["tr_lam"][4])


def test_csr_mask_and_geometry():
    inst = workloads.random_small(46, 3000, 25, 4, iters=50)
    rng = np.random.default_rng(46)
    mask = (rng.random((1, inst.nnz)) < 0.5).astype(np.uint8)
    mask[0, inst.offsets[:-1]] = 1
    inst.feasible = mask
    _say("csr mask + geometry")
    ref = oracle.Oracle(inst).solve(trace_choice=True)
    for nb, sw in ((0, 0), (1, 1), (7, 0)):
        s = esp.Solver(inst, blocks_per_cluster=nb, sweep_order=sw)
        g = s.solve(s.prices(inst.lam0), inst.iters, trace=True, trace_choice=True)
        torch.cuda.synchronize()
        _check_trace(g, ref, inst.iters)
        s.close()


# ---------------------------------------------------------------------------
# Penalty Gamma of the ESP score (Eq. 7)
# ---------------------------------------------------------------------------

PEN_CASES = {
    "dense_k64_r8": lambda: workloads.with_penalties(workloads.make("large", n_jobs=2051), 81, switch_cost=0.5),
    "dense_batched": lambda: workloads.with_penalties(workloads.make("batched", n_jobs=300, n_clusters=3), 82),
    "csr_ragged": lambda: workloads.with_penalties(workloads.make("ragged", n_jobs=9000), 83, switch_cost=0.2),
    "switch_only": lambda: _switch_only(),
    "penalty_only_dyadic": lambda: _penalty_only(),
}


def _switch_only():
    inst = workloads.with_penalties(workloads.random_small(84, 900, 16, 3, dense=True, iters=80), 84)
    inst.penalty = None
    return inst


def _penalty_only():
    inst = workloads.random_small(85, 700, 12, 2, dyadic=True, iters=80, rule=workloads.STEP_CONST, eta0=0.125)
    workloads.with_penalties(inst, 85, dyadic=True)
    inst.current = None
    inst.switch_cost = None
    return inst


@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("name", sorted(PEN_CASES))
def test_penalty_trace_matches_oracle(name, mode):
    inst = PEN_CASES[name]()
    T = min(inst.iters, 80)
    _say(f"penalty {name} mode={mode}")
    s = esp.Solver(inst, mode=MODES[mode])
    g = s.solve(s.prices(inst.lam0), T, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    ref = oracle.Oracle(inst).solve(iters=T, trace_choice=True)
    _check_trace(g, ref, T)


def test_hand_penalty_trace_on_gpu():
    from tests._helpers import golden_instance, read_golden
    g = read_golden("hand_penalty.txt")
    inst = golden_instance(g)
    _say("hand penalty trace")
    s = esp.Solver(inst)
    out = s.solve(s.prices(inst.lam0), inst.iters, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    for i, row in enumerate(g["trace"]):
        assert list(out["tr_choice"][i, 0].cpu().numpy()) == [int(x) for x in row[2]]
        assert np.array_equal(out["tr_lam"][i, 0].cpu().numpy(), np.array(row[4]))
    assert list(out["choice"][0].cpu().numpy()) == [int(x) for x in g["final_choice"]]


def test_set_penalties_between_rounds():
    """Alg. 1 updates Gamma between ESP-IAC rounds: esp_set_penalties then a
    warm-started solve equals the oracle on the updated problem."""
    inst = workloads.with_penalties(workloads.make("large", n_jobs=1500), 86)
    _say("set penalties")
    s = esp.Solver(inst)
    lam = s.prices(inst.lam0)
    s.solve(lam, 20)
    new = workloads.with_penalties(workloads.make("large", n_jobs=1500), 87, switch_cost=0.3)
    s.set_penalties(new.current, new.switch_cost, new.penalty)
    g = s.solve(lam, 25, t_start=21, trace=True, trace_choice=True)
    torch.cuda.synchronize()
    ref1 = oracle.Oracle(inst).solve(iters=20)
    ref2 = oracle.Oracle(new).solve(lam0=ref1["lam"], iters=25, t_start=21, trace_choice=True)
    _check_trace(g, ref2, 25)
    plain = esp.Solver(workloads.make("tiny"))
    with pytest.raises(esp.EspError) as e:
        plain.set_penalties(None, None, np.zeros((1, 512), np.float32))
    assert e.value.code == esp.ESP_ERR_STATE
