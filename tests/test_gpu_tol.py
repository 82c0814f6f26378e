"""GPU: the early-stop rule against the hand-derived trace (hand_tol.txt),
in both loop drivers, with one workgroup per cluster and with many (the
deferred completion), and the boundary's remaining error paths: a
cooperative grid the device cannot hold (ESP_ERR_DEVICE, nothing launched),
the persistent driver under graph capture (ESP_ERR_INVALID_ARG, nothing
recorded), and -0.0 prices stored back as +0.0."""
import struct

import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads
from tests._helpers import golden_instance, read_golden

pytestmark = pytest.mark.gpu

MODES = {"stream": esp.ESP_MODE_STREAM, "persistent": esp.ESP_MODE_PERSISTENT}


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _replicated(g, n, k):
    """The fixture's job repeated n times with k identical configurations
    each: capacities times n and the step divided by n (n and k powers of
    two), so every price, demand ratio and stop test is the fixture's exactly;
    ties between the k copies go to configuration 0."""
    inst = golden_instance(g)
    R = inst.R
    util = np.full((1, n * k), inst.utility[0, 0], np.float32)
    dem = np.tile(inst.demand[0, 0], (n * k, 1))[None].astype(np.float32)
    cap = inst.capacity * n
    eta0 = inst.eta0 / n
    out = workloads.Instance("hand_tol_x", 0, workloads.uniform_offsets(n, k), util, dem, cap, eta0, inst.rule,
                             inst.lam0.copy(), inst.iters)
    if k in (4, 8, 16, 32, 64):
        out.dense_k = k
    assert out.R == R
    return out


CASES = {
    "fixture": lambda g: golden_instance(g),
    "csr_65536x1": lambda g: _replicated(g, 65536, 1),          # 64 workgroups, deferred completion
    "dense_65536x4": lambda g: _replicated(g, 65536, 4),        # 192 workgroups, deferred completion
}


@pytest.mark.parametrize("mode", sorted(MODES))
@pytest.mark.parametrize("case", sorted(CASES))
def test_tol_stop_matches_hand_trace(case, mode):
    g = read_golden("hand_tol.txt")
    inst = CASES[case](g)
    tol = g["tol"][0]
    done = int(g["iters_done"][0])
    _say(f"tol stop {case} mode={mode} N={inst.N} T={inst.iters}")
    s = esp.Solver(inst, mode=MODES[mode])
    out = s.solve(s.prices(inst.lam0), inst.iters, tol=tol, trace=True)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    assert int(out["iters_done"][0]) == done
    tr_lam, tr_U = out["tr_lam"][:, 0].cpu().numpy(), out["tr_U"][:, 0].cpu().numpy()
    n = inst.N
    for i, row in enumerate(g["trace"]):
        assert np.array_equal(tr_lam[i], np.array(row[4])), i
        assert np.array_equal(tr_U[i], np.array(row[3]) * n), i
    assert np.isnan(tr_lam[done:]).all() and np.isnan(tr_U[done:]).all()
    assert np.array_equal(out["lam"][0].cpu().numpy(), np.array(g["final_lam"]))
    assert np.array_equal(out["U"][0].cpu().numpy(), np.array(g["final_U"]) * n)
    assert (out["choice"].cpu().numpy() == 0).all()
    for c_tol, c_n, c_lam in g["cases"]:
        r = s.solve(s.prices(inst.lam0), inst.iters, tol=c_tol[0])
        torch.cuda.synchronize()
        assert int(r["iters_done"][0]) == int(c_n[0]), c_tol
        assert np.array_equal(r["lam"][0].cpu().numpy(), np.array(c_lam)), c_tol
    # the oracle agrees on the replicated problem as well
    ref = oracle.Oracle(inst).solve(tol=tol)
    assert int(ref["iters_done"][0]) == done
    assert np.array_equal(ref["lam"], out["lam"].cpu().numpy())
    s.close()


def _bits(x: float) -> int:
    return struct.unpack("<Q", struct.pack("<d", x))[0]


@pytest.mark.parametrize("layout", ["dense", "csr"])
def test_negative_zero_prices_are_stored_as_positive_zero(layout):
    inst = (workloads.random_small(41, 500, 8, 4, dense=True, iters=5) if layout == "dense"
            else workloads.random_small(42, 400, 9, 4, iters=5))
    lam0 = np.array([[-0.0, 0.25, -0.0, 0.0]])
    _say(f"-0.0 prices, iters = 0, {layout}")
    s = esp.Solver(inst)
    lam = s.prices(lam0)
    g = s.solve(lam, 0)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    got = g["lam"].cpu().numpy()[0]
    assert [_bits(x) for x in got] == [_bits(x) for x in (0.0, 0.25, 0.0, 0.0)]
    ref = oracle.Oracle(inst).solve(lam0=np.abs(lam0), iters=0)
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    assert np.array_equal(g["U"].cpu().numpy(), ref["U"])
    # with iterations too: the trajectory is the one from +0.0
    lam = s.prices(lam0)
    g = s.solve(lam, 5, trace=True)
    torch.cuda.synchronize()
    ref = oracle.Oracle(inst).solve(lam0=np.abs(lam0), iters=5)
    assert np.array_equal(g["tr_lam"].cpu().numpy(), ref["tr_lam"])
    assert np.array_equal(g["lam"].cpu().numpy(), ref["lam"])
    s.close()


def _too_wide():
    """512 clusters x 1024 jobs x 16 configurations, R = 1, 16 workgroups per
    cluster: 8192 workgroups of 4 wavefronts, more than the 256 compute units
    can hold at once (32 per SIMD)."""
    return workloads.random_small(43, 1024, 16, 1, dense=True, n_clusters=512, iters=20)


def test_refused_cooperative_grid_is_a_device_error():
    inst = _too_wide()
    _say("persistent driver, grid beyond co-residency: refused on the host")
    s = esp.Solver(inst, mode=esp.ESP_MODE_PERSISTENT, blocks_per_cluster=16)
    lam = s.prices(inst.lam0)
    with pytest.raises(esp.EspError) as e:
        s.solve(lam, 20)
    assert e.value.code == esp.ESP_ERR_DEVICE
    torch.cuda.synchronize()
    assert s.device_status() == 0
    # the context stays usable: a one-launch-per-iteration solve afterwards
    s.close()
    s = esp.Solver(inst, mode=esp.ESP_MODE_STREAM, blocks_per_cluster=16)
    g = s.solve(s.prices(inst.lam0), 20, trace=True)
    torch.cuda.synchronize()
    ref = oracle.Oracle(inst).solve(iters=20)
    assert np.array_equal(g["tr_lam"].cpu().numpy(), ref["tr_lam"])
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    s.close()


def test_auto_falls_back_when_the_grid_is_refused():
    """AUTO with a tolerance asks for the persistent driver; the refused grid
    falls back to one launch per iteration with the same results."""
    inst = _too_wide()
    _say("AUTO + tol, grid beyond co-residency: falls back to one launch per iteration")
    s = esp.Solver(inst, mode=esp.ESP_MODE_AUTO, blocks_per_cluster=16)
    g = s.solve(s.prices(inst.lam0), 20, tol=1e-3, trace=True)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    assert s.loop_driver() == esp.ESP_MODE_STREAM
    ref = oracle.Oracle(inst).solve(iters=20, tol=1e-3)
    assert np.array_equal(g["iters_done"].cpu().numpy(), ref["iters_done"])
    assert np.array_equal(g["lam"].cpu().numpy(), ref["lam"])
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    s.close()


def test_persistent_driver_under_capture_is_refused():
    inst = workloads.make("tiny")
    _say("persistent driver under graph capture")
    s = esp.Solver(inst, mode=esp.ESP_MODE_PERSISTENT)
    lam = s.prices(inst.lam0)
    graph = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    codes = []
    torch.cuda.synchronize()
    with torch.cuda.graph(graph, stream=stream):
        lam.mul_(2.0)
        try:
            esp.esp_solve(s.ctx, lam, 10, 1, 0.0, None, None, None, None, torch.cuda.current_stream())
        except esp.EspError as e:
            codes.append(e.code)
    assert codes == [esp.ESP_ERR_INVALID_ARG]
    lam.fill_(0.5)
    graph.replay()                               # holds the multiplication only
    torch.cuda.synchronize()
    assert (lam.cpu().numpy() == 1.0).all()
    # eager solves on the same context are unaffected
    g = s.solve(s.prices(inst.lam0), inst.iters, trace=True)
    torch.cuda.synchronize()
    ref = oracle.Oracle(inst).solve()
    assert np.array_equal(g["tr_lam"].cpu().numpy(), ref["tr_lam"])
    assert s.device_status() == 0
    s.close()
