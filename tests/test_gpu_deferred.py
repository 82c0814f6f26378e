"""GPU parity of the deferred completion of price iterations (several
workgroups per cluster): every workgroup completes iteration t (U^t and the
Eq. 8 update) at the start of iteration t + 1, or in the closing launch after
the last one.  Covers clusters that meet the stop tolerance at different
iterations (including the first), the closing launch with and without the
final re-selection, group sizes of the persistent barrier, and persistent
solves longer than one cooperative launch."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads

pytestmark = pytest.mark.gpu

MODES = {"stream": esp.ESP_MODE_STREAM, "persistent": esp.ESP_MODE_PERSISTENT}


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _staggered():
    """Four clusters whose step sizes make them meet tol = 1e-3 after 1, 3
    and 108 updates (oracle), the fourth not within T = 120."""
    inst = workloads.random_small(31, 1500, 16, 3, dense=True, n_clusters=4, iters=120, eta0=0.02)
    inst.eta0 = np.array([1e-5, 4e-5, 1e-3, 0.05], dtype=np.float64)
    return inst


def _check_rows(g, ref, n_per_cluster):
    """Trace rows up to each cluster's own stop, then final state."""
    tl, tu = g["tr_lam"].cpu().numpy(), g["tr_U"].cpu().numpy()
    for b, n in enumerate(n_per_cluster):
        assert np.array_equal(tl[:n, b], ref["tr_lam"][:n, b]), b
        assert np.array_equal(tu[:n, b], ref["tr_U"][:n, b]), b
    assert np.array_equal(g["lam"].cpu().numpy(), ref["lam"])
    assert np.array_equal(g["iters_done"].cpu().numpy(), ref["iters_done"])


@pytest.mark.parametrize("blocks", [4, 7, 19])
@pytest.mark.parametrize("mode", sorted(MODES))
def test_staggered_stop_matches_oracle(mode, blocks):
    inst = _staggered()
    ref = oracle.Oracle(inst).solve(tol=1e-3, trace=True)
    n = [int(x) for x in ref["iters_done"]]
    assert n[0] == 1 and n[1] == 3 and n[2] == 108 and n[3] == inst.iters
    _say(f"staggered stop {mode} blocks={blocks} stops={n}")
    s = esp.Solver(inst, mode=MODES[mode], blocks_per_cluster=blocks)
    g = s.solve(s.prices(inst.lam0), inst.iters, tol=1e-3, trace=True)
    torch.cuda.synchronize()
    _check_rows(g, ref, n)
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    assert np.array_equal(g["U"].cpu().numpy(), ref["U"])
    assert s.device_status() == 0
    s.close()


@pytest.mark.parametrize("mode", sorted(MODES))
def test_closing_launch_without_reselection(mode):
    """No final choice or demand asked for: the closing launch only
    completes the last iteration (prices, trace, iteration counts)."""
    inst = _staggered()
    ref = oracle.Oracle(inst).solve(tol=1e-3, trace=True)
    _say(f"closing launch without re-selection {mode}")
    s = esp.Solver(inst, mode=MODES[mode], blocks_per_cluster=5)
    g = s.solve(s.prices(inst.lam0), inst.iters, tol=1e-3, trace=True, final_select=False)
    torch.cuda.synchronize()
    assert "choice" not in g
    _check_rows(g, ref, [int(x) for x in ref["iters_done"]])
    # without a tolerance every cluster runs all T updates
    ref0 = oracle.Oracle(inst).solve(iters=37, trace=True)
    g0 = s.solve(s.prices(inst.lam0), 37, trace=True, final_select=False)
    torch.cuda.synchronize()
    _check_rows(g0, ref0, [37] * inst.B)
    assert s.device_status() == 0


def test_persistent_solve_longer_than_one_launch():
    """1,100 iterations on Small (128 workgroups): two cooperative launches
    (1,024 + 76 iterations); the second starts by completing the first's
    last iteration.  Bitwise equal to one launch per iteration and to the
    oracle."""
    inst = workloads.make("small")
    T = 1100
    _say(f"persistent T={T} small")
    ref = oracle.Oracle(inst).solve(iters=T, trace=True)
    outs = []
    for mode in (esp.ESP_MODE_PERSISTENT, esp.ESP_MODE_STREAM):
        s = esp.Solver(inst, mode=mode)
        g = s.solve(s.prices(inst.lam0), T, trace=True)
        torch.cuda.synchronize()
        outs.append(g)
        _check_rows(g, ref, [T] * inst.B)
        assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
        assert s.device_status() == 0
        s.close()
    assert torch.equal(outs[0]["tr_lam"], outs[1]["tr_lam"])


def test_warm_start_across_deferred_solves():
    """A solve split in two (t_start) equals one solve, with several
    workgroups per cluster and the persistent driver."""
    inst = workloads.make("large", n_jobs=6000)
    _say("warm start deferred large_6000")
    s = esp.Solver(inst, mode=esp.ESP_MODE_PERSISTENT, blocks_per_cluster=12)
    full = s.solve(s.prices(inst.lam0), 60, trace=True)
    lam = s.prices(inst.lam0)
    a = s.solve(lam, 25, trace=True)
    b = s.solve(lam, 35, t_start=26, trace=True)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([a["tr_lam"], b["tr_lam"]]), full["tr_lam"])
    assert torch.equal(torch.cat([a["tr_U"], b["tr_U"]]), full["tr_U"])
    assert torch.equal(b["choice"], full["choice"])
    assert s.device_status() == 0
