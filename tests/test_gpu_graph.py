"""GPU: device-computed step sizes equal the host's IEEE values, and a
stream-mode esp_solve captured in a HIP graph replays bit for bit."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def test_device_step_sizes_are_the_ieee_values():
    """lambda = 0 and U - C = 1: the update returns eta_t itself, which must
    equal eta0 / sqrt(t) rounded as on the host, for t up to 2^31 - 1."""
    inst = workloads.random_small(3, 10, 4, 1, rule=workloads.STEP_INV_SQRT)
    rng = np.random.default_rng(0)
    ts = sorted(set([1, 2, 3, 4, 5, 7, 9, 10, 16, 99, 1000, 2 ** 20, 10 ** 9 + 7, 2 ** 31 - 1] +
                    [int(x) for x in rng.integers(1, 2 ** 31 - 1, 200)]))
    _say(f"step sizes at {len(ts)} values of t")
    for e0 in (0.01, 1.0, 0.3, 2.0 ** -20, 12345.678):
        inst.eta0 = np.array([e0])
        s = esp.Solver(inst)
        for t in ts:
            lam = s.prices(np.zeros((1, 1)))
            U = s.prices(inst.capacity + 1.0)
            s.update_prices(U, t, lam)
            got = float(lam.cpu().numpy()[0, 0])
            assert got == oracle.eta(workloads.STEP_INV_SQRT, e0, t), (e0, t)
        s.close()


@pytest.mark.parametrize("name", ["small", "ragged_3000"])
def test_captured_solve_replays_bitwise(name):
    inst = workloads.make("small") if name == "small" else workloads.make("ragged", n_jobs=3000)
    T = 30
    _say(f"graph capture {name}")
    s = esp.Solver(inst)
    lam0 = s.prices(inst.lam0)
    eager = s.solve(lam0.clone(), T, trace=True)
    torch.cuda.synchronize()
    ref = {k: eager[k].cpu().numpy() for k in ("lam", "U", "choice", "tr_lam")}
    # static buffers, then capture on a side stream
    lam = lam0.clone()
    choice = torch.empty((s.B, s.N), dtype=torch.int32, device="cuda")
    U = torch.empty((s.B, s.R), dtype=torch.float64, device="cuda")
    tr_lam = torch.empty((T, s.B, s.R), dtype=torch.float64, device="cuda")
    tr = esp.esp_trace(tr_lam.data_ptr(), None, None)
    g = torch.cuda.CUDAGraph()
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.graph(g, stream=stream):
        lam.copy_(lam0)
        esp.esp_solve(s.ctx, lam, T, 1, 0.0, choice, U, tr, None, torch.cuda.current_stream())
    other = s.prices(np.full((s.B, s.R), 0.05))
    for rep in range(4):
        lam.fill_(123.0)                                   # eager work between the replays
        s.solve(other.clone(), 5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(lam.cpu().numpy(), ref["lam"]), rep
        assert np.array_equal(U.cpu().numpy(), ref["U"]), rep
        assert np.array_equal(choice.cpu().numpy(), ref["choice"]), rep
        assert np.array_equal(tr_lam.cpu().numpy(), ref["tr_lam"]), rep
    assert s.device_status() == 0
