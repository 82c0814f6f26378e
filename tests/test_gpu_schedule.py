"""GPU parity of the outer ESP-IAC rounds (Sec. 3.4, Alg. 1) through the
C-ABI against the oracle: rounds run, violating pairs, prices, choices,
the GPU occupancy lists and the final penalties, all bit-exact."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads
from tests._helpers import schedule_fixture

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _with_penalty_inputs(inst):
    """A context needs the penalty column for Alg. 1: zero interference
    penalties (Alg. 1 resets them anyway), no switching cost."""
    if inst.penalty is None:
        inst.penalty = np.zeros((inst.B, inst.nnz), np.float32)
    return inst


def _compare(inst, model, M, T, tol=0.0, clusters=None):
    s = esp.Solver(_with_penalty_inputs(inst))
    lam = s.prices(inst.lam0)
    g = s.schedule(model, lam, M, T, tol)
    torch.cuda.synchronize()
    pen = s.read_penalties()
    assert s.device_status() == 0
    o = oracle.Oracle(inst)
    gj = g["gpu_jobs"].cpu().numpy()
    for b in (range(inst.B) if clusters is None else clusters):
        r = o.schedule(b, model, M, T, tol)
        G = int(model.gpus[b])
        assert int(g["rounds"][b]) == r["rounds"], b
        assert int(g["violations"][b]) == r["violations"], b
        assert np.array_equal(g["choice"][b].cpu().numpy(), r["choice"]), b
        assert np.array_equal(g["lam"][b].cpu().numpy(), r["lam"]), b
        assert np.array_equal(gj[b, :G], r["occ"]), b
        assert (gj[b, G:] == -1).all()
        assert np.array_equal(pen[b], r["penalty"]), b
    s.close()
    return g


def test_hand_example_on_gpu():
    inst, m, results = schedule_fixture()
    _say("schedule hand example")
    for M, nr, V, ch, g0, g1, pen in results:
        g = _compare(inst, m, int(M[0]), inst.iters)
        assert int(g["rounds"][0]) == int(nr[0]) and int(g["violations"][0]) == int(V[0])


CASES = {
    "tiny": lambda: workloads.make("tiny"),
    "small_600": lambda: workloads.make("small", n_jobs=600),
    "small_2000": lambda: workloads.make("small", n_jobs=2000),
    "batched_3x700": lambda: workloads.make("batched", n_jobs=700, n_clusters=3),
    "ragged_shape_r6": lambda: workloads.make("ragged", n_jobs=1500),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_schedule_matches_oracle(name):
    inst = CASES[name]()
    model = workloads.iac_model(inst, gpus=None if name != "ragged_shape_r6" else [600])
    _say(f"schedule {name}: B={inst.B} N={inst.N} R={inst.R} G={list(model.gpus)}")
    for M, T in ((1, 40), (3, 60)):
        _compare(inst, model, M, T)


def test_schedule_with_switching_cost_and_tolerance():
    """Switching costs stay through Gamma's reset; rounds use a stop
    tolerance (the persistent driver)."""
    inst = workloads.with_penalties(workloads.make("small", n_jobs=800), 3)
    model = workloads.iac_model(inst)
    _say("schedule small_800 with switching cost, tol")
    _compare(inst, model, 3, 200, tol=1e-3)


def test_schedule_errors():
    inst = workloads.make("tiny")
    _say("schedule errors")
    s = esp.Solver(inst)                             # no penalty column
    model = workloads.iac_model(inst)
    with pytest.raises(esp.EspError) as e:
        s.schedule(model, s.prices(inst.lam0), 2, 10)
    assert e.value.code == esp.ESP_ERR_STATE
    s2 = esp.Solver(_with_penalty_inputs(workloads.make("tiny")))
    for field, value in (("gpus", np.array([0])), ("gpus", np.array([5000])), ("r_sm", 7), ("kappa", -1.0),
                         ("u_target", 0.0)):
        bad = workloads.iac_model(inst)
        setattr(bad, field, value)
        with pytest.raises(esp.EspError) as e:
            s2.schedule(bad, s2.prices(inst.lam0), 2, 10)
        assert e.value.code == esp.ESP_ERR_INVALID_ARG, field
    bad = workloads.iac_model(inst)
    bad.beta = float("nan")
    with pytest.raises(esp.EspError) as e:
        s2.schedule(bad, s2.prices(inst.lam0), 2, 10)
    assert e.value.code == esp.ESP_ERR_NONFINITE
    torch.cuda.synchronize()
    assert s2.device_status() == 0


def test_fullsize_batched_rounds():
    """The Batched workload (256 clusters x 16,384 jobs x 64 configurations,
    256..1024 GPUs each) with 3 rounds of 20 iterations, in the launch
    configuration bench.py uses; four clusters checked against the oracle."""
    inst = workloads.make("batched")
    model = workloads.iac_model(inst)
    _say("schedule full-size batched, M=3, T=20")
    _compare(inst, model, 3, 20, clusters=(0, 1, 131, inst.B - 1))
