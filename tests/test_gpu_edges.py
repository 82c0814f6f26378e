"""GPU parity on the edges of the input space: every resource count, a
single job, zero iterations, and demand columns whose bit span needs the
128-bit accumulators.  All results bitwise equal to the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_07971_amd as esp
import workloads

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _parity(inst, T, mode=esp.ESP_MODE_AUTO):
    s = esp.Solver(inst, mode=mode)
    g = s.solve(s.prices(inst.lam0), T, trace=T > 0, trace_choice=T > 0)
    torch.cuda.synchronize()
    ref = oracle.Oracle(inst).solve(iters=T, trace_choice=T > 0, trace=T > 0)
    if T > 0:
        assert np.array_equal(g["tr_choice"].cpu().numpy(), ref["tr_choice"])
        assert np.array_equal(g["tr_U"].cpu().numpy(), ref["tr_U"])
        assert np.array_equal(g["tr_lam"].cpu().numpy(), ref["tr_lam"])
    assert np.array_equal(g["choice"].cpu().numpy(), ref["choice"])
    assert np.array_equal(g["U"].cpu().numpy(), ref["U"])
    assert np.array_equal(g["lam"].cpu().numpy(), ref["lam"])
    assert s.device_status() == 0
    s.close()


@pytest.mark.parametrize("R", list(range(1, 9)))
@pytest.mark.parametrize("layout", ["dense_k8", "csr"])
def test_every_resource_count(R, layout):
    inst = (workloads.random_small(60 + R, 900, 8, R, dense=True, iters=40) if layout == "dense_k8"
            else workloads.random_small(70 + R, 700, 23, R, iters=40))
    _say(f"R={R} {layout}")
    # both drivers explicitly: the persistent one is a cooperative launch of
    # the whole grid, which the kernel's registers must let the device hold
    for mode in (esp.ESP_MODE_STREAM, esp.ESP_MODE_PERSISTENT):
        _parity(inst, 40, mode)


@pytest.mark.parametrize("layout", ["dense", "csr"])
def test_single_job(layout):
    # K = 16 takes the dense kernel; K = 7 (no dense variant) the CSR kernel
    inst = workloads.random_small(80 if layout == "dense" else 81, 1, 16 if layout == "dense" else 7, 3,
                                  dense=True, iters=30)
    _say(f"single job {layout}")
    for mode in (esp.ESP_MODE_STREAM, esp.ESP_MODE_PERSISTENT):
        _parity(inst, 30, mode)


def test_zero_iterations_reselects_at_the_given_prices():
    inst = workloads.make("small", n_jobs=1000)
    inst.lam0 = np.full((1, inst.R), 0.01)
    _say("T = 0")
    _parity(inst, 0)


def _wide(inst, seed, span=36):
    """Demands multiplied by 2^U{-span..span} per entry: a column spans more
    than 63 bits with log2(N + 1), so the packer picks 128-bit sums."""
    rng = np.random.default_rng(seed)
    inst.demand = (inst.demand.astype(np.float64) *
                   np.exp2(rng.integers(-span, span + 1, inst.demand.shape))).astype(np.float32)
    return inst


@pytest.mark.parametrize("layout", ["dense_k16", "dense_k64_r8", "csr", "csr_batched", "csr_r8"])
def test_wide_spans_use_128_bit_sums(layout):
    inst = {
        "dense_k16": lambda: workloads.random_small(90, 3000, 16, 5, dense=True, iters=60),
        "dense_k64_r8": lambda: workloads.random_small(91, 700, 64, 8, dense=True, iters=60),
        "csr": lambda: workloads.random_small(92, 2500, 30, 6, iters=60),
        "csr_batched": lambda: workloads.random_small(93, 800, 30, 4, n_clusters=3, iters=60),
        "csr_r8": lambda: workloads.random_small(94, 1200, 40, 8, iters=60),
    }[layout]()
    _wide(inst, 5)
    inst.eta0 = np.full(inst.B, 1e-12)                   # prices stay in a useful range for 2^36 demands
    _say(f"128-bit sums {layout}")
    for mode in (esp.ESP_MODE_STREAM, esp.ESP_MODE_PERSISTENT):
        _parity(inst, 60, mode)
