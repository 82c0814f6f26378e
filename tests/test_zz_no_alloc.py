"""GPU: esp_solve_noalloc (per-solve scratch in the library's static device
array) against esp_solve (scratch in the context's workspace) on the same
contexts, through the C-ABI: bitwise equal outputs on calls in a row, each
later call on a smaller problem than the one before, so stale contents of
the shared array would show; and the size limit refused on the host."""
import numpy as np
import pytest
import torch

import paper_2608_07971_amd as esp
import workloads

pytestmark = pytest.mark.gpu


def _say(msg):
    print(f"[gpu-case] {msg}", flush=True)


def _outputs(s, T):
    dev = s.device
    return {
        "lam": None,
        "choice": torch.full((s.B, s.N), -7, dtype=torch.int32, device=dev),
        "U": torch.full((s.B, s.R), -7.0, dtype=torch.float64, device=dev),
        "tr_lam": torch.full((max(T, 1), s.B, s.R), -7.0, dtype=torch.float64, device=dev),
        "tr_U": torch.full((max(T, 1), s.B, s.R), -7.0, dtype=torch.float64, device=dev),
        "tr_choice": torch.full((max(T, 1), s.B, s.N), -7, dtype=torch.int32, device=dev),
        "iters_done": torch.full((s.B,), -7, dtype=torch.int32, device=dev),
    }


def _call(fn, s, lam0, T, tol, out):
    out["lam"] = s.prices(lam0)
    tr = esp.esp_trace(out["tr_lam"].data_ptr(), out["tr_U"].data_ptr(), out["tr_choice"].data_ptr())
    torch.cuda.synchronize()
    before = torch.cuda.memory_stats().get("allocation.all.allocated", 0)
    fn(s.ctx, out["lam"], T, 1, tol, out["choice"], out["U"], tr, out["iters_done"], torch.cuda.current_stream())
    after = torch.cuda.memory_stats().get("allocation.all.allocated", 0)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    return after - before


# Largest first: every later call runs on a smaller problem (fewer clusters,
# workgroups or jobs) than the call before it.
CASES = [
    ("batched_4x3000_tol", lambda: workloads.make("batched", n_jobs=3000, n_clusters=4), esp.ESP_MODE_AUTO, 40, 1e-4),
    ("large_4099", lambda: workloads.make("large", n_jobs=4099), esp.ESP_MODE_STREAM, 40, 0.0),
    ("ragged_20000", lambda: workloads.make("ragged", n_jobs=20000), esp.ESP_MODE_STREAM, 50, 0.0),
    ("ragged_20000_persistent", lambda: workloads.make("ragged", n_jobs=20000), esp.ESP_MODE_PERSISTENT, 50, 0.0),
    ("small", lambda: workloads.make("small"), esp.ESP_MODE_AUTO, 60, 0.0),
    ("tiny", lambda: workloads.make("tiny"), esp.ESP_MODE_AUTO, 200, 0.0),
    ("tiny_tol", lambda: workloads.make("tiny"), esp.ESP_MODE_AUTO, 200, 1e-3),
]


def test_noalloc_solve_matches_solve_on_calls_in_a_row():
    for name, make, mode, T, tol in CASES:
        inst = make()
        _say(f"noalloc vs solve: {name} B={inst.B} N={inst.N} R={inst.R} T={T} tol={tol}")
        s = esp.Solver(inst, mode=mode)
        ref, got = _outputs(s, T), _outputs(s, T)
        _call(esp.esp_solve, s, inst.lam0, T, tol, ref)
        grew = _call(esp.esp_solve_noalloc, s, inst.lam0, T, tol, got)
        assert grew == 0, f"{name}: the call allocated through torch"
        for k in ref:
            assert torch.equal(ref[k], got[k]), f"{name}: {k} differs"
        if tol == 0.0:
            assert (got["iters_done"].cpu().numpy() == T).all()
        # the same solve once more through the static array: unchanged results
        again = _outputs(s, T)
        _call(esp.esp_solve_noalloc, s, inst.lam0, T, tol, again)
        for k in ref:
            assert torch.equal(ref[k], again[k]), f"{name}: {k} differs on the second call"
        s.close()


def test_noalloc_refuses_problems_beyond_its_scratch():
    """512 clusters need more than ESP_NOALLOC_SCRATCH_BYTES (barrier words
    alone take 4352 bytes per cluster): refused on the host, nothing runs."""
    inst = workloads.random_small(44, 64, 8, 4, dense=True, n_clusters=512, iters=5)
    _say("noalloc: 512 clusters, beyond the static scratch")
    s = esp.Solver(inst)
    lam = s.prices(inst.lam0)
    keep = lam.clone()
    with pytest.raises(esp.EspError) as e:
        esp.esp_solve_noalloc(s.ctx, lam, 5)
    assert e.value.code == esp.ESP_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert torch.equal(lam, keep)
    # the workspace path still serves it
    g = s.solve(lam, 5)
    torch.cuda.synchronize()
    assert s.device_status() == 0 and (g["iters_done"].cpu().numpy() == 5).all()
    s.close()
