"""Python binding of the MI355X Elastic Shadow Pricing library (libesp.so).

The functions below carry the names of the C-ABI in include/esp.h and only
marshal arguments: every step of the method runs in the HIP kernels of
csrc/.  PyTorch provides device memory (the workspace and per-call tensors)
and streams.  There is no CPU fallback: importing the binding without a built
libesp.so raises, and so does calling it without a GPU.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np
import torch  # loaded first so libesp.so binds to the HIP runtime torch uses

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libesp.so")

ESP_OK = 0
ESP_ERR_INVALID_ARG = 1
ESP_ERR_SHAPE = 2
ESP_ERR_NONFINITE = 3
ESP_ERR_NEGATIVE_DEMAND = 4
ESP_ERR_EMPTY_FAMILY = 5
ESP_ERR_WORKSPACE = 6
ESP_ERR_RANGE = 7
ESP_ERR_DEVICE = 8
ESP_ERR_STATE = 9

ESP_STEP_CONST = 0
ESP_STEP_INV_SQRT = 1

ESP_MODE_AUTO = 0
ESP_MODE_STREAM = 1
ESP_MODE_PERSISTENT = 2
ESP_MODE_RESIDENT = 3
ESP_OPT_PROFILE_STORE = 1


class EspError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: {status_string(code)} (status {code})")


class esp_problem(C.Structure):
    _fields_ = [
        ("num_clusters", C.c_int32), ("num_jobs", C.c_int32), ("num_resources", C.c_int32),
        ("configs_per_job", C.c_int32), ("family_offsets", C.c_void_p), ("utility", C.c_void_p),
        ("demand", C.c_void_p), ("capacity", C.c_void_p), ("feasible", C.c_void_p),
        ("current", C.c_void_p), ("switch_cost", C.c_void_p), ("penalty", C.c_void_p),
    ]


class esp_step_rule(C.Structure):
    _fields_ = [("rule", C.c_int32), ("eta0", C.c_void_p)]


class esp_options(C.Structure):
    _fields_ = [("blocks_per_cluster", C.c_int32), ("sweep_order", C.c_int32), ("mode", C.c_int32),
                ("flags", C.c_int32), ("reserved", C.c_int32 * 4)]


class esp_iac_model(C.Structure):
    _fields_ = [("gpus", C.c_void_p), ("gpu_memory", C.c_double), ("gpu_compute", C.c_double),
                ("r_gpus", C.c_int32), ("r_mem", C.c_int32), ("r_sm", C.c_int32),
                ("sensitivity", C.c_void_p), ("pressure", C.c_void_p), ("tau_base", C.c_void_p),
                ("beta", C.c_double), ("beta_max", C.c_double), ("u_target", C.c_double), ("kappa", C.c_double)]


ESP_MAX_GPUS = 2048
ESP_MAX_PER_GPU = 4


class esp_trace(C.Structure):
    _fields_ = [("prices", C.c_void_p), ("demand", C.c_void_p), ("choice", C.c_void_p)]


_lib = None

# Every entry point of include/esp.h with its ctypes signature.
_SIGS = {
    "esp_workspace_size": ([C.c_void_p, C.c_void_p, C.POINTER(C.c_size_t)], C.c_int),
    "esp_create": ([C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p,
                    C.POINTER(C.c_void_p)], C.c_int),
    "esp_score_select": ([C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
    "esp_reduce_demand": ([C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
    "esp_update_prices": ([C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p], C.c_int),
    "esp_solve": ([C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_double, C.c_void_p, C.c_void_p,
                   C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
    "esp_solve_noalloc": ([C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_double, C.c_void_p, C.c_void_p,
                           C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
    "esp_set_penalties": ([C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
    "esp_device_status": ([C.c_void_p, C.c_void_p], C.c_int),
    "esp_loop_driver": ([C.c_void_p, C.POINTER(C.c_int32)], C.c_int),
    "esp_set_capacity": ([C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
    "esp_read_penalties": ([C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
    "esp_schedule": ([C.c_void_p, C.c_void_p, C.c_int32, C.c_int32, C.c_double, C.c_void_p, C.c_void_p, C.c_void_p,
                      C.c_void_p, C.c_void_p, C.c_void_p], C.c_int),
    "esp_nearest_profile": ([C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p],
                            C.c_int),
    "esp_effective_capacity": ([C.c_void_p, C.c_void_p, C.c_void_p, C.c_double, C.c_void_p, C.c_void_p],
                               C.c_int),
    "esp_destroy": ([C.c_void_p], C.c_int),
    "esp_status_string": ([C.c_int], C.c_char_p),
}


def lib():
    """Load libesp.so (raises when it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(there is no CPU fallback)")
        L = C.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().esp_status_string(code).decode()


def _check(code: int, where: str) -> None:
    if code != ESP_OK:
        raise EspError(code, where)


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, torch.Tensor):
        if not t.is_cuda:
            raise ValueError("device tensor expected")
        if not t.is_contiguous():
            raise ValueError("contiguous tensor expected")
        return t.data_ptr()
    return int(t)


# ---------------------------------------------------------------------------
# C-ABI entry points (same names as include/esp.h)
# ---------------------------------------------------------------------------

class Problem:
    """Host arrays of an esp_problem kept alive for the duration of a call."""

    def __init__(self, offsets, utility, demand, capacity, feasible=None, dense_k: Optional[int] = None,
                 current=None, switch_cost=None, penalty=None):
        self.current = None if current is None else np.ascontiguousarray(current, dtype=np.int32)
        self.switch_cost = None if switch_cost is None else np.ascontiguousarray(switch_cost, dtype=np.float64)
        self.penalty = None if penalty is None else np.ascontiguousarray(penalty, dtype=np.float32)
        self.utility = np.ascontiguousarray(utility, dtype=np.float32)
        self.demand = np.ascontiguousarray(demand, dtype=np.float32)
        self.capacity = np.ascontiguousarray(capacity, dtype=np.float64)
        self.feasible = None if feasible is None else np.ascontiguousarray(feasible, dtype=np.uint8)
        self.offsets = None if dense_k else np.ascontiguousarray(offsets, dtype=np.int64)
        B = self.utility.shape[0]
        R = self.demand.shape[-1]
        N = (self.utility.shape[1] // dense_k) if dense_k else self.offsets.size - 1
        self.B, self.N, self.R = B, N, R
        self.c = esp_problem(B, N, R, int(dense_k or 0),
                             None if self.offsets is None else self.offsets.ctypes.data,
                             self.utility.ctypes.data, self.demand.ctypes.data, self.capacity.ctypes.data,
                             None if self.feasible is None else self.feasible.ctypes.data,
                             _np_ptr(self.current), _np_ptr(self.switch_cost), _np_ptr(self.penalty))

    @classmethod
    def from_instance(cls, inst) -> "Problem":
        return cls(inst.offsets, inst.utility, inst.demand, inst.capacity, inst.feasible,
                   dense_k=getattr(inst, "dense_k", None), current=getattr(inst, "current", None),
                   switch_cost=getattr(inst, "switch_cost", None), penalty=getattr(inst, "penalty", None))


def _np_ptr(a):
    return None if a is None else a.ctypes.data


def esp_workspace_size(problem: Problem, options: Optional[esp_options] = None) -> int:
    n = C.c_size_t(0)
    _check(lib().esp_workspace_size(C.addressof(problem.c), None if options is None else C.addressof(options),
                                    C.byref(n)), "esp_workspace_size")
    return int(n.value)


def esp_create(problem: Problem, rule: int, eta0, workspace, options: Optional[esp_options] = None,
               stream=None) -> int:
    e0 = np.ascontiguousarray(eta0, dtype=np.float64)
    step = esp_step_rule(int(rule), e0.ctypes.data)
    out = C.c_void_p(None)
    _check(lib().esp_create(C.addressof(problem.c), C.addressof(step),
                            None if options is None else C.addressof(options), _ptr(workspace),
                            workspace.numel() * workspace.element_size(), _stream(stream), C.byref(out)),
           "esp_create")
    return int(out.value)


def esp_score_select(ctx: int, prices, choice, stream=None) -> None:
    _check(lib().esp_score_select(ctx, _ptr(prices), _ptr(choice), _stream(stream)), "esp_score_select")


def esp_reduce_demand(ctx: int, choice, demand, stream=None) -> None:
    _check(lib().esp_reduce_demand(ctx, _ptr(choice), _ptr(demand), _stream(stream)), "esp_reduce_demand")


def esp_update_prices(ctx: int, demand, t: int, prices, stream=None) -> None:
    _check(lib().esp_update_prices(ctx, _ptr(demand), int(t), _ptr(prices), _stream(stream)),
           "esp_update_prices")


def esp_solve(ctx: int, prices, iters: int, t_start: int = 1, tol: float = 0.0, choice=None, demand=None,
              trace: Optional[esp_trace] = None, iters_done=None, stream=None) -> None:
    _check(lib().esp_solve(ctx, _ptr(prices), int(iters), int(t_start), float(tol), _ptr(choice), _ptr(demand),
                           None if trace is None else C.addressof(trace), _ptr(iters_done), _stream(stream)),
           "esp_solve")


def esp_solve_noalloc(ctx: int, prices, iters: int, t_start: int = 1, tol: float = 0.0, choice=None, demand=None,
                      trace: Optional[esp_trace] = None, iters_done=None, stream=None) -> None:
    _check(lib().esp_solve_noalloc(ctx, _ptr(prices), int(iters), int(t_start), float(tol), _ptr(choice),
                                   _ptr(demand), None if trace is None else C.addressof(trace), _ptr(iters_done),
                                   _stream(stream)), "esp_solve_noalloc")


def esp_set_penalties(ctx: int, current=None, switch_cost=None, penalty=None, stream=None) -> None:
    cur = None if current is None else np.ascontiguousarray(current, dtype=np.int32)
    swc = None if switch_cost is None else np.ascontiguousarray(switch_cost, dtype=np.float64)
    pen = None if penalty is None else np.ascontiguousarray(penalty, dtype=np.float32)
    _check(lib().esp_set_penalties(ctx, _np_ptr(cur), _np_ptr(swc), _np_ptr(pen), _stream(stream)),
           "esp_set_penalties")


def esp_device_status(ctx: int, stream=None) -> int:
    return int(lib().esp_device_status(ctx, _stream(stream)))


def esp_loop_driver(ctx: int) -> int:
    mode = C.c_int32(0)
    _check(lib().esp_loop_driver(ctx, C.byref(mode)), "esp_loop_driver")
    return int(mode.value)


def esp_set_capacity(ctx: int, capacity, stream=None) -> None:
    cap = np.ascontiguousarray(capacity, dtype=np.float64)
    _check(lib().esp_set_capacity(ctx, _np_ptr(cap), _stream(stream)), "esp_set_capacity")


def esp_effective_capacity(ctx: int, queue: Optional[int], queued, gamma: float, capacity_eff=None,
                           stream=None) -> None:
    _check(lib().esp_effective_capacity(ctx, queue, _ptr(queued), float(gamma), _ptr(capacity_eff),
                                        _stream(stream)), "esp_effective_capacity")


def esp_read_penalties(ctx: int, nnz_total: int, stream=None) -> np.ndarray:
    out = np.empty(nnz_total, dtype=np.float32)
    _check(lib().esp_read_penalties(ctx, out.ctypes.data, _stream(stream)), "esp_read_penalties")
    return out


def esp_schedule(ctx: int, model: esp_iac_model, max_rounds: int, iters: int, tol: float, prices, choice,
                 gpu_jobs, rounds_used, violations, stream=None) -> None:
    _check(lib().esp_schedule(ctx, C.addressof(model), int(max_rounds), int(iters), float(tol), _ptr(prices),
                              _ptr(choice), _ptr(gpu_jobs), _ptr(rounds_used), _ptr(violations), _stream(stream)),
           "esp_schedule")


def esp_nearest_profile(store: int, num_queries: int, family, query, nearest, estimate=None, stream=None) -> None:
    _check(lib().esp_nearest_profile(store, int(num_queries), _ptr(family), _ptr(query), _ptr(nearest),
                                     _ptr(estimate), _stream(stream)), "esp_nearest_profile")


def esp_destroy(ctx: int) -> None:
    _check(lib().esp_destroy(ctx), "esp_destroy")


# ---------------------------------------------------------------------------
# Convenience wrapper: owns the workspace tensor and the context
# ---------------------------------------------------------------------------

class Solver:
    """A packed problem on one GPU.  `inst` is any object with the fields of a
    logical problem (offsets, utility, demand, capacity, feasible, eta0, rule,
    dense_k)."""

    def __init__(self, inst, device="cuda:0", blocks_per_cluster: int = 0, sweep_order: int = 0,
                 mode: int = ESP_MODE_AUTO, stream=None, flags: int = 0):
        if not torch.cuda.is_available():
            raise RuntimeError("no GPU: the ESP library has no CPU path")
        self.device = torch.device(device)
        self.problem = Problem.from_instance(inst)
        self.B, self.N, self.R = self.problem.B, self.problem.N, self.problem.R
        self.nnz = int(self.problem.utility.shape[1])
        self.options = esp_options(int(blocks_per_cluster), int(sweep_order), int(mode), int(flags))
        nbytes = esp_workspace_size(self.problem, self.options)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=self.device)
        with torch.cuda.device(self.device):
            self.ctx = esp_create(self.problem, int(inst.rule), inst.eta0, self.workspace, self.options, stream)
        self.problem = None            # host arrays are no longer needed

    def close(self) -> None:
        if getattr(self, "ctx", None):
            esp_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def prices(self, lam) -> torch.Tensor:
        return torch.as_tensor(np.asarray(lam, dtype=np.float64).reshape(self.B, self.R),
                               device=self.device).contiguous()

    def score_select(self, prices: torch.Tensor, stream=None) -> torch.Tensor:
        ch = torch.empty((self.B, self.N), dtype=torch.int32, device=self.device)
        esp_score_select(self.ctx, prices, ch, stream)
        return ch

    def reduce_demand(self, choice: torch.Tensor, stream=None) -> torch.Tensor:
        U = torch.empty((self.B, self.R), dtype=torch.float64, device=self.device)
        esp_reduce_demand(self.ctx, choice, U, stream)
        return U

    def update_prices(self, demand: torch.Tensor, t: int, prices: torch.Tensor, stream=None) -> None:
        esp_update_prices(self.ctx, demand, t, prices, stream)

    def solve(self, prices: torch.Tensor, iters: int, t_start: int = 1, tol: float = 0.0, trace: bool = False,
              trace_choice: bool = False, stream=None, final_select: bool = True) -> dict:
        """Run `iters` iterations in place on `prices`; returns device tensors.
        final_select=False omits the re-selection at the final prices (no
        "choice" / "U" outputs)."""
        out = {"iters_done": torch.empty(self.B, dtype=torch.int32, device=self.device)}
        if final_select:
            out["choice"] = torch.empty((self.B, self.N), dtype=torch.int32, device=self.device)
            out["U"] = torch.empty((self.B, self.R), dtype=torch.float64, device=self.device)
        tr = None
        if trace or trace_choice:
            T = max(int(iters), 1)
            if trace:
                out["tr_lam"] = torch.full((T, self.B, self.R), float("nan"), dtype=torch.float64,
                                           device=self.device)
                out["tr_U"] = torch.full((T, self.B, self.R), float("nan"), dtype=torch.float64, device=self.device)
            if trace_choice:
                out["tr_choice"] = torch.full((T, self.B, self.N), -1, dtype=torch.int32, device=self.device)
            tr = esp_trace(_ptr(out.get("tr_lam")), _ptr(out.get("tr_U")), _ptr(out.get("tr_choice")))
        esp_solve(self.ctx, prices, iters, t_start, tol, out.get("choice"), out.get("U"), tr, out["iters_done"],
                  stream)
        out["lam"] = prices
        return out

    def set_penalties(self, current=None, switch_cost=None, penalty=None, stream=None) -> None:
        esp_set_penalties(self.ctx, current, switch_cost, penalty, stream)

    def device_status(self, stream=None) -> int:
        return esp_device_status(self.ctx, stream)

    def read_penalties(self, stream=None) -> np.ndarray:
        """Current interference penalties Gamma, [B, nnz] float32 (host)."""
        return esp_read_penalties(self.ctx, self.B * self.nnz, stream).reshape(self.B, self.nnz)

    def schedule(self, model, prices, max_rounds: int, iters: int, tol: float = 0.0, stream=None) -> dict:
        """Alg. 1 rounds in place on `prices`.  `model` has the fields of
        esp_iac_model (gpus host int array [B]; sensitivity, pressure
        float32 [B, nnz] and tau_base float64 [B, N], host or device)."""
        dev = self.device

        def on_dev(x, dt):
            t = torch.as_tensor(np.asarray(x) if not isinstance(x, torch.Tensor) else x).to(dev, dt)
            return t.contiguous()

        gpus = np.ascontiguousarray(model.gpus, dtype=np.int32).reshape(self.B)
        keep = {"sa": on_dev(model.sensitivity, torch.float32), "pr": on_dev(model.pressure, torch.float32),
                "tb": on_dev(model.tau_base, torch.float64)}
        m = esp_iac_model(gpus.ctypes.data, float(model.gpu_memory), float(model.gpu_compute), int(model.r_gpus),
                          int(model.r_mem), int(model.r_sm), _ptr(keep["sa"]), _ptr(keep["pr"]), _ptr(keep["tb"]),
                          float(model.beta), float(model.beta_max), float(model.u_target), float(model.kappa))
        gmax = int(gpus.max())
        out = {
            "choice": torch.empty((self.B, self.N), dtype=torch.int32, device=dev),
            "gpu_jobs": torch.empty((self.B, gmax, ESP_MAX_PER_GPU), dtype=torch.int32, device=dev),
            "rounds": torch.empty(self.B, dtype=torch.int32, device=dev),
            "violations": torch.empty(self.B, dtype=torch.int32, device=dev),
        }
        esp_schedule(self.ctx, m, max_rounds, iters, tol, prices, out["choice"], out["gpu_jobs"], out["rounds"],
                     out["violations"], stream)
        out["lam"] = prices
        out["_keep"] = keep
        return out

    def nearest_profile(self, family, query, stream=None):
        """RST fallback with this context as the profile store: family
        int32 [B, Q] and query float32 [B, Q, R] device tensors -> (nearest
        int32 [B, Q], estimate float32 [B, Q])."""
        assert family.dtype == torch.int32 and query.dtype == torch.float32
        assert family.is_contiguous() and query.is_contiguous()
        assert family.dim() == 2 and family.shape[0] == self.B
        Q = family.shape[1]
        assert tuple(query.shape) == (self.B, Q, self.R)
        nearest = torch.empty((self.B, Q), dtype=torch.int32, device=self.device)
        est = torch.empty((self.B, Q), dtype=torch.float32, device=self.device)
        esp_nearest_profile(self.ctx, Q, family, query, nearest, est, stream)
        return nearest, est

    def loop_driver(self) -> int:
        return esp_loop_driver(self.ctx)

    def set_capacity(self, capacity, stream=None) -> None:
        esp_set_capacity(self.ctx, capacity, stream)

    def effective_capacity(self, queue: Optional["Solver"], gamma: float, queued=None, stream=None):
        """Eq. 12 with `queue` holding the pending jobs (None: no pending
        job); installs C_eff as this context's capacity and returns it as a
        [B, R] float64 tensor.  queued: optional uint8 [B, N_queue] tensor on
        the device (nonzero = pending)."""
        out = torch.empty((self.B, self.R), dtype=torch.float64, device=self.device)
        if queued is not None:
            assert queued.dtype == torch.uint8 and queued.is_contiguous() and queued.device == out.device
            assert queue is not None and tuple(queued.shape) == (queue.B, queue.N)
        esp_effective_capacity(self.ctx, None if queue is None else queue.ctx, queued, gamma, out, stream)
        return out
