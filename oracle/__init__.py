"""CPU oracle for Elastic Shadow Pricing -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The HIP library and its Python binding
never import it; the two share no code.

A thin ctypes layer over ``esp_oracle.c`` (plain single-threaded C, fp64,
``-ffp-contract=off``), which follows the paper's Sec. 3.2 (Eq. 6-8): per-job
argmax of utility minus price-weighted demand, exact aggregate demand, and the
projected-subgradient price update; Sec. 3.4's effective capacity (Eq. 12);
and RST's nearest-profile fallback (Sec. 3.1.2).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "esp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle_esp.so")

CFLAGS = ["-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
          "-Wall", "-Wextra"]


def build(force: bool = True) -> str:
    """Compile the oracle library with gcc (x86-64 SSE2 binary64, no contraction)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.run(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


MAX_PER_GPU = 4
MAX_SHARDS = 8


class _Iac(C.Structure):
    _fields_ = [
        ("G", C.c_int32), ("gpu_memory", C.c_double), ("gpu_compute", C.c_double),
        ("r_gpus", C.c_int32), ("r_mem", C.c_int32), ("r_sm", C.c_int32),
        ("sensitivity", C.c_void_p), ("pressure", C.c_void_p), ("tau_base", C.c_void_p),
        ("beta", C.c_double), ("beta_max", C.c_double), ("u_target", C.c_double), ("kappa", C.c_double),
    ]


class _Problem(C.Structure):
    _fields_ = [
        ("B", C.c_int32), ("N", C.c_int32), ("R", C.c_int32), ("nnz", C.c_int64),
        ("offsets", C.c_void_p), ("utility", C.c_void_p), ("demand", C.c_void_p),
        ("feasible", C.c_void_p), ("capacity", C.c_void_p), ("eta0", C.c_void_p),
        ("rule", C.c_int32), ("current", C.c_void_p), ("switch_cost", C.c_void_p),
        ("penalty", C.c_void_p),
    ]


_lib = None


def bind(path: str):
    """Load an oracle library build and declare its signatures."""
    L = C.CDLL(path)
    _declare(L)
    return L


def lib():
    global _lib
    if _lib is None:
        build(force=False)
        _lib = bind(_LIB)
    return _lib


def _declare(L):
    vp, i32, i64, dbl = C.c_void_p, C.c_int32, C.c_int64, C.c_double
    L.orc_exact_sum_f32.argtypes = [vp, i64]
    L.orc_exact_sum_f32.restype = dbl
    L.orc_score.argtypes = [vp, C.c_int, i64, i32, vp]
    L.orc_score.restype = dbl
    L.orc_select.argtypes = [vp, C.c_int, vp, vp]
    L.orc_select.restype = None
    L.orc_demand.argtypes = [vp, C.c_int, vp, vp]
    L.orc_demand.restype = None
    L.orc_eta.argtypes = [C.c_int, dbl, i64]
    L.orc_eta.restype = dbl
    L.orc_update.argtypes = [C.c_int, vp, vp, dbl, vp]
    L.orc_update.restype = None
    L.orc_dual_value.argtypes = [vp, C.c_int, vp, vp]
    L.orc_dual_value.restype = dbl
    L.orc_primal_value.argtypes = [vp, C.c_int, vp]
    L.orc_primal_value.restype = dbl
    L.orc_solve.argtypes = [vp, vp, i32, i32, dbl, vp, vp, vp, vp, vp, vp, vp, vp]
    L.orc_solve.restype = C.c_int
    L.orc_effective_capacity.argtypes = [vp, C.c_int, vp, vp, dbl, vp]
    L.orc_effective_capacity.restype = C.c_int
    L.orc_binpack.argtypes = [vp, C.c_int, vp, vp, vp]
    L.orc_binpack.restype = i64
    L.orc_iac_eval.argtypes = [vp, C.c_int, vp, vp, vp, vp]
    L.orc_iac_eval.restype = i64
    L.orc_schedule.argtypes = [vp, C.c_int, vp, i32, i32, dbl, vp, vp, vp, vp, vp, vp]
    L.orc_schedule.restype = C.c_int
    L.orc_nearest.argtypes = [vp, C.c_int, i64, vp, vp]
    L.orc_nearest.restype = i32
    L.orc_nearest_batch.argtypes = [vp, C.c_int, i64, vp, vp, vp, vp]
    L.orc_nearest_batch.restype = None


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def exact_sum_f32(values, L=None) -> float:
    """Exact sum of non-negative float32 values, rounded once to float64."""
    v = np.ascontiguousarray(values, dtype=np.float32)
    return float((L or lib()).orc_exact_sum_f32(_p(v), v.size))


def eta(rule: int, eta0: float, t: int, L=None) -> float:
    return float((L or lib()).orc_eta(rule, eta0, t))


def update(U, Cap, eta_t: float, lam, L=None) -> np.ndarray:
    U = np.ascontiguousarray(U, dtype=np.float64)
    Cap = np.ascontiguousarray(Cap, dtype=np.float64)
    out = np.array(lam, dtype=np.float64, copy=True)
    (L or lib()).orc_update(out.size, _p(U), _p(Cap), eta_t, _p(out))
    return out


class Oracle:
    """Oracle bound to one logical instance (a ``workloads.Instance`` or any
    object with the same fields)."""

    def __init__(self, inst, L=None):
        self.L = L or lib()
        self.inst = inst
        self.offsets = np.ascontiguousarray(inst.offsets, dtype=np.int64)
        self.utility = np.ascontiguousarray(inst.utility, dtype=np.float32)
        self.demand = np.ascontiguousarray(inst.demand, dtype=np.float32)
        self.capacity = np.ascontiguousarray(inst.capacity, dtype=np.float64)
        self.eta0 = np.ascontiguousarray(inst.eta0, dtype=np.float64)
        self.feasible = (None if inst.feasible is None
                         else np.ascontiguousarray(inst.feasible, dtype=np.uint8))
        self.B, self.N, self.R = self.utility.shape[0], self.offsets.size - 1, self.demand.shape[2]
        self.rule = int(inst.rule)
        cur = getattr(inst, "current", None)
        pen = getattr(inst, "penalty", None)
        self.current = None if cur is None else np.ascontiguousarray(cur, dtype=np.int32)
        self.switch_cost = (None if cur is None else
                            np.ascontiguousarray(getattr(inst, "switch_cost"), dtype=np.float64))
        self.penalty = None if pen is None else np.ascontiguousarray(pen, dtype=np.float32)
        self._prob = _Problem(self.B, self.N, self.R, int(self.offsets[-1]),
                              _p(self.offsets), _p(self.utility), _p(self.demand),
                              _p(self.feasible), _p(self.capacity), _p(self.eta0), self.rule,
                              _p(self.current), _p(self.switch_cost), _p(self.penalty))
        self._pp = C.addressof(self._prob)

    # single steps -------------------------------------------------------
    def score(self, b: int, j: int, k: int, lam) -> float:
        lam = np.ascontiguousarray(lam, dtype=np.float64)
        return float(self.L.orc_score(self._pp, b, j, k, _p(lam)))

    def select(self, b: int, lam) -> np.ndarray:
        lam = np.ascontiguousarray(lam, dtype=np.float64)
        ch = np.empty(self.N, dtype=np.int32)
        self.L.orc_select(self._pp, b, _p(lam), _p(ch))
        return ch

    def demand_sum(self, b: int, choice) -> np.ndarray:
        ch = np.ascontiguousarray(choice, dtype=np.int32)
        U = np.empty(self.R, dtype=np.float64)
        self.L.orc_demand(self._pp, b, _p(ch), _p(U))
        return U

    def eta(self, b: int, t: int) -> float:
        return eta(self.rule, float(self.eta0[b]), t, self.L)

    def step(self, b: int, lam, t: int):
        """One iteration at lambda^t: (choice c^t, U^t, lambda^{t+1})."""
        ch = self.select(b, lam)
        U = self.demand_sum(b, ch)
        return ch, U, update(U, self.capacity[b], self.eta(b, t), lam, self.L)

    def dual_value(self, b: int, lam, choice) -> float:
        lam = np.ascontiguousarray(lam, dtype=np.float64)
        ch = np.ascontiguousarray(choice, dtype=np.int32)
        return float(self.L.orc_dual_value(self._pp, b, _p(lam), _p(ch)))

    def primal_value(self, b: int, choice) -> float:
        ch = np.ascontiguousarray(choice, dtype=np.int32)
        return float(self.L.orc_primal_value(self._pp, b, _p(ch)))

    def effective_capacity(self, b: int, capacity, gamma: float, queued=None) -> np.ndarray:
        """Eq. 12 with this instance as the pending jobs of cluster b:
        capacity - gamma * (exact sum over pending jobs of their componentwise
        smallest demand vector).  queued: optional [N] mask (nonzero = pending)."""
        cap = np.ascontiguousarray(capacity, dtype=np.float64)
        q = None if queued is None else np.ascontiguousarray(queued, dtype=np.uint8)
        out = np.empty(self.R, dtype=np.float64)
        rc = self.L.orc_effective_capacity(self._pp, b, _p(q), _p(cap), float(gamma), _p(out))
        if rc != 0:
            raise ValueError("oracle: a pending job has no allowed configuration")
        return out

    def nearest(self, b: int, family: int, q):
        """RST nearest-profile fallback for one query: (index within the
        family or -1, squared l2 distance of the winner)."""
        q = np.ascontiguousarray(q, dtype=np.float32)
        d2 = C.c_double(0.0)
        k = int(self.L.orc_nearest(self._pp, b, int(family), _p(q), C.byref(d2)))
        return k, float(d2.value)

    def nearest_batch(self, b: int, family, queries):
        """Batch of queries (family [Q] int32, queries [Q, R] float32):
        (nearest index [Q] int32, throughput estimate [Q] float32)."""
        fam = np.ascontiguousarray(family, dtype=np.int32)
        q = np.ascontiguousarray(queries, dtype=np.float32).reshape(fam.size, self.R)
        k = np.empty(fam.size, dtype=np.int32)
        est = np.empty(fam.size, dtype=np.float32)
        self.L.orc_nearest_batch(self._pp, b, fam.size, _p(fam), _p(q), _p(k), _p(est))
        return k, est

    # Alg. 1 outer rounds ---------------------------------------------------
    def _iac(self, model, b):
        sa = np.ascontiguousarray(model.sensitivity, dtype=np.float32)
        pr = np.ascontiguousarray(model.pressure, dtype=np.float32)
        tb = np.ascontiguousarray(model.tau_base, dtype=np.float64)
        keep = (sa, pr, tb)
        m = _Iac(int(model.gpus[b]), float(model.gpu_memory), float(model.gpu_compute), int(model.r_gpus),
                 int(model.r_mem), int(model.r_sm), _p(sa), _p(pr), _p(tb), float(model.beta),
                 float(model.beta_max), float(model.u_target), float(model.kappa))
        return m, keep

    def binpack(self, b: int, model, choice):
        """First-fit BinPack of cluster b's selection: (occupants [G, 4], shares placed)."""
        m, keep = self._iac(model, b)
        ch = np.ascontiguousarray(choice, dtype=np.int32)
        occ = np.empty((m.G, MAX_PER_GPU), dtype=np.int32)
        placed = int(self.L.orc_binpack(self._pp, b, C.byref(m), _p(ch), _p(occ)))
        return occ, placed

    def iac_eval(self, b: int, model, choice, occ):
        """Co-located pairs against Eq. 11: (violating pairs, largest excess per job [N])."""
        m, keep = self._iac(model, b)
        ch = np.ascontiguousarray(choice, dtype=np.int32)
        oc = np.ascontiguousarray(occ, dtype=np.int32)
        inc = np.empty(self.N, dtype=np.float64)
        V = int(self.L.orc_iac_eval(self._pp, b, C.byref(m), _p(ch), _p(oc), _p(inc)))
        return V, inc

    def schedule(self, b: int, model, rounds: int, iters: int, tol: float = 0.0, lam0=None) -> dict:
        """Alg. 1 on cluster b: prices, choice, occupants of the last round,
        rounds run, violating pairs of the last round, final penalties."""
        m, keep = self._iac(model, b)
        lam = np.array(self.inst.lam0[b] if lam0 is None else lam0, dtype=np.float64).reshape(self.R).copy()
        # the instance's interference penalties as the starting Gamma (Alg. 1 resets them)
        pen = (np.zeros(int(self.offsets[-1]), dtype=np.float32) if self.penalty is None
               else self.penalty[b].copy())
        ch = np.empty(self.N, dtype=np.int32)
        occ = np.empty((m.G, MAX_PER_GPU), dtype=np.int32)
        nr = C.c_int32(0)
        nv = C.c_int64(0)
        rc = self.L.orc_schedule(self._pp, b, C.byref(m), int(rounds), int(iters), float(tol), _p(lam), _p(pen),
                                 _p(ch), _p(occ), C.byref(nr), C.byref(nv))
        if rc != 0:
            raise ValueError(f"oracle: schedule failed (rc={rc})")
        return {"lam": lam, "penalty": pen, "choice": ch, "occ": occ, "rounds": int(nr.value),
                "violations": int(nv.value)}

    # whole loop ---------------------------------------------------------
    def solve(self, lam0=None, iters: Optional[int] = None, t_start: int = 1, tol: float = 0.0,
              trace: bool = True, trace_choice: bool = False, duals: bool = True) -> dict:
        """The loop of Sec. 3.2.3 from lam0 for `iters` iterations starting at
        step index t_start.  trace: per-iteration prices and demand (and, with
        duals, the dual and primal values); trace_choice: per-iteration
        selections.  A solve continued from another's final prices with
        t_start advanced reproduces the longer solve's iterates."""
        T = int(self.inst.iters if iters is None else iters)
        B, N, R = self.B, self.N, self.R
        lam = np.array(self.inst.lam0 if lam0 is None else lam0, dtype=np.float64).reshape(B, R).copy()
        out = {
            "choice": np.empty((B, N), dtype=np.int32),
            "U": np.empty((B, R), dtype=np.float64),
            "iters_done": np.empty(B, dtype=np.int32),
        }
        if trace:
            out["tr_lam"] = np.full((T, B, R), np.nan)
            out["tr_U"] = np.full((T, B, R), np.nan)
            if duals:
                out["tr_dual"] = np.full((T, B), np.nan)
                out["tr_primal"] = np.full((T, B), np.nan)
        if trace_choice:
            out["tr_choice"] = np.full((T, B, N), -1, dtype=np.int32)
        rc = self.L.orc_solve(self._pp, _p(lam), T, t_start, tol,
                             _p(out.get("tr_lam")), _p(out.get("tr_U")), _p(out.get("tr_choice")),
                             _p(out.get("tr_dual")), _p(out.get("tr_primal")),
                             _p(out["choice"]), _p(out["U"]), _p(out["iters_done"]))
        if rc != 0:
            raise ValueError(f"oracle: a job family has no allowed configuration (rc={rc})")
        out["lam"] = lam
        return out
