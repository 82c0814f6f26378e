"""Test helpers: golden-fixture parsing, brute-force optimum, LP bound.

None of this is the method: brute force enumerates Eq. 1-3 directly and the LP
is the continuous relaxation of Eq. 1-3 solved by SciPy's HiGHS.
"""
from __future__ import annotations

import itertools
import os
from fractions import Fraction

import numpy as np

import workloads

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def read_golden(name: str) -> dict:
    """Parse a golden text fixture: 'key v1 v2 ...' lines, '|' groups, '#' comments."""
    out: dict = {"trace": []}
    with open(os.path.join(GOLDEN, name)) as f:
        for ln in f:
            ln = ln.split("#", 1)[0].strip()
            if not ln:
                continue
            key, _, rest = ln.partition(" ")
            if key in ("case", "query", "masked_query", "result"):
                out.setdefault(key + "s" if key != "case" else "cases", []).append(
                    [[float(x) for x in g.split()] for g in rest.split("|")])
            elif key == "trace":
                out["trace"].append([[float(x) for x in g.split()] for g in rest.split("|")])
            elif "|" in rest:
                out[key] = [[float(x) for x in g.split()] for g in rest.split("|")]
            else:
                vals = rest.split()
                try:
                    out[key] = [float(x) for x in vals]
                except ValueError:
                    out[key] = vals
    return out


def golden_instance(g: dict) -> workloads.Instance:
    offsets = np.array(g["offsets"], dtype=np.int64)
    nnz = int(offsets[-1])
    util = np.array(g["utility"], dtype=np.float32).reshape(1, nnz)
    dem = np.array(g["demand"], dtype=np.float32).reshape(1, nnz, -1)
    R = dem.shape[2]
    cap = np.array(g["capacity"], dtype=np.float64).reshape(1, R)
    rule = workloads.STEP_CONST if g["rule"] == ["const"] else workloads.STEP_INV_SQRT
    lam0 = np.array(g.get("lam0", [0.0] * R), dtype=np.float64).reshape(1, R)
    inst = workloads.Instance("golden", 0, offsets, util, dem, cap,
                              np.array(g["eta0"], dtype=np.float64), rule, lam0, int(g["iters"][0]))
    if "current" in g:
        inst.current = np.array(g["current"], dtype=np.int32).reshape(1, -1)
        inst.switch_cost = np.array(g["switch_cost"], dtype=np.float64)
    if "penalty" in g:
        inst.penalty = np.array(g["penalty"], dtype=np.float32).reshape(1, nnz)
    return inst


def penalized_utility(inst, b, j, k) -> Fraction:
    """u_jk less the penalty of Eq. 7 (switching cost, interference), exactly."""
    e = int(inst.offsets[j]) + k
    v = Fraction(float(inst.utility[b, e]))
    cur = getattr(inst, "current", None)
    if cur is not None and cur[b, j] >= 0 and k != cur[b, j]:
        v -= Fraction(float(inst.switch_cost[b]))
    pen = getattr(inst, "penalty", None)
    if pen is not None:
        v -= Fraction(float(pen[b, e]))
    return v


def brute_force_optimum(inst: workloads.Instance, b: int = 0):
    """max sum_j u_{j,c_j} (less Eq. 7's penalty when given) over all
    selections with sum_j d_{j,c_j} <= C (Eq. 1-3), in exact rational
    arithmetic.  Returns (P*, argmax tuple) or (None, None) when no selection
    is feasible."""
    off = inst.offsets
    N, R = inst.N, inst.R
    fam = [range(int(off[j + 1] - off[j])) for j in range(N)]
    u = [[penalized_utility(inst, b, j, k) for k in fam[j]] for j in range(N)]
    d = [[[Fraction(float(inst.demand[b, off[j] + k, r])) for r in range(R)] for k in fam[j]]
         for j in range(N)]
    cap = [Fraction(float(c)) for c in inst.capacity[b]]
    allowed = None if inst.feasible is None else inst.feasible[b]
    best, arg = None, None
    for combo in itertools.product(*fam):
        if allowed is not None and any(allowed[off[j] + k] == 0 for j, k in enumerate(combo)):
            continue
        ok = True
        for r in range(R):
            if sum(d[j][k][r] for j, k in enumerate(combo)) > cap[r]:
                ok = False
                break
        if not ok:
            continue
        v = sum(u[j][k] for j, k in enumerate(combo))
        if best is None or v > best:
            best, arg = v, combo
    return best, arg


def lp_optimum(inst: workloads.Instance, b: int = 0) -> float:
    """Continuous relaxation of Eq. 1-3 (x_jk in [0,1], sum_k x_jk = 1),
    solved by scipy.optimize.linprog with the HiGHS method."""
    from scipy.optimize import linprog
    off = inst.offsets
    N, R, nnz = inst.N, inst.R, inst.nnz
    c = -np.array([float(penalized_utility(inst, b, j, k)) for j in range(N)
                   for k in range(int(off[j + 1] - off[j]))])
    A_eq = np.zeros((N, nnz))
    for j in range(N):
        A_eq[j, off[j]:off[j + 1]] = 1.0
    A_ub = inst.demand[b].astype(np.float64).T
    ub = [(0.0, 0.0) if (inst.feasible is not None and inst.feasible[b, e] == 0) else (0.0, None)
          for e in range(nnz)]
    res = linprog(c, A_ub=A_ub, b_ub=inst.capacity[b], A_eq=A_eq, b_eq=np.ones(N), bounds=ub,
                  method="highs")
    assert res.status in (0, 2), res.message
    return float("nan") if res.status == 2 else -float(res.fun)


def exact_score(inst, b, e, lam, j=None) -> Fraction:
    """Exact rational score of entry e (job j), penalties included."""
    if j is None:
        j = int(np.searchsorted(inst.offsets, e, side="right") - 1)
    s = penalized_utility(inst, b, j, e - int(inst.offsets[j]))
    for r in range(inst.R):
        s -= Fraction(float(lam[r])) * Fraction(float(inst.demand[b, e, r]))
    return s


def queue_instance(offsets, demand, feasible=None, capacity=None) -> workloads.Instance:
    """An instance holding pending jobs' families (demand only: the utility of
    a pending job does not enter Eq. 12)."""
    offsets = np.asarray(offsets, dtype=np.int64)
    nnz = int(offsets[-1])
    dem = np.asarray(demand, dtype=np.float32).reshape(1, nnz, -1)
    R = dem.shape[2]
    cap = (np.zeros((1, R)) if capacity is None else np.asarray(capacity, dtype=np.float64).reshape(1, R))
    inst = workloads.Instance("queue", 0, offsets, np.zeros((1, nnz), np.float32), dem, cap,
                              np.array([0.1]), workloads.STEP_CONST, np.zeros((1, R)), 1)
    if feasible is not None:
        inst.feasible = np.asarray(feasible, dtype=np.uint8).reshape(1, nnz)
    return inst


def brute_effective_capacity(inst, b, capacity, gamma, queued=None) -> np.ndarray:
    """Eq. 12 in exact rationals: per pending job the componentwise minimum over
    its allowed configurations, summed exactly, rounded once (Python's
    correctly rounded Fraction -> float), then gamma * S and C - that in
    binary64."""
    off = inst.offsets
    out = np.empty(inst.R)
    for r in range(inst.R):
        S = Fraction(0)
        for j in range(inst.N):
            if queued is not None and not queued[j]:
                continue
            vals = [Fraction(float(inst.demand[b, e, r])) for e in range(off[j], off[j + 1])
                    if inst.feasible is None or inst.feasible[b, e]]
            S += min(vals)
        out[r] = float(capacity[r]) - float(gamma) * float(S)
    return out


def store_instance(offsets, utility, demand, feasible=None) -> workloads.Instance:
    """An instance used as a profile store: family f = job type f, utility =
    profiled throughput, demand = resource vector."""
    offsets = np.asarray(offsets, dtype=np.int64)
    nnz = int(offsets[-1])
    dem = np.asarray(demand, dtype=np.float32).reshape(1, nnz, -1)
    R = dem.shape[2]
    inst = workloads.Instance("store", 0, offsets, np.asarray(utility, np.float32).reshape(1, nnz), dem,
                              np.zeros((1, R)), np.array([0.1]), workloads.STEP_CONST, np.zeros((1, R)), 1)
    if feasible is not None:
        inst.feasible = np.asarray(feasible, dtype=np.uint8).reshape(1, nnz)
    return inst


def exact_sq_dist(q, v) -> Fraction:
    return sum((Fraction(float(a)) - Fraction(float(b))) ** 2 for a, b in zip(q, v))


def schedule_fixture(name: str = "hand_schedule.txt"):
    """The instance, the IAC model and the expected results of a hand-derived
    Alg. 1 fixture."""
    g = read_golden(name)
    inst = golden_instance(g)
    B, nnz, N = 1, inst.nnz, inst.N
    m = workloads.IacModel(np.array([int(g["gpus"][0])], np.int32), g["gpu_memory"][0], g["gpu_compute"][0],
                           *[int(x) for x in g["resources"]],
                           np.array(g["sensitivity"], np.float32).reshape(B, nnz),
                           np.array(g["pressure"], np.float32).reshape(B, nnz),
                           np.array(g["tau_base"], np.float64).reshape(B, N),
                           g["beta"][0], g["beta_max"][0], g["u_target"][0], g["kappa"][0])
    return inst, m, g["results"]


def check_first_fit(inst, b, model, choice, occ):
    """Checks that occ is the first-fit packing of the selection: capacities
    respected, and replaying the jobs in index order, each job sits on the
    first g GPUs that had room, or is absent when fewer than g had room."""
    G = int(model.gpus[b])
    mem = [float(model.gpu_memory)] * G
    sm = [float(model.gpu_compute)] * G
    cnt = [0] * G
    where = {}
    for h in range(G):
        for i, j in enumerate(occ[h]):
            if j >= 0:
                where.setdefault(int(j), []).append((h, i))
    for j in range(inst.N):
        e = inst.offsets[j] + choice[j]
        gv = float(inst.demand[b, e, model.r_gpus])
        placeable = 1.0 <= gv <= 8.0 and gv == int(gv)
        if not placeable:
            assert j not in where
            continue
        g = int(gv)
        nm = float(inst.demand[b, e, model.r_mem]) / gv
        ns = float(inst.demand[b, e, model.r_sm]) / gv
        room = [h for h in range(G) if cnt[h] < 4 and mem[h] >= nm and sm[h] >= ns]
        if len(room) < g:
            assert j not in where, j
            continue
        got = sorted(h for h, _ in where[j])
        assert got == room[:g], (j, got, room[:g])
        for h, i in where[j]:
            assert i == cnt[h]                      # placement order on the GPU
            mem[h] -= nm
            sm[h] -= ns
            cnt[h] += 1
    for h in range(G):
        assert all(x == -1 for x in occ[h][cnt[h]:])
