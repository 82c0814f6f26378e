"""Seeded synthetic ESP instances: job x configuration tables of utilities and
resource vectors, per-resource capacities, step rules and iteration counts.

This module is the ONLY code shared by the HIP path's tests/bench and the CPU
oracle.  It draws inputs; it holds none of the method's arithmetic (no scores,
no selection, no demand sums at prices, no price updates).

Random numbers come from a counter-based SplitMix64 (Steele, Lea & Flood,
"Fast splittable pseudorandom number generators", OOPSLA 2014): the value for
(seed, stream, index) is the SplitMix64 output function applied to
``key(seed, stream) + (index + 1) * 0x9E3779B97F4A7C15``, so any single draw
can be recomputed without generating the ones before it.  Every value is
computed in float64 and rounded once to float32 (tables) or kept in float64
(capacities, step sizes, prices).  Parity never depends on libm agreement
across hosts: both sides consume the same in-memory arrays.

The five named workloads follow the paper's problem statement (Sec. 3.2.1,
Eq. 1-5) and the shapes of its workload table (Table 2: 8 training + 4
offline-inference workloads, 12-198 profiles per family, checkpointing / AMP /
micro-batch / batch-size knobs), scaled up.  The paper's profiled tables and
cluster traces are not available; these generators stand in for them.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from typing import Optional

import numpy as np

__all__ = [
    "Instance", "make", "NAMES", "random_small", "uniform_offsets", "with_penalties",
    "STEP_CONST", "STEP_INV_SQRT",
]

STEP_CONST = 0       # eta_t = eta0            (Sec. 3.2.3, Eq. 8 "fixed")
STEP_INV_SQRT = 1    # eta_t = eta0 / sqrt(t)  (Sec. 3.2.3, Eq. 8 "diminishing")

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def _mix(z: np.ndarray) -> np.ndarray:
    """SplitMix64 output function on a uint64 array (wrapping arithmetic)."""
    z = z.copy()
    z ^= z >> np.uint64(30)
    z *= _M1
    z ^= z >> np.uint64(27)
    z *= _M2
    z ^= z >> np.uint64(31)
    return z


def _key(seed: int, stream: int) -> np.uint64:
    k = np.array([(seed * 0x100000001B3 + stream * 0x632BE59BD9B4E019) & ((1 << 64) - 1)],
                 dtype=np.uint64)
    return _mix(k)[0]


def _uniform(seed: int, stream: int, idx: np.ndarray) -> np.ndarray:
    """U[0,1) float64 draws for counter indices ``idx`` (int64/uint64 array)."""
    with np.errstate(over="ignore"):
        z = _key(seed, stream) + (idx.astype(np.uint64) + np.uint64(1)) * _GAMMA
        z = _mix(z)
    return (z >> np.uint64(11)).astype(np.float64) * (1.0 / 9007199254740992.0)


def _normal(seed: int, stream: int, idx: np.ndarray) -> np.ndarray:
    """Standard normal draws by Box-Muller (1958) from two counter streams."""
    u1 = 1.0 - _uniform(seed, stream, idx)          # (0, 1]
    u2 = _uniform(seed, stream + 1000, idx)
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * math.pi * u2)


# Stream ids: one per random field, so fields never share draws.
_S_B, _S_M, _S_S, _S_F, _S_P, _S_Q, _S_CPU, _S_IO = 10, 12, 13, 14, 15, 16, 17, 18
_S_K, _S_TYPE, _S_OFF, _S_STRIDE, _S_BINF, _S_BSAT, _S_W, _S_KV = 20, 21, 22, 23, 24, 25, 26, 27
_S_G, _S_ETA, _S_TINY_U, _S_TINY_D, _S_TINY_K, _S_TINY_C = 30, 31, 40, 41, 42, 43
_S_CUR, _S_PEN = 50, 52
_S_QUEUE = 60
_S_NNF, _S_NNB, _S_NNZ, _S_NNX = 70, 71, 72, 73
_S_IA, _S_IB, _S_IT = 80, 81, 82


@dataclasses.dataclass
class Instance:
    """A logical ESP problem (Sec. 3.2.1): B independent clusters sharing one
    family layout.

    offsets  int64 [N+1]   CSR family boundaries; job j owns entries
                           offsets[j] .. offsets[j+1]-1 (config k = entry - offsets[j]).
    utility  float32 [B, nnz]     u_jk (w_j T_j(c) of Eq. 1, or T/Tmax - Gamma of Eq. 7)
    demand   float32 [B, nnz, R]  R_j(c)[r] >= 0 (Eq. 3)
    capacity float64 [B, R]       C_r (or C_eff of Eq. 12)
    eta0     float64 [B]          step-size scale (Eq. 8)
    lam0     float64 [B, R]       initial prices lambda^1 >= 0
    """
    name: str
    seed: int
    offsets: np.ndarray
    utility: np.ndarray
    demand: np.ndarray
    capacity: np.ndarray
    eta0: np.ndarray
    rule: int
    lam0: np.ndarray
    iters: int
    feasible: Optional[np.ndarray] = None      # uint8 [B, nnz] (Eq. 4 mask) or None
    dense_k: Optional[int] = None              # K when every family has K configs
    # Penalty Gamma of the ESP score (Eq. 7), optional:
    current: Optional[np.ndarray] = None       # int32 [B, N] current configuration, -1 = none
    switch_cost: Optional[np.ndarray] = None   # float64 [B] switching cost gamma_0
    penalty: Optional[np.ndarray] = None       # float32 [B, nnz] interference penalty

    @property
    def B(self) -> int:
        return int(self.utility.shape[0])

    @property
    def N(self) -> int:
        return int(self.offsets.shape[0] - 1)

    @property
    def R(self) -> int:
        return int(self.demand.shape[2])

    @property
    def nnz(self) -> int:
        return int(self.offsets[-1])

    def table_bytes(self) -> int:
        """Bytes of the job x config table one price iteration must read:
        utility plus R demand columns, fp32, for every configuration."""
        return self.B * self.nnz * (1 + self.R) * 4

    def fingerprint(self) -> str:
        h = hashlib.sha256()
        for a in (self.offsets, self.utility, self.demand, self.capacity, self.eta0, self.lam0):
            h.update(np.ascontiguousarray(a).tobytes())
        for extra in (self.feasible, self.current, self.switch_cost, self.penalty):
            if extra is not None:
                h.update(np.ascontiguousarray(extra).tobytes())
        h.update(f"{self.rule}:{self.iters}".encode())
        return h.hexdigest()


def uniform_offsets(n: int, k: int) -> np.ndarray:
    return np.arange(n + 1, dtype=np.int64) * k


def _f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


# ---------------------------------------------------------------------------
# Tiny: 64 x 8 x 4
# ---------------------------------------------------------------------------

def _tiny(seed: int = 0, n_jobs: int = 64) -> Instance:
    """64 jobs x 8 configs x 4 resources (GPU count, GPU memory GB, SM share,
    host memory GB).  Config k enumerates GPU count g = 2^(k mod 4) and the
    checkpoint flag c = k div 4; the SM share s in {0.5, 1} is drawn per
    (job, config).  u = b g^0.85 (1 - 0.25c) s^0.7 with b ~ LogNormal(0, 0.5)
    per job; d = (g, m (1 - 0.4c) g^0.4, g s, 16 g) with m ~ U[8, 70] GB."""
    N, K, R = n_jobs, 8, 4
    j = np.arange(N, dtype=np.int64)
    b = np.exp(0.5 * _normal(seed, _S_B, j))
    m = 8.0 + 62.0 * _uniform(seed, _S_M, j)
    e = np.arange(N * K, dtype=np.int64)
    jj, kk = e // K, e % K
    g = (2.0 ** (kk % 4)).astype(np.float64)
    c = (kk // 4).astype(np.float64)
    s = np.where(_uniform(seed, _S_S, e) < 0.5, 0.5, 1.0)
    u = b[jj] * g ** 0.85 * (1.0 - 0.25 * c) * s ** 0.7
    d = np.stack([g, g * m[jj] * (1.0 - 0.4 * c) / g ** 0.6, g * s, 16.0 * g], axis=1)
    cap = np.array([[64.0, 64.0 * 80.0, 64.0, 64.0 * 512.0]])
    return Instance("tiny", seed, uniform_offsets(N, K), _f32(u)[None], _f32(d)[None], cap,
                    np.array([0.01]), STEP_INV_SQRT, np.zeros((1, R)), 200, dense_k=K)


# ---------------------------------------------------------------------------
# Small: 4096 x 32 x 4
# ---------------------------------------------------------------------------

_MS = np.array([1.0, 0.8, 0.6, 0.45])


def _small(seed: int = 1, n_jobs: int = 4096) -> Instance:
    """4096 jobs x 32 configs x 4 resources.  Config k enumerates
    g = 2^(k div 8), s = (0.5, 1)[(k div 4) mod 2] and a pipeline/recompute
    memory scale ms = (1, 0.8, 0.6, 0.45)[k mod 4], which takes the place of the
    checkpoint flag: memory factor ms, throughput factor 1 - 0.625 (1 - ms)
    (so ms = 0.6 gives the 0.75 of the checkpointed tiny configuration).
    Capacity: 512 GPUs of 80 GB (SM 1 and host memory 512 GB per GPU)."""
    N, K, R = n_jobs, 32, 4
    j = np.arange(N, dtype=np.int64)
    b = np.exp(0.5 * _normal(seed, _S_B, j))
    m = 8.0 + 62.0 * _uniform(seed, _S_M, j)
    e = np.arange(N * K, dtype=np.int64)
    jj, kk = e // K, e % K
    g = 2.0 ** (kk // 8)
    s = np.where((kk // 4) % 2 == 0, 0.5, 1.0)
    ms = _MS[kk % 4]
    u = b[jj] * g ** 0.85 * (1.0 - 0.625 * (1.0 - ms)) * s ** 0.7
    d = np.stack([g, g * m[jj] * ms / g ** 0.6, g * s, 16.0 * g], axis=1)
    cap = np.array([[512.0, 512.0 * 80.0, 512.0, 512.0 * 512.0]])
    return Instance("small", seed, uniform_offsets(N, K), _f32(u)[None], _f32(d)[None], cap,
                    np.array([0.01]), STEP_INV_SQRT, np.zeros((1, R)), 500, dense_k=K)


# ---------------------------------------------------------------------------
# Large / Batched training families: 64 configs, up to 8 resources
# ---------------------------------------------------------------------------

def _training64(seed: int, jobs: np.ndarray, nres: int) -> tuple[np.ndarray, np.ndarray]:
    """Utility [n*64] and demand [n*64, nres] for training jobs with global ids
    ``jobs`` and 64 configs each: k = ((gi*2 + si)*4 + mi)*2 + ai enumerates
    GPU count 2^gi, SM share (0.5, 1)[si], memory scale ms[mi] and AMP ai.
    Resources (first nres of): GPU count, GPU memory GB, SM share, host memory
    GB, PCIe share, NVLink share, host CPU cores, storage-I/O share.  With
    nres == 6 the NVLink and storage columns are left out.  A co-location
    interference factor f ~ U[0.6, 1] per (job, config) multiplies u."""
    K = 64
    n = jobs.shape[0]
    b = np.exp(0.5 * _normal(seed, _S_B, jobs))
    m = 8.0 + 62.0 * _uniform(seed, _S_M, jobs)
    p = 0.05 + 0.45 * _uniform(seed, _S_P, jobs)
    q = 0.05 + 0.55 * _uniform(seed, _S_Q, jobs)
    cpu = np.floor(2.0 + 7.0 * _uniform(seed, _S_CPU, jobs))      # 2..8 cores per GPU
    io = 0.01 + 0.19 * _uniform(seed, _S_IO, jobs)
    kk = np.tile(np.arange(K, dtype=np.int64), n)
    jl = np.repeat(np.arange(n, dtype=np.int64), K)
    e = np.repeat(jobs, K) * K + kk
    a = (kk % 2).astype(np.float64)
    ms = _MS[(kk // 2) % 4]
    s = np.where((kk // 8) % 2 == 0, 0.5, 1.0)
    g = 2.0 ** (kk // 16)
    f = 0.6 + 0.4 * _uniform(seed, _S_F, e)
    thr = b[jl] * g ** 0.85 * (1.0 - 0.625 * (1.0 - ms)) * s ** 0.7 * (1.0 + 0.3 * a)
    u = thr * f
    cols = [
        g,
        g * m[jl] * ms * (1.0 - 0.25 * a) / g ** 0.6,
        g * s,
        16.0 * g,
        g * p[jl] * s,
        g * q[jl] * (1.5 - 0.5 * ms),
        g * cpu[jl],
        io[jl] * np.sqrt(g) * (1.0 + 0.3 * a),
    ]
    if nres == 6:
        cols = [cols[i] for i in (0, 1, 2, 3, 4, 6)]
    else:
        cols = cols[:nres]
    return _f32(u), _f32(np.stack(cols, axis=1))


def _large(seed: int = 2, n_jobs: int = 262144) -> Instance:
    """262,144 jobs x 64 configs x 8 resources; capacity C_r = 0.6 sum_j min_k
    d_jkr (sequential float64 sum); eta = 0.01/sqrt(t); 1000 iterations."""
    N, K, R = n_jobs, 64, 8
    u, d = _training64(seed, np.arange(N, dtype=np.int64), R)
    mins = d.reshape(N, K, R).min(axis=1).astype(np.float64)
    cap = 0.6 * np.sum(mins, axis=0)
    return Instance("large", seed, uniform_offsets(N, K), u[None], d[None], cap[None],
                    np.array([0.01]), STEP_INV_SQRT, np.zeros((1, R)), 1000, dense_k=K)


def _batched(seed: int = 4, n_clusters: int = 256, n_jobs: int = 16384) -> Instance:
    """256 independent clusters of 16,384 jobs x 64 configs x 6 resources.
    Cluster b has G_b ~ U{256..1024} GPUs; capacity per GPU: 1 GPU, 80 GB,
    1 SM, 512 GB host memory, 1 PCIe share, 16 CPU cores.  Step scale
    eta0_b drawn from {0.005, 0.01, 0.02}; eta = eta0_b/sqrt(t); 500 iterations."""
    B, N, K, R = n_clusters, n_jobs, 64, 6
    nnz = N * K
    util = np.empty((B, nnz), dtype=np.float32)
    dem = np.empty((B, nnz, R), dtype=np.float32)
    for bi in range(B):
        u, d = _training64(seed, np.arange(N, dtype=np.int64) + bi * N, R)
        util[bi] = u
        dem[bi] = d
    cl = np.arange(B, dtype=np.int64)
    G = np.floor(256.0 + 769.0 * _uniform(seed, _S_G, cl))
    cap = np.stack([G, 80.0 * G, G, 512.0 * G, G, 16.0 * G], axis=1)
    eta0 = np.array([0.005, 0.01, 0.02])[np.minimum((3.0 * _uniform(seed, _S_ETA, cl)).astype(np.int64), 2)]
    return Instance("batched", seed, uniform_offsets(N, K), util, dem, cap, eta0,
                    STEP_INV_SQRT, np.zeros((B, R)), 500, dense_k=K)


# ---------------------------------------------------------------------------
# Ragged: 1,048,576 jobs, Geometric(0.08) family sizes clipped to [1, 256], CSR
# ---------------------------------------------------------------------------

def _ragged(seed: int = 3, n_jobs: int = 1048576) -> Instance:
    """CSR families of K_j = 1 + floor(ln U / ln 0.92) configs, clipped to
    [1, 256] (mean about 12.5); 6 resources (GPU count, GPU memory, SM share,
    host memory, PCIe share, host CPU cores).  A third of the jobs are offline
    inference (utility = tokens/s), the rest training (utility = throughput x
    interference factor, as in the 64-config training generator).

    Training family: K_j distinct points of a 256-point knob grid
    g(4) x ms(4) x s(2) x AMP(2) x micro-batch mb in {1,2,4,8}, visited as
    (o + i*st) mod 256 with a per-job offset o and odd stride st.
    Inference family: K_j distinct batch sizes from 1..256 (same visiting rule),
    sorted ascending; tokens/s = b_inf B / (1 + B / B_sat); GPU memory =
    weights + KV-per-sequence x B.
    Capacity C_r = S_min + (S_max - S_min)/2 with S_min = sum_j min_k d_jkr and
    S_max = sum_j max_k d_jkr (feasible, and binding for typical prices)."""
    N, R = n_jobs, 6
    j = np.arange(N, dtype=np.int64)
    uk = _uniform(seed, _S_K, j)
    K = 1 + np.floor(np.log1p(-uk) / math.log(1.0 - 0.08)).astype(np.int64)
    K = np.clip(K, 1, 256)
    offsets = np.zeros(N + 1, dtype=np.int64)
    np.cumsum(K, out=offsets[1:])
    nnz = int(offsets[-1])
    infer = _uniform(seed, _S_TYPE, j) < (1.0 / 3.0)
    o = np.floor(256.0 * _uniform(seed, _S_OFF, j)).astype(np.int64)
    st = 2 * np.floor(128.0 * _uniform(seed, _S_STRIDE, j)).astype(np.int64) + 1
    jl = np.repeat(j, K)
    kk = np.arange(nnz, dtype=np.int64) - offsets[jl]
    pt = (o[jl] + kk * st[jl]) % 256                     # grid point / batch-1
    # training knobs
    b = np.exp(0.5 * _normal(seed, _S_B, j))
    m = 8.0 + 62.0 * _uniform(seed, _S_M, j)
    p = 0.05 + 0.45 * _uniform(seed, _S_P, j)
    cpu = np.floor(2.0 + 7.0 * _uniform(seed, _S_CPU, j))
    g = 2.0 ** (pt // 64)
    ms = _MS[(pt // 16) % 4]
    s = np.where((pt // 8) % 2 == 0, 0.5, 1.0)
    a = ((pt // 4) % 2).astype(np.float64)
    mb = 2.0 ** (pt % 4)
    f = 0.6 + 0.4 * _uniform(seed, _S_F, np.arange(nnz, dtype=np.int64))
    thr = b[jl] * g ** 0.85 * (1.0 - 0.625 * (1.0 - ms)) * s ** 0.7 * (1.0 + 0.3 * a) * (mb / 8.0) ** 0.25
    t_u = thr * f
    t_d = [g, g * m[jl] * ms * (1.0 - 0.25 * a) * (0.5 + 0.5 * mb / 8.0) / g ** 0.6, g * s,
           16.0 * g, g * p[jl] * s, g * cpu[jl]]
    # inference knobs: batch sizes sorted ascending within the family
    bs = (pt + 1).astype(np.float64)
    bs_sorted = bs.copy()
    inf_entries = infer[jl]
    if inf_entries.any():
        # sort batch sizes inside each inference family (stable, per job)
        order = np.lexsort((bs, jl))
        bs_sorted = bs[order]
    binf = 50.0 * np.exp(0.5 * _normal(seed, _S_BINF, j))
    bsat = 16.0 + 112.0 * _uniform(seed, _S_BSAT, j)
    w = 4.0 + 16.0 * _uniform(seed, _S_W, j)
    kv = 0.02 + 0.18 * _uniform(seed, _S_KV, j)
    B_ = bs_sorted
    i_u = binf[jl] * B_ / (1.0 + B_ / bsat[jl])
    i_d = [np.ones(nnz), w[jl] + kv[jl] * B_, np.minimum(1.0, 0.2 + 0.8 * B_ / 256.0),
           8.0 + 0.05 * B_, p[jl] * B_ / 256.0, np.full(nnz, 2.0)]
    u = np.where(inf_entries, i_u, t_u)
    d = np.stack([np.where(inf_entries, i_d[r], t_d[r]) for r in range(R)], axis=1)
    u32, d32 = _f32(u), _f32(d)
    # capacity between the all-min and all-max selections
    dd = d32.astype(np.float64)
    smin = np.minimum.reduceat(dd, offsets[:-1], axis=0).sum(axis=0)
    smax = np.maximum.reduceat(dd, offsets[:-1], axis=0).sum(axis=0)
    cap = smin + 0.5 * (smax - smin)
    return Instance("ragged", seed, offsets, u32[None], d32[None], cap[None],
                    np.array([0.01]), STEP_INV_SQRT, np.zeros((1, R)), 300)


NAMES = ("tiny", "small", "large", "ragged", "batched")


# ---------------------------------------------------------------------------
# Epochs: active jobs + a pending queue, for the warm-start experiment
# ---------------------------------------------------------------------------

def epoch_market(n_jobs: int = 1048576, queue_frac: float = 0.125, seed: int = 3):
    """Active jobs and a pending queue for repeated scheduling epochs
    (Sec. 3.4: C_eff of Eq. 12 at the start of every epoch; Sec. 3.4's
    complexity paragraph: prices carried over between epochs).

    Both are Ragged-shaped families (generator of the Ragged workload, the
    queue with its own seed and queue_frac * n_jobs jobs).  Every resource is
    rescaled so that the active jobs' capacity is n_jobs: one unit per job on
    average.  Then one step size serves all resources and prices are O(1):
    eta0 = 2 / n_jobs with the 1/sqrt(t) rule (the Ragged workload's absolute
    units, 1 to 10^6 per resource, make a single eta overshoot and oscillate).
    Returns (active, queue)."""
    act = _ragged(seed, n_jobs)
    que = _ragged(seed + 1000, max(1, int(round(n_jobs * queue_frac))))
    scale = float(n_jobs) / act.capacity[0]
    act.demand = _f32(act.demand.astype(np.float64) * scale[None, None, :])
    que.demand = _f32(que.demand.astype(np.float64) * scale[None, None, :])
    R = act.R
    act.capacity = np.full((1, R), float(n_jobs))
    que.capacity = act.capacity.copy()
    act.eta0 = np.array([2.0 / n_jobs])
    act.rule = STEP_INV_SQRT
    act.iters = 1000
    act.name, que.name = "epoch_active", "epoch_queue"
    return act, que


def epoch_pending(n_queue: int, n_epochs: int, seed: int = 3, start: float = 0.5, churn: float = 0.1):
    """Pending-job masks [n_epochs, n_queue] (uint8): about `start` of the
    queue is pending in epoch 0; in each later epoch about `churn` of the
    jobs change state (arrivals and admissions)."""
    j = np.arange(n_queue, dtype=np.int64)
    m = (_uniform(seed, _S_QUEUE, j) < start).astype(np.uint8)
    out = np.empty((n_epochs, n_queue), dtype=np.uint8)
    for e in range(n_epochs):
        if e > 0:
            m = m ^ (_uniform(seed, _S_QUEUE, j + (e * n_queue)) < churn).astype(np.uint8)
        out[e] = m
    return out


# ---------------------------------------------------------------------------
# Outer ESP-IAC rounds (Alg. 1): cluster model and synthetic slowdown inputs
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class IacModel:
    """GPU-level cluster model for BinPack and the inputs of the predicted
    slowdown S_x|y = 1 + a_x b_y of a co-located pair (a synthetic stand-in
    for the trained predictor of Sec. 3.3.2), with the Eq. 11 thresholds."""
    gpus: np.ndarray              # int32 [B] GPUs per cluster
    gpu_memory: float             # per-GPU capacity of resource r_mem
    gpu_compute: float            # per-GPU capacity of resource r_sm
    r_gpus: int                   # resource holding the GPU count (whole numbers)
    r_mem: int
    r_sm: int
    sensitivity: np.ndarray       # float32 [B, nnz] a: how much a configuration suffers
    pressure: np.ndarray          # float32 [B, nnz] b: how much it disturbs its neighbour
    tau_base: np.ndarray          # float64 [B, N] baseline tolerance
    beta: float = 0.5
    beta_max: float = 0.1
    u_target: float = 0.8
    kappa: float = 0.5


def iac_model(inst: Instance, seed: int = 11, gpus=None, gpu_memory: float = 80.0,
              gpu_compute: float = 1.0) -> IacModel:
    """Synthetic interference inputs for `inst` (resources 0, 1, 2 = GPU
    count, GPU memory, compute share, as in every workload here):
    sensitivity a ~ U[0, 0.6) per configuration; pressure b = (compute share
    per GPU) x U[0.5, 1); tau_base ~ U[1.1, 1.4) per job; GPUs per cluster =
    the capacity's GPU count unless given."""
    B, N, nnz = inst.B, inst.N, inst.nnz
    e = np.arange(B * nnz, dtype=np.int64)
    a = 0.6 * _uniform(seed, _S_IA, e)
    d = inst.demand.reshape(B * nnz, inst.R).astype(np.float64)
    share = d[:, 2] / np.maximum(d[:, 0], 1.0)
    bb = share * (0.5 + 0.5 * _uniform(seed, _S_IB, e))
    tb = 1.1 + 0.3 * _uniform(seed, _S_IT, np.arange(B * N, dtype=np.int64))
    if gpus is None:
        gpus = np.rint(inst.capacity[:, 0]).astype(np.int32)
    return IacModel(np.asarray(gpus, dtype=np.int32).reshape(B), gpu_memory, gpu_compute, 0, 1, 2,
                    _f32(a).reshape(B, nnz), _f32(bb).reshape(B, nnz), tb.reshape(B, N))


# ---------------------------------------------------------------------------
# Queries of the nearest-profile fallback (RST)
# ---------------------------------------------------------------------------

def nn_queries(store: Instance, n_queries: int, seed: int = 5, exact_frac: float = 0.1, sigma: float = 0.25):
    """Unprofiled configurations for the profile store `store` (family f =
    job type f): per query a job type drawn uniformly, a base entry of its
    family drawn uniformly, and the base's resource vector multiplied per
    resource by exp(sigma Z) (a knob combination between profiled ones); a
    fraction exact_frac are exact copies of a profiled vector (store hits).
    Returns (family int32 [B, Q], query float32 [B, Q, R])."""
    B, N, R = store.B, store.N, store.R
    i = np.arange(B * n_queries, dtype=np.int64)
    fam = np.minimum(np.floor(N * _uniform(seed, _S_NNF, i)).astype(np.int64), N - 1)
    off = store.offsets
    size = off[fam + 1] - off[fam]
    k = np.minimum(np.floor(size * _uniform(seed, _S_NNB, i)).astype(np.int64), size - 1)
    b = i // n_queries
    base = store.demand[b, off[fam] + k].astype(np.float64)
    z = _normal(seed, _S_NNZ, np.arange(B * n_queries * R, dtype=np.int64)).reshape(-1, R)
    factor = np.exp(sigma * z)
    factor[_uniform(seed, _S_NNX, i) < exact_frac] = 1.0
    q = _f32(base * factor)
    return fam.astype(np.int32).reshape(B, n_queries), q.reshape(B, n_queries, R)


def make(name: str, **kw) -> Instance:
    """Build a named workload.  Keyword overrides shrink it for tests
    (``n_jobs`` for all, ``n_clusters`` for batched, ``seed``)."""
    fn = {"tiny": _tiny, "small": _small, "large": _large, "ragged": _ragged,
          "batched": _batched}[name]
    return fn(**kw)


# ---------------------------------------------------------------------------
# Small random instances for brute force / property tests
# ---------------------------------------------------------------------------

def with_penalties(inst: Instance, seed: int, switch_cost: float = 0.05, penalty_scale: float = 0.2,
                   frac_current: float = 0.8, dyadic: bool = False) -> Instance:
    """Attach Eq. 7 penalty inputs to an instance: a current configuration for
    a fraction of the jobs (-1 for the rest), a switching cost per cluster and
    an interference penalty U[0, penalty_scale) per configuration (multiples
    of 1/64 when ``dyadic``).  Returns the same instance, modified."""
    B, N, nnz = inst.B, inst.N, inst.nnz
    j = np.arange(B * N, dtype=np.int64)
    sizes = np.tile(np.diff(inst.offsets), B)
    cur = np.floor(_uniform(seed, _S_CUR, j) * sizes).astype(np.int64)
    cur = np.where(_uniform(seed, _S_CUR + 1, j) < frac_current, cur, -1)
    inst.current = cur.reshape(B, N).astype(np.int32)
    inst.switch_cost = np.full(B, float(switch_cost))
    pen = penalty_scale * _uniform(seed, _S_PEN, np.arange(B * nnz, dtype=np.int64))
    if dyadic:
        pen = np.floor(pen * 64.0) / 64.0
    inst.penalty = _f32(pen).reshape(B, nnz)
    return inst


def random_small(seed: int, n_jobs: int, max_k: int, n_res: int, *, dense: bool = False,
                 dyadic: bool = False, n_clusters: int = 1, eta0: float = 0.05,
                 rule: int = STEP_INV_SQRT, iters: int = 50) -> Instance:
    """A tiny instance whose optimum can be enumerated: K_j ~ U{1..max_k}
    (or max_k for all jobs when ``dense``), utilities U[0, 2), demands
    U[0, 4) (multiples of 1/8 when ``dyadic``), capacity halfway between the
    all-min and the all-max selection of each resource."""
    N, R, B = n_jobs, n_res, n_clusters
    j = np.arange(N, dtype=np.int64)
    if dense:
        K = np.full(N, max_k, dtype=np.int64)
    else:
        K = 1 + np.floor(max_k * _uniform(seed, _S_TINY_K, j)).astype(np.int64)
    offsets = np.zeros(N + 1, dtype=np.int64)
    np.cumsum(K, out=offsets[1:])
    nnz = int(offsets[-1])
    idx = np.arange(B * nnz, dtype=np.int64)
    u = 2.0 * _uniform(seed, _S_TINY_U, idx)
    d = 4.0 * _uniform(seed, _S_TINY_D, np.arange(B * nnz * R, dtype=np.int64))
    if dyadic:
        u = np.floor(u * 8.0) / 8.0
        d = np.floor(d * 8.0) / 8.0
    u32 = _f32(u).reshape(B, nnz)
    d32 = _f32(d).reshape(B, nnz, R)
    dd = d32.astype(np.float64)
    cap = np.empty((B, R))
    for bi in range(B):
        smin = np.minimum.reduceat(dd[bi], offsets[:-1], axis=0).sum(axis=0)
        smax = np.maximum.reduceat(dd[bi], offsets[:-1], axis=0).sum(axis=0)
        cap[bi] = smin + 0.5 * (smax - smin)
    if dyadic:
        cap = np.floor(cap * 8.0) / 8.0
    return Instance(f"random{seed}", seed, offsets, u32, d32, cap, np.full(B, eta0), rule,
                    np.zeros((B, R)), iters, dense_k=(max_k if dense else None))
