"""Benchmark of the ESP hot path on one MI355X.

A step is one esp_solve of the named workload: T price iterations (score ->
select -> exact demand -> Eq. 8 update, one fused pass of the kernel each) plus
the re-selection at the final prices, with the table resident in HBM.  The
library picks the loop driver: one launch per pass for the large tables, one
persistent launch for all passes of the small ones.

Prints one JSON line:
  value        job-configurations scored per second (whole job)
  roofline     the fused kernel's algorithmic bytes per pass (the table:
               (1 + R) * 4 bytes per job-configuration) over its average pass
               duration, against the 8 TB/s HBM peak
  cpu_baseline the CPU oracle (single-threaded C) on a bounded sample of the
               same workload, in the same unit
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def _parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="large", choices=["tiny", "small", "large", "ragged", "batched"])
    ap.add_argument("--iters", type=int, default=0, help="override T (0 = the workload's own)")
    ap.add_argument("--blocks", type=int, default=0, help="workgroups per cluster (0 = library default)")
    ap.add_argument("--sweep", type=int, default=0, help="0 = alternate sweep direction, 1 = forward only")
    ap.add_argument("--mode", type=int, default=0,
                    help="loop driver: 0 auto, 1 one launch per iteration, 2 persistent (table streamed every "
                         "iteration), 3 resident (tiles held in registers)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step (price reset + esp_solve, one launch per pass) in a HIP graph and time "
                         "its replays")
    ap.add_argument("--penalties", action="store_true",
                    help="add Eq. 7 penalty inputs (current configurations, switching cost, interference penalty)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES (10 times): the reference kernel "
                         "whose FETCH_SIZE / WRITE_SIZE counters scale the fused kernel's")
    ap.add_argument("--calibrate-stream", default="", metavar="CONFIG",
                    help="only time the read-only streaming probe (libesp_calib.so: the fused dense kernel's load "
                         "pattern with no work) over a table laid out like CONFIG's packed table, on the fused "
                         "kernel's grid; prints the ceiling in GB/s")
    ap.add_argument("--stream-mb", type=float, default=0.0,
                    help="with --calibrate-stream: resize the table to about this many MB (memory-side cache "
                         "check); 0 = CONFIG's size")
    ap.add_argument("--epochs", type=int, default=0, metavar="E",
                    help="instead of the default line: E scheduling epochs of an active market plus a pending "
                         "queue (C_eff of Eq. 12 each epoch, then esp_solve to tol 1e-3 from cold and from "
                         "warm prices); prints iterations to converge and epoch times")
    ap.add_argument("--nearest", type=int, default=0, metavar="Q",
                    help="instead of the default line: Q nearest-profile queries (RST fallback) against the "
                         "Ragged table used as the profile store; prints queries/s and the gather roofline")
    ap.add_argument("--store-layout", choices=("aos", "soa"), default="aos",
                    help="profile-store layout of --nearest: the entry-major copy (ESP_OPT_PROFILE_STORE, "
                         "default) or the structure-of-arrays columns of the price loop")
    ap.add_argument("--schedule", default="", metavar="CONFIG",
                    help="instead of the default line: Alg. 1 outer rounds (tatonnement, first-fit BinPack, "
                         "co-located pair checks, penalty updates) on CONFIG; --iters per round (default 5), "
                         "--rounds rounds")
    ap.add_argument("--rounds", type=int, default=3, help="max rounds M of --schedule")
    ap.add_argument("--epoch-jobs", type=int, default=1048576, help="active jobs of the --epochs market")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic_large.json"),
                    help="HBM bytes per launch measured with rocprofv3 counters, if present")
    return ap.parse_args()


def _cpu_baseline(inst, budget_s: float) -> dict:
    import numpy as np

    import oracle

    o = oracle.Oracle(inst)
    lam = np.array(inst.lam0[0], dtype=np.float64)
    n, t0 = 0, time.perf_counter()
    while True:
        _, _, lam = o.step(0, lam, n + 1)
        n += 1
        el = time.perf_counter() - t0
        if el >= budget_s or n >= inst.iters:
            break
    per_iter = el / n
    return {
        "value": inst.nnz / per_iter,
        "unit": "job-configs/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"{inst.name}: first {n} price iterations of cluster 0 from lambda^1 = 0 "
                  f"({el:.1f} s, single-threaded C oracle, fp64)",
        "iters_per_s": 1.0 / per_iter,
        "host": _host_cpu(),
    }


def _host_cpu() -> str:
    """CPU model and logical CPU count of the host the baseline ran on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{model}, {os.cpu_count()} logical CPUs (the baseline uses one thread)"


def main() -> int:
    args = _parse()
    if args.gpus != 1:
        print(f"bench.py: runs on one GPU only (asked for --gpus {args.gpus}); "
              "the path shards over jobs but no multi-GPU code is built", file=sys.stderr)
        return 2
    import numpy as np
    import torch

    if args.calibrate_copy:
        n = args.calibrate_copy // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n * 4, "copies": 10}), flush=True)
        return 0

    if args.calibrate_stream:
        return _calibrate_stream(args, np, torch)

    import paper_2608_07971_amd as esp
    import workloads

    if args.epochs:
        return _epochs(args, esp, workloads, np, torch)
    if args.nearest:
        return _nearest(args, esp, workloads, np, torch)
    if args.schedule:
        return _schedule(args, esp, workloads, np, torch)

    t_gen = time.perf_counter()
    kw = {}
    inst = workloads.make(args.config, **kw)
    if args.penalties:
        workloads.with_penalties(inst, inst.seed + 100)
    T = args.iters or inst.iters
    print(f"[bench] {args.config}: B={inst.B} N={inst.N} R={inst.R} nnz={inst.nnz} T={T} "
          f"(generated in {time.perf_counter() - t_gen:.1f} s)", file=sys.stderr, flush=True)
    solver = esp.Solver(inst, "cuda:0", blocks_per_cluster=args.blocks, sweep_order=args.sweep, mode=args.mode)
    stream = torch.cuda.Stream()
    lam0 = solver.prices(inst.lam0)
    lam = lam0.clone()
    torch.cuda.synchronize()

    def step():
        lam.copy_(lam0)
        solver.solve(lam, T, stream=stream)

    run = step
    if args.graph:
        # static output buffers, one captured step; replays rerun it on them
        graph = torch.cuda.CUDAGraph()
        choice = torch.empty((solver.B, solver.N), dtype=torch.int32, device="cuda:0")
        demand = torch.empty((solver.B, solver.R), dtype=torch.float64, device="cuda:0")
        with torch.cuda.graph(graph, stream=stream):
            lam.copy_(lam0)
            esp.esp_solve(solver.ctx, lam, T, 1, 0.0, choice, demand, None, None, torch.cuda.current_stream())
        run = graph.replay
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            run()
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        evs[0].record(stream)
        for i in range(args.steps):
            run()
            evs[i + 1].record(stream)
    torch.cuda.synchronize()
    ms_total = evs[0].elapsed_time(evs[-1])
    step_ms = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
    assert solver.device_status() == 0
    ms_per_step = ms_total / args.steps
    sec = ms_total / 1e3
    configs = inst.B * inst.nnz
    passes = (T + 1) * args.steps                    # T fused iterations + the final re-selection
    driver = solver.loop_driver()
    persistent = driver == esp.ESP_MODE_PERSISTENT and not args.graph
    resident = driver == esp.ESP_MODE_RESIDENT and not args.graph
    # algorithmic bytes: the fp32 table read once per iteration, plus the
    # family boundaries (one 4-byte offset per job) for ragged families
    csr = inst.dense_k is None or inst.dense_k not in (4, 8, 16, 32, 64)
    pen_col = 1 if (inst.current is not None or inst.penalty is not None) else 0
    bytes_per_pass = configs * (1 + inst.R + pen_col) * 4 + (4 * (inst.N + 1) if csr else 0)
    avg_pass_s = sec / passes
    achieved = bytes_per_pass / avg_pass_s / 1e9
    traffic = None
    if os.path.exists(args.traffic_json):
        try:
            tj = json.load(open(args.traffic_json))
            if tj.get("config") == args.config and tj.get("kernel_source_sha") == _kernel_sha():
                traffic = tj.get("bytes_per_pass")
        except Exception:
            traffic = None
    out = {
        "metric": "job-configs scored/sec and price iterations/sec at 262k x 64 x 8; % HBM peak",
        "value": configs * T * args.steps / sec,
        "unit": "job-configs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "step_ms": {"min": step_ms[0], "median": step_ms[len(step_ms) // 2], "max": step_ms[-1]},
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": f"{args.config}: {inst.B} x {inst.N} jobs x "
                               f"{inst.dense_k or 'CSR'} configs x {inst.R} resources, T={T}, fp32 table",
                   "clusters": inst.B, "jobs": inst.N, "configs_per_job": inst.dense_k,
                   "resources": inst.R, "iterations": T, "seed": inst.seed},
        "iters_per_s": T * args.steps / sec,
        "pct_hbm_peak": 100.0 * achieved / HBM_PEAK_GBS,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": ("k_csr" if csr else "k_dense") + " (fused score/select/demand/update)",
                     "driver": ("graph: replays of a captured step, one launch per pass" if args.graph
                                else "persistent: one cooperative launch runs the T passes" if persistent
                                else "resident: one launch runs the T passes over tiles held in registers"
                                if resident else "stream: one launch per pass"),
                     "bytes_per_pass": bytes_per_pass, "avg_pass_us": avg_pass_s * 1e6,
                     "passes_per_launch": T if (persistent or resident) else 1},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = _cpu_baseline(inst, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    solver.close()
    return 0


def _epochs(args, esp, workloads, np, torch) -> int:
    """Scheduling epochs (Sec. 3.4, Alg. 1 first step and warm start): each
    epoch recomputes C_eff from the epoch's pending set (gamma = 0.5), then
    runs the tatonnement to tol = 1e-3 (at most 1000 iterations) from
    lambda = 0 (cold) and from the previous epoch's prices (warm, t restarts
    at 1).  Times with HIP events on the solve stream; the first epoch is
    also run once untimed."""
    E, TOL, GAMMA, TMAX = args.epochs, 1e-3, 0.5, 1000
    act, que = workloads.epoch_market(args.epoch_jobs)
    pend = torch.from_numpy(workloads.epoch_pending(que.N, E)).cuda().contiguous()
    a = esp.Solver(act, mode=args.mode)
    q = esp.Solver(que, mode=args.mode)
    stream = torch.cuda.Stream()
    print(f"[bench] epochs: active N={act.N} nnz={act.nnz} queue N={que.N} nnz={que.nnz} R={act.R} E={E}",
          file=sys.stderr, flush=True)

    def timed(fn):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(stream):
            e0.record(stream)
            out = fn()
            e1.record(stream)
        torch.cuda.synchronize()
        return out, e0.elapsed_time(e1)

    def solve(lam0):
        lam = lam0.clone()
        g = a.solve(lam, TMAX, tol=TOL, stream=stream)
        return lam, g

    zero = a.prices(np.zeros((1, act.R)))
    # untimed warm-up of every kernel involved
    a.effective_capacity(q, GAMMA, pend[0:1].clone())
    solve(zero)
    torch.cuda.synchronize()
    rows, lam_w = [], None
    for e in range(E):
        pe = pend[e:e + 1].clone()
        _, ms_c = timed(lambda: a.effective_capacity(q, GAMMA, pe, stream=stream))
        (lam_c, gc), ms_cold = timed(lambda: solve(zero))
        (lam_w, gw), ms_warm = timed(lambda: solve(lam_c if lam_w is None else lam_w))
        rows.append((ms_c, int(gc["iters_done"][0]), ms_cold, int(gw["iters_done"][0]), ms_warm))
        print(f"[bench] epoch {e}: C_eff {ms_c * 1e3:.1f} us, cold {rows[-1][1]} it {ms_cold:.3f} ms, "
              f"warm {rows[-1][3]} it {ms_warm:.3f} ms", file=sys.stderr, flush=True)
    assert a.device_status() == 0 and q.device_status() == 0
    later = rows[1:] if E > 1 else rows
    mean = lambda i: sum(r[i] for r in later) / len(later)
    ceff_bytes = que.nnz * (1 + que.R) * 4 + que.N
    out = {
        "metric": "price iterations to converge per scheduling epoch (tol 1e-3), warm vs cold start",
        "value": mean(3),
        "unit": "iterations (warm start, mean over epochs 1..E-1)",
        "higher_is_better": False,
        "n_gpus": 1, "steps": E, "warmup": 1, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"epoch market: {act.N} active jobs x Geo(0.08) configs x {act.R} resources "
                               f"(unit share per job), queue {que.N} jobs, gamma {GAMMA}, tol {TOL}",
                   "epochs": E},
        "cold_iters": mean(1), "warm_iters": mean(3),
        "epoch_ms_cold": mean(0) + mean(2), "epoch_ms_warm": mean(0) + mean(4),
        "ceff_us": 1e3 * mean(0),
        "ceff_gbs": ceff_bytes / (mean(0) * 1e-3) / 1e9,
        "ceff_bytes": ceff_bytes,
        "per_epoch": [{"ceff_us": 1e3 * r[0], "cold_iters": r[1], "cold_ms": r[2], "warm_iters": r[3],
                       "warm_ms": r[4]} for r in rows],
    }
    print(json.dumps(out), flush=True)
    a.close()
    q.close()
    return 0


def _nearest(args, esp, workloads, np, torch) -> int:
    """RST's nearest-profile fallback (Sec. 3.1.2): Q queries, each naming a
    job type of the Ragged table (the profile store) and a perturbed resource
    vector; one esp_nearest_profile call per step, timed with HIP events."""
    store = workloads.make("ragged")
    fam_np, q_np = workloads.nn_queries(store, args.nearest, seed=9)
    fam = torch.from_numpy(fam_np).cuda()
    q = torch.from_numpy(q_np).cuda()
    flags = esp.ESP_OPT_PROFILE_STORE if args.store_layout == "aos" else 0
    s = esp.Solver(store, mode=args.mode, flags=flags)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for _ in range(max(1, args.warmup)):
            s.nearest_profile(fam, q, stream=stream)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        e0.record(stream)
        for _ in range(args.steps):
            s.nearest_profile(fam, q, stream=stream)
        e1.record(stream)
    torch.cuda.synchronize()
    assert s.device_status() == 0
    sec = e0.elapsed_time(e1) / 1e3
    Q, R = args.nearest, store.R
    sizes = (store.offsets[1:] - store.offsets[:-1])[fam_np[0]]
    # algorithmic bytes: family id, query vector, family slot (8 B), the
    # family's utility and R demand columns, and the two outputs
    bytes_per_call = int(Q * (4 + 4 * R + 8 + 8) + 4 * (1 + R) * int(sizes.sum()))
    per_call = sec / args.steps
    out = {
        "metric": "nearest-profile queries/sec (RST fallback, l2 within the job type's family)",
        "value": Q / per_call, "unit": "queries/s", "higher_is_better": True,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"store: Ragged table ({store.N} job types, {store.nnz} profiles, R={R}); "
                               f"{Q} queries, uniform job type, log-normal(0.25) perturbation, 10% exact hits",
                   "store_layout": args.store_layout},
        "ms_per_step": per_call * 1e3,
        "roofline": {"bound": "hbm", "achieved": bytes_per_call / per_call / 1e9, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": bytes_per_call / per_call / 1e9 / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "k_nearest", "bytes_per_launch": bytes_per_call,
                     "avg_launch_us": per_call * 1e6},
    }
    print(json.dumps(out), flush=True)
    s.close()
    return 0


def _schedule(args, esp, workloads, np, torch) -> int:
    """Alg. 1 (Sec. 3.4): one esp_schedule call per step (Gamma reset, then up
    to M rounds of tatonnement + BinPack + pair checks + penalty updates),
    from the same starting prices each step; HIP events on the stream."""
    inst = workloads.make(args.schedule)
    inst.penalty = np.zeros((inst.B, inst.nnz), np.float32)
    model = workloads.iac_model(inst)
    # the interference inputs stay resident on the device like the table
    model.sensitivity = torch.from_numpy(model.sensitivity).cuda()
    model.pressure = torch.from_numpy(model.pressure).cuda()
    model.tau_base = torch.from_numpy(model.tau_base).cuda()
    T = args.iters or 5
    s = esp.Solver(inst, mode=args.mode)
    lam0 = s.prices(inst.lam0)
    lam = lam0.clone()
    stream = torch.cuda.Stream()

    def step():
        lam.copy_(lam0)
        return s.schedule(model, lam, args.rounds, T, stream=stream)

    with torch.cuda.stream(stream):
        for _ in range(max(1, args.warmup)):
            step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # the same work with the pack/IAC step left out: M plain solves
    with torch.cuda.stream(stream):
        e0.record(stream)
        for _ in range(args.steps):
            lam.copy_(lam0)
            for _ in range(args.rounds):
                s.solve(lam, T, stream=stream)
        e1.record(stream)
    torch.cuda.synchronize()
    ms_solves = e0.elapsed_time(e1) / args.steps
    with torch.cuda.stream(stream):
        e0.record(stream)
        for _ in range(args.steps):
            g = step()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    assert s.device_status() == 0
    rounds = g["rounds"].cpu().numpy()
    viol = g["violations"].cpu().numpy()
    out = {
        "metric": "Alg. 1 scheduling passes/sec (ESP-IAC rounds: tatonnement, first-fit BinPack, pair checks, "
                  "penalty updates)",
        "value": 1e3 / ms, "unit": "schedules/s", "higher_is_better": True,
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"{args.schedule}: {inst.B} x {inst.N} jobs x {inst.dense_k or 'CSR'} configs x "
                               f"{inst.R} resources, GPUs per cluster {int(model.gpus.min())}..{int(model.gpus.max())}, "
                               f"M={args.rounds}, T={T} per round"},
        "ms_per_step": ms,
        "ms_same_solves_without_pack_iac": ms_solves,
        "rounds_used": {"mean": float(rounds.mean()), "max": int(rounds.max())},
        "violations_last_round": {"clusters_with_violations": int((viol > 0).sum()), "pairs": int(viol.sum())},
    }
    print(json.dumps(out), flush=True)
    s.close()
    return 0


def _calibrate_stream(args, np, torch) -> int:
    """Streaming ceiling of the packed-table layout: the probe kernel reads a
    table of CONFIG's shape (its columns and tiles; dense families) with the
    fused kernel's access pattern and grid, and nothing else."""
    import ctypes

    import workloads

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2608_07971_amd", "libesp_calib.so"))
    lib.esp_calib_stream.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_int, ctypes.c_int,
                                     ctypes.c_void_p, ctypes.c_void_p]
    lib.esp_calib_stream.restype = ctypes.c_int
    inst = workloads.make(args.calibrate_stream)
    if inst.dense_k not in (4, 8, 16, 32, 64):
        print("bench.py: --calibrate-stream takes a dense workload (tiny, small, large, batched)", file=sys.stderr)
        return 2
    ncol = 1 + inst.R
    jobs_per_tile = 64 // (inst.dense_k // 4)
    tiles = -(-inst.N // jobs_per_tile)
    if args.stream_mb > 0:
        tiles = max(1, int(round(args.stream_mb * 1e6 / (ncol * 256 * 4))))
    col_len = (tiles + 7) * 256                            # the packer's column pad
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    blocks = args.blocks or max(1, min(3 * cus // 4, -(-tiles // 4)))
    table = torch.ones(ncol * col_len, dtype=torch.float32, device="cuda:0")
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda:0")
    stream = torch.cuda.Stream()
    h = ctypes.c_void_p(stream.cuda_stream)

    def launch():
        rc = lib.esp_calib_stream(table.data_ptr(), ncol, col_len, tiles, blocks, sink.data_ptr(), h)
        assert rc == 0, rc

    passes = max(1, args.steps) * 20
    with torch.cuda.stream(stream):
        for _ in range(max(1, args.warmup) * 5):
            launch()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(passes):
            launch()
        e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / passes
    nbytes = tiles * 256 * ncol * 4
    gbs = nbytes / (us * 1e-6) / 1e9
    print(json.dumps({"calibrate_stream": args.calibrate_stream, "kernel": "k_stream_probe (libesp_calib.so)",
                      "columns": ncol, "tiles": tiles, "blocks": blocks, "bytes_per_pass": nbytes,
                      "passes": passes, "avg_pass_us": us, "GB/s": gbs, "frac_of_hbm_peak": gbs / HBM_PEAK_GBS}),
          flush=True)
    return 0


def _kernel_sha() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in ("esp_kernels.hpp", "esp_kernels.hip", "esp_device.hpp", "esp_internal.hpp", "esp_inst_dense12.hip",
              "esp_inst_dense34.hip", "esp_inst_dense56.hip", "esp_inst_dense78.hip", "esp_inst_csr1234.hip",
              "esp_inst_csr5678.hip"):
        h.update(open(os.path.join(ROOT, "paper_2608_07971_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    sys.exit(main())
