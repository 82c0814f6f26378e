// gfx950 kernels of the Elastic Shadow Pricing hot path (paper Sec. 3.2), as
// templates; esp_kernels.hip dispatches on R at run time and the
// esp_inst_*.hip files instantiate the fused kernels (split by R so that
// they compile in parallel).
//
// One price iteration = one launch of a fused kernel:
//   score   s_jk = u_jk - sum_r lambda_r d_jkr          (Sec. 3.2.2, bracket of Eq. 6)
//   select  c_j  = argmax_k s_jk, lowest k on ties     (Sec. 3.2.2 per-job subproblem)
//   demand  U_r  = sum_j d_{j,c_j,r}, exact             (Sec. 3.2.3, under Eq. 8)
//   update  lambda_r <- max(0, lambda_r + eta_t (U_r - C_r))  (Eq. 8)
//
// With several workgroups per cluster, a solve iteration ends once every
// workgroup has published its exact demand sums; every workgroup of the
// cluster then computes U and the update itself at the start of the next
// iteration (integer sums: all obtain the same bits), so no workgroup waits
// for a last one to finish the update.  With one workgroup per cluster the
// workgroup updates at the end of its own iteration.
//
// Table layout (built by the packer): per cluster, one fp32 column for the
// utility and one per resource, each a sequence of 256-entry tiles.  A
// wavefront scores one tile per step with one 128-bit load per lane per
// column (lane l holds entries 4l .. 4l+3 of the tile).
//
// Arithmetic contract: binary64, no contraction (`fp contract(off)` below and
// -ffp-contract=off on the command line), rent summed left to right over r.
// The demand sum is exact: each fp32 demand is turned into a 128-bit integer
// multiple of 2^shift (the column's lowest set bit, fixed by the packer),
// integers are added in any order, and the total is rounded once to binary64
// (round-to-nearest-even).  No floating-point atomics are used.
#pragma once

#include <algorithm>
#include <type_traits>

#include "esp_device.hpp"

#pragma clang fp contract(off)

namespace esp {

// ---------------------------------------------------------------------------
// Cluster completion: per-workgroup sums -> last workgroup -> U, Eq. 8 update
// ---------------------------------------------------------------------------

// eta_t of Eq. 8 for the launch's step index t: eta0 or eta0 / sqrt(t), one
// IEEE division and one correctly rounded square root in binary64 (no fast
// math), so the value equals the host's.
__device__ __forceinline__ double step_size(const KArgs &a, int cl, int t) {
    const double e0 = a.eta0[cl];
    return a.rule == 1 ? e0 / sqrt(static_cast<double>(t)) : e0;
}

// U_r from the cluster's exact total, the Eq. 8 update and the stop test for
// resource r (one thread per resource of the cluster's last workgroup).
// lam_cur (LDS) holds the prices the iteration selected at.  Gather: the
// launch is esp_reduce_demand's, whose workgroups flag invalid choices
// (flag 4) during the launch; no other launch sets that flag.  An update
// (lam_out set) happens only with one workgroup per cluster (deferred
// completion otherwise), so the prices, the trace rows and the iteration
// count each have one writer in a launch; the next launch reads them after
// the launch boundary: plain stores.
template <int R, bool Gather>
__device__ __forceinline__ void complete_resource(const KArgs &a, int cl, int r, u128 tot, const double *lam_cur,
                                                  int *s_ok, double *s_newlam) {
    const bool bad =
        Gather && a.flags && (__hip_atomic_load(&a.flags[cl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 4);
    const double U = bad ? __builtin_nan("") : fx_to_double(tot, a.shift[cl * R + r]);
    if (a.demand_out) a.demand_out[cl * R + r] = U;
    if (a.tr_U) a.tr_U[cl * R + r] = U;
    int ok = 1;
    if (a.lam_out) {
        const double lo = lam_cur[r];
        const double g = U - a.cap[cl * R + r];
        const double x = lo + step_size(a, cl, a.t) * g;
        const double ln = (x > 0.0) ? x : 0.0;
        a.lam_out[cl * R + r] = ln;
        if (a.tr_lam) a.tr_lam[cl * R + r] = ln;
        s_newlam[r] = ln;
        const double diff = fabs(ln - lo);
        const double scale = lo > 1.0 ? lo : 1.0;
        ok = diff <= a.tol * scale;
    }
    s_ok[r] = ok;
}

// Per-cluster bookkeeping after the update (thread 0 of the last workgroup).
// Returns whether the cluster stops (tol reached).
template <int R, bool Gather>
__device__ __forceinline__ int complete_cluster(const KArgs &a, int cl, const int *s_ok) {
    int stop = 0;
    if (Gather && a.flags && (a.flags[cl] & 4)) atomicAnd(&a.flags[cl], ~4);
    if (a.lam_out) {
        if (a.iters_done) a.iters_done[cl] = a.iter_no;
        int all = 1;
        for (int r = 0; r < R; ++r) all &= s_ok[r];
        if (a.tol > 0.0 && all && a.flags) {
            atomicOr(&a.flags[cl], kFlagStopped);
            stop = 1;
        }
    }
    return stop;
}

// The demand sums of one iteration: U, the Eq. 8 update and the per-cluster
// bookkeeping in the last workgroup.  s_newlam / s_stop (LDS) receive the new
// prices and the stop decision there.
template <int R, bool Gather>
__device__ bool finish_cluster(const KArgs &a, int cl, int blk, const u128 *bsum, const double *lam_cur,
                               double *s_newlam, int *s_stop) {
    __shared__ int s_ok[R];
    const bool last = cluster_sums<R>(a, cl, blk, bsum, [&](int r, u128 tot) {
        complete_resource<R, Gather>(a, cl, r, tot, lam_cur, s_ok, s_newlam);
    });
    if (!last) return false;
    if (threadIdx.x == 0) *s_stop = complete_cluster<R, Gather>(a, cl, s_ok);
    __syncthreads();
    return true;
}

// ---------------------------------------------------------------------------
// Deferred completion (several workgroups per cluster)
// ---------------------------------------------------------------------------

// Complete iteration m of cluster cl (step index t_m) from the sums it
// published into buffer m & 1, whose first loads (partial_loads) are in v:
// U_m, lambda_{m+1} of Eq. 8 and the stop test.  lam_m (LDS) holds the
// prices iteration m selected at; lam_next (LDS) receives lambda_{m+1};
// s_red is LDS scratch.  All threads take part and get whether the tolerance
// is met.  The writer (workgroup 0 of the cluster) also stores
// lambda_{m+1} into the caller's prices and lam_ws, the trace rows of
// iteration m, the iteration count, and m as the stop iteration.
template <int R, typename A, bool Coherent>
__device__ bool complete_iteration(const KArgs &a, int cl, int m, int t_m, bool writer, const double *lam_m,
                                   double *lam_next, u128 *s_red, const A (&v)[kSumLoads]) {
    __shared__ int s_ok[R];
    partial_totals<R, A, Coherent>(a, m & 1, cl, v, s_red);
    const int t = threadIdx.x;
    if (t < R) {
        const size_t i = static_cast<size_t>(cl) * R + t;
        const double U = fx_to_double(s_red[t], a.shift[i]);
        const double lo = lam_m[t];
        const double g = U - a.cap[i];
        const double x = lo + step_size(a, cl, t_m) * g;
        const double ln = (x > 0.0) ? x : 0.0;
        lam_next[t] = ln;
        const double diff = fabs(ln - lo);
        const double scale = lo > 1.0 ? lo : 1.0;
        s_ok[t] = diff <= a.tol * scale;
        if (writer) {
            const size_t BR = static_cast<size_t>(a.B) * R;
            a.lam_dst[i] = ln;
            a.lam_ws[static_cast<size_t>((m + 1) & 1) * BR + i] = ln;
            if (a.trace_U) a.trace_U[static_cast<size_t>(m - 1) * BR + i] = U;
            if (a.trace_lam) a.trace_lam[static_cast<size_t>(m - 1) * BR + i] = ln;
        }
    }
    __syncthreads();
    int all = 1;
#pragma unroll
    for (int r = 0; r < R; ++r) all &= s_ok[r];
    const bool stop = a.tol > 0.0 && all;
    if (writer && t == 0) {
        if (a.iters_done) a.iters_done[cl] = m;
        if (stop) __hip_atomic_store(&a.conv_at[cl], m, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return stop;
}

// The loads of a launch's pending completion (pend_m > 0).  They are issued
// before the first tiles' loads, so they return first and the completion
// runs while the tiles are still in flight; they are issued whether or not
// the completion turns out to be needed.
template <int R, typename A>
struct Pending {
    A v[kSumLoads];      // this thread's first published sums of iteration pend_m
    double lam_m = 0.0;  // thread t < R: lambda_{pend_m}[t]
    int conv = 0;        // conv_at[cl]
};

// conv: conv_at[cl], read by the caller at the start of the launch together
// with the cluster's flags.  Within a launch conv_at changes only from 0 to
// pend_m (workgroup 0 completing pend_m itself), and both values lead to the
// same path, so a value read before that store is as good as one read after.
// The loads are issued whether or not a completion is pending, from valid
// addresses and without branches, so that the compiler waits for exactly
// these loads (and not for the tile loads issued after them) where they are
// used.
template <int R, typename A>
__device__ __forceinline__ void pending_loads(const KArgs &a, int cl, int conv, Pending<R, A> &p) {
    const int k = a.pend_m & 1;
    p.conv = conv;
    p.lam_m = a.lam_ws[static_cast<size_t>(k) * a.B * R + static_cast<size_t>(cl) * R + threadIdx.x % R];
    partial_loads<R, A, false>(a, k, cl, p.v);
}

// Prices of the launch's first iteration, into s_lam (LDS).  A launch with a
// pending completion first completes iteration pend_m, unless the cluster
// met the tolerance at an earlier iteration (conv_at 0 or pend_m: complete
// it here; every workgroup then reaches the same decision).  Returns false
// when the cluster has nothing left to do in this launch (it has converged
// and the launch runs solve iterations).
template <int R, typename A>
__device__ bool launch_prices(const KArgs &a, int cl, int blk, const Pending<R, A> &p, double *s_lam,
                              double *s_tmp, u128 *s_red) {
    const int t = threadIdx.x;
    if (a.pend_m > 0) {
        if (p.conv == 0 || p.conv >= a.pend_m) {
            if (t < R) s_tmp[t] = p.lam_m;
            __syncthreads();
            const bool stop =
                complete_iteration<R, A, false>(a, cl, a.pend_m, a.pend_t, blk == 0, s_tmp, s_lam, s_red, p.v);
            return !(stop && a.defer);
        }
        if (a.defer) return false;
        // met the tolerance earlier: the caller's prices are final and are not
        // written in this launch
    }
    if (t < R) s_lam[t] = a.lam_in[cl * R + t];
    __syncthreads();
    return true;
}

// Barrier word i of cluster cl (see kSyncSlots).
__device__ __forceinline__ uint32_t *sync_word(const KArgs &a, int cl, int i) {
    return a.sync + (static_cast<size_t>(cl) * kSyncSlots + i) * kSyncStride;
}

// End of iteration m in a deferred launch: publish the workgroup's sums
// (bsum, LDS) into buffer m & 1.  A one-iteration launch stores plainly: the
// next launch reads the sums after the launch boundary.  A persistent launch
// publishes with completed agent-scope exchanges and then arrives at the
// cluster's barrier: one atomic add on its group's counter (blk mod
// kSyncGroups); the group's last arrival adds one to the count of complete
// groups, and the last group releases every group by storing m into the
// groups' release words.  Adds to one address are serialized at the device
// coherence point (about 11 ns each), so no word takes more than one add per
// group member per iteration, and each group polls its own release word.
template <int R, bool Persist>
__device__ __forceinline__ void publish_iteration(const KArgs &a, int cl, int blk, int m, const u128 *bsum) {
    const int t = threadIdx.x;
    if constexpr (Persist) {
        if (t < kWaveSize) {
            publish_sums<R>(a, m & 1, cl, blk, bsum);
            if (t == 0) {
                const int g = blk % kSyncGroups;
                const int groups = a.nblk < kSyncGroups ? a.nblk : kSyncGroups;
                const uint32_t size = static_cast<uint32_t>((a.nblk - g + kSyncGroups - 1) / kSyncGroups);
                const uint32_t um = static_cast<uint32_t>(m);
                const uint32_t n = __hip_atomic_fetch_add(sync_word(a, cl, g), 1u, __ATOMIC_RELAXED,
                                                          __HIP_MEMORY_SCOPE_AGENT);
                if (n + 1u == size * um) {
                    const uint32_t c = __hip_atomic_fetch_add(sync_word(a, cl, kSyncGroups), 1u, __ATOMIC_RELAXED,
                                                              __HIP_MEMORY_SCOPE_AGENT);
                    if (c + 1u == static_cast<uint32_t>(groups) * um)
                        for (int h = 0; h < groups; ++h)
                            __hip_atomic_store(sync_word(a, cl, kSyncGroups + 1 + h), um, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        }
    } else if (t < R) {
        uint64_t *p = partials_of<R>(a, m & 1, cl) + (static_cast<size_t>(blk) * R + t) * 2;
        const u128 v = bsum[t];
        p[0] = static_cast<uint64_t>(v);
        p[1] = static_cast<uint64_t>(v >> 64);
    }
}

// Inside a persistent launch: wait until the workgroup's group is released
// for iteration m (its release word reaches m, compared modulo 2^32), i.e.
// every workgroup of the cluster has published iteration m.  The release
// word is stored only after the last arrival add returned, every arrival add
// is issued after the workgroup's exchanges completed, and the sums are
// loaded only after the release value is back, all with agent-scope atomics
// performed at the memory-side coherence point: the loads return the
// published sums (the argument is spelled out at publish_sums).  Bounded: about
// 2 s of the 100 MHz real-time counter, or until another workgroup has
// recorded an error; then the status records a timeout and the function
// returns false in every waiting workgroup.
__device__ bool wait_iteration(const KArgs &a, int cl, int blk, int m, int *s_go) {
    if (threadIdx.x == 0) {
        const uint32_t *w = sync_word(a, cl, kSyncGroups + 1 + blk % kSyncGroups);
        int go = 1;
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        while (static_cast<int32_t>(__hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) -
                                    static_cast<uint32_t>(m)) < 0) {
            __builtin_amdgcn_s_sleep(4);
            if (__hip_atomic_load(a.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
                __builtin_amdgcn_s_memrealtime() - t0 > 200000000ull) {
                atomicCAS(a.status, 0, kStatusTimeout);
                go = 0;
                break;
            }
        }
        *s_go = go;
    }
    __syncthreads();
    return *s_go != 0;
}

// ---------------------------------------------------------------------------
// Resident launches with several workgroups per cluster: the exact sums of
// iteration m are exchanged through tagged words, and every workgroup
// completes the iteration itself.
// ---------------------------------------------------------------------------

// Workgroup w's sum for resource r is split into a.limbs limbs of kLimbBits
// bits; limb l travels in one 64-bit word whose top 16 bits carry the tag of
// the iteration, (m - 1) mod 65535 + 1 (never 0, the value the solve's
// prologue clears the words to, and different for m and m - 2).  Tag and
// limb are one single-copy-atomic 64-bit store, so a reader that sees the
// tag of iteration m sees that iteration's limb: the exchange needs no fence
// and no counter.  Words of iteration m live in half m & 1 of a.xch
// ([2][B][nblk][R * limbs]); a workgroup writes half m & 1 again (iteration
// m + 2) only after it has read every workgroup's words of iteration m + 1,
// which each workgroup wrote after it had read all words of iteration m.
constexpr int kLimbBits = 48;
constexpr uint64_t kLimbMask = (1ull << kLimbBits) - 1;

__device__ __forceinline__ uint64_t *xch_words(const KArgs &a, int cl, int m) {
    return a.xch + (static_cast<size_t>(m & 1) * a.B + cl) * static_cast<size_t>(a.nblk) * a.xch_stride;
}

__device__ __forceinline__ double readlane_d(double v, int lane) {
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane(static_cast<int>(static_cast<unsigned>(b)), lane);
    const int hi = __builtin_amdgcn_readlane(static_cast<int>(b >> 32), lane);
    return __longlong_as_double(static_cast<long long>(
        (static_cast<unsigned long long>(static_cast<unsigned>(hi)) << 32) | static_cast<unsigned>(lo)));
}

// Step sizes eta_t of all iterations of a resident launch, computed once at
// its start by the whole workgroup (the same IEEE operations as step_size, so
// the same bits), so that no division or square root lies on an iteration's
// path.  The caller synchronizes the workgroup before the first read.
__device__ __forceinline__ const double *resident_etas(const KArgs &a, int cl) {
    __shared__ double s_eta[kLaunchChunk];
    for (int i = threadIdx.x; i < a.n_iters; i += kBlockThreads) s_eta[i] = step_size(a, cl, a.t + i);
    return s_eta;
}

// End of iteration a.iter_no in a resident launch.  `acc` is this lane's
// exact partial sum for resource lane % R (acc_lane: the lane accumulates);
// lam holds the iteration's prices and receives lambda_{m+1}.  Every
// wavefront completes the iteration itself, with one workgroup barrier (two
// when the workgroups of a cluster exchange their sums):
//  1. each wavefront totals its lanes' sums per resource through LDS (lanes
//     r < R hold them) and posts them; after the barrier every wavefront adds
//     the four wavefronts' sums;
//  2. with several workgroups per cluster, wavefront 0 publishes the
//     workgroup's sums as tagged limbs and all four wavefronts read every
//     workgroup's words (wavefront w the workgroups w, w + 4, ...; each lane
//     one limb position of up to kXchPerThread workgroups, its loads in
//     flight together, polling until every tag matches, bounded by about 2 s
//     of the real-time counter); after a second barrier every wavefront adds
//     the four partial totals;
//  3. lanes r < R compute U_r (exact total rounded once), lambda_r of Eq. 8
//     and the stop test, and the new prices reach every lane by readlane, in
//     the same bits in every wavefront and workgroup; wavefront 0 of
//     workgroup 0 writes the prices, trace rows, update count and stop flag.
// Returns false when the cluster stops here or a wait timed out.
template <int R, typename A>
__device__ bool resident_complete(const KArgs &a, int cl, int blk, int wave, int lane, A acc, bool acc_lane,
                                  double eta, double (&lam)[R]) {
    constexpr int Q = kWaveSize / R;
    __shared__ A s_lane[kBlockWaves][kWaveSize];
    __shared__ A s_wave[2][kBlockWaves][R];
    __shared__ unsigned long long s_limb[kBlockWaves][kWaveSize];
    __shared__ unsigned long long s_xw[2][kBlockWaves][R * kMaxLimbs];
    __shared__ int s_go;
    const int m = a.iter_no;
    const int par = m & 1;
    // 1. wavefront sums per resource
    s_lane[wave][lane] = acc_lane ? acc : A(0);
    wave_sync();
    // (every partial sum fits the accumulator type A: the packer sized A for
    // the whole column's total)
    if (lane < R) {
        A ws = 0;
#pragma unroll
        for (int q = 0; q < Q; ++q) ws += s_lane[wave][q * R + lane];
        s_wave[par][wave][lane] = ws;
    }
    if (threadIdx.x == 0) s_go = 1;
    __syncthreads();
    A tot = 0;
    if (lane < R) {
#pragma unroll
        for (int w = 0; w < kBlockWaves; ++w) tot += s_wave[par][w][lane];
    }
    if (a.nblk > 1) {
        // 2. the exchange between the workgroups of the cluster
        const int L = a.limbs;
        const int RL = R * L;
        const uint64_t tag = static_cast<uint64_t>((m - 1) % 65535 + 1);
        uint64_t *words = xch_words(a, cl, m);
        if (wave == 0 && lane < R) {
            for (int l = 0; l < L; ++l) {
                const uint64_t v = static_cast<uint64_t>(static_cast<u128>(tot) >> (kLimbBits * l)) & kLimbMask;
                __hip_atomic_store(words + static_cast<size_t>(blk) * a.xch_stride + lane * L + l,
                                   (tag << kLimbBits) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        const int G = kWaveSize / RL;                 // lane groups per wavefront
        const int g = lane / RL, q = lane - g * RL;
        unsigned long long sum = 0;
        if (g < G) {
            const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
            while (true) {
                bool all = true;
                sum = 0;
#pragma unroll
                for (int u = 0; u < kXchPerThread; ++u) {
                    const int b = wave + kBlockWaves * (g + G * u);
                    const int bc = b < a.nblk ? b : a.nblk - 1;          // clamped: no branch around the load
                    const uint64_t x = __hip_atomic_load(words + static_cast<size_t>(bc) * a.xch_stride + q,
                                                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    const bool valid = b < a.nblk;
                    all &= !valid | ((x >> kLimbBits) == tag);
                    sum += valid ? (x & kLimbMask) : 0ull;
                }
                if (all) break;
                if (__hip_atomic_load(a.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
                    __builtin_amdgcn_s_memrealtime() - t0 > 200000000ull) {
                    atomicCAS(a.status, 0, kStatusTimeout);
                    s_go = 0;                          // every wavefront still reaches the barrier
                    break;
                }
            }
        }
        s_limb[wave][lane] = sum;
        wave_sync();
        if (lane < RL) {
            unsigned long long ps = 0;
            for (int gg = 0; gg < G; ++gg) ps += s_limb[wave][gg * RL + lane];
            s_xw[par][wave][lane] = ps;
        }
        __syncthreads();
        if (s_go == 0) return false;
        tot = 0;
        if (lane < R) {
            u128 t128 = 0;
            for (int l = 0; l < L; ++l) {
                u128 ls = 0;
#pragma unroll
                for (int w = 0; w < kBlockWaves; ++w) ls += s_xw[par][w][lane * L + l];
                t128 += ls << (kLimbBits * l);
            }
            tot = static_cast<A>(t128);          // the exact total, which fits A
        }
    }
    // 3. U, Eq. 8 and the stop test in lanes r < R
    double lo = lam[0];
#pragma unroll
    for (int r = 1; r < R; ++r) lo = (lane == r) ? lam[r] : lo;
    double U = 0.0, ln = 0.0;
    bool ok = true;
    if (lane < R) {
        const size_t i = static_cast<size_t>(cl) * R + lane;
        U = fx_to_double(tot, a.shift[i]);
        const double gd = U - a.cap[i];
        const double x = lo + eta * gd;
        ln = (x > 0.0) ? x : 0.0;
        const double scale = lo > 1.0 ? lo : 1.0;
        ok = fabs(ln - lo) <= a.tol * scale;
        if (wave == 0 && blk == 0) {
            a.lam_out[i] = ln;
            if (a.tr_lam) a.tr_lam[i] = ln;
            if (a.tr_U) a.tr_U[i] = U;
        }
    }
    const bool stop = (a.tol > 0.0) & (__ballot(!ok) == 0);      // wave-uniform, the same in every wavefront
    if (wave == 0 && blk == 0 && lane == 0) {
        if (a.iters_done) a.iters_done[cl] = m;
        if (stop) atomicOr(&a.flags[cl], kFlagStopped);
    }
#pragma unroll
    for (int r = 0; r < R; ++r) lam[r] = readlane_d(ln, r);
    return !stop;
}

// Per-iteration view of the arguments of a persistent launch.
template <int R>
__device__ __forceinline__ KArgs iteration_args(const KArgs &a, int it) {
    KArgs ai = a;
    const size_t i = static_cast<size_t>(it);
    ai.t = a.t + it;
    if (a.tr_lam) ai.tr_lam = a.tr_lam + i * a.B * R;
    if (a.tr_U) ai.tr_U = a.tr_U + i * a.B * R;
    if (a.choice) ai.choice = a.choice + i * a.B * a.N;
    ai.iter_no = a.iter_no + it;
    ai.reverse = a.reverse ^ (a.sweep_alt & it & 1);
    return ai;
}

// Between the iterations of a persistent launch with one workgroup per
// cluster: the workgroup computed the new prices itself (s_newlam) and
// continues with them unless the cluster has stopped.
template <int R>
__device__ __forceinline__ bool next_prices_local(double *s_lam, const double *s_newlam, const int *s_stop) {
    __syncthreads();
    if (*s_stop) return false;
    if (threadIdx.x < R) s_lam[threadIdx.x] = s_newlam[threadIdx.x];
    __syncthreads();
    return true;
}

// ---------------------------------------------------------------------------
// Dense families: K = 4 * LPJ configurations per job, LPJ lanes per job
// ---------------------------------------------------------------------------

// Launch modes of the fused kernels, one instance each, so that the
// one-iteration instance does without the code (and the registers) of the
// multi-iteration ones.
constexpr int kOnePass = 0;          // one iteration or one selection per launch
constexpr int kPersistLocal = 1;     // several iterations, one workgroup per cluster
constexpr int kPersistDeferred = 2;  // cooperative, several iterations, deferred completion between them
// Several iterations over tiles held in registers for the whole launch (each
// wavefront has at most two: no table loads inside the loop); the launch
// completes every iteration itself, with one workgroup per cluster or
// through the tagged exchange between the workgroups of a cluster.
constexpr int kResident = 3;

template <int R, int LPJ, typename A, int Mode>
__global__ __launch_bounds__(kBlockThreads) void k_dense(KArgs a) {
    constexpr int JPT = kWaveSize / LPJ;       // jobs per tile
    constexpr int Q = kWaveSize / R;           // accumulating lanes per resource
    __shared__ float s_stage[kBlockWaves][JPT][R];
    __shared__ u128 s_acc[kBlockThreads];
    __shared__ u128 s_wsum[kBlockWaves][R];
    __shared__ u128 s_bsum[R];
    __shared__ double s_lam[R];
    __shared__ double s_newlam[R];
    __shared__ int s_go;
    __shared__ int s_stop;

    const int cl = blockIdx.x / a.nblk;
    const int blk = blockIdx.x - cl * a.nblk;
    const int conv = a.conv_at[cl];            // with the flags: one wait for both
    if (a.flags && (a.flags[cl] & a.skip_mask)) return;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (threadIdx.x == 0) s_stop = 0;

    double lam[R];                             // prices of the current iteration

    const float *col = a.table + cl * a.cluster_stride;
    const int my_r = lane % R;
    const int my_q = lane / R;
    const bool acc_lane = lane < Q * R;
    const int my_shift = a.shift[cl * R + my_r];
    const int gl = lane % LPJ;                 // lane within its job group
    const int jt = lane / LPJ;                 // job within the tile
    A acc = 0;

    const int stride = a.nblk * kBlockWaves;
    const size_t lane_off = static_cast<size_t>(lane) * 4;
    // Tiles are swept front to back, or back to front when `rev` is set; the
    // exact demand sum does not depend on the order.
    const int last = a.tiles - 1;
    const double sw = a.has_pen ? a.switch_cost[cl] : 0.0;
    auto load_tile = [&](int t, int rev, f4 &u, f4 (&d)[R], f4 &pn) {
        const int tl = rev ? last - t : t;
        const float *p = col + static_cast<size_t>(tl) * kTileEntries + lane_off;
        u = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p));
#pragma unroll
        for (int r = 0; r < R; ++r)
            d[r] = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p + (r + 1) * a.col_len));
        if (a.has_pen) pn = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p + (R + 1) * a.col_len));
    };
    // Score, select and stage one tile held in registers.
    auto process = [&](const KArgs &ai, int t, const f4 &u, const f4 (&d)[R], const f4 &pn) {
        const int tl = ai.reverse ? last - t : t;
        double best = 0.0;
        int bi = 0;
        // The lane's best of its 4 entries (lowest index on ties); the
        // penalty test is taken once per tile (a uniform branch), not per entry.
        auto lane_best = [&](auto pen) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                double rent = static_cast<double>(d[0][i]) * lam[0];
#pragma unroll
                for (int r = 1; r < R; ++r) rent = rent + static_cast<double>(d[r][i]) * lam[r];
                double sc = static_cast<double>(u[i]) - rent;
                if constexpr (decltype(pen)::value) sc = penalize(sc, pn[i], sw);
                if (i == 0 || sc > best) { best = sc; bi = i; }
            }
        };
        if (a.has_pen) lane_best(std::true_type{});
        else lane_best(std::false_type{});
        int k = gl * 4 + bi;
        group_argmax<LPJ>(best, k);
        const int j = tl * JPT + jt;
        const bool owner = ((k >> 2) == gl) & (j < ai.N);   // this lane holds the winning entry
        if (ai.choice && owner) ai.choice[static_cast<size_t>(cl) * ai.N + j] = k;
        if (ai.reduce) {
            const int w = k & 3;
            float v[R];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const float lo = (w & 1) ? d[r][1] : d[r][0];
                const float hi = (w & 1) ? d[r][3] : d[r][2];
                v[r] = (w & 2) ? hi : lo;
            }
            if ((j >= ai.N) & (gl == 0)) {
#pragma unroll
                for (int r = 0; r < R; ++r) s_stage[wave][jt][r] = 0.0f;   // jobs past N add nothing
            }
            if (owner) {
#pragma unroll
                for (int r = 0; r < R; ++r) s_stage[wave][jt][r] = v[r];
            }
            wave_sync();
            if (acc_lane) {
#pragma unroll 1
                for (int q = my_q; q < JPT; q += Q) acc += fx_of<A>(s_stage[wave][q][my_r], my_shift);
            }
            wave_sync();
        }
    };
    // Three register buffers, rotated by unrolling: while one tile is scored
    // the loads of the next two are in flight (18 KB per wavefront at R = 8).
    // In a persistent launch the first two loads of the next iteration are
    // issued before the wait for its prices.
    f4 ua, ub, uc, pa = {}, pb = {}, pc = {};
    f4 da[R], db[R], dc[R];
    const int tile0 = blk * kBlockWaves + wave;
    // Loads of tiles past the end are clamped to the last tile (never
    // processed): no branches, so that the compiler's waits for earlier loads
    // do not wait for these.
    auto prefetch_two = [&](int rev) {
        load_tile(min(tile0, last), rev, ua, da, pa);
        load_tile(min(tile0 + stride, last), rev, ub, db, pb);
    };
    Pending<R, A> pend;
    if constexpr (Mode != kResident) pending_loads<R, A>(a, cl, conv, pend);   // issued first: they return first
    prefetch_two(a.reverse);                   // in flight during a pending completion; a resident
                                               // launch's tiles for all its iterations
    const double *etas = nullptr;
    if constexpr (Mode == kResident) etas = resident_etas(a, cl);   // read after launch_prices' barrier
    if (!launch_prices<R, A>(a, cl, blk, pend, s_lam, s_newlam, s_acc)) return;
#pragma unroll
    for (int r = 0; r < R; ++r) lam[r] = s_lam[r];
    for (int it = 0; it < a.n_iters; ++it) {
        const KArgs ai = iteration_args<R>(a, it);
        const int rev = ai.reverse;
        if constexpr (Mode == kResident) {
            // the wavefront's tiles stay in ua / ub (loaded front to back)
            if (tile0 < a.tiles) process(ai, tile0, ua, da, pa);
            if (tile0 + stride < a.tiles) process(ai, tile0 + stride, ub, db, pb);
        } else {
            // Loads past the end are clamped to the last tile (never
            // processed): without branches around them the compiler waits
            // for each tile's own loads only.
            for (int tile = tile0; tile < a.tiles; tile += 3 * stride) {
                const int t1 = tile + stride, t2 = tile + 2 * stride;
                load_tile(min(t2, last), rev, uc, dc, pc);
                process(ai, tile, ua, da, pa);
                load_tile(min(t2 + stride, last), rev, ua, da, pa);
                if (t1 < a.tiles) process(ai, t1, ub, db, pb);
                load_tile(min(t2 + 2 * stride, last), rev, ub, db, pb);
                if (t2 < a.tiles) process(ai, t2, uc, dc, pc);
            }
        }
        if (!ai.reduce) return;
        if constexpr (Mode == kResident) {
            const bool go = resident_complete<R, A>(ai, cl, blk, wave, lane, acc, acc_lane, etas[it], lam);
            acc = 0;
            if (!go || it + 1 == a.n_iters) break;
            continue;
        }

        // Workgroup sum per resource (integer adds: any order gives the same value).
        s_acc[threadIdx.x] = acc_lane ? static_cast<u128>(acc) : static_cast<u128>(0);
        acc = 0;
        __syncthreads();
        if (threadIdx.x < kBlockWaves * R) {
            const int w = threadIdx.x / R, r = threadIdx.x % R;
            u128 v = 0;
#pragma unroll   // independent LDS loads, all in flight
            for (int q = 0; q < Q; ++q) v += s_acc[w * kWaveSize + q * R + r];
            s_wsum[w][r] = v;
        }
        __syncthreads();
        if (threadIdx.x < R) {
            u128 v = 0;
#pragma unroll
            for (int w = 0; w < kBlockWaves; ++w) v += s_wsum[w][threadIdx.x];
            s_bsum[threadIdx.x] = v;
        }
        __syncthreads();
        if (Mode == kPersistDeferred || (Mode == kOnePass && a.defer)) {
            publish_iteration<R, Mode == kPersistDeferred>(ai, cl, blk, ai.iter_no, s_bsum);
            if (Mode == kOnePass || it + 1 == a.n_iters) break;    // the next launch completes it
            prefetch_two(rev ^ a.sweep_alt);
            if (!wait_iteration(a, cl, blk, ai.iter_no, &s_go)) break;
            A v[kSumLoads];
            partial_loads<R, A, true>(ai, ai.iter_no & 1, cl, v);
            if (complete_iteration<R, A, true>(ai, cl, ai.iter_no, ai.t, blk == 0, s_lam, s_newlam, s_acc, v)) break;
            if (threadIdx.x < R) s_lam[threadIdx.x] = s_newlam[threadIdx.x];
            __syncthreads();
        } else {
            // the next iteration's first tiles do not depend on the prices
            if (Mode == kPersistLocal && it + 1 < a.n_iters) prefetch_two(rev ^ a.sweep_alt);
            finish_cluster<R, false>(ai, cl, blk, s_bsum, s_lam, s_newlam, &s_stop);
            if (Mode == kOnePass || it + 1 == a.n_iters) break;
            if (!next_prices_local<R>(s_lam, s_newlam, &s_stop)) break;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) lam[r] = s_lam[r];
    }
}

// ---------------------------------------------------------------------------
// CSR families (ragged sizes 1..256): whole families packed into tiles
// ---------------------------------------------------------------------------

constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;
constexpr int kDppWaveShr1 = 0x138;

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_or_i(int old, int v) {
    return __builtin_amdgcn_update_dpp(old, v, CTRL, ROW_MASK, 0xf, false);
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_or_d(double old, double v) {
    const long long ob = __double_as_longlong(old), vb = __double_as_longlong(v);
    const int lo = dpp_or_i<CTRL, ROW_MASK>(static_cast<int>(static_cast<unsigned>(ob)),
                                            static_cast<int>(static_cast<unsigned>(vb)));
    const int hi = dpp_or_i<CTRL, ROW_MASK>(static_cast<int>(ob >> 32), static_cast<int>(vb >> 32));
    return __longlong_as_double(static_cast<long long>(
        (static_cast<unsigned long long>(static_cast<unsigned>(hi)) << 32) | static_cast<unsigned>(lo)));
}

// acc plus the number of set bits of a wave-wide mask in the lanes below this one.
__device__ __forceinline__ unsigned below_lane(uint64_t m, unsigned acc) {
    return __builtin_amdgcn_mbcnt_hi(static_cast<unsigned>(m >> 32),
                                     __builtin_amdgcn_mbcnt_lo(static_cast<unsigned>(m), acc));
}

// One step of an inclusive segmented max-scan over lanes of (best score,
// segment-start flag): a lane without a segment start combines the value
// arriving from lower lanes.  A lane with no source receives its own score
// and a clear flag, which changes nothing.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ void seg_scan_step(double &s, int &f) {
    const double os = dpp_or_d<CTRL, ROW_MASK>(s, s);
    const int of = dpp_or_i<CTRL, ROW_MASK>(0, f);
    // selects and bitwise operators, not branches (the lanes diverge on f)
    s = ((f == 0) & (os > s)) ? os : s;
    f = f | of;
}

// Two wavefronts per SIMD at least (at most 256 registers): the CSR grid holds
// two workgroups per CU, and a cooperative launch needs them all resident
// (the persistent instances at R = 8 would otherwise take a few more).  The
// resident instance keeps two tiles live through every iteration and runs
// one workgroup per CU at most: it may use the whole register file.
template <int R, typename A, int Mode>
__global__ __launch_bounds__(kBlockThreads, Mode == kResident ? 1 : 2) void k_csr(KArgs a) {
    constexpr int Q = kWaveSize / R;           // accumulating lanes per resource
    __shared__ float s_stage[kBlockWaves][kTileEntries][R];
    __shared__ u128 s_acc[kBlockThreads];
    __shared__ u128 s_wsum[kBlockWaves][R];
    __shared__ u128 s_bsum[R];
    __shared__ double s_lam[R];
    __shared__ double s_newlam[R];
    __shared__ int s_go;
    __shared__ int s_stop;

    const int cl = blockIdx.x / a.nblk;
    const int blk = blockIdx.x - cl * a.nblk;
    const int conv = a.conv_at[cl];            // with the flags: one wait for both
    if (a.flags && (a.flags[cl] & a.skip_mask)) return;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (threadIdx.x == 0) s_stop = 0;

    double lam[R];                             // prices of the current iteration
    const int my_r = lane % R;
    const int my_q = lane / R;
    const bool acc_lane = lane < Q * R;
    const int my_shift = a.shift[cl * R + my_r];
    A acc = 0;

    const float *col = a.table + cl * a.cluster_stride;
    const size_t lane_off = static_cast<size_t>(lane) * 4;
    const int hshift = (lane & 7) * 4;                   // this lane's 4 head bits in its word
    const uint64_t above = lane == kWaveSize - 1 ? 0ull : ~0ull << (lane + 1);   // the lanes above this one
    const double sw = a.has_pen ? a.switch_cost[cl] : 0.0;
    const int stride = a.nblk * kBlockWaves;
    const int last = a.tiles - 1;
    auto load_tile = [&](int t, int rev, f4 &u, f4 (&d)[R], f4 &pn, uint32_t &hw) {
        const int tl = rev ? last - t : t;
        const float *p = col + static_cast<size_t>(tl) * kTileEntries + lane_off;
        u = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p));
#pragma unroll
        for (int r = 0; r < R; ++r)
            d[r] = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p + (r + 1) * a.col_len));
        if (a.has_pen) pn = __builtin_nontemporal_load(reinterpret_cast<const f4 *>(p + (R + 1) * a.col_len));
        hw = a.meta[tl].head[lane >> 3];
    };
    // Score one tile, find every family's winner and stage the winners'
    // demands (or write the choices).
    auto process = [&](const KArgs &ai, int t, const f4 &u, const f4 (&d)[R], const f4 &pn, uint32_t hw) {
        const int tl = ai.reverse ? last - t : t;
        const uint32_t hbits = (hw >> hshift) & 0xFu;
        double sc[4];
        // the penalty test is taken once per tile (a uniform branch)
        auto scores = [&](auto pen) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                double rent = static_cast<double>(d[0][i]) * lam[0];
#pragma unroll
                for (int r = 1; r < R; ++r) rent = rent + static_cast<double>(d[r][i]) * lam[r];
                sc[i] = static_cast<double>(u[i]) - rent;
                if constexpr (decltype(pen)::value) sc[i] = penalize(sc[i], pn[i], sw);
            }
        };
        if (a.has_pen) scores(std::true_type{});
        else scores(std::false_type{});
        // Lane-local pass: one running best (lowest entry on ties) that
        // restarts at every head.  At a head the run so far is either a
        // segment that began at an earlier head of this lane (complete: its
        // winner is marked) or, before the lane's first head, this lane's
        // part of a segment from lower lanes (pre).  At the end the run is
        // the segment left open at the lane's end.
        // (selects, not branches: the lanes diverge on their head bits)
        const bool h0 = hbits & 1u;
        double run_s = sc[0], pre_s = sc[0];
        int run_i = 0, pre_i = 0;
        bool open = h0;
        uint32_t local_win = 0;
#pragma unroll
        for (int i = 1; i < 4; ++i) {
            const bool head = (hbits >> i) & 1u;
            local_win |= static_cast<uint32_t>(head & open) << run_i;
            const bool first = head & !open;
            pre_s = first ? run_s : pre_s;
            pre_i = first ? run_i : pre_i;
            const bool take = head | (sc[i] > run_s);
            run_s = take ? sc[i] : run_s;
            run_i = take ? i : run_i;
            open = open | head;
        }
        const bool has_head = hbits != 0;
        const bool has_pre = has_head & !h0;
        // Segment maxima across lanes: after the scan, ps is the largest score
        // of the segment open at this lane's end, over its slots up to here.
        double ps = run_s;
        int pf = has_head ? 1 : 0;
        seg_scan_step<kDppRowShr1, 0xf>(ps, pf);
        seg_scan_step<kDppRowShr2, 0xf>(ps, pf);
        seg_scan_step<kDppRowShr4, 0xf>(ps, pf);
        seg_scan_step<kDppRowShr8, 0xf>(ps, pf);
        seg_scan_step<kDppRowBcast15, 0xa>(ps, pf);
        seg_scan_step<kDppRowBcast31, 0xc>(ps, pf);
        // the same at the previous lane (lane 0: its own value)
        const double qs = dpp_or_d<kDppWaveShr1, 0xf>(ps, ps);
        // Each winner is marked by the lane that holds it.  The winner of a
        // segment is its first slot with the segment's largest score: in the
        // lane where the running maximum last rose (a head, or a run strictly
        // above everything before it: lane `jump`), its run's best, unless the
        // part of the next head lane before its first head (slots above all
        // of the segment's others) beats it strictly (`pre_wins` there).
        const bool jump = has_head | (ps > qs) | (lane == 0);
        const bool pre_wins = has_pre & (pre_s > qs);
        const uint64_t m_head = __ballot(has_head);
        const uint64_t m_rise = __ballot(jump);
        const uint64_t m_keep = m_head & ~__ballot(pre_wins);   // head lanes whose pre part loses
        // the next lane above this one where the maximum rises or a segment starts
        const uint64_t later = m_rise & above;
        const int nxt = later ? __builtin_ctzll(later) : kWaveSize;
        const bool run_wins = jump & ((nxt == kWaveSize) | (((m_keep >> (nxt & (kWaveSize - 1))) & 1ull) != 0ull));
        const uint32_t wbits = local_win | (pre_wins ? 1u << pre_i : 0u) | (run_wins ? 1u << run_i : 0u);
        // Rank of this lane's first winner among the tile's winners (slot
        // order: lane, then entry): the winners in lower lanes, counted from
        // one ballot per entry position; n_win is the same for every lane.
        const uint64_t b0 = __ballot(wbits & 1u), b1 = __ballot(wbits & 2u);
        const uint64_t b2 = __ballot(wbits & 4u), b3 = __ballot(wbits & 8u);
        int rank = static_cast<int>(below_lane(b3, below_lane(b2, below_lane(b1, below_lane(b0, 0u)))));
        const int n_win = __popcll(b0) + __popcll(b1) + __popcll(b2) + __popcll(b3);
        if (wbits) {
            uint32_t hwm[8];
            if (ai.choice) {
#pragma unroll
                for (int q = 0; q < 8; ++q) hwm[q] = a.meta[tl].head[q];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                if (!((wbits >> i) & 1u)) continue;
                if (ai.reduce) {
#pragma unroll
                    for (int r = 0; r < R; ++r) s_stage[wave][rank][r] = d[r][i];
                }
                ++rank;
                if (ai.choice) {
                    // job = first_job + (heads at or before the slot) - 1;
                    // config = slot - (the last head at or before it)
                    const int slot = lane * 4 + i;
                    const int w = slot >> 5;
                    int cnt = 0, hs = -1;
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        uint32_t m = hwm[q];
                        if (q == w) m &= 0xffffffffu >> (31 - (slot & 31));
                        if (q <= w) {
                            cnt += __popc(m);
                            if (m) hs = q * 32 + 31 - __clz(m);
                        }
                    }
                    const int j = static_cast<int>(a.meta[tl].first_job) + cnt - 1;
                    ai.choice[static_cast<size_t>(cl) * a.N + j] = slot - hs;
                }
            }
        }
        if (ai.reduce) {
            wave_sync();
            if (acc_lane) {
#pragma unroll 1
                for (int q = my_q; q < n_win; q += Q) acc += fx_of<A>(s_stage[wave][q][my_r], my_shift);
            }
            wave_sync();
        }
    };
    // One tile of prefetch: the next tile's loads are in flight while the
    // current one is scored (a deeper prefetch measured no faster).  Two
    // register sets take turns (the loop body appears twice), so the
    // prefetched tile is scored where it landed, without copies.
    f4 nu, npn = {}, bu, bpn = {};
    f4 nd[R], bd[R];
    uint32_t nhw = 0, bhw = 0;
    const int tile0 = blk * kBlockWaves + wave;
    Pending<R, A> pend;
    if constexpr (Mode != kResident) pending_loads<R, A>(a, cl, conv, pend);   // issued first: they return first
    load_tile(min(tile0, last), a.reverse, nu, nd, npn, nhw);   // in flight during a pending completion (clamped: no branch)
    if constexpr (Mode == kResident)
        load_tile(min(tile0 + stride, last), a.reverse, bu, bd, bpn, bhw);   // the launch's second tile
    const double *etas = nullptr;
    if constexpr (Mode == kResident) etas = resident_etas(a, cl);   // read after launch_prices' barrier
    if (!launch_prices<R, A>(a, cl, blk, pend, s_lam, s_newlam, s_acc)) return;
#pragma unroll
    for (int r = 0; r < R; ++r) lam[r] = s_lam[r];
    for (int it = 0; it < a.n_iters; ++it) {
        const KArgs ai = iteration_args<R>(a, it);
        const int rev = ai.reverse;
        if constexpr (Mode == kResident) {
            // the wavefront's tiles stay in the two register sets (loaded front to back)
            if (tile0 < a.tiles) process(ai, tile0, nu, nd, npn, nhw);
            if (tile0 + stride < a.tiles) process(ai, tile0 + stride, bu, bd, bpn, bhw);
        } else {
            for (int tile = tile0; tile < a.tiles; tile += 2 * stride) {
                load_tile(min(tile + stride, last), rev, bu, bd, bpn, bhw);   // clamped: no branch
                process(ai, tile, nu, nd, npn, nhw);
                if (tile + stride >= a.tiles) break;
                load_tile(min(tile + 2 * stride, last), rev, nu, nd, npn, nhw);
                process(ai, tile + stride, bu, bd, bpn, bhw);
            }
        }
        if (!ai.reduce) return;
        if constexpr (Mode == kResident) {
            const bool go = resident_complete<R, A>(ai, cl, blk, wave, lane, acc, acc_lane, etas[it], lam);
            acc = 0;
            if (!go || it + 1 == a.n_iters) break;
            continue;
        }

        s_acc[threadIdx.x] = acc_lane ? static_cast<u128>(acc) : static_cast<u128>(0);
        acc = 0;
        __syncthreads();
        if (threadIdx.x < kBlockWaves * R) {
            const int w = threadIdx.x / R, r = threadIdx.x % R;
            u128 v = 0;
#pragma unroll   // independent LDS loads, all in flight
            for (int q = 0; q < Q; ++q) v += s_acc[w * kWaveSize + q * R + r];
            s_wsum[w][r] = v;
        }
        __syncthreads();
        if (threadIdx.x < R) {
            u128 v = 0;
#pragma unroll
            for (int w = 0; w < kBlockWaves; ++w) v += s_wsum[w][threadIdx.x];
            s_bsum[threadIdx.x] = v;
        }
        __syncthreads();
        if (Mode == kPersistDeferred || (Mode == kOnePass && a.defer)) {
            publish_iteration<R, Mode == kPersistDeferred>(ai, cl, blk, ai.iter_no, s_bsum);
            if (Mode == kOnePass || it + 1 == a.n_iters) break;    // the next launch completes it
            load_tile(min(tile0, last), rev ^ a.sweep_alt, nu, nd, npn, nhw);
            if (!wait_iteration(a, cl, blk, ai.iter_no, &s_go)) break;
            A v[kSumLoads];
            partial_loads<R, A, true>(ai, ai.iter_no & 1, cl, v);
            if (complete_iteration<R, A, true>(ai, cl, ai.iter_no, ai.t, blk == 0, s_lam, s_newlam, s_acc, v)) break;
            if (threadIdx.x < R) s_lam[threadIdx.x] = s_newlam[threadIdx.x];
            __syncthreads();
        } else {
            // the next iteration's first tile does not depend on the prices
            if (Mode == kPersistLocal && it + 1 < a.n_iters)
                load_tile(min(tile0, last), rev ^ a.sweep_alt, nu, nd, npn, nhw);
            finish_cluster<R, false>(ai, cl, blk, s_bsum, s_lam, s_newlam, &s_stop);
            if (Mode == kOnePass || it + 1 == a.n_iters) break;
            if (!next_prices_local<R>(s_lam, s_newlam, &s_stop)) break;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) lam[r] = s_lam[r];
    }
}

// ---------------------------------------------------------------------------
// Gather: U from caller-supplied choices (granular esp_reduce_demand)
// ---------------------------------------------------------------------------

template <int R, typename A>
__global__ __launch_bounds__(kBlockThreads) void k_gather(KArgs a) {
    __shared__ u128 s_red[kBlockThreads];
    __shared__ u128 s_bsum[R];
    __shared__ int s_bad;
    const int cl = blockIdx.x / a.nblk;
    const int blk = blockIdx.x - cl * a.nblk;
    const float *col = a.table + cl * a.cluster_stride;
    A acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] = 0;
    int sh[R];
#pragma unroll
    for (int r = 0; r < R; ++r) sh[r] = a.shift[cl * R + r];
    if (threadIdx.x == 0) s_bad = 0;
    __syncthreads();
    bool bad = false;
    for (int j = blk * kBlockThreads + threadIdx.x; j < a.N; j += a.nblk * kBlockThreads) {
        const int c = a.choice_in[static_cast<size_t>(cl) * a.N + j];
        uint32_t slot, size;
        if (a.K > 0) {
            slot = static_cast<uint32_t>(j) * static_cast<uint32_t>(a.K);
            size = static_cast<uint32_t>(a.K);
        } else {
            slot = a.jobs[j].slot;
            size = a.jobs[j].size;
        }
        if (c < 0 || static_cast<uint32_t>(c) >= size) { bad = true; continue; }
        const size_t e = static_cast<size_t>(slot) + static_cast<uint32_t>(c);
#pragma unroll
        for (int r = 0; r < R; ++r) acc[r] += fx_of<A>(col[(r + 1) * a.col_len + e], sh[r]);
    }
    if (bad) s_bad = 1;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        s_red[threadIdx.x] = static_cast<u128>(acc[r]);
        __syncthreads();
#pragma unroll 1
        for (int st = kBlockThreads / 2; st > 0; st >>= 1) {
            if (threadIdx.x < st) s_red[threadIdx.x] += s_red[threadIdx.x + st];
            __syncthreads();
        }
        if (threadIdx.x == 0) s_bsum[r] = s_red[0];
        __syncthreads();
    }
    if (threadIdx.x == 0 && s_bad) {
        atomicOr(&a.flags[cl], 4);
        atomicCAS(a.status, 0, kStatusInvalid);
    }
    __shared__ double s_newlam[R];
    __shared__ int s_stop;
    finish_cluster<R, true>(a, cl, blk, s_bsum, nullptr, s_newlam, &s_stop);
}

// ---------------------------------------------------------------------------
// Granular price update (esp_update_prices) and price validation
// ---------------------------------------------------------------------------

__device__ __forceinline__ bool price_ok(double x) {
    return x >= 0.0 && x <= 0x1p400;            // false for NaN and +-Inf
}

template <int R>
__global__ void k_update(KArgs a, const double *demand_in, int B) {
    const int cl = blockIdx.x * blockDim.x + threadIdx.x;
    if (cl >= B) return;
    bool ok = true;
    for (int r = 0; r < R; ++r) {
        const double U = demand_in[cl * R + r];
        ok = ok && price_ok(a.lam_in[cl * R + r]) && (U >= -0x1p200 && U <= 0x1p200);
    }
    if (!ok) {
        atomicCAS(a.status, 0, kStatusNonfinite);
        return;
    }
    for (int r = 0; r < R; ++r) {
        const double lo = a.lam_in[cl * R + r];
        const double g = demand_in[cl * R + r] - a.cap[cl * R + r];
        const double x = lo + step_size(a, cl, a.t) * g;
        a.lam_out[cl * R + r] = (x > 0.0) ? x : 0.0;
    }
}

// Validate prices before a solve or a selection; mark bad clusters.  A valid
// price -0.0 is stored back as +0.0 when `canon` is set (the solve's in/out
// prices; never -0.0 afterwards, as after the projection of Eq. 8).  For a
// solve (iters_done set) also reset the per-solve counters and store the
// starting prices as lambda_1 (lam_ws[1]) for the first deferred completion.
template <int R>
__global__ void k_prepare(KArgs a, const double *lam, double *canon, int B) {
    const int cl = blockIdx.x * blockDim.x + threadIdx.x;
    // the resident exchange words start at tag 0 (a.xch_clear words, or none)
    for (size_t i = cl; i < a.xch_clear; i += static_cast<size_t>(gridDim.x) * blockDim.x) a.xch[i] = 0ull;
    if (cl >= B) return;
    bool ok = true;
    for (int r = 0; r < R; ++r) ok = ok && price_ok(lam[cl * R + r]);
    a.flags[cl] = (a.flags[cl] & kFlagFrozen) | (ok ? 0 : kFlagError);
    if (ok && canon) {
        for (int r = 0; r < R; ++r)
            if (__double_as_longlong(lam[cl * R + r]) == static_cast<long long>(0x8000000000000000ull))
                canon[cl * R + r] = 0.0;
    }
    if (a.iters_done) {
        a.iters_done[cl] = 0;
        a.tickets[cl] = 0u;          // 0 between launches; cleared for scratch shared between solves
        for (int i = 0; i < kSyncSlots; ++i) a.sync[(static_cast<size_t>(cl) * kSyncSlots + i) * kSyncStride] = 0u;
        a.conv_at[cl] = 0;
        for (int r = 0; r < R; ++r) {
            const double v = lam[cl * R + r];
            a.lam_ws[static_cast<size_t>(B) * R + static_cast<size_t>(cl) * R + r] = (v == 0.0) ? 0.0 : v;
        }
    }
    if (!ok) atomicCAS(a.status, 0, kStatusNonfinite);
}

// Closing launch of a deferred solve without a final selection: one
// workgroup per cluster completes the solve's last iteration (pend_m).
template <int R>
__global__ __launch_bounds__(kBlockThreads) void k_finish(KArgs a) {
    __shared__ u128 s_red[kBlockThreads];
    __shared__ double s_tmp[R];
    __shared__ double s_lam[R];
    const int cl = blockIdx.x;
    if (a.flags && (a.flags[cl] & a.skip_mask)) return;
    Pending<R, u128> pend;
    pending_loads<R, u128>(a, cl, a.conv_at[cl], pend);
    (void)launch_prices<R, u128>(a, cl, 0, pend, s_lam, s_tmp, s_red);
}

// ---------------------------------------------------------------------------
// Launchers (runtime R / LPJ -> template instance)
// ---------------------------------------------------------------------------

template <int R, typename A>
hipError_t launch_dense_ra(int lpj, const KArgs &a, int B, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(B) * a.nblk), block(kBlockThreads);
    switch (lpj) {
        case 1: hipLaunchKernelGGL((k_dense<R, 1, A, kOnePass>), grid, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL((k_dense<R, 2, A, kOnePass>), grid, block, 0, s, a); break;
        case 4: hipLaunchKernelGGL((k_dense<R, 4, A, kOnePass>), grid, block, 0, s, a); break;
        case 8: hipLaunchKernelGGL((k_dense<R, 8, A, kOnePass>), grid, block, 0, s, a); break;
        case 16: hipLaunchKernelGGL((k_dense<R, 16, A, kOnePass>), grid, block, 0, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int R>
hipError_t launch_dense_r(int lpj, const KArgs &a, int B, hipStream_t s) {
    return a.acc128 ? launch_dense_ra<R, u128>(lpj, a, B, s) : launch_dense_ra<R, uint64_t>(lpj, a, B, s);
}

// A cooperative launch of `blocks` workgroups of kernel f: refused on the host
// when the device cannot hold them all at once (nothing is enqueued then).
inline hipError_t launch_cooperative(const void *f, unsigned blocks, const KArgs &a, hipStream_t s) {
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, f, kBlockThreads, 0) != hipSuccess)
        return hipErrorInvalidValue;
    if (static_cast<int64_t>(blocks) > static_cast<int64_t>(per_cu) * cus) return hipErrorCooperativeLaunchTooLarge;
    KArgs copy = a;
    void *args[] = {&copy};
    return hipLaunchCooperativeKernel(f, dim3(blocks), dim3(kBlockThreads), args, 0, s);
}

// A multi-iteration launch of kernel f.  With one workgroup per cluster no
// workgroup waits for another: an ordinary launch.  Otherwise a cooperative
// one, so that the workgroups of a cluster are co-resident.
inline hipError_t launch_multi(const void *f, unsigned blocks, const KArgs &a, hipStream_t s) {
    if (a.nblk == 1) {
        KArgs copy = a;
        void *args[] = {&copy};
        return hipLaunchKernel(f, dim3(blocks), dim3(kBlockThreads), args, 0, s);
    }
    return launch_cooperative(f, blocks, a, s);
}

template <int R, int LPJ, typename A>
const void *dense_multi_kernel(const KArgs &a, bool resident) {
    if (resident) return reinterpret_cast<const void *>(&k_dense<R, LPJ, A, kResident>);
    return a.defer ? reinterpret_cast<const void *>(&k_dense<R, LPJ, A, kPersistDeferred>)
                   : reinterpret_cast<const void *>(&k_dense<R, LPJ, A, kPersistLocal>);
}

template <int R, typename A>
hipError_t launch_dense_coop_ra(int lpj, const KArgs &a, int B, bool resident, hipStream_t s) {
    const void *f = nullptr;
    switch (lpj) {
        case 1: f = dense_multi_kernel<R, 1, A>(a, resident); break;
        case 2: f = dense_multi_kernel<R, 2, A>(a, resident); break;
        case 4: f = dense_multi_kernel<R, 4, A>(a, resident); break;
        case 8: f = dense_multi_kernel<R, 8, A>(a, resident); break;
        case 16: f = dense_multi_kernel<R, 16, A>(a, resident); break;
        default: return hipErrorInvalidValue;
    }
    return launch_multi(f, static_cast<unsigned>(B) * a.nblk, a, s);
}

template <int R>
hipError_t launch_dense_coop_r(int lpj, const KArgs &a, int B, bool resident, hipStream_t s) {
    // several workgroups need deferred completion, or the resident exchange
    if (!resident && !a.defer && a.nblk != 1) return hipErrorInvalidValue;
    return a.acc128 ? launch_dense_coop_ra<R, u128>(lpj, a, B, resident, s)
                    : launch_dense_coop_ra<R, uint64_t>(lpj, a, B, resident, s);
}

template <int R>
hipError_t launch_gather_r(const KArgs &a, int B, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(B) * a.nblk), block(kBlockThreads);
    if (a.acc128)
        hipLaunchKernelGGL((k_gather<R, u128>), grid, block, 0, s, a);
    else
        hipLaunchKernelGGL((k_gather<R, uint64_t>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <int R>
hipError_t launch_update_r(const KArgs &a, const double *demand_in, int B, hipStream_t s) {
    hipLaunchKernelGGL((k_update<R>), dim3((B + 255) / 256), dim3(256), 0, s, a, demand_in, B);
    return hipGetLastError();
}

template <int R>
hipError_t launch_prepare_r(const KArgs &a, const double *lam, double *canon, int B, hipStream_t s) {
    const size_t blocks = std::max<size_t>((static_cast<size_t>(B) + 255) / 256,
                                           std::min<size_t>((a.xch_clear + 255) / 256, 256));
    hipLaunchKernelGGL((k_prepare<R>), dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s, a, lam, canon, B);
    return hipGetLastError();
}

template <int R>
hipError_t launch_finish_r(const KArgs &a, int B, hipStream_t s) {
    hipLaunchKernelGGL((k_finish<R>), dim3(static_cast<unsigned>(B)), dim3(kBlockThreads), 0, s, a);
    return hipGetLastError();
}

template <int R>
hipError_t launch_csr_r(const KArgs &a, int B, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(B) * a.nblk), block(kBlockThreads);
    if (a.acc128)
        hipLaunchKernelGGL((k_csr<R, u128, kOnePass>), grid, block, 0, s, a);
    else
        hipLaunchKernelGGL((k_csr<R, uint64_t, kOnePass>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <int R, typename A>
const void *csr_multi_kernel(const KArgs &a, bool resident) {
    if (resident) return reinterpret_cast<const void *>(&k_csr<R, A, kResident>);
    return a.defer ? reinterpret_cast<const void *>(&k_csr<R, A, kPersistDeferred>)
                   : reinterpret_cast<const void *>(&k_csr<R, A, kPersistLocal>);
}

template <int R>
hipError_t launch_csr_coop_r(const KArgs &a, int B, bool resident, hipStream_t s) {
    // several workgroups need deferred completion, or the resident exchange
    if (!resident && !a.defer && a.nblk != 1) return hipErrorInvalidValue;
    const void *f = a.acc128 ? csr_multi_kernel<R, u128>(a, resident) : csr_multi_kernel<R, uint64_t>(a, resident);
    return launch_multi(f, static_cast<unsigned>(B) * a.nblk, a, s);
}


// Instances compiled in the esp_inst_*.hip files.
#define ESP_FUSED_LAUNCHERS(X) \
    X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8)
#define ESP_DENSE_DECL(RR, EXT)                                                                      \
    EXT template hipError_t launch_dense_r<RR>(int, const KArgs &, int, hipStream_t);                  \
    EXT template hipError_t launch_dense_coop_r<RR>(int, const KArgs &, int, bool, hipStream_t);
#define ESP_CSR_DECL(RR, EXT)                                                                        \
    EXT template hipError_t launch_csr_r<RR>(const KArgs &, int, hipStream_t);                         \
    EXT template hipError_t launch_csr_coop_r<RR>(const KArgs &, int, bool, hipStream_t);

}  // namespace esp
