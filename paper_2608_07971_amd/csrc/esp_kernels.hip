// gfx950 kernels of the Elastic Shadow Pricing hot path (paper Sec. 3.2).
//
// One price iteration = one launch of a fused kernel:
//   score   s_jk = u_jk - sum_r lambda_r d_jkr          (Sec. 3.2.2, bracket of Eq. 6)
//   select  c_j  = argmax_k s_jk, lowest k on ties     (Sec. 3.2.2 per-job subproblem)
//   demand  U_r  = sum_j d_{j,c_j,r}, exact             (Sec. 3.2.3, under Eq. 8)
//   update  lambda_r <- max(0, lambda_r + eta_t (U_r - C_r)) in the last
//           workgroup of each cluster                   (Eq. 8)
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
#include <algorithm>

#include "esp_internal.hpp"

#pragma clang fp contract(off)

namespace esp {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef unsigned __int128 u128;

// ---------------------------------------------------------------------------
// Wavefront primitives
// ---------------------------------------------------------------------------

// DPP lane moves inside 16-lane rows.
constexpr int kDppXor1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;   // lane i <- lane 7-i within each 8 lanes
constexpr int kDppMirror = 0x140;       // lane i <- lane 15-i within each row

template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xf, 0xf, false);
}

template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
    const long long b = __double_as_longlong(v);
    const int lo = dpp_i<CTRL>(static_cast<int>(static_cast<unsigned>(b)));
    const int hi = dpp_i<CTRL>(static_cast<int>(b >> 32));
    return __longlong_as_double(static_cast<long long>(
        (static_cast<unsigned long long>(static_cast<unsigned>(hi)) << 32) | static_cast<unsigned>(lo)));
}

// (os, ok) replaces (s, k) when its score is larger, or equal with a lower
// configuration index.  This is a total order on (score, -index) for the
// non-NaN scores the kernels produce, so any reduction tree returns the
// entry a sequential lowest-index scan would.
__device__ __forceinline__ void take_better(double &s, int &k, double os, int ok) {
    const bool b = (os > s) || (os == s && ok < k);
    s = b ? os : s;
    k = b ? ok : k;
}

// The penalty of the ESP score (Eq. 7) after the rent: the switching cost when
// the stored penalty's sign bit marks "not the current configuration", then
// the interference penalty |p|.
__device__ __forceinline__ double penalize(double sc, float p, double sw) {
    if (__float_as_uint(p) >> 31) sc = sc - sw;
    return sc - static_cast<double>(fabsf(p));
}

// Argmax over aligned groups of LPJ lanes (LPJ in {1,2,4,8,16}); afterwards
// every lane of a group holds the group's winner.
template <int LPJ>
__device__ __forceinline__ void group_argmax(double &s, int &k) {
    if constexpr (LPJ >= 2) take_better(s, k, dpp_d<kDppXor1>(s), dpp_i<kDppXor1>(k));
    if constexpr (LPJ >= 4) take_better(s, k, dpp_d<kDppXor2>(s), dpp_i<kDppXor2>(k));
    if constexpr (LPJ >= 8) take_better(s, k, dpp_d<kDppHalfMirror>(s), dpp_i<kDppHalfMirror>(k));
    if constexpr (LPJ >= 16) take_better(s, k, dpp_d<kDppMirror>(s), dpp_i<kDppMirror>(k));
}

// Compiler-level ordering of LDS traffic inside one wavefront.
__device__ __forceinline__ void wave_sync() {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_wave_barrier();
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// ---------------------------------------------------------------------------
// Exact fixed-point demand accumulation
// ---------------------------------------------------------------------------

// v (finite, +0.0 or positive) as an integer multiple of 2^sh in an
// accumulator type A (64- or 128-bit, chosen by the packer per problem).  The
// packer guarantees that every nonzero value of the column has its lowest set
// bit at or above 2^sh and its highest below 2^(sh + bits(A) - 1 -
// ceil(log2(N + 1))), so the shift is exact and N of them cannot overflow A.
template <typename A>
__device__ __forceinline__ A fx_of(float v, int sh) {
    constexpr int kMax = static_cast<int>(sizeof(A)) * 8 - 1;
    const uint32_t bits = __float_as_uint(v);
    const uint32_t e = bits >> 23;
    const uint32_t m = (bits & 0x7fffffu) | (e ? 0x800000u : 0u);
    int s = (e ? static_cast<int>(e) : 1) - 150 - sh;
    if (m == 0) return 0;
    s = s > kMax ? kMax : (s < -kMax ? -kMax : s);
    const A mm = m;
    return s >= 0 ? (mm << s) : (mm >> (-s));
}

// Round a * 2^sh to the nearest binary64, ties to even.
__device__ __forceinline__ double fx_to_double(u128 a, int sh) {
    if (a == 0) return 0.0;
    const uint64_t hi = static_cast<uint64_t>(a >> 64);
    const uint64_t lo = static_cast<uint64_t>(a);
    const int h = hi ? 127 - __clzll(hi) : 63 - __clzll(lo);
    if (h <= 52) return ldexp(static_cast<double>(lo), sh);
    const int drop = h - 52;
    uint64_t m = static_cast<uint64_t>(a >> drop);
    const u128 rem = a & ((static_cast<u128>(1) << drop) - 1);
    const u128 half = static_cast<u128>(1) << (drop - 1);
    if (rem > half || (rem == half && (m & 1u))) m += 1;   // m <= 2^53: exact as a double
    return ldexp(static_cast<double>(m), drop + sh);
}

// ---------------------------------------------------------------------------
// Cluster completion: per-workgroup sums -> last workgroup -> U, Eq. 8 update
// ---------------------------------------------------------------------------

// U_r from the cluster's exact total, the Eq. 8 update and the stop test for
// resource r (one thread per resource of the cluster's last workgroup).
template <int R>
__device__ __forceinline__ void complete_resource(const KArgs &a, int cl, int r, u128 tot, int *s_ok,
                                                  double *s_newlam) {
    const bool bad = a.flags && (__hip_atomic_load(&a.flags[cl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & 4);
    const double U = bad ? __builtin_nan("") : fx_to_double(tot, a.shift[cl * R + r]);
    if (a.demand_out) a.demand_out[cl * R + r] = U;
    if (a.tr_U) a.tr_U[cl * R + r] = U;
    int ok = 1;
    if (a.lam_out) {
        const double lo = a.lam_in[cl * R + r];
        const double g = U - a.cap[cl * R + r];
        const double x = lo + a.eta[cl] * g;
        const double ln = (x > 0.0) ? x : 0.0;
        // agent-scope exchange: visible at the coherence point to the other
        // workgroups of a persistent launch once it has returned
        const double prev = __hip_atomic_exchange(&a.lam_out[cl * R + r], ln, __ATOMIC_RELAXED,
                                                  __HIP_MEMORY_SCOPE_AGENT);
        asm volatile("s_waitcnt vmcnt(0)" : : "v"(prev) : "memory");
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
template <int R>
__device__ __forceinline__ int complete_cluster(const KArgs &a, int cl, const int *s_ok) {
    int stop = 0;
    if (a.flags && (a.flags[cl] & 4)) atomicAnd(&a.flags[cl], ~4);
    if (a.lam_out) {
        // one writer per iteration, but not the same workgroup (or XCD) every
        // time: a coherent exchange, so the last iteration's value is the one kept
        if (a.iters_done) (void)__hip_atomic_exchange(&a.iters_done[cl], a.iter_no, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT);
        int all = 1;
        for (int r = 0; r < R; ++r) all &= s_ok[r];
        if (a.tol > 0.0 && all && a.flags) {
            atomicOr(&a.flags[cl], kFlagStopped);
            stop = 1;
        }
    }
    return stop;
}

// Cross-workgroup exact sums of one cluster.  bsum[r] (LDS) holds this
// workgroup's 128-bit sum for resource r.  In the workgroup that finishes
// last, thread r < R runs done(r, total_r) with the cluster's total; the
// function returns true there (after a workgroup barrier) and false in every
// other workgroup.
//
// Ordering across the 8 XCDs (each with its own L2) without cache-wide
// writeback or invalidation: wavefront 0 publishes the partial with
// agent-scope atomic exchanges, which are performed at the device coherence
// point and have completed once their old values are back; it waits for them
// (s_waitcnt vmcnt(0) on the returned values) before it takes a ticket with
// an agent-scope atomic add.  The workgroup that draws the last ticket reads
// every partial with agent-scope atomic loads, which bypass the non-coherent
// caches, and resets the ticket for the next use.
template <int R, typename Done>
__device__ __forceinline__ bool cluster_sums(const KArgs &a, int cl, int blk, const u128 *bsum, Done &&done) {
    __shared__ int s_last;
    __shared__ u128 s_red[kBlockThreads];
    const int t = threadIdx.x;
    if (a.nblk == 1) {
        // One workgroup per cluster: its own sums are the totals.
        if (t < R) s_red[t] = bsum[t];
        __syncthreads();
        if (t < R) done(t, s_red[t]);
        __syncthreads();
        return true;
    }
    if (t < kWaveSize) {
        uint64_t old = 0;
        if (t < R) {
            uint64_t *p = a.partials + ((static_cast<size_t>(cl) * a.nblk + blk) * R + t) * 2;
            const u128 v = bsum[t];
            old ^= __hip_atomic_exchange(p, static_cast<uint64_t>(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            old ^= __hip_atomic_exchange(p + 1, static_cast<uint64_t>(v >> 64), __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
        }
        asm volatile("s_waitcnt vmcnt(0)" : : "v"(old) : "memory");
        if (t == 0) {
            const unsigned prev = __hip_atomic_fetch_add(&a.tickets[cl], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_last = (prev == static_cast<unsigned>(a.nblk) - 1u);
        }
    }
    __syncthreads();
    if (!s_last) return false;

    // Sum the nblk partials of each resource: thread (g, r) takes blocks
    // g, g+G, g+2G, ...; eight independent loads in flight per thread.
    constexpr int G = kBlockThreads / R;
    constexpr int U = 8;
    u128 s = 0;
    if (t < G * R) {
        const int r = t % R, g = t / R;
        const uint64_t *base = a.partials + (static_cast<size_t>(cl) * a.nblk * R + r) * 2;
#pragma unroll 1
        for (int b0 = g; b0 < a.nblk; b0 += U * G) {
            u128 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int b = b0 + u * G;
                v[u] = 0;
                if (b < a.nblk) {
                    uint64_t *p = const_cast<uint64_t *>(base) + static_cast<size_t>(b) * R * 2;
                    const uint64_t lo = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    const uint64_t hi = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    v[u] = (static_cast<u128>(hi) << 64) | lo;
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) s += v[u];
        }
    }
    s_red[t] = s;
    __syncthreads();
    if (t < R) {
        u128 tot = 0;
#pragma unroll 1
        for (int g = 0; g < G; ++g) tot += s_red[g * R + t];
        done(t, tot);
    }
    if (t == 0) {
        // ready for the next use
        const unsigned o = __hip_atomic_exchange(&a.tickets[cl], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        asm volatile("s_waitcnt vmcnt(0)" : : "v"(o) : "memory");
    }
    __syncthreads();
    return true;
}

// The demand sums of one iteration: U, the Eq. 8 update and the per-cluster
// bookkeeping in the last workgroup.  s_newlam / s_stop (LDS) receive the new
// prices and the stop decision there.
template <int R>
__device__ bool finish_cluster(const KArgs &a, int cl, int blk, const u128 *bsum, double *s_newlam, int *s_stop) {
    __shared__ int s_ok[R];
    const bool last = cluster_sums<R>(a, cl, blk, bsum, [&](int r, u128 tot) {
        complete_resource<R>(a, cl, r, tot, s_ok, s_newlam);
    });
    if (!last) return false;
    if (threadIdx.x == 0) *s_stop = complete_cluster<R>(a, cl, s_ok);
    __syncthreads();
    return true;
}

// ---------------------------------------------------------------------------
// Persistent launches: one launch runs n_iters iterations
// ---------------------------------------------------------------------------

// Per-iteration view of the arguments of a persistent launch.
template <int R>
__device__ __forceinline__ KArgs iteration_args(const KArgs &a, int it) {
    KArgs ai = a;
    const size_t i = static_cast<size_t>(it);
    ai.eta = a.eta + i * a.B;
    if (a.tr_lam) ai.tr_lam = a.tr_lam + i * a.B * R;
    if (a.tr_U) ai.tr_U = a.tr_U + i * a.B * R;
    if (a.choice) ai.choice = a.choice + i * a.B * a.N;
    ai.iter_no = a.iter_no + it;
    ai.reverse = a.reverse ^ (a.sweep_alt & it & 1);
    return ai;
}

// After iteration `it` of a persistent launch: thread 0 of the last
// workgroup has published the new prices (atomic exchanges) and reset the
// ticket; it now bumps the cluster's epoch.  Every workgroup then waits for
// the epoch (bounded: a timeout records an error and ends the launch) and
// reads the new prices and the stop flag with agent-scope atomic loads.
// Returns false when the workgroup must leave the iteration loop.
template <int R>
__device__ bool persist_barrier(const KArgs &a, int cl, int it, bool was_last, double *s_lam, int *s_go,
                                const double *s_newlam, const int *s_stop) {
    const int t = threadIdx.x;
    if (a.nblk == 1) {
        // The only workgroup of the cluster computed the prices itself.
        __syncthreads();
        if (*s_stop) return false;
        if (t < R) s_lam[t] = s_newlam[t];
        __syncthreads();
        return true;
    }
    const uint32_t target = a.epoch_base + static_cast<uint32_t>(it) + 1u;
    if (t == 0) {
        if (was_last) {
            asm volatile("s_waitcnt vmcnt(0)" : : : "memory");   // flag updates complete
            __hip_atomic_fetch_add(&a.epoch[cl], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        int go = 1;
        // Bounded wait: about 2 s of the 100 MHz real-time counter, or until
        // another workgroup has recorded an error.
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        while (__hip_atomic_load(&a.epoch[cl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
            __builtin_amdgcn_s_sleep(2);
            if (__hip_atomic_load(a.status, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
                __builtin_amdgcn_s_memrealtime() - t0 > 200000000ull) {
                atomicCAS(a.status, 0, kStatusTimeout);
                go = 0;
                break;
            }
        }
        if (go && a.flags &&
            (__hip_atomic_load(&a.flags[cl], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) & (kFlagStopped | kFlagError)))
            go = 0;
        *s_go = go;
    }
    __syncthreads();
    if (!*s_go) return false;
    if (t < R)
        s_lam[t] = __hip_atomic_load(const_cast<double *>(&a.lam_in[cl * R + t]), __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    return true;
}

// ---------------------------------------------------------------------------
// Dense families: K = 4 * LPJ configurations per job, LPJ lanes per job
// ---------------------------------------------------------------------------

template <int R, int LPJ, typename A>
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
    if (a.flags && (a.flags[cl] & a.skip_mask)) return;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (threadIdx.x == 0) s_stop = 0;

    double lam[R];
#pragma unroll
    for (int r = 0; r < R; ++r) lam[r] = a.lam_in[cl * R + r];

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
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            double rent = static_cast<double>(d[0][i]) * lam[0];
#pragma unroll
            for (int r = 1; r < R; ++r) rent = rent + static_cast<double>(d[r][i]) * lam[r];
            double sc = static_cast<double>(u[i]) - rent;
            if (a.has_pen) sc = penalize(sc, pn[i], sw);
            if (i == 0 || sc > best) { best = sc; bi = i; }
        }
        int k = gl * 4 + bi;
        group_argmax<LPJ>(best, k);
        const int j = tl * JPT + jt;
        const bool owner = ((k >> 2) == gl) && (j < ai.N);  // this lane holds the winning entry
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
            if (!(j < ai.N) && gl == 0) {
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
    auto prefetch_two = [&](int rev) {
        if (tile0 < a.tiles) load_tile(tile0, rev, ua, da, pa);
        if (tile0 + stride < a.tiles) load_tile(tile0 + stride, rev, ub, db, pb);
    };
    prefetch_two(a.reverse);
    for (int it = 0; it < a.n_iters; ++it) {
        const KArgs ai = iteration_args<R>(a, it);
        const int rev = ai.reverse;
        for (int tile = tile0; tile < a.tiles; tile += 3 * stride) {
            const int t1 = tile + stride, t2 = tile + 2 * stride;
            if (t2 < a.tiles) load_tile(t2, rev, uc, dc, pc);
            process(ai, tile, ua, da, pa);
            if (t2 + stride < a.tiles) load_tile(t2 + stride, rev, ua, da, pa);
            if (t1 < a.tiles) process(ai, t1, ub, db, pb);
            if (t2 + 2 * stride < a.tiles) load_tile(t2 + 2 * stride, rev, ub, db, pb);
            if (t2 < a.tiles) process(ai, t2, uc, dc, pc);
        }
        if (!ai.reduce) return;

        // Workgroup sum per resource (integer adds: any order gives the same value).
        s_acc[threadIdx.x] = acc_lane ? static_cast<u128>(acc) : static_cast<u128>(0);
        acc = 0;
        __syncthreads();
        if (threadIdx.x < kBlockWaves * R) {
            const int w = threadIdx.x / R, r = threadIdx.x % R;
            u128 v = 0;
#pragma unroll 1
            for (int q = 0; q < Q; ++q) v += s_acc[w * kWaveSize + q * R + r];
            s_wsum[w][r] = v;
        }
        __syncthreads();
        if (threadIdx.x < R) {
            u128 v = 0;
#pragma unroll 1
            for (int w = 0; w < kBlockWaves; ++w) v += s_wsum[w][threadIdx.x];
            s_bsum[threadIdx.x] = v;
        }
        __syncthreads();
        const bool was_last = finish_cluster<R>(ai, cl, blk, s_bsum, s_newlam, &s_stop);
        if (it + 1 == a.n_iters) break;
        prefetch_two(rev ^ a.sweep_alt);
        if (!persist_barrier<R>(a, cl, it, was_last, s_lam, &s_go, s_newlam, &s_stop)) break;
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

// One step of an inclusive segmented scan over lanes of (best score, slot,
// segment-start flag): a lane without a segment start combines the value
// arriving from lower lanes (lanes with no source receive the identity
// (-inf, INT_MAX, 0)).  Lower slots come from lower lanes, so equal scores
// keep the lower slot, as the sequential scan does.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ void seg_scan_step(double &s, int &k, int &f) {
    const double os = dpp_or_d<CTRL, ROW_MASK>(-__builtin_inf(), s);
    const int ok = dpp_or_i<CTRL, ROW_MASK>(0x7fffffff, k);
    const int of = dpp_or_i<CTRL, ROW_MASK>(0, f);
    if (!f) {
        take_better(s, k, os, ok);
        f = of;
    }
}

template <int R, typename A>
__global__ __launch_bounds__(kBlockThreads) void k_csr(KArgs a) {
    constexpr int Q = kWaveSize / R;           // accumulating lanes per resource
    __shared__ uint32_t s_win[kBlockWaves][8];
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
    if (a.flags && (a.flags[cl] & a.skip_mask)) return;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (threadIdx.x == 0) s_stop = 0;

    double lam[R];
#pragma unroll
    for (int r = 0; r < R; ++r) lam[r] = a.lam_in[cl * R + r];
    const int my_r = lane % R;
    const int my_q = lane / R;
    const bool acc_lane = lane < Q * R;
    const int my_shift = a.shift[cl * R + my_r];
    A acc = 0;

    const float *col = a.table + cl * a.cluster_stride;
    const size_t lane_off = static_cast<size_t>(lane) * 4;
    const int hshift = (lane & 7) * 4;                   // this lane's 4 head bits in its word
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
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            double rent = static_cast<double>(d[0][i]) * lam[0];
#pragma unroll
            for (int r = 1; r < R; ++r) rent = rent + static_cast<double>(d[r][i]) * lam[r];
            sc[i] = static_cast<double>(u[i]) - rent;
            if (a.has_pen) sc[i] = penalize(sc[i], pn[i], sw);
        }
        // Lane-local pass: the part before this lane's first head (it belongs to
        // a segment from lower lanes), segments complete inside the lane, and
        // the segment left open at the lane's end.
        double pre_s = -__builtin_inf(), cur_s = -__builtin_inf();
        int pre_k = 0x7fffffff, cur_k = 0x7fffffff;
        bool has_pre = false, open = false;
        uint32_t local_win = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int slot = lane * 4 + i;
            if ((hbits >> i) & 1u) {
                if (open) local_win |= 1u << (cur_k - lane * 4);
                open = true;
                cur_s = sc[i];
                cur_k = slot;
            } else if (open) {
                if (sc[i] > cur_s) { cur_s = sc[i]; cur_k = slot; }
            } else {
                if (!has_pre || sc[i] > pre_s) { pre_s = sc[i]; pre_k = slot; }
                has_pre = true;
            }
        }
        const bool has_head = hbits != 0;
        double ps = has_head ? cur_s : pre_s;
        int pk = has_head ? cur_k : pre_k;
        int pf = has_head ? 1 : 0;
        seg_scan_step<kDppRowShr1, 0xf>(ps, pk, pf);
        seg_scan_step<kDppRowShr2, 0xf>(ps, pk, pf);
        seg_scan_step<kDppRowShr4, 0xf>(ps, pk, pf);
        seg_scan_step<kDppRowShr8, 0xf>(ps, pk, pf);
        seg_scan_step<kDppRowBcast15, 0xa>(ps, pk, pf);
        seg_scan_step<kDppRowBcast31, 0xc>(ps, pk, pf);
        // Value of the scan at the previous lane (the segment that ends inside this lane).
        double qs = dpp_or_d<kDppWaveShr1, 0xf>(-__builtin_inf(), ps);
        int qk = dpp_or_i<kDppWaveShr1, 0xf>(0x7fffffff, pk);

        // Winner mask of the tile (one bit per slot), built in LDS.
        if (lane < 8) s_win[wave][lane] = 0u;
        wave_sync();
        if (local_win) atomicOr(&s_win[wave][lane >> 3], local_win << hshift);
        if (has_head && lane > 0) {
            if (has_pre) take_better(qs, qk, pre_s, pre_k);
            atomicOr(&s_win[wave][qk >> 5], 1u << (qk & 31));
        }
        if (lane == kWaveSize - 1) atomicOr(&s_win[wave][pk >> 5], 1u << (pk & 31));
        wave_sync();
        uint32_t wm[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) wm[q] = s_win[wave][q];
        wave_sync();
        const uint32_t wbits = (wm[lane >> 3] >> hshift) & 0xFu;
        // Rank of this lane's first winner among the tile's winners (slot order).
        int rank = __popc(wm[lane >> 3] & ((1u << hshift) - 1u));
        int n_win = 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            n_win += __popc(wm[q]);
            if (q < (lane >> 3)) rank += __popc(wm[q]);
        }
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
    // current one is scored (the loop body is large; unrolling it costs more
    // than the deeper prefetch gains).
    f4 nu, npn = {};
    f4 nd[R];
    uint32_t nhw = 0;
    const int tile0 = blk * kBlockWaves + wave;
    if (tile0 < a.tiles) load_tile(tile0, a.reverse, nu, nd, npn, nhw);
    for (int it = 0; it < a.n_iters; ++it) {
        const KArgs ai = iteration_args<R>(a, it);
        const int rev = ai.reverse;
        for (int tile = tile0; tile < a.tiles; tile += stride) {
            const f4 u = nu, pn = npn;
            f4 d[R];
#pragma unroll
            for (int r = 0; r < R; ++r) d[r] = nd[r];
            const uint32_t hw = nhw;
            if (tile + stride < a.tiles) load_tile(tile + stride, rev, nu, nd, npn, nhw);
            process(ai, tile, u, d, pn, hw);
        }
        if (!ai.reduce) return;

        s_acc[threadIdx.x] = acc_lane ? static_cast<u128>(acc) : static_cast<u128>(0);
        acc = 0;
        __syncthreads();
        if (threadIdx.x < kBlockWaves * R) {
            const int w = threadIdx.x / R, r = threadIdx.x % R;
            u128 v = 0;
#pragma unroll 1
            for (int q = 0; q < Q; ++q) v += s_acc[w * kWaveSize + q * R + r];
            s_wsum[w][r] = v;
        }
        __syncthreads();
        if (threadIdx.x < R) {
            u128 v = 0;
#pragma unroll 1
            for (int w = 0; w < kBlockWaves; ++w) v += s_wsum[w][threadIdx.x];
            s_bsum[threadIdx.x] = v;
        }
        __syncthreads();
        const bool was_last = finish_cluster<R>(ai, cl, blk, s_bsum, s_newlam, &s_stop);
        if (it + 1 == a.n_iters) break;
        if (tile0 < a.tiles) load_tile(tile0, rev ^ a.sweep_alt, nu, nd, npn, nhw);
        if (!persist_barrier<R>(a, cl, it, was_last, s_lam, &s_go, s_newlam, &s_stop)) break;
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
    finish_cluster<R>(a, cl, blk, s_bsum, s_newlam, &s_stop);
}

// ---------------------------------------------------------------------------
// Effective capacity (Sec. 3.4, Eq. 12)
// ---------------------------------------------------------------------------

// C_eff_r = C_r - gamma * S_r, S_r = sum over pending jobs j of
// min over j's allowed configurations of d_jkr (the componentwise smallest
// footprint), over the pending jobs' own packed table.  A wavefront takes one
// tile at a time: each lane folds its 4 entries into one minimum per job
// piece (entries of one job are adjacent) and merges it into the tile's
// per-job minima in LDS with an unsigned atomic minimum (demands are
// non-negative floats with +0.0 for zero, whose bit patterns order like the
// values); the lanes then add the minima of pending jobs to exact fixed-point
// accumulators.  Masked configurations and padding carry a utility of -inf
// (dense padding: job index >= N) and are skipped.
template <int R, typename A>
__global__ __launch_bounds__(kBlockThreads) void k_reserve(KArgs a, ReserveArgs ra) {
    constexpr uint32_t kInf = 0x7f800000u;
    __shared__ uint32_t s_min[kBlockWaves][kTileEntries][R];
    __shared__ u128 s_part[kBlockWaves][R];
    __shared__ u128 s_bsum[R];
    const int cl = blockIdx.x / a.nblk;
    const int blk = blockIdx.x - cl * a.nblk;
    const int lane = threadIdx.x & (kWaveSize - 1);
    const int wave = threadIdx.x / kWaveSize;
    const float *col = a.table + cl * a.cluster_stride;
    const uint8_t *pend = ra.queued ? ra.queued + static_cast<size_t>(cl) * a.N : nullptr;
    int sh[R];
    A acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        sh[r] = a.shift[cl * R + r];
        acc[r] = 0;
    }
    uint32_t *mins = &s_min[wave][0][0];
    for (int i = lane; i < kTileEntries * R; i += kWaveSize) mins[i] = kInf;
    wave_sync();
    const int jpt = a.K > 0 ? kTileEntries / a.K : 0;          // dense: jobs per tile
    for (int tile = blk * kBlockWaves + wave; tile < a.tiles; tile += a.nblk * kBlockWaves) {
        const size_t base = static_cast<size_t>(tile) * kTileEntries + static_cast<size_t>(lane) * 4;
        const f4 u = *reinterpret_cast<const f4 *>(col + base);
        f4 d[R];
#pragma unroll
        for (int r = 0; r < R; ++r) d[r] = *reinterpret_cast<const f4 *>(col + (r + 1) * a.col_len + base);
        int first_job, njobs, jt;
        uint32_t heads;                        // bit i: entry 4*lane + i starts a job
        if (a.K > 0) {
            first_job = tile * jpt;
            njobs = min(jpt, a.N - first_job);
            jt = (lane * 4) / a.K;
            heads = 0;                         // K >= 4: a lane's 4 entries share one job
        } else {
            const TileMeta &m = a.meta[tile];
            const int e0 = lane * 4, w = e0 >> 5, bit = e0 & 31;
            int before = 0, total = 0;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int c = __popc(m.head[q]);
                total += c;
                before += (q < w) ? c : 0;
            }
            const uint32_t word = m.head[w];
            const uint32_t upto = (bit == 31) ? 0xffffffffu : ((2u << bit) - 1u);
            first_job = static_cast<int>(m.first_job);
            njobs = total;
            jt = before + __popc(word & upto) - 1; // entry 0 of a tile always starts a job
            heads = (word >> bit) & 0xfu;
        }
        uint32_t mn[R];
#pragma unroll
        for (int r = 0; r < R; ++r) mn[r] = kInf;
        auto flush = [&]() {
#pragma unroll
            for (int r = 0; r < R; ++r)
                if (mn[r] != kInf) atomicMin(&s_min[wave][jt][r], mn[r]);
        };
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if (i > 0 && ((heads >> i) & 1u)) {
                flush();
                ++jt;
#pragma unroll
                for (int r = 0; r < R; ++r) mn[r] = kInf;
            }
            const bool valid = (u[i] != -__builtin_inff()) && (jt < njobs);
            if (valid) {
#pragma unroll
                for (int r = 0; r < R; ++r) mn[r] = min(mn[r], __float_as_uint(d[r][i]));
            }
        }
        flush();
        wave_sync();
        for (int q = lane; q < njobs; q += kWaveSize) {
            const bool take = !pend || pend[first_job + q] != 0;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const uint32_t m = s_min[wave][q][r];
                s_min[wave][q][r] = kInf;
                if (take && m != kInf) acc[r] += fx_of<A>(__uint_as_float(m), sh[r]);
            }
        }
        wave_sync();
    }
    // workgroup sums: wavefront tree over lanes, then the 4 wavefronts in order
#pragma unroll
    for (int r = 0; r < R; ++r) {
        u128 v = static_cast<u128>(acc[r]);
#pragma unroll
        for (int off = kWaveSize / 2; off > 0; off >>= 1) {
            const unsigned long long lo = __shfl_down(static_cast<unsigned long long>(v), off);
            const unsigned long long hi = __shfl_down(static_cast<unsigned long long>(v >> 64), off);
            v += (static_cast<u128>(hi) << 64) | lo;
        }
        if (lane == 0) s_part[wave][r] = v;
    }
    __syncthreads();
    if (threadIdx.x < R) {
        u128 t = 0;
        for (int w = 0; w < kBlockWaves; ++w) t += s_part[w][threadIdx.x];
        s_bsum[threadIdx.x] = t;
    }
    __syncthreads();
    cluster_sums<R>(a, cl, blk, s_bsum, [&](int r, u128 tot) {
        const double S = fx_to_double(tot, a.shift[cl * R + r]);
        const double g = ra.gamma * S;
        const double ce = ra.cap_phys[cl * R + r] - g;
        ra.cap_eff[cl * R + r] = ce;
        if (ra.out) ra.out[cl * R + r] = ce;
    });
}

// ---------------------------------------------------------------------------
// Nearest-profile fallback of RST (Sec. 3.1.2, Sec. 4.1)
// ---------------------------------------------------------------------------

constexpr int kNearestLanes = 16;                     // lanes per query (one DPP row)

// Query i of a cluster names a job type f and an unprofiled configuration's
// resource vector q.  The 16 lanes of one DPP row serve one query: lane s
// takes entries s, s+16, ... of family f, skips masked ones (utility -inf),
// and keeps the smallest squared l2 distance, computed in binary64 in a fixed
// order (e_0 = q_0 - d_0, acc = e_0 e_0, acc = acc + e_r e_r for r = 1..R-1).
// The row then takes the argmax of the negated distance with lowest-index
// ties (group_argmax), i.e. the nearest entry with the lowest index among
// equals; lane 0 writes its index and its throughput (the utility column).
// A family index out of range or a non-finite query component gives -1 /
// NaN and records an error.
template <int R>
__global__ __launch_bounds__(kBlockThreads) void k_nearest(KArgs a, NearestArgs na) {
    constexpr int kPerBlock = kBlockThreads / kNearestLanes;
    const int sub = threadIdx.x & (kNearestLanes - 1);
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kPerBlock;
    // every lane of a row shares gi, so rows stay whole for the DPP steps
    for (int64_t gi = static_cast<int64_t>(blockIdx.x) * kPerBlock + threadIdx.x / kNearestLanes; gi < na.total;
         gi += stride) {
        const int cl = static_cast<int>(gi / na.Q);
        const float *col = a.table + cl * a.cluster_stride;
        const int f = na.family[gi];
        double q[R];
        bool ok = f >= 0 && f < a.N;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const float v = na.query[gi * R + r];
            ok = ok && (fabsf(v) <= 3.402823466e38f);     // false for NaN and +-inf
            q[r] = static_cast<double>(v);
        }
        double best = -__builtin_inf();
        int bk = 0x7fffffff;
        uint32_t slot = 0;
        if (ok) {
            uint32_t size;
            if (a.K > 0) {
                slot = static_cast<uint32_t>(f) * static_cast<uint32_t>(a.K);
                size = static_cast<uint32_t>(a.K);
            } else {
                slot = a.jobs[f].slot;
                size = a.jobs[f].size;
            }
            for (uint32_t k = sub; k < size; k += kNearestLanes) {
                const size_t e = static_cast<size_t>(slot) + k;
                if (col[e] == -__builtin_inff()) continue;     // masked configuration
                double x = q[0] - static_cast<double>(col[a.col_len + e]);
                double acc = x * x;
#pragma unroll
                for (int r = 1; r < R; ++r) {
                    x = q[r] - static_cast<double>(col[(r + 1) * a.col_len + e]);
                    acc = acc + x * x;
                }
                take_better(best, bk, -acc, static_cast<int>(k));
            }
        }
        group_argmax<kNearestLanes>(best, bk);
        if (sub == 0) {
            const bool found = ok && bk != 0x7fffffff;
            na.nearest[gi] = found ? bk : -1;
            if (na.estimate)
                na.estimate[gi] = found ? col[static_cast<size_t>(slot) + static_cast<uint32_t>(bk)] : __builtin_nanf("");
            if (!ok) atomicCAS(a.status, 0, (f >= 0 && f < a.N) ? kStatusNonfinite : kStatusInvalid);
        }
    }
}

// ---------------------------------------------------------------------------
// Outer ESP-IAC rounds (Sec. 3.4, Alg. 1; thresholds of Eq. 11)
// ---------------------------------------------------------------------------

// One wavefront per cluster, after the round's tatonnement and re-selection:
//  BinPack  jobs in index order; job j at its chosen configuration needs
//           g = d[r_gpus] GPUs (a whole number in 1..8, else not placeable)
//           and d[r_mem] / g memory and d[r_sm] / g compute on each; it takes
//           the g lowest-index GPUs with room for one share (all or
//           nothing).  Jobs are gathered 64 at a time (one per lane) and
//           placed in order; each lane tests 4 consecutive GPUs, so one step
//           covers 256, only in blocks whose summary (largest residuals,
//           fewest jobs) admits the share, and ballots rank the fitting
//           GPUs.  Residuals live in LDS, updated in job order (binary64,
//           the oracle's operations).
//  IAC      every pair of jobs sharing a GPU: S_x|y = 1 + a_x b_y against
//           tau_x = tau_base_x + min(beta (U / U_target - 1), beta_max),
//           U = busy GPUs / G; a pair violates when either slowdown exceeds
//           its threshold.  Each job keeps its largest excess (atomic max on
//           the bit patterns of non-negative doubles).
//  Gamma    each violating job's chosen configuration: penalty <-
//           fp32(penalty + kappa * excess), in the packed penalty column
//           (its sign bit, the switching-cost mark, is kept).
// A cluster without violations is frozen: later rounds' kernels skip it.
// Wave-uniform copies of lane t's value (t uniform).
__device__ __forceinline__ int lane_i(int v, int t) { return __builtin_amdgcn_readlane(v, t); }
__device__ __forceinline__ double lane_d(double v, int t) {
    const long long b = __double_as_longlong(v);
    const unsigned lo = static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(static_cast<unsigned>(b)), t));
    const unsigned hi = static_cast<unsigned>(__builtin_amdgcn_readlane(static_cast<int>(b >> 32), t));
    return __longlong_as_double(static_cast<long long>((static_cast<unsigned long long>(hi) << 32) | lo));
}

// Maximum of x and minimum of c over the 64 lanes (all active): DPP inside
// each 16-lane row, then the four row results.
__device__ __forceinline__ void wave_max2_min(double &x, double &y, int &c) {
    x = fmax(x, dpp_d<kDppXor1>(x));
    y = fmax(y, dpp_d<kDppXor1>(y));
    c = min(c, dpp_i<kDppXor1>(c));
    x = fmax(x, dpp_d<kDppXor2>(x));
    y = fmax(y, dpp_d<kDppXor2>(y));
    c = min(c, dpp_i<kDppXor2>(c));
    x = fmax(x, dpp_d<kDppHalfMirror>(x));
    y = fmax(y, dpp_d<kDppHalfMirror>(y));
    c = min(c, dpp_i<kDppHalfMirror>(c));
    x = fmax(x, dpp_d<kDppMirror>(x));
    y = fmax(y, dpp_d<kDppMirror>(y));
    c = min(c, dpp_i<kDppMirror>(c));
    x = fmax(fmax(lane_d(x, 0), lane_d(x, 16)), fmax(lane_d(x, 32), lane_d(x, 48)));
    y = fmax(fmax(lane_d(y, 0), lane_d(y, 16)), fmax(lane_d(y, 32), lane_d(y, 48)));
    c = min(min(lane_i(c, 0), lane_i(c, 16)), min(lane_i(c, 32), lane_i(c, 48)));
}

template <int R>
__global__ __launch_bounds__(kWaveSize) void k_pack_iac(KArgs a, IacArgs m) {
    constexpr int kPerLane = 4;                          // GPUs per lane in one scan step
    constexpr int kStep = kWaveSize * kPerLane;          // GPUs per scan step
    constexpr int kBlocks = kMaxGpus / kStep;
    __shared__ double s_mem[kMaxGpus];
    __shared__ double s_sm[kMaxGpus];
    __shared__ int s_cnt[kMaxGpus];
    __shared__ int s_occ[kMaxGpus][kMaxPerGpu];
    __shared__ int s_sel[kMaxShards];
    static_assert(kBlocks <= kWaveSize, "one lane per block summary");
    const int cl = blockIdx.x;
    const int lane = threadIdx.x;
    if (a.flags[cl] & kFlagFrozen) return;
    const int G = m.gpus[cl];
    const int nblk = (G + kStep - 1) / kStep;
    const int N = a.N;
    float *col = const_cast<float *>(a.table) + cl * a.cluster_stride;
    const int32_t *ch = m.choice + static_cast<size_t>(cl) * N;
    // GPUs beyond G get no room at all (count kMaxPerGpu), so they never fit
    for (int h = lane; h < nblk * kStep; h += kWaveSize) {
        s_mem[h] = m.gpu_memory;
        s_sm[h] = m.gpu_compute;
        s_cnt[h] = h < G ? 0 : kMaxPerGpu;
#pragma unroll
        for (int i = 0; i < kMaxPerGpu; ++i) s_occ[h][i] = -1;
    }
    // Lane c < nblk keeps block c's summary in registers: largest residual
    // memory and compute over its GPUs that can still take a job, fewest
    // jobs.  A block failing any of the three cannot hold the share, so
    // skipping it is exact.
    double sum_m = m.gpu_memory, sum_s = m.gpu_compute;
    int sum_c = lane < nblk ? 0 : kMaxPerGpu;
    wave_sync();
    const uint64_t below = (1ull << lane) - 1ull;
    // Jobs 64 at a time: each lane gathers one job's share (GPU count,
    // memory and compute per GPU), then the wavefront places them in order.
    for (int j0 = 0; j0 < N; j0 += kWaveSize) {
        int g_l = 0;
        double nm_l = 0.0, ns_l = 0.0;
        const int jl = j0 + lane;
        if (jl < N) {
            const int k = ch[jl];
            if (k >= 0) {
                const size_t e =
                    (a.K > 0 ? static_cast<size_t>(jl) * a.K : static_cast<size_t>(a.jobs[jl].slot)) + k;
                const double gv = static_cast<double>(col[(m.r_gpus + 1) * a.col_len + e]);
                if (gv >= 1.0 && gv <= static_cast<double>(kMaxShards) && gv == floor(gv)) {
                    g_l = static_cast<int>(gv);
                    nm_l = static_cast<double>(col[(m.r_mem + 1) * a.col_len + e]) / gv;
                    ns_l = static_cast<double>(col[(m.r_sm + 1) * a.col_len + e]) / gv;
                }
            }
        }
        const int cnt = min(kWaveSize, N - j0);
        for (int t = 0; t < cnt; ++t) {
            const int g = lane_i(g_l, t);
            if (g == 0) continue;                          // not placeable
            const double nm = lane_d(nm_l, t);
            const double ns = lane_d(ns_l, t);
            uint64_t cand = __ballot((sum_c < kMaxPerGpu) & (sum_m >= nm) & (sum_s >= ns));
            int found = 0;
            while (cand != 0ull && found < g) {
                const int c = __builtin_ctzll(cand);
                cand &= cand - 1ull;
                // lane l tests GPUs c*256 + 4l .. 4l+3 (ascending with the lane)
                const int h0 = c * kStep + lane * kPerLane;
                bool fit[kPerLane];
                uint64_t bal[kPerLane];
                int before = 0, total = 0;
                int cv[kPerLane];
                double mv[kPerLane], sv[kPerLane];
#pragma unroll
                for (int i = 0; i < kPerLane; ++i) {
                    cv[i] = s_cnt[h0 + i];
                    mv[i] = s_mem[h0 + i];
                    sv[i] = s_sm[h0 + i];
                }
#pragma unroll
                for (int i = 0; i < kPerLane; ++i) {
                    fit[i] = (cv[i] < kMaxPerGpu) & (mv[i] >= nm) & (sv[i] >= ns);
                    bal[i] = __ballot(fit[i]);
                    before += __popcll(bal[i] & below);
                    total += __popcll(bal[i]);
                }
                int rank = found + before;
#pragma unroll
                for (int i = 0; i < kPerLane; ++i) {
                    if (fit[i]) {
                        if (rank < g) s_sel[rank] = h0 + i;
                        ++rank;
                    }
                }
                found += total;
            }
            wave_sync();
            if (found < g) continue;                       // all or nothing
            if (lane < g) {
                const int h = s_sel[lane];
                const double mh = s_mem[h], sh_ = s_sm[h];
                const int ch_ = s_cnt[h];
                s_mem[h] = mh - nm;
                s_sm[h] = sh_ - ns;
                s_occ[h][ch_] = j0 + t;
                s_cnt[h] = ch_ + 1;
            }
            wave_sync();
            // refresh the summaries of the blocks that changed
            int last = -1;
            for (int i = 0; i < g; ++i) {
                const int c = s_sel[i] / kStep;
                if (c == last) continue;
                last = c;
                const int h0 = c * kStep + lane * kPerLane;
                double xm = -__builtin_inf(), xs = -__builtin_inf();
                int xc = kMaxPerGpu;
#pragma unroll
                for (int q = 0; q < kPerLane; ++q) {
                    const int cq = s_cnt[h0 + q];
                    const double mq = s_mem[h0 + q], sq = s_sm[h0 + q];
                    const bool open = cq < kMaxPerGpu;           // GPUs that can still take a job
                    xm = open ? fmax(xm, mq) : xm;
                    xs = open ? fmax(xs, sq) : xs;
                    xc = min(xc, cq);
                }
                wave_max2_min(xm, xs, xc);
                if (lane == c) {
                    sum_m = xm;
                    sum_s = xs;
                    sum_c = xc;
                }
            }
        }
    }
    // thresholds of Eq. 11
    int used = 0;
    for (int h = lane; h < G; h += kWaveSize) used += s_cnt[h] > 0;
#pragma unroll
    for (int off = kWaveSize / 2; off > 0; off >>= 1) used += __shfl_xor(used, off);
    double q = static_cast<double>(used) / static_cast<double>(G);
    q = q / m.u_target;
    const double w = q - 1.0;
    double add = m.beta * w;
    if (add > m.beta_max) add = m.beta_max;
    const float *sa = m.sensitivity + static_cast<size_t>(cl) * m.nnz;
    const float *pb = m.pressure + static_cast<size_t>(cl) * m.nnz;
    const double *tb = m.tau_base + static_cast<size_t>(cl) * N;
    unsigned long long *inc = reinterpret_cast<unsigned long long *>(m.inc) + static_cast<size_t>(cl) * N;
    int V = 0;
    for (int h = lane; h < G; h += kWaveSize) {
        const int n = s_cnt[h];
        for (int x = 0; x < n; ++x)
            for (int y = x + 1; y < n; ++y) {
                const int jx = s_occ[h][x], jy = s_occ[h][y];
                const int64_t ex = m.offsets[jx] + ch[jx], ey = m.offsets[jy] + ch[jy];
                double sxy = static_cast<double>(sa[ex]) * static_cast<double>(pb[ey]);
                sxy = 1.0 + sxy;
                double syx = static_cast<double>(sa[ey]) * static_cast<double>(pb[ex]);
                syx = 1.0 + syx;
                const double ox = sxy - (tb[jx] + add);
                const double oy = syx - (tb[jy] + add);
                if (ox > 0.0) atomicMax(&inc[jx], static_cast<unsigned long long>(__double_as_longlong(ox)));
                if (oy > 0.0) atomicMax(&inc[jy], static_cast<unsigned long long>(__double_as_longlong(oy)));
                V += (ox > 0.0 || oy > 0.0) ? 1 : 0;
            }
    }
#pragma unroll
    for (int off = kWaveSize / 2; off > 0; off >>= 1) V += __shfl_xor(V, off);
    __threadfence();                                   // the maxima are complete before they are read
    float *pcol = col + static_cast<size_t>(R + 1) * a.col_len;
    for (int j = lane; j < N; j += kWaveSize) {
        const unsigned long long bits = __hip_atomic_load(&inc[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (bits == 0ull) continue;
        __hip_atomic_store(&inc[j], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const double x = __longlong_as_double(static_cast<long long>(bits));
        const size_t e = (a.K > 0 ? static_cast<size_t>(j) * a.K : static_cast<size_t>(a.jobs[j].slot)) + ch[j];
        const uint32_t old = __float_as_uint(pcol[e]);
        const float mag = __uint_as_float(old & 0x7fffffffu);
        const float nv = __double2float_rn(static_cast<double>(mag) + m.kappa * x);
        pcol[e] = __uint_as_float(__float_as_uint(nv) | (old & 0x80000000u));
    }
    int32_t *gj = m.gpu_jobs + static_cast<size_t>(cl) * m.gmax * kMaxPerGpu;
    for (int h = lane; h < m.gmax; h += kWaveSize)
#pragma unroll
        for (int i = 0; i < kMaxPerGpu; ++i) gj[h * kMaxPerGpu + i] = h < G ? s_occ[h][i] : -1;
    if (lane == 0) {
        m.violations[cl] = V;
        m.rounds_used[cl] = m.round;
        if (V == 0) a.flags[cl] = a.flags[cl] | kFlagFrozen;
    }
}

// Gamma <- 0 over the packed penalty columns (sign bits kept) and/or clear
// the frozen flags.
__global__ void k_iac_reset(float *table, size_t cluster_stride, size_t col_len, int R, int B, int32_t *flags,
                            int zero_gamma) {
    const size_t tid = static_cast<size_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    const size_t stride = static_cast<size_t>(gridDim.x) * blockDim.x;
    if (zero_gamma) {
        const size_t total = static_cast<size_t>(B) * col_len;
        for (size_t i = tid; i < total; i += stride) {
            const size_t b = i / col_len, e = i - b * col_len;
            float *p = table + b * cluster_stride + static_cast<size_t>(R + 1) * col_len + e;
            *p = __uint_as_float(__float_as_uint(*p) & 0x80000000u);
        }
    }
    for (size_t b = tid; b < static_cast<size_t>(B); b += stride) flags[b] = flags[b] & ~kFlagFrozen;
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
        const double x = lo + a.eta[cl] * g;
        a.lam_out[cl * R + r] = (x > 0.0) ? x : 0.0;
    }
}

// Validate prices before a solve or a selection; mark bad clusters.
template <int R>
__global__ void k_prepare(const double *lam, int32_t *flags, int32_t *iters_done, uint32_t *epoch, int32_t *status,
                          int B) {
    const int cl = blockIdx.x * blockDim.x + threadIdx.x;
    if (cl >= B) return;
    bool ok = true;
    for (int r = 0; r < R; ++r) ok = ok && price_ok(lam[cl * R + r]);
    flags[cl] = (flags[cl] & kFlagFrozen) | (ok ? 0 : kFlagError);
    if (iters_done) iters_done[cl] = 0;
    if (epoch) epoch[cl] = 0u;
    if (!ok) atomicCAS(status, 0, kStatusNonfinite);
}

// ---------------------------------------------------------------------------
// Launchers (runtime R / LPJ -> template instance)
// ---------------------------------------------------------------------------

template <int R, typename A>
static hipError_t launch_dense_ra(int lpj, const KArgs &a, int B, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(B) * a.nblk), block(kBlockThreads);
    switch (lpj) {
        case 1: hipLaunchKernelGGL((k_dense<R, 1, A>), grid, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL((k_dense<R, 2, A>), grid, block, 0, s, a); break;
        case 4: hipLaunchKernelGGL((k_dense<R, 4, A>), grid, block, 0, s, a); break;
        case 8: hipLaunchKernelGGL((k_dense<R, 8, A>), grid, block, 0, s, a); break;
        case 16: hipLaunchKernelGGL((k_dense<R, 16, A>), grid, block, 0, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int R>
static hipError_t launch_dense_r(int lpj, const KArgs &a, int B, hipStream_t s) {
    return a.acc128 ? launch_dense_ra<R, u128>(lpj, a, B, s) : launch_dense_ra<R, uint64_t>(lpj, a, B, s);
}

template <int R, typename A>
static hipError_t launch_dense_coop_ra(int lpj, const KArgs &a, int B, hipStream_t s) {
    const void *f = nullptr;
    switch (lpj) {
        case 1: f = reinterpret_cast<const void *>(&k_dense<R, 1, A>); break;
        case 2: f = reinterpret_cast<const void *>(&k_dense<R, 2, A>); break;
        case 4: f = reinterpret_cast<const void *>(&k_dense<R, 4, A>); break;
        case 8: f = reinterpret_cast<const void *>(&k_dense<R, 8, A>); break;
        case 16: f = reinterpret_cast<const void *>(&k_dense<R, 16, A>); break;
        default: return hipErrorInvalidValue;
    }
    KArgs copy = a;
    void *args[] = {&copy};
    return hipLaunchCooperativeKernel(f, dim3(static_cast<unsigned>(B) * a.nblk), dim3(kBlockThreads), args, 0, s);
}

template <int R>
static hipError_t launch_dense_coop_r(int lpj, const KArgs &a, int B, hipStream_t s) {
    return a.acc128 ? launch_dense_coop_ra<R, u128>(lpj, a, B, s) : launch_dense_coop_ra<R, uint64_t>(lpj, a, B, s);
}

#define ESP_DISPATCH_R(R, CALL)              \
    switch (R) {                             \
        case 1: return CALL(1);              \
        case 2: return CALL(2);              \
        case 3: return CALL(3);              \
        case 4: return CALL(4);              \
        case 5: return CALL(5);              \
        case 6: return CALL(6);              \
        case 7: return CALL(7);              \
        case 8: return CALL(8);              \
        default: return hipErrorInvalidValue; \
    }

hipError_t launch_dense(int R, int lpj, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_dense_r<RR>(lpj, a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_dense_persistent(int R, int lpj, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_dense_coop_r<RR>(lpj, a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

template <int R>
static hipError_t launch_gather_r(const KArgs &a, int B, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(B) * a.nblk), block(kBlockThreads);
    if (a.acc128)
        hipLaunchKernelGGL((k_gather<R, u128>), grid, block, 0, s, a);
    else
        hipLaunchKernelGGL((k_gather<R, uint64_t>), grid, block, 0, s, a);
    return hipGetLastError();
}

hipError_t launch_gather(int R, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_gather_r<RR>(a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

template <int R>
static hipError_t launch_nearest_r(const KArgs &a, const NearestArgs &na, hipStream_t s) {
    constexpr int kPerBlock = kBlockThreads / kNearestLanes;
    const int64_t need = (na.total + kPerBlock - 1) / kPerBlock;
    const int64_t cap = 256 * 32;                    // enough resident queries to cover gather latency
    const dim3 grid(static_cast<unsigned>(need < cap ? need : cap)), block(kBlockThreads);
    hipLaunchKernelGGL((k_nearest<R>), grid, block, 0, s, a, na);
    return hipGetLastError();
}

hipError_t launch_nearest(int R, const KArgs &a, const NearestArgs &na, hipStream_t s) {
#define CALL(RR) launch_nearest_r<RR>(a, na, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

template <int R>
static hipError_t launch_pack_iac_r(const KArgs &a, const IacArgs &m, int B, hipStream_t s) {
    hipLaunchKernelGGL((k_pack_iac<R>), dim3(static_cast<unsigned>(B)), dim3(kWaveSize), 0, s, a, m);
    return hipGetLastError();
}

hipError_t launch_pack_iac(int R, const KArgs &a, const IacArgs &m, int B, hipStream_t s) {
#define CALL(RR) launch_pack_iac_r<RR>(a, m, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_iac_reset(int R, const KArgs &a, int B, int zero_gamma, hipStream_t s) {
    const size_t work = zero_gamma ? static_cast<size_t>(B) * a.col_len : static_cast<size_t>(B);
    const size_t blocks = std::min<size_t>((work + 255) / 256, 4096);
    hipLaunchKernelGGL(k_iac_reset, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, s,
                       const_cast<float *>(a.table), a.cluster_stride, a.col_len, R, B, a.flags, zero_gamma);
    return hipGetLastError();
}

template <int R>
static hipError_t launch_reserve_r(const KArgs &a, const ReserveArgs &ra, int B, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(B) * a.nblk), block(kBlockThreads);
    if (a.acc128)
        hipLaunchKernelGGL((k_reserve<R, u128>), grid, block, 0, s, a, ra);
    else
        hipLaunchKernelGGL((k_reserve<R, uint64_t>), grid, block, 0, s, a, ra);
    return hipGetLastError();
}

hipError_t launch_reserve(int R, const KArgs &a, const ReserveArgs &ra, int B, hipStream_t s) {
#define CALL(RR) launch_reserve_r<RR>(a, ra, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

template <int R>
static hipError_t launch_update_r(const KArgs &a, const double *demand_in, int B, hipStream_t s) {
    hipLaunchKernelGGL((k_update<R>), dim3((B + 255) / 256), dim3(256), 0, s, a, demand_in, B);
    return hipGetLastError();
}

hipError_t launch_update(int R, const KArgs &a, const double *demand_in, int B, hipStream_t s) {
#define CALL(RR) launch_update_r<RR>(a, demand_in, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

template <int R>
static hipError_t launch_prepare_r(const double *lam, int32_t *flags, int32_t *iters_done, uint32_t *epoch,
                                   int32_t *status, int B, hipStream_t s) {
    hipLaunchKernelGGL((k_prepare<R>), dim3((B + 255) / 256), dim3(256), 0, s, lam, flags, iters_done, epoch, status,
                       B);
    return hipGetLastError();
}

hipError_t launch_prepare(int R, const double *lam, int32_t *flags, int32_t *iters_done, uint32_t *epoch,
                          int32_t *status, int B, hipStream_t s) {
#define CALL(RR) launch_prepare_r<RR>(lam, flags, iters_done, epoch, status, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

template <int R>
static hipError_t launch_csr_r(const KArgs &a, int B, hipStream_t s) {
    const dim3 grid(static_cast<unsigned>(B) * a.nblk), block(kBlockThreads);
    if (a.acc128)
        hipLaunchKernelGGL((k_csr<R, u128>), grid, block, 0, s, a);
    else
        hipLaunchKernelGGL((k_csr<R, uint64_t>), grid, block, 0, s, a);
    return hipGetLastError();
}

template <int R>
static hipError_t launch_csr_coop_r(const KArgs &a, int B, hipStream_t s) {
    const void *f = a.acc128 ? reinterpret_cast<const void *>(&k_csr<R, u128>)
                             : reinterpret_cast<const void *>(&k_csr<R, uint64_t>);
    KArgs copy = a;
    void *args[] = {&copy};
    return hipLaunchCooperativeKernel(f, dim3(static_cast<unsigned>(B) * a.nblk), dim3(kBlockThreads), args, 0, s);
}

hipError_t launch_csr_persistent(int R, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_csr_coop_r<RR>(a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

hipError_t launch_csr(int R, const KArgs &a, int B, hipStream_t s) {
#define CALL(RR) launch_csr_r<RR>(a, B, s)
    ESP_DISPATCH_R(R, CALL)
#undef CALL
}

}  // namespace esp
