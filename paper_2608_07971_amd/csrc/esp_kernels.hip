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
#include "esp_device.hpp"

#pragma clang fp contract(off)

namespace esp {

// ---------------------------------------------------------------------------
// Cluster completion: per-workgroup sums -> last workgroup -> U, Eq. 8 update
// ---------------------------------------------------------------------------

// eta_t of Eq. 8 for the launch's step index t: eta0 or eta0 / sqrt(t), one
// IEEE division and one correctly rounded square root in binary64 (no fast
// math), so the value equals the host's.
__device__ __forceinline__ double step_size(const KArgs &a, int cl) {
    const double e0 = a.eta0[cl];
    return a.rule == 1 ? e0 / sqrt(static_cast<double>(a.t)) : e0;
}

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
        const double x = lo + step_size(a, cl) * g;
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
    ai.t = a.t + it;
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
        const double x = lo + step_size(a, cl) * g;
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
