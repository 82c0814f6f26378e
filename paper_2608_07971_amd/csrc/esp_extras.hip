// gfx950 kernels beyond the price loop: the effective capacity of Eq. 12,
// the outer ESP-IAC rounds of Alg. 1 and RST's nearest-profile fallback.
#include <algorithm>

#include "esp_device.hpp"
#include "esp_extras.hpp"

#pragma clang fp contract(off)

namespace esp {

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
            const bool valid = (u[i] != -__builtin_inff()) & (jt < njobs);
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
                if (take & (m != kInf)) acc[r] += fx_of<A>(__uint_as_float(m), sh[r]);
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

// Sum over the 16 lanes of a DPP row, in every lane of the row.
__device__ __forceinline__ uint32_t row_sum(uint32_t v) {
    constexpr int kRowRor8 = 0x128, kRowRor4 = 0x124, kRowRor2 = 0x122, kRowRor1 = 0x121;
    v += static_cast<uint32_t>(dpp_i<kRowRor8>(static_cast<int>(v)));
    v += static_cast<uint32_t>(dpp_i<kRowRor4>(static_cast<int>(v)));
    v += static_cast<uint32_t>(dpp_i<kRowRor2>(static_cast<int>(v)));
    v += static_cast<uint32_t>(dpp_i<kRowRor1>(static_cast<int>(v)));
    return v;
}

// Query i of a cluster names a job type f and an unprofiled configuration's
// resource vector q.  The 16 lanes of one DPP row serve a query: lane s takes
// entries s, s+16, ... of family f, skips masked ones (utility -inf), and
// keeps the smallest squared l2 distance, computed in binary64 in a fixed
// order (e_0 = q_0 - d_0, acc = e_0 e_0, acc = acc + e_r e_r for r = 1..R-1).
// The row then takes the argmax of the negated distance with lowest-index
// ties (group_argmax), i.e. the nearest entry with the lowest index among
// equals.  Lane 0 writes the index; the lane that found the entry writes its
// throughput (the utility), which it still holds in a register.  A family
// index out of range or a non-finite query component gives -1 / NaN and
// records an error.
//
// The family is read from the store's entry-major copy (AOS: each entry's
// utility and demands contiguous, so the family is one contiguous run that
// starts on a cache line) or from the structure-of-arrays columns of the
// price loop's table.  With the copy, the row finds the run from the
// directory record of the family's group of 60: lane 0 holds the group's
// first line, lanes 1..15 hold four one-byte family sizes each, and two row
// sums give the run's first line (the group's first line plus the lines of
// the families before f) and the family's size.  The directory (64 bytes per
// 60 families) stays in L2.
//
// Each query is a chain of dependent gathers (query -> family extent ->
// entries), so a row works on three queries at once: while it reads the
// entries of query i it has the extent of query i+1 and the family index of
// query i+2 in flight, and every step waits for one memory round trip
// instead of three.
template <int R, bool AOS>
__global__ __launch_bounds__(kBlockThreads) void k_nearest(KArgs a, NearestArgs na) {
    constexpr int kPerBlock = kBlockThreads / kNearestLanes;
    constexpr uint32_t kEntryBytes = 4 * (R + 1);
    const int sub = threadIdx.x & (kNearestLanes - 1);
    // The workgroup takes queries [lo, lo + chunk), kPerBlock at a time (one
    // per row), so the cache lines of the query and output arrays it touches
    // are its own.
    constexpr int64_t stride = kPerBlock;
    const int64_t lo = static_cast<int64_t>(blockIdx.x) * na.chunk;
    const int64_t last = min(lo + na.chunk, na.total) - 1;
    auto family_of = [&](int64_t g) { return na.family[g < last ? g : last]; };
    auto query_of = [&](int64_t g, float (&v)[R]) {
        const float *p = na.query + (g < last ? g : last) * R;
#pragma unroll
        for (int r = 0; r < R; ++r) v[r] = p[r];
    };
    auto in_range = [&](int f) { return (f >= 0) & (f < a.N); };
    // The extent lookup of a family (any value: out-of-range ones read family 0).
    // AOS: this lane's word of the family's directory record; else the family's
    // slot and size in the columns.
    auto extent_load = [&](int f) -> uint64_t {
        const int fc = in_range(f) ? f : 0;
        if constexpr (AOS) {
            return na.dir[static_cast<size_t>(fc / kDirFamilies) * kDirWords + sub];
        } else {
            if (a.K > 0) return (static_cast<uint64_t>(a.K) << 32) | (static_cast<uint32_t>(fc) * static_cast<uint32_t>(a.K));
            const JobSlot js = a.jobs[fc];
            return (static_cast<uint64_t>(js.size) << 32) | js.slot;
        }
    };
    // every lane of a row shares gi, so rows stay whole for the DPP steps
    int64_t gi = lo + threadIdx.x / kNearestLanes;
    if (gi > last) return;
    int f = family_of(gi);
    float q[R];
    query_of(gi, q);
    uint64_t ext = extent_load(f);
    int f1 = family_of(gi + stride);
    for (; gi <= last; gi += stride) {
        bool ok = in_range(f);
#pragma unroll
        for (int r = 0; r < R; ++r) ok = ok & (fabsf(q[r]) <= 3.402823466e38f);   // false for NaN and +-inf
        // next steps of the pipeline: the query and extent of gi + stride, the family of gi + 2 stride
        const uint64_t ext1 = extent_load(f1);
        const int f2 = family_of(gi + 2 * stride);
        float q1[R];
        query_of(gi + stride, q1);
        int size = 0;
        const float *base = nullptr;       // the family's first entry (AOS) or its slot in column 0
        const int cl = static_cast<int>(gi / na.Q);
        if constexpr (AOS) {
            const uint32_t w = static_cast<uint32_t>(ext);
            const int i = (in_range(f) ? f : 0) % kDirFamilies;
            const int first = 4 * (sub - 1);                 // family of byte 0 of this word
            uint32_t before = w, own = 0;                    // lane 0: the group's first line
            if (sub > 0) {
                before = 0;
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const uint32_t k = ((w >> (8 * m)) & 0xffu) + 1u;      // family size, 1..256
                    if (first + m < i) before += (k * kEntryBytes + (kStoreLine - 1)) / kStoreLine;
                    if (first + m == i) own = k;
                }
            }
            before = row_sum(before);
            own = row_sum(own);
            if (ok) {
                size = static_cast<int>(own);
                base = na.aos + (static_cast<size_t>(cl) * na.aos_lines + before) * (kStoreLine / 4);
            }
        } else if (ok) {
            size = static_cast<int>(ext >> 32);
            base = a.table + cl * a.cluster_stride + static_cast<uint32_t>(ext);
        }
        double best = -__builtin_inf();
        int bk = 0x7fffffff;
        float bu = 0.0f;
        for (int k = sub; k < size; k += kNearestLanes) {
            float d[R + 1];                                  // utility, then the R demands
            if constexpr (AOS) {
                __builtin_memcpy(d, base + static_cast<size_t>(k) * (R + 1), sizeof d);
            } else {
#pragma unroll
                for (int r = 0; r <= R; ++r) d[r] = base[r * a.col_len + k];
            }
            double x = static_cast<double>(q[0]) - static_cast<double>(d[1]);
            double acc = x * x;
#pragma unroll
            for (int r = 1; r < R; ++r) {
                x = static_cast<double>(q[r]) - static_cast<double>(d[r + 1]);
                acc = acc + x * x;
            }
            // Masked configurations (utility -inf) are no candidates.  k ascends
            // within a lane, so keeping the first of equal distances keeps the
            // lowest index.  Selects, not a branch: all of the entry's loads
            // are issued before the mask is tested.
            const bool take = (d[0] != -__builtin_inff()) & (-acc > best);
            best = take ? -acc : best;
            bk = take ? k : bk;
            bu = take ? d[0] : bu;
        }
        const int mine = bk;
        group_argmax<kNearestLanes>(best, bk);
        const bool found = ok && bk != 0x7fffffff;
        if (sub == 0) {
            na.nearest[gi] = found ? bk : -1;
            if (na.estimate && !found) na.estimate[gi] = __builtin_nanf("");
            if (!ok) atomicCAS(a.status, 0, in_range(f) ? kStatusNonfinite : kStatusInvalid);
        }
        // the entry's own lane (entries k of lane s satisfy k = s mod 16)
        if (found && na.estimate && mine == bk) na.estimate[gi] = bu;
        f = f1;
        ext = ext1;
        f1 = f2;
#pragma unroll
        for (int r = 0; r < R; ++r) q[r] = q1[r];
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
//           GPUs.  A job needing at least as much as a share that already
//           failed in this round is skipped without a scan.  Residuals live
//           in LDS, updated in job order (binary64, the oracle's operations).
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
    // jobs, or bounds on them (upper, upper, lower).  A block failing any of
    // the three cannot hold the share, so skipping it is exact.
    double sum_m = m.gpu_memory, sum_s = m.gpu_compute;
    int sum_c = lane < nblk ? 0 : kMaxPerGpu;
    // Lane l remembers a share that found no room in this round (GPU count,
    // memory and compute per GPU; the lanes are filled in turn).  Residuals
    // only shrink and counts only grow while jobs are placed, so a job that
    // needs at least as much in all three as a remembered failure cannot be
    // placed either: it is skipped without a scan.
    int fail_g = 0x7fffffff;
    double fail_m = __builtin_inf(), fail_s = __builtin_inf();
    int n_fail = 0;
    wave_sync();
    const uint64_t below = (1ull << lane) - 1ull;
    // Jobs 64 at a time: each lane gathers one job's share (GPU count,
    // memory and compute per GPU), then the wavefront places them in order.
    // The gathers run one batch ahead: while a batch is placed (LDS and
    // registers only), the next batch's table values and the choices and
    // family slots of the batch after it are in flight.  Indices past N are
    // clamped (loaded, then ignored), so every load stays in bounds.
    auto job_entry = [&](int j0, int &k, size_t &base) {
        const int jl = min(j0 + lane, N - 1);
        k = ch[jl];
        base = a.K > 0 ? static_cast<size_t>(jl) * a.K : static_cast<size_t>(a.jobs[jl].slot);
    };
    auto share_of = [&](int k, size_t base, float &gv, float &mv, float &sv) {
        const size_t e = base + static_cast<size_t>(k > 0 ? k : 0);
        gv = col[(m.r_gpus + 1) * a.col_len + e];
        mv = col[(m.r_mem + 1) * a.col_len + e];
        sv = col[(m.r_sm + 1) * a.col_len + e];
    };
    int k_cur, k_next;
    size_t b_cur, b_next;
    float gv_cur, mv_cur, sv_cur;
    job_entry(0, k_cur, b_cur);
    share_of(k_cur, b_cur, gv_cur, mv_cur, sv_cur);
    job_entry(kWaveSize, k_next, b_next);
    for (int j0 = 0; j0 < N; j0 += kWaveSize) {
        float gv_n, mv_n, sv_n;
        share_of(k_next, b_next, gv_n, mv_n, sv_n);
        int k_after;
        size_t b_after;
        job_entry(j0 + 2 * kWaveSize, k_after, b_after);
        int g_l = 0;
        double nm_l = 0.0, ns_l = 0.0;
        const double gv = static_cast<double>(gv_cur);
        if ((j0 + lane < N) & (k_cur >= 0) & (gv >= 1.0) & (gv <= static_cast<double>(kMaxShards)) &
            (gv == floor(gv))) {
            g_l = static_cast<int>(gv);
            nm_l = static_cast<double>(mv_cur) / gv;
            ns_l = static_cast<double>(sv_cur) / gv;
        }
        k_cur = k_next;
        gv_cur = gv_n;
        mv_cur = mv_n;
        sv_cur = sv_n;
        k_next = k_after;
        b_next = b_after;
        const int cnt = min(kWaveSize, N - j0);
        // jobs of the batch already ruled out by the failures remembered so
        // far (each lane tests its own job against every remembered one)
        bool ruled_out = g_l == 0;
        for (int f = 0; f < min(n_fail, kWaveSize); ++f) {
            const int fg = lane_i(fail_g, f);
            const double fm = lane_d(fail_m, f), fs = lane_d(fail_s, f);
            ruled_out = ruled_out | ((g_l >= fg) & (nm_l >= fm) & (ns_l >= fs));
        }
        const uint64_t skip = __ballot(ruled_out);
        for (int t = 0; t < cnt; ++t) {
            if ((skip >> t) & 1ull) continue;             // not placeable, or needs more than a failure
            const int g = lane_i(g_l, t);
            const double nm = lane_d(nm_l, t);
            const double ns = lane_d(ns_l, t);
            // failures remembered within this batch
            if (__ballot((g >= fail_g) & (nm >= fail_m) & (ns >= fail_s)) != 0ull) continue;
            uint64_t cand = __ballot((sum_c < kMaxPerGpu) & (sum_m >= nm) & (sum_s >= ns));
            int found = 0, visited = 0;
            // the last visited block's GPUs of this lane, and which of them fit
            int c = 0, h0 = 0, before = 0;
            bool fit[kPerLane];
            int cv[kPerLane];
            double mv[kPerLane], sv[kPerLane];
            while ((cand != 0ull) & (found < g)) {
                c = __builtin_ctzll(cand);
                cand &= cand - 1ull;
                ++visited;
                // lane l tests GPUs c*256 + 4l .. 4l+3 (ascending with the lane)
                h0 = c * kStep + lane * kPerLane;
                int total = 0;
                before = 0;
#pragma unroll
                for (int i = 0; i < kPerLane; ++i) {
                    cv[i] = s_cnt[h0 + i];
                    mv[i] = s_mem[h0 + i];
                    sv[i] = s_sm[h0 + i];
                }
#pragma unroll
                for (int i = 0; i < kPerLane; ++i) {
                    fit[i] = (cv[i] < kMaxPerGpu) & (mv[i] >= nm) & (sv[i] >= ns);
                    const uint64_t bal = __ballot(fit[i]);
                    before += __popcll(bal & below);
                    total += __popcll(bal);
                }
                int rank = found + before;
#pragma unroll
                for (int i = 0; i < kPerLane; ++i) {
                    if (fit[i]) {
                        if (rank < g) s_sel[rank] = h0 + i;
                        ++rank;
                    }
                }
                if (found + total < g) {
                    // the block cannot complete the share: make its summary
                    // exact from the values just read
                    double xm = -__builtin_inf(), xs = -__builtin_inf();
                    int xc = kMaxPerGpu;
#pragma unroll
                    for (int i = 0; i < kPerLane; ++i) {
                        const bool open = cv[i] < kMaxPerGpu;
                        xm = open ? fmax(xm, mv[i]) : xm;
                        xs = open ? fmax(xs, sv[i]) : xs;
                        xc = min(xc, cv[i]);
                    }
                    wave_max2_min(xm, xs, xc);
                    if (lane == c) {
                        sum_m = xm;
                        sum_s = xs;
                        sum_c = xc;
                    }
                }
                found += total;
            }
            if (found < g) {                               // all or nothing
                if (lane == (n_fail & (kWaveSize - 1))) {
                    fail_g = g;
                    fail_m = nm;
                    fail_s = ns;
                }
                ++n_fail;
                wave_sync();
                continue;
            }
            if (visited == 1) {
                // The share lies in one block: each selected GPU's lane updates
                // it from the values it holds (no second round trip through
                // LDS).  The block's summary is left as it was: residuals only
                // shrink and counts only grow, so it stays an upper bound, and
                // skipping the blocks it rules out stays exact; it is made exact
                // again when a visit finds the block unable to complete a share.
                int rank = before;
#pragma unroll
                for (int i = 0; i < kPerLane; ++i) {
                    const bool take = fit[i] & (rank < g);
                    rank += fit[i] ? 1 : 0;
                    if (take) {
                        s_mem[h0 + i] = mv[i] - nm;
                        s_sm[h0 + i] = sv[i] - ns;
                        s_occ[h0 + i][cv[i]] = j0 + t;
                        s_cnt[h0 + i] = cv[i] + 1;
                    }
                }
                wave_sync();
                continue;
            }
            wave_sync();
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
                const int cb = s_sel[i] / kStep;
                if (cb == last) continue;
                last = cb;
                const int hb = cb * kStep + lane * kPerLane;
                double xm = -__builtin_inf(), xs = -__builtin_inf();
                int xc = kMaxPerGpu;
#pragma unroll
                for (int q = 0; q < kPerLane; ++q) {
                    const int cq = s_cnt[hb + q];
                    const double mq = s_mem[hb + q], sq = s_sm[hb + q];
                    const bool open = cq < kMaxPerGpu;           // GPUs that can still take a job
                    xm = open ? fmax(xm, mq) : xm;
                    xs = open ? fmax(xs, sq) : xs;
                    xc = min(xc, cq);
                }
                wave_max2_min(xm, xs, xc);
                if (lane == cb) {
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
// Launchers
// ---------------------------------------------------------------------------

template <int R>
static hipError_t launch_nearest_r(const KArgs &a, const NearestArgs &na, hipStream_t s) {
    constexpr int kPerBlock = kBlockThreads / kNearestLanes;
    constexpr int64_t kLineQueries = 32;             // one 128-byte line of 4-byte outputs
    const int64_t cap = 256 * 32;                    // enough resident queries to cover gather latency
    const int64_t need = (na.total + kPerBlock - 1) / kPerBlock;
    NearestArgs nb = na;
    nb.chunk = (na.total + (need < cap ? need : cap) - 1) / (need < cap ? need : cap);
    nb.chunk = (nb.chunk + kLineQueries - 1) / kLineQueries * kLineQueries;
    const dim3 grid(static_cast<unsigned>((na.total + nb.chunk - 1) / nb.chunk)), block(kBlockThreads);
    if (na.aos)
        hipLaunchKernelGGL((k_nearest<R, true>), grid, block, 0, s, a, nb);
    else
        hipLaunchKernelGGL((k_nearest<R, false>), grid, block, 0, s, a, nb);
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

}  // namespace esp
