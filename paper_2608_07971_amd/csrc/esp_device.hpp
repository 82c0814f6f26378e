// Device helpers shared by the gfx950 kernels of the Elastic Shadow Pricing
// library: DPP lane moves and the lowest-index argmax, exact fixed-point
// sums, and the cross-workgroup completion of a cluster's sums.
#pragma once

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
    // bitwise, not short-circuit, operators: no branches where lanes diverge
    const bool b = (os > s) | ((os == s) & (ok < k));
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
    s = s > kMax ? kMax : (s < -kMax ? -kMax : s);       // (zero: m = 0 shifts to 0 either way)
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

// The same for a 64-bit accumulator (fewer instructions where the sums are
// known to fit 64 bits).
__device__ __forceinline__ double fx_to_double(uint64_t a, int sh) {
    if (a == 0) return 0.0;
    const int h = 63 - __clzll(a);
    if (h <= 52) return ldexp(static_cast<double>(a), sh);
    const int drop = h - 52;
    uint64_t m = a >> drop;
    const uint64_t rem = a & ((1ull << drop) - 1);
    const uint64_t half = 1ull << (drop - 1);
    if (rem > half || (rem == half && (m & 1u))) m += 1;   // m <= 2^53: exact as a double
    return ldexp(static_cast<double>(m), drop + sh);
}

// Partial-sum buffer k of cluster cl: [nblk][R][2] 64-bit words (low, high).
template <int R>
__device__ __forceinline__ uint64_t *partials_of(const KArgs &a, int k, int cl) {
    return a.partials + (static_cast<size_t>(k) * a.B + cl) * static_cast<size_t>(a.nblk) * R * 2;
}

// Publish this workgroup's sums bsum[r] (LDS) into buffer k with agent-scope
// atomic exchanges, which are performed at the device coherence point, and
// wait until they have completed (their old values are back).  Runs in
// wavefront 0; the caller orders the rest of the workgroup.
//
// Why a reader elsewhere on the device then sees these sums (the argument
// for publish_sums / cluster_sums here and for the persistent barrier of the
// kernels; it rests on how gfx950 performs agent-scope atomics, not on a
// release/acquire pair, whose cache-wide writeback and invalidation cost
// 12 us per iteration at 256 workgroups):
//  1. The 8 XCDs each have their own L2, which is not coherent with the
//     others.  Agent-scope atomic operations are not performed in an XCD's
//     L2: they travel to the memory-side coherence point of their address
//     (shared by all XCDs), and one that returns a value returns it only
//     after it has been performed there.  Agent-scope atomic loads read from
//     that point as well, never from a stale L2 line.
//  2. s_waitcnt vmcnt(0) on the returned values therefore means every
//     exchange below has been performed at the coherence point before the
//     workgroup issues anything after it: the ticket or arrival add that
//     signals "published" is issued later, so it is performed later.
//  3. A reader learns "all published" from the value another atomic
//     returned (the last ticket, or a release word stored only after the
//     last arrival add had returned), and issues its loads of the sums only
//     after that value is back (the loads depend on it).  They are performed
//     after every exchange was, at the same point, so they return the
//     published sums.
// What would break it: workgroup scope (performed in one XCD's L2), plain
// stores (held in the writer's L2 until evicted), plain loads (a stale line
// in the reader's L2), a non-returning add or a missing wait (the signal
// could overtake the sums on their way to the coherence point).
template <int R>
__device__ __forceinline__ void publish_sums(const KArgs &a, int k, int cl, int blk, const u128 *bsum) {
    const int t = threadIdx.x;
    uint64_t old = 0;
    if (t < R) {
        uint64_t *p = partials_of<R>(a, k, cl) + (static_cast<size_t>(blk) * R + t) * 2;
        const u128 v = bsum[t];
        old ^= __hip_atomic_exchange(p, static_cast<uint64_t>(v), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        old ^= __hip_atomic_exchange(p + 1, static_cast<uint64_t>(v >> 64), __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
    }
    asm volatile("s_waitcnt vmcnt(0)" : : "v"(old) : "memory");
}

// Totals over the nblk published sums of buffer k.  Thread (g, r), g < G =
// kBlockThreads / R, takes blocks g, g+G, g+2G, ...: partial_loads issues the
// first kSumLoads of them (so that a caller can start them early, before
// other loads), partial_totals loads the rest, adds, and runs a tree over g
// in LDS; afterwards s_red[r] holds the cluster's total for resource r (all
// threads take part; ends with a workgroup barrier).  With 64-bit
// accumulators every sum fits in the low word, the high word is not read.
// Coherent: agent-scope atomic loads, which bypass the non-coherent caches
// (sums published in the same launch); otherwise plain loads (sums of an
// earlier launch, made visible by the launch boundary).
constexpr int kSumLoads = 8;

template <typename A, bool Coherent>
__device__ __forceinline__ A load_sum(uint64_t *p) {
    uint64_t lo, hi = 0;
    if constexpr (Coherent) {
        lo = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if constexpr (sizeof(A) > 8) hi = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
        lo = p[0];
        if constexpr (sizeof(A) > 8) hi = p[1];
    }
    if constexpr (sizeof(A) > 8) return (static_cast<A>(hi) << 64) | lo;
    else return static_cast<A>(lo);
}

// Every thread loads kSumLoads sums without branches (addresses past the
// last block are clamped to it and the value replaced by zero), so that the
// compiler can wait for exactly these loads.
template <int R, typename A, bool Coherent>
__device__ __forceinline__ void partial_loads(const KArgs &a, int k, int cl, A (&v)[kSumLoads]) {
    constexpr int G = kBlockThreads / R;
    const int t = threadIdx.x;
    const int r = t % R, g = t / R;
    uint64_t *base = partials_of<R>(a, k, cl) + static_cast<size_t>(r) * 2;
#pragma unroll
    for (int u = 0; u < kSumLoads; ++u) {
        const int b = g + u * G;
        const A x = load_sum<A, Coherent>(base + static_cast<size_t>(min(b, a.nblk - 1)) * R * 2);
        v[u] = (t < G * R && b < a.nblk) ? x : A(0);
    }
}

template <int R, typename A, bool Coherent>
__device__ __forceinline__ void partial_totals(const KArgs &a, int k, int cl, const A (&v)[kSumLoads],
                                               u128 *s_red) {
    constexpr int G = kBlockThreads / R;
    const int t = threadIdx.x;
    u128 s = 0;
#pragma unroll
    for (int u = 0; u < kSumLoads; ++u) s += static_cast<u128>(v[u]);
    if (t < G * R) {
        const int r = t % R, g = t / R;
        uint64_t *base = partials_of<R>(a, k, cl) + static_cast<size_t>(r) * 2;
#pragma unroll 1
        for (int b0 = g + kSumLoads * G; b0 < a.nblk; b0 += kSumLoads * G) {
            A w[kSumLoads];
#pragma unroll
            for (int u = 0; u < kSumLoads; ++u) {
                const int b = b0 + u * G;
                w[u] = b < a.nblk ? load_sum<A, Coherent>(base + static_cast<size_t>(b) * R * 2) : A(0);
            }
#pragma unroll
            for (int u = 0; u < kSumLoads; ++u) s += static_cast<u128>(w[u]);
        }
    }
    s_red[t] = s;
    __syncthreads();
    // tree over the G groups (integer adds: the order does not matter)
#pragma unroll
    for (int h = 128; h >= 1; h >>= 1) {
        if (h < G) {
            if (t < h * R && t + h * R < G * R) s_red[t] += s_red[t + h * R];
            __syncthreads();
        }
    }
}

// Cross-workgroup exact sums of one cluster within one launch.  bsum[r]
// (LDS) holds this workgroup's 128-bit sum for resource r.  In the workgroup
// that finishes last, thread r < R runs done(r, total_r) with the cluster's
// total; the function returns true there (after a workgroup barrier) and
// false in every other workgroup.
//
// Ordering across the 8 XCDs (each with its own L2) without cache-wide
// writeback or invalidation: the sums are published with agent-scope atomic
// exchanges that have completed before the workgroup takes a ticket with an
// agent-scope atomic add.  The workgroup that draws the last ticket reads
// every sum with agent-scope atomic loads and resets the ticket for the next
// use.
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
        publish_sums<R>(a, kInLaunchBuffer, cl, blk, bsum);
        if (t == 0) {
            const unsigned prev = __hip_atomic_fetch_add(&a.tickets[cl], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_last = (prev == static_cast<unsigned>(a.nblk) - 1u);
        }
    }
    __syncthreads();
    if (!s_last) return false;
    u128 v[kSumLoads];
    partial_loads<R, u128, true>(a, kInLaunchBuffer, cl, v);
    partial_totals<R, u128, true>(a, kInLaunchBuffer, cl, v, s_red);
    if (t < R) done(t, s_red[t]);
    if (t == 0) {
        // ready for the next use
        const unsigned o = __hip_atomic_exchange(&a.tickets[cl], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        asm volatile("s_waitcnt vmcnt(0)" : : "v"(o) : "memory");
    }
    __syncthreads();
    return true;
}

}  // namespace esp

// Runtime R -> template instance of a launcher.
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
