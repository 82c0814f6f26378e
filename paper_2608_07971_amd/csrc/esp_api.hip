// Host side of the Elastic Shadow Pricing C-ABI (include/esp.h): argument
// validation, the packer that lays the job x configuration table out as
// structure-of-arrays tiles in the caller's device workspace, and the drivers
// that enqueue the kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/esp.h"
#include "esp_extras.hpp"
#include "esp_internal.hpp"

#pragma clang fp contract(off)

using namespace esp;

namespace {

constexpr uint32_t kMagic = 0x45535031u;   // "ESP1"
static_assert(ESP_MAX_GPUS == kMaxGpus && ESP_MAX_PER_GPU == kMaxPerGpu, "public limits match the kernels");
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Launch plan and workspace layout derived from the problem's shapes.
struct Plan {
    int B = 0, N = 0, R = 0;
    int K = 0;          // dense family size handled by the dense kernel, else 0
    int lpj = 0;        // lanes per job of the dense kernel
    bool csr = false;
    bool pen = false;   // a penalty column follows the demand columns
    int64_t nnz = 0;
    int tiles = 0;      // per cluster
    size_t col_len = 0; // floats per column
    int nblk = 0;       // workgroups per cluster
    int aos_stride = 0; // floats per entry of the entry-major copy, 0 when there is none
    int64_t aos_lines = 0;  // kStoreLine-byte lines of one cluster's entry-major copy
    // workspace offsets (bytes)
    size_t o_table = 0, o_meta = 0, o_jobs = 0, o_shift = 0, o_cap = 0, o_eta = 0, o_part = 0,
           o_tick = 0, o_flags = 0, o_iters = 0, o_sync = 0, o_swc = 0, o_status = 0, o_capp = 0, o_offs = 0, o_inc = 0, o_gpus = 0,
           o_aos = 0, o_dir = 0, o_lamws = 0, o_conv = 0, o_xch = 0, total = 0;
    size_t columns() const { return static_cast<size_t>(R) + 1 + (pen ? 1 : 0); }
};

// Compute units of the current device (256 on MI355X); 256 when no device
// can be queried (workspace sizing on a host without a GPU).
int device_cus() {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
    return n;
}

bool dense_fast_k(int K) { return K == 4 || K == 8 || K == 16 || K == 32 || K == 64; }

// Entry-major copy: lines of a family of k configurations, records of the directory.
int64_t store_lines(int64_t k, int stride) {
    return (k * stride * static_cast<int64_t>(sizeof(float)) + kStoreLine - 1) / kStoreLine;
}
int64_t dir_records(int N) { return (static_cast<int64_t>(N) + kDirFamilies - 1) / kDirFamilies; }

// Family sizes of the problem (dense or CSR) and validation of the offsets.
esp_status family_layout(const esp_problem *p, std::vector<int64_t> *sizes_out, int *uniform_k) {
    const int N = p->num_jobs;
    *uniform_k = 0;
    if (p->family_offsets == nullptr) {
        if (p->configs_per_job < 1 || p->configs_per_job > kMaxFamily) return ESP_ERR_SHAPE;
        *uniform_k = p->configs_per_job;
        return ESP_OK;
    }
    const int64_t *off = p->family_offsets;
    if (off[0] != 0) return ESP_ERR_SHAPE;
    int64_t k0 = -1;
    bool uniform = true;
    for (int j = 0; j < N; ++j) {
        const int64_t k = off[j + 1] - off[j];
        if (k < 1 || k > kMaxFamily) return ESP_ERR_SHAPE;
        if (k0 < 0) k0 = k;
        uniform = uniform && (k == k0);
    }
    if (uniform) *uniform_k = static_cast<int>(k0);
    if (sizes_out) {
        sizes_out->resize(N);
        for (int j = 0; j < N; ++j) (*sizes_out)[j] = off[j + 1] - off[j];
    }
    return ESP_OK;
}

esp_status make_plan(const esp_problem *p, const esp_options *opt, Plan *pl) {
    if (p == nullptr) return ESP_ERR_INVALID_ARG;
    if (opt) {
        if (opt->blocks_per_cluster < 0) return ESP_ERR_INVALID_ARG;
        if (opt->sweep_order != 0 && opt->sweep_order != 1) return ESP_ERR_INVALID_ARG;
        if (opt->mode < ESP_MODE_AUTO || opt->mode > ESP_MODE_RESIDENT) return ESP_ERR_INVALID_ARG;
        if ((opt->flags & ~ESP_OPT_PROFILE_STORE) != 0) return ESP_ERR_INVALID_ARG;
        for (int i = 0; i < 4; ++i)
            if (opt->reserved[i] != 0) return ESP_ERR_INVALID_ARG;
    }
    if (p->num_clusters < 1 || p->num_jobs < 1 || p->num_resources < 1 || p->num_resources > kMaxR)
        return ESP_ERR_SHAPE;
    const int64_t BN = static_cast<int64_t>(p->num_clusters) * p->num_jobs;
    if (BN > INT32_MAX) return ESP_ERR_SHAPE;
    int uk = 0;
    esp_status st = family_layout(p, nullptr, &uk);
    if (st != ESP_OK) return st;
    pl->B = p->num_clusters;
    pl->N = p->num_jobs;
    pl->R = p->num_resources;
    pl->pen = p->current != nullptr || p->penalty != nullptr;
    if (uk > 0 && dense_fast_k(uk)) {
        pl->K = uk;
        pl->lpj = uk / 4;
        const int jpt = kWaveSize / pl->lpj;
        pl->nnz = static_cast<int64_t>(pl->N) * uk;
        pl->tiles = static_cast<int>((static_cast<int64_t>(pl->N) + jpt - 1) / jpt);
    } else {
        // CSR tiles: whole families packed greedily into 256-entry tiles.
        const int N = pl->N;
        int64_t tiles = 0, fill = kTileEntries, nnz = 0;
        for (int j = 0; j < N; ++j) {
            const int64_t k = p->family_offsets ? p->family_offsets[j + 1] - p->family_offsets[j]
                                                : p->configs_per_job;
            if (fill + k > kTileEntries) { ++tiles; fill = 0; }
            fill += k;
            nnz += k;
        }
        pl->csr = true;
        pl->nnz = nnz;
        if (tiles > INT32_MAX / 2) return ESP_ERR_SHAPE;
        pl->tiles = static_cast<int>(tiles);
    }
    // Columns are kColumnPadTiles tiles longer than the table, so that the
    // 1 + R columns of a cluster do not start at the same offset modulo large
    // powers of two (one wavefront reads the same tile of every column at
    // once).  Measured on Large: 93.9 us per pass with the pad, 96.9 without.
    pl->col_len = (static_cast<size_t>(pl->tiles) + kColumnPadTiles) * kTileEntries;
    if (pl->col_len >= (static_cast<size_t>(1) << 32)) return ESP_ERR_SHAPE;
    // Workgroups over the whole device, split across clusters (every
    // workgroup sweeps many tiles).  The CSR kernel does more VALU work per
    // tile and runs two workgroups per compute unit.  The dense kernel runs
    // one per compute unit on three quarters of the units: with every unit
    // streaming, the workgroups finish further apart and a pass takes longer
    // (Large: 90 us per pass at 192 workgroups, 94 us at 256).
    const int max_useful = std::max(1, (pl->tiles + kBlockWaves - 1) / kBlockWaves);
    const int cus = device_cus();
    const int total = pl->csr ? 2 * cus : std::max(1, 3 * cus / 4);
    int nblk = (opt && opt->blocks_per_cluster > 0) ? opt->blocks_per_cluster
                                                     : std::max(1, (total + pl->B - 1) / pl->B);
    pl->nblk = std::min(nblk, max_useful);
    if (static_cast<int64_t>(pl->nblk) * pl->B > INT32_MAX) return ESP_ERR_SHAPE;

    const size_t B = pl->B, R = pl->R;
    size_t o = 0;
    pl->o_table = o; o = align_up(o + B * pl->columns() * pl->col_len * sizeof(float));
    pl->o_meta = o;  o = align_up(o + (pl->csr ? static_cast<size_t>(pl->tiles) * sizeof(TileMeta) : 0));
    pl->o_jobs = o;  o = align_up(o + (pl->csr ? static_cast<size_t>(pl->N) * sizeof(JobSlot) : 0));
    pl->o_shift = o; o = align_up(o + B * R * sizeof(int32_t));
    pl->o_cap = o;   o = align_up(o + B * R * sizeof(double));
    pl->o_eta = o;   o = align_up(o + B * sizeof(double));
    pl->o_part = o;  o = align_up(o + kPartialBuffers * B * pl->nblk * R * 2 * sizeof(uint64_t));
    pl->o_tick = o;  o = align_up(o + B * sizeof(uint32_t));
    pl->o_flags = o; o = align_up(o + B * sizeof(int32_t));
    pl->o_iters = o; o = align_up(o + B * sizeof(int32_t));
    pl->o_sync = o;  o = align_up(o + B * kSyncSlots * kSyncStride * sizeof(uint32_t));
    pl->o_swc = o;   o = align_up(o + B * sizeof(double));
    pl->o_status = o; o = align_up(o + sizeof(int32_t));
    pl->o_capp = o;  o = align_up(o + B * R * sizeof(double));
    pl->o_offs = o;  o = align_up(o + (static_cast<size_t>(pl->N) + 1) * sizeof(int64_t));
    pl->o_inc = o;   o = align_up(o + B * static_cast<size_t>(pl->N) * sizeof(uint64_t));
    pl->o_gpus = o;  o = align_up(o + B * sizeof(int32_t));
    size_t dir_bytes = 0;
    if (opt && (opt->flags & ESP_OPT_PROFILE_STORE)) {
        pl->aos_stride = pl->R + 1;
        int64_t lines = 0;
        for (int j = 0; j < pl->N; ++j)
            lines += store_lines(p->family_offsets ? p->family_offsets[j + 1] - p->family_offsets[j]
                                                   : p->configs_per_job, pl->aos_stride);
        if (lines > static_cast<int64_t>(UINT32_MAX)) return ESP_ERR_SHAPE;   // 32-bit line numbers
        pl->aos_lines = lines;
        dir_bytes = static_cast<size_t>(dir_records(pl->N)) * kDirWords * sizeof(uint32_t);
    }
    pl->o_aos = o;   o = align_up(o + B * static_cast<size_t>(pl->aos_lines) * kStoreLine);
    pl->o_dir = o;   o = align_up(o + dir_bytes);
    pl->o_lamws = o; o = align_up(o + 2 * B * R * sizeof(double));
    pl->o_conv = o;  o = align_up(o + B * sizeof(int32_t));
    pl->o_xch = o;   o = align_up(o + 2 * B * pl->nblk * R * kMaxLimbs * sizeof(uint64_t));
    pl->total = o;
    return ESP_OK;
}

// Lowest set bit exponent and bit length of a positive finite float:
// v = m * 2^x with m odd; top = exponent of the bit above the highest set bit.
void float_bits(float v, int *low, int *top) {
    uint32_t b;
    std::memcpy(&b, &v, 4);
    const uint32_t e = b >> 23;
    const uint32_t m = (b & 0x7fffffu) | (e ? 0x800000u : 0u);
    const int x = (e ? static_cast<int>(e) : 1) - 150;
    *low = x + __builtin_ctz(m);
    *top = x + (32 - __builtin_clz(m));
}

struct PinnedPair {
    float *buf[2] = {nullptr, nullptr};
    hipEvent_t ev[2] = {nullptr, nullptr};
    bool pending[2] = {false, false};
    size_t cap = 0;
    ~PinnedPair() {
        for (int i = 0; i < 2; ++i) {
            if (ev[i]) { if (pending[i]) (void)hipEventSynchronize(ev[i]); (void)hipEventDestroy(ev[i]); }
            if (buf[i]) (void)hipHostFree(buf[i]);
        }
    }
};

}  // namespace

// Scratch of esp_solve_noalloc: one array per GPU, in the library's code
// object, held until the process ends.  Host code never uses `scratch`
// itself (on the host it is a stand-in, not a device address): each device's
// address comes from hipGetSymbolAddress, resolved once per device with that
// device current, when a context is created on it.
static __device__ __align__(256) unsigned char scratch[ESP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char *g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch` (NULL when it cannot be resolved).
char *resolve_scratch(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) == hipSuccess) g_scratch_ptr[dev] = static_cast<char *>(p);
        else (void)hipGetLastError();
    }
    return g_scratch_ptr[dev];
}

// Byte offsets of the per-solve scratch regions of a plan inside the static
// array, each 256-byte aligned; the last value is the size.
struct ScratchLayout {
    size_t part = 0, tick = 0, iters = 0, sync = 0, lamws = 0, conv = 0, xch = 0, total = 0;
};

ScratchLayout scratch_layout(const Plan &pl) {
    const size_t B = pl.B, R = pl.R;
    ScratchLayout L;
    size_t o = 0;
    L.part = o;  o = align_up(o + kPartialBuffers * B * pl.nblk * R * 2 * sizeof(uint64_t));
    L.tick = o;  o = align_up(o + B * sizeof(uint32_t));
    L.iters = o; o = align_up(o + B * sizeof(int32_t));
    L.sync = o;  o = align_up(o + B * kSyncSlots * kSyncStride * sizeof(uint32_t));
    L.lamws = o; o = align_up(o + 2 * B * R * sizeof(double));
    L.conv = o;  o = align_up(o + B * sizeof(int32_t));
    L.xch = o;   o = align_up(o + 2 * B * pl.nblk * R * kMaxLimbs * sizeof(uint64_t));
    L.total = o;
    return L;
}

}  // namespace

struct esp_ctx {
    uint32_t magic = kMagic;
    char *scratch = nullptr;           // this device's address of `scratch`, or NULL
    Plan pl;
    int rule = 0;
    std::vector<double> eta0;
    char *ws = nullptr;
    double *h_stage = nullptr;         // pinned staging for capacities and GPU counts
    hipEvent_t stage_ev = nullptr;     // recorded after the last copy out of h_stage
    bool stage_pending = false;
    int sweep = 0;                     // 0: alternate the sweep direction, 1: always forward
    int mode = ESP_MODE_AUTO;
    bool auto_mode = false;            // the caller asked for ESP_MODE_AUTO
    bool fell_back = false;            // AUTO: the device refused a co-resident grid
    bool resident_ok = false;          // persistent solves may hold the tiles in registers
    std::vector<int64_t> off;          // family offsets (host copy)
    std::vector<int64_t> slot_of;      // first table slot of each family
    KArgs base{};
};

namespace {

// Validate the penalty inputs of Eq. 7 against the family layout.
esp_status validate_penalties(int B, int N, int64_t nnz, const std::vector<int64_t> &off, const int32_t *current,
                              const double *switch_cost, const float *penalty) {
    if ((current == nullptr) != (switch_cost == nullptr)) return ESP_ERR_INVALID_ARG;
    if (current) {
        for (int b = 0; b < B; ++b) {
            const double g = switch_cost[b];
            if (!std::isfinite(g)) return ESP_ERR_NONFINITE;
            if (!(g >= 0.0)) return ESP_ERR_INVALID_ARG;
            if (g > 0x1p100) return ESP_ERR_RANGE;
            for (int j = 0; j < N; ++j) {
                const int32_t c = current[static_cast<size_t>(b) * N + j];
                if (c < -1 || c >= off[j + 1] - off[j]) return ESP_ERR_INVALID_ARG;
            }
        }
    }
    if (penalty) {
        for (size_t e = 0; e < static_cast<size_t>(B) * nnz; ++e) {
            const float v = penalty[e];
            if (!std::isfinite(v)) return ESP_ERR_NONFINITE;
            if (v < 0.0f) return ESP_ERR_INVALID_ARG;
        }
    }
    return ESP_OK;
}

// Penalty column of cluster b into h (col_len floats): |penalty| with the sign
// bit set on entries that pay the switching cost.
void fill_penalty_column(float *h, size_t col_len, int b, int N, int64_t nnz, const std::vector<int64_t> &off,
                         const std::vector<int64_t> &slot_of, const int32_t *current, const float *penalty) {
    std::fill(h, h + col_len, 0.0f);
    for (int j = 0; j < N; ++j) {
        const int64_t k = off[j + 1] - off[j];
        const int32_t cur = current ? current[static_cast<size_t>(b) * N + j] : -1;
        for (int64_t i = 0; i < k; ++i) {
            float v = penalty ? penalty[static_cast<size_t>(b) * nnz + off[j] + i] : 0.0f;
            v = (v == 0.0f) ? 0.0f : v;                 // +0.0 for either zero
            h[slot_of[j] + i] = (cur >= 0 && i != cur) ? -v : v;   // -0.0 when the penalty is zero
        }
    }
}

esp_status check_ctx(const esp_ctx *c) {
    return (c != nullptr && c->magic == kMagic) ? ESP_OK : ESP_ERR_STATE;
}

esp_status dev(hipError_t e) { return e == hipSuccess ? ESP_OK : ESP_ERR_DEVICE; }

// Wait until h_stage may be rewritten.
esp_status stage_wait(esp_ctx *c) {
    if (c->stage_pending) {
        if (hipEventSynchronize(c->stage_ev) != hipSuccess) return ESP_ERR_DEVICE;
        c->stage_pending = false;
    }
    return ESP_OK;
}

hipError_t launch_select(const esp_ctx *c, const KArgs &a, hipStream_t s) {
    return c->pl.csr ? launch_csr(c->pl.R, a, c->pl.B, s) : launch_dense(c->pl.R, c->pl.lpj, a, c->pl.B, s);
}

}  // namespace

namespace {

// The body of esp_solve and esp_solve_noalloc.  `kb` is the context's launch
// arguments with the per-solve scratch (partial sums, tickets, barrier words,
// lambda_m, stop iteration) pointing into the context's workspace or into the
// static scratch array; d_iters (device [B]) counts the updates.
esp_status solve_with(esp_ctx *c, const KArgs &kb, int32_t *d_iters, double *prices, int32_t iters,
                      int32_t t_start, double tol, int32_t *choice, double *demand, const esp_trace *trace,
                      int32_t *iters_done, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (prices == nullptr || iters < 0 || t_start < 1 || !(tol >= 0.0) || !std::isfinite(tol))
        return ESP_ERR_INVALID_ARG;
    if (static_cast<int64_t>(t_start) + iters - 1 > INT32_MAX) return ESP_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int B = c->pl.B, R = c->pl.R, N = c->pl.N;
    // Persistent launches (one cooperative launch per chunk of up to
    // kLaunchChunk iterations); one launch per iteration in stream mode, when
    // the device cannot hold the grid co-resident, or while `stream` is being
    // captured into a graph (a cooperative launch cannot be captured).  The
    // capture is checked before anything is enqueued, so a refused call
    // records nothing.
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(s, &cap) != hipSuccess) return ESP_ERR_DEVICE;
    const bool capturing = cap != hipStreamCaptureStatusNone;
    if (capturing && (c->mode == ESP_MODE_PERSISTENT || c->mode == ESP_MODE_RESIDENT)) return ESP_ERR_INVALID_ARG;
    // The loop driver: persistent launches (one per chunk of up to
    // kLaunchChunk iterations) or one launch per iteration.  Persistent
    // launches run over register-resident tiles when every wavefront of the
    // grid holds at most two tiles (tables of up to a few MB, where the
    // latency of an iteration, not the bandwidth, sets the pace): each launch
    // then completes all of its iterations itself.
    bool persistent =
        !capturing && !c->fell_back && (c->mode != ESP_MODE_STREAM || (c->auto_mode && tol > 0.0));
    bool resident = persistent && (c->mode == ESP_MODE_RESIDENT || (c->auto_mode && c->resident_ok));
    {
        // validates the prices, turns -0.0 into +0.0 in place, resets the
        // per-solve state (and the exchange words of a resident solve)
        KArgs p = kb;
        p.iters_done = d_iters;
        p.xch_clear = (resident && c->pl.nblk > 1)
                          ? 2 * static_cast<size_t>(B) * c->pl.nblk * static_cast<size_t>(kb.xch_stride) : 0;
        if ((st = dev(launch_prepare(R, p, prices, prices, B, s))) != ESP_OK) return st;
    }
    // With several workgroups per cluster and no resident launch, every
    // iteration only publishes its sums; the next launch (or the closing
    // one) completes it.  With one workgroup per cluster, or in a resident
    // launch, the iteration is completed where it runs.
    bool defer = false;
    KArgs base;
    auto setup = [&]() {
        defer = !resident && c->pl.nblk > 1;
        base = kb;
        base.lam_in = prices;
        base.lam_dst = prices;
        base.iters_done = d_iters;
        base.tol = tol;
        base.defer = defer ? 1 : 0;
        base.xch_clear = 0;
        if (defer) {
            base.lam_out = nullptr;
            base.skip_mask = kFlagError | kFlagFrozen;
            if (trace) {
                base.trace_lam = trace->prices;
                base.trace_U = trace->demand;
            }
        } else {
            base.lam_out = prices;
            base.skip_mask = kFlagError | kFlagStopped | kFlagFrozen;
        }
        if (resident) base.sweep_alt = 0;      // a wavefront keeps the same tiles
    };
    setup();
    // Launch arguments for solve iterations i .. i + n - 1 (0-based).
    auto iteration_launch = [&](int32_t i, int32_t n) {
        KArgs a = base;
        a.n_iters = n;
        a.t = t_start + i;
        a.iter_no = i + 1;
        a.reduce = 1;
        a.reverse = (c->sweep == 0 && !resident) ? static_cast<int32_t>(i & 1) : 0;
        if (defer && i > 0) {
            a.pend_m = i;
            a.pend_t = t_start + i - 1;
        }
        if (trace) {
            if (!defer && trace->prices) a.tr_lam = trace->prices + static_cast<size_t>(i) * B * R;
            if (!defer && trace->demand) a.tr_U = trace->demand + static_cast<size_t>(i) * B * R;
            if (trace->choice) a.choice = trace->choice + static_cast<size_t>(i) * B * N;
        }
        return a;
    };
    for (int32_t i0 = 0; i0 < iters; i0 += kLaunchChunk) {
        const int n = std::min<int32_t>(kLaunchChunk, iters - i0);
        if (persistent) {
            const KArgs a = iteration_launch(i0, n);
            hipError_t e;
            if (resident)
                e = c->pl.csr ? launch_csr_resident(R, a, B, s) : launch_dense_resident(R, c->pl.lpj, a, B, s);
            else
                e = c->pl.csr ? launch_csr_persistent(R, a, B, s) : launch_dense_persistent(R, c->pl.lpj, a, B, s);
            if (e == hipSuccess) continue;
            (void)hipGetLastError();           // not left for the next launch's error check
            // A refused grid enqueues nothing.  AUTO falls back to one launch
            // per iteration: from here on for deferred persistent launches
            // (same completion scheme), from the first iteration for resident
            // ones (which can only be refused at their first launch).
            if (!c->auto_mode || (resident && i0 > 0)) return ESP_ERR_DEVICE;
            persistent = false;
            c->fell_back = true;
            if (resident) {
                resident = false;
                setup();
            }
        }
        for (int i = 0; i < n; ++i)
            if ((st = dev(launch_select(c, iteration_launch(i0 + i, 1), s))) != ESP_OK) return st;
    }
    // Closing launch: completes the last iteration of a deferred solve, and
    // re-selects at the final prices (no update) when asked to.
    KArgs a = base;
    a.lam_out = nullptr;
    a.tr_lam = a.tr_U = nullptr;
    a.defer = 0;
    a.n_iters = 1;
    a.skip_mask = kFlagError | kFlagFrozen;
    if (defer && iters > 0) {
        a.pend_m = iters;
        a.pend_t = t_start + iters - 1;
    }
    if (choice || demand) {
        a.choice = choice;
        a.demand_out = demand;
        a.reduce = demand ? 1 : 0;
        a.reverse = (c->sweep == 0) ? static_cast<int32_t>(iters & 1) : 0;
        if ((st = dev(launch_select(c, a, s))) != ESP_OK) return st;
    } else if (a.pend_m > 0) {
        if ((st = dev(launch_finish(R, a, B, s))) != ESP_OK) return st;
    }
    if (iters_done &&
        hipMemcpyAsync(iters_done, d_iters, sizeof(int32_t) * B, hipMemcpyDeviceToDevice, s) != hipSuccess)
        return ESP_ERR_DEVICE;
    return ESP_OK;
}

}  // namespace

extern "C" {

const char *esp_status_string(esp_status st) {
    switch (st) {
        case ESP_OK: return "ok";
        case ESP_ERR_INVALID_ARG: return "invalid argument";
        case ESP_ERR_SHAPE: return "inconsistent or unsupported shape";
        case ESP_ERR_NONFINITE: return "non-finite input value";
        case ESP_ERR_NEGATIVE_DEMAND: return "negative demand";
        case ESP_ERR_EMPTY_FAMILY: return "job with no allowed configuration";
        case ESP_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
        case ESP_ERR_RANGE: return "value range not supported";
        case ESP_ERR_DEVICE: return "HIP runtime error";
        case ESP_ERR_STATE: return "invalid context";
    }
    return "unknown status";
}

esp_status esp_workspace_size(const esp_problem *problem, const esp_options *options, size_t *bytes) {
    if (bytes == nullptr) return ESP_ERR_INVALID_ARG;
    Plan pl;
    esp_status st = make_plan(problem, options, &pl);
    if (st != ESP_OK) return st;
    *bytes = pl.total;
    return ESP_OK;
}

esp_status esp_create(const esp_problem *p, const esp_step_rule *step, const esp_options *options,
                      void *workspace, size_t workspace_bytes, void *stream, esp_ctx **out) {
    if (out == nullptr) return ESP_ERR_INVALID_ARG;
    *out = nullptr;
    if (p == nullptr || step == nullptr || p->utility == nullptr || p->demand == nullptr ||
        p->capacity == nullptr || step->eta0 == nullptr)
        return ESP_ERR_INVALID_ARG;
    if (step->rule != ESP_STEP_CONST && step->rule != ESP_STEP_INV_SQRT) return ESP_ERR_INVALID_ARG;
    Plan pl;
    esp_status st = make_plan(p, options, &pl);
    if (st != ESP_OK) return st;
    const int B = pl.B, N = pl.N, R = pl.R;
    const int64_t nnz = pl.nnz;

    // ---- validate values (host) ----
    for (int b = 0; b < B; ++b) {
        const double e0 = step->eta0[b];
        if (!std::isfinite(e0)) return ESP_ERR_NONFINITE;
        if (!(e0 > 0.0)) return ESP_ERR_INVALID_ARG;
        if (e0 > 0x1p100) return ESP_ERR_RANGE;
        for (int r = 0; r < R; ++r) {
            const double cr = p->capacity[static_cast<size_t>(b) * R + r];
            if (!std::isfinite(cr)) return ESP_ERR_NONFINITE;
            if (std::fabs(cr) > 0x1p200) return ESP_ERR_RANGE;
        }
    }
    std::vector<int64_t> off(static_cast<size_t>(N) + 1);
    for (int j = 0; j <= N; ++j)
        off[j] = p->family_offsets ? p->family_offsets[j] : static_cast<int64_t>(j) * p->configs_per_job;
    const size_t BNNZ = static_cast<size_t>(B) * static_cast<size_t>(nnz);
    for (size_t e = 0; e < BNNZ; ++e)
        if (!std::isfinite(p->utility[e])) return ESP_ERR_NONFINITE;
    for (size_t e = 0; e < BNNZ * R; ++e) {
        const float v = p->demand[e];
        if (!std::isfinite(v)) return ESP_ERR_NONFINITE;
        if (v < 0.0f) return ESP_ERR_NEGATIVE_DEMAND;
    }
    if (p->feasible) {
        for (int b = 0; b < B; ++b)
            for (int j = 0; j < N; ++j) {
                bool any = false;
                for (int64_t e = off[j]; e < off[j + 1] && !any; ++e)
                    any = p->feasible[static_cast<size_t>(b) * nnz + e] != 0;
                if (!any) return ESP_ERR_EMPTY_FAMILY;
            }
    }
    if (pl.pen && (st = validate_penalties(B, N, nnz, off, p->current, p->switch_cost, p->penalty)) != ESP_OK)
        return st;
    // Fixed-point window per (cluster, resource): lowest set bit over the
    // column.  The highest bit plus log2(N + 1) fixes the accumulator width:
    // 64-bit when it is at most 63 for every column, 128-bit when at most 127.
    std::vector<int32_t> shift(static_cast<size_t>(B) * R, 0);
    int need_bits = 0;
    int lgN = 0;
    while ((static_cast<int64_t>(1) << lgN) < static_cast<int64_t>(N) + 1) ++lgN;
    for (int b = 0; b < B; ++b)
        for (int r = 0; r < R; ++r) {
            int lo = INT32_MAX, hi = INT32_MIN;
            const float *d = p->demand + static_cast<size_t>(b) * nnz * R + r;
            for (int64_t e = 0; e < nnz; ++e) {
                const float v = d[static_cast<size_t>(e) * R];
                if (v == 0.0f) continue;
                int l, t;
                float_bits(v, &l, &t);
                lo = std::min(lo, l);
                hi = std::max(hi, t);
            }
            if (lo == INT32_MAX) { shift[static_cast<size_t>(b) * R + r] = 0; continue; }
            if (hi - lo + lgN > 127) return ESP_ERR_RANGE;
            need_bits = std::max(need_bits, hi - lo + lgN);
            shift[static_cast<size_t>(b) * R + r] = lo;
        }

    // Resident persistent launches (ESP_MODE_RESIDENT): every wavefront of
    // the grid holds at most two tiles, and with several workgroups per
    // cluster each lane reads at most kXchPerThread exchange words (sums in
    // 48-bit limbs) per round: wavefront w of a workgroup reads workgroups
    // w, w + 4, ..., with 64 / (R limbs) lanes per limb position.
    const int limbs = std::max(1, (need_bits + 47) / 48);
    bool resident_ok = false;
    {
        const int64_t waves = static_cast<int64_t>(pl.nblk) * kBlockWaves;
        const int groups = kWaveSize / (R * limbs);
        resident_ok = static_cast<int64_t>(pl.tiles) <= 2 * waves &&
                      (pl.nblk == 1 || (groups >= 1 && pl.nblk <= kXchPerThread * kBlockWaves * groups));
    }
    if (options && options->mode == ESP_MODE_RESIDENT && !resident_ok) return ESP_ERR_SHAPE;

    // ---- workspace ----
    if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0 || workspace_bytes < pl.total)
        return ESP_ERR_WORKSPACE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    char *ws = static_cast<char *>(workspace);

    esp_ctx *c = new (std::nothrow) esp_ctx();
    if (c == nullptr) return ESP_ERR_DEVICE;
    c->pl = pl;
    {
        int dev = 0;
        if (hipGetDevice(&dev) == hipSuccess) c->scratch = resolve_scratch(dev);
    }
    c->rule = step->rule;
    c->eta0.assign(step->eta0, step->eta0 + B);
    c->ws = ws;
    c->sweep = options ? options->sweep_order : 0;
    c->mode = options ? options->mode : ESP_MODE_AUTO;
    c->auto_mode = c->mode == ESP_MODE_AUTO;
    // AUTO stays AUTO (persistent, falling back to one launch per iteration
    // when the grid cannot be co-resident) only for short passes; solves with
    // a stop tolerance use the persistent driver in any case (the loop then
    // ends on the device as soon as every cluster has converged).
    if (c->mode == ESP_MODE_AUTO &&
        static_cast<size_t>(B) * pl.columns() * pl.col_len * sizeof(float) > ESP_AUTO_PERSISTENT_BYTES)
        c->mode = ESP_MODE_STREAM;
    auto fail = [&](esp_status e) {
        if (c->h_stage) (void)hipHostFree(c->h_stage);
        if (c->stage_ev) (void)hipEventDestroy(c->stage_ev);
        delete c;
        return e;
    };
    if (hipHostMalloc(reinterpret_cast<void **>(&c->h_stage), sizeof(double) * B * kMaxR) != hipSuccess)
        return fail(ESP_ERR_DEVICE);
    if (hipEventCreateWithFlags(&c->stage_ev, hipEventDisableTiming) != hipSuccess) return fail(ESP_ERR_DEVICE);

    // ---- pack the table: one column at a time through two pinned buffers ----
    std::vector<TileMeta> meta;
    std::vector<JobSlot> jobs;
    std::vector<int64_t> slot_of(N);
    std::vector<uint32_t> dir;          // directory of the entry-major copy (copied on `s` below)
    if (pl.csr) {
        meta.assign(pl.tiles, TileMeta{});
        jobs.resize(N);
        int64_t tile = -1, fill = kTileEntries;
        for (int j = 0; j < N; ++j) {
            const int64_t k = off[j + 1] - off[j];
            if (fill + k > kTileEntries) {
                ++tile;
                fill = 0;
                meta[tile].first_job = static_cast<uint32_t>(j);
            }
            meta[tile].head[fill / 32] |= 1u << (fill % 32);
            slot_of[j] = tile * kTileEntries + fill;
            jobs[j].slot = static_cast<uint32_t>(slot_of[j]);
            jobs[j].size = static_cast<uint32_t>(k);
            fill += k;
        }
    } else {
        for (int j = 0; j < N; ++j) slot_of[j] = static_cast<int64_t>(j) * pl.K;
    }
    {
        PinnedPair pp;
        pp.cap = std::max<size_t>(pl.col_len, store_lines(kMaxFamily, kMaxR + 1) * kStoreLine / sizeof(float));   // a column, or the longest family run
        for (int i = 0; i < 2; ++i) {
            if (hipHostMalloc(reinterpret_cast<void **>(&pp.buf[i]), sizeof(float) * pp.cap) != hipSuccess)
                return fail(ESP_ERR_DEVICE);
            if (hipEventCreateWithFlags(&pp.ev[i], hipEventDisableTiming) != hipSuccess) return fail(ESP_ERR_DEVICE);
        }
        const float neg_inf = -__builtin_inff();
        const float pad_u = pl.csr ? neg_inf : 0.0f;
        int which = 0;
        const int ncol = static_cast<int>(pl.columns());
        for (int b = 0; b < B; ++b) {
            for (int a = 0; a < ncol; ++a) {
                if (pp.pending[which]) {
                    if (hipEventSynchronize(pp.ev[which]) != hipSuccess) return fail(ESP_ERR_DEVICE);
                    pp.pending[which] = false;
                }
                float *h = pp.buf[which];
                if (a == R + 1) {
                    fill_penalty_column(h, pl.col_len, b, N, nnz, off, slot_of, p->current, p->penalty);
                } else {
                    std::fill(h, h + pl.col_len, a == 0 ? pad_u : 0.0f);
                    const float *u = p->utility + static_cast<size_t>(b) * nnz;
                    const float *d = p->demand + static_cast<size_t>(b) * nnz * R + (a - 1);
                    const uint8_t *f = p->feasible ? p->feasible + static_cast<size_t>(b) * nnz : nullptr;
                    for (int j = 0; j < N; ++j) {
                        const int64_t e0 = off[j], k = off[j + 1] - off[j];
                        float *dst = h + slot_of[j];
                        if (a == 0) {
                            for (int64_t i = 0; i < k; ++i)
                                dst[i] = (f && f[e0 + i] == 0) ? neg_inf : u[e0 + i];
                        } else {
                            for (int64_t i = 0; i < k; ++i) {
                                const float v = d[static_cast<size_t>(e0 + i) * R];
                                dst[i] = (v == 0.0f) ? 0.0f : v;     // -0.0 -> +0.0
                            }
                        }
                    }
                }
                float *dcol = reinterpret_cast<float *>(ws + pl.o_table) +
                              (static_cast<size_t>(b) * ncol + a) * pl.col_len;
                if (hipMemcpyAsync(dcol, h, sizeof(float) * pl.col_len, hipMemcpyHostToDevice, s) != hipSuccess ||
                    hipEventRecord(pp.ev[which], s) != hipSuccess)
                    return fail(ESP_ERR_DEVICE);
                pp.pending[which] = true;
                which ^= 1;
            }
        }
        // Entry-major copy (ESP_OPT_PROFILE_STORE): family j of cluster b is a
        // run of slots of 1 + R floats (the utility, -inf when masked, then
        // the R demands) starting on a kStoreLine-byte line; the slots after
        // its last configuration, up to the end of its last line, are masked
        // entries.  Whole families are staged, then copied.
        if (pl.aos_stride > 0) {
            const size_t st = static_cast<size_t>(pl.aos_stride);
            constexpr size_t kLineFloats = kStoreLine / sizeof(float);
            float *dst0 = reinterpret_cast<float *>(ws + pl.o_aos);
            float *h = nullptr;
            size_t n = 0, out = 0;                      // floats staged in h; floats of the copy written
            auto flush = [&]() -> bool {
                if (n > 0) {
                    if (hipMemcpyAsync(dst0 + out, h, sizeof(float) * n, hipMemcpyHostToDevice, s) != hipSuccess ||
                        hipEventRecord(pp.ev[which], s) != hipSuccess)
                        return false;
                    pp.pending[which] = true;
                    which ^= 1;
                    out += n;
                }
                h = nullptr;
                n = 0;
                return true;
            };
            for (int b = 0; b < B; ++b) {
                const float *u = p->utility + static_cast<size_t>(b) * nnz;
                const float *d = p->demand + static_cast<size_t>(b) * nnz * R;
                const uint8_t *f = p->feasible ? p->feasible + static_cast<size_t>(b) * nnz : nullptr;
                for (int j = 0; j < N; ++j) {
                    const int64_t e0 = off[j], k = off[j + 1] - off[j];
                    const size_t fl = static_cast<size_t>(store_lines(k, pl.aos_stride)) * kLineFloats;
                    if (h != nullptr && n + fl > pp.cap && !flush()) return fail(ESP_ERR_DEVICE);
                    if (h == nullptr) {
                        if (pp.pending[which]) {
                            if (hipEventSynchronize(pp.ev[which]) != hipSuccess) return fail(ESP_ERR_DEVICE);
                            pp.pending[which] = false;
                        }
                        h = pp.buf[which];
                    }
                    float *run = h + n;
                    std::fill(run, run + fl, 0.0f);
                    for (size_t i = 0; i < fl / st; ++i) {
                        float *slot = run + i * st;
                        if (static_cast<int64_t>(i) >= k) {
                            slot[0] = neg_inf;
                            continue;
                        }
                        const size_t e = static_cast<size_t>(e0) + i;
                        slot[0] = (f && f[e] == 0) ? neg_inf : u[e];
                        for (int r = 0; r < R; ++r) {
                            const float v = d[e * R + r];
                            slot[1 + r] = (v == 0.0f) ? 0.0f : v;     // -0.0 -> +0.0
                        }
                    }
                    n += fl;
                }
                if (!flush()) return fail(ESP_ERR_DEVICE);
            }
            // directory: first line of each group of kDirFamilies families, then
            // each family's size - 1 (1..kMaxFamily configurations) in a byte
            dir.assign(static_cast<size_t>(dir_records(N)) * kDirWords, 0u);
            int64_t line = 0;
            for (int j = 0; j < N; ++j) {
                const int64_t k = off[j + 1] - off[j];
                uint32_t *rec = dir.data() + static_cast<size_t>(j / kDirFamilies) * kDirWords;
                const int i = j % kDirFamilies;
                if (i == 0) rec[0] = static_cast<uint32_t>(line);
                rec[1 + i / 4] |= static_cast<uint32_t>(k - 1) << (8 * (i % 4));
                line += store_lines(k, pl.aos_stride);
            }
        }
        std::vector<double> cap(p->capacity, p->capacity + static_cast<size_t>(B) * R);
        std::vector<double> swc(B, 0.0);
        if (p->switch_cost) swc.assign(p->switch_cost, p->switch_cost + B);
        bool ok = hipMemcpyAsync(ws + pl.o_shift, shift.data(), sizeof(int32_t) * shift.size(),
                                 hipMemcpyHostToDevice, s) == hipSuccess &&
                  hipMemcpyAsync(ws + pl.o_cap, cap.data(), sizeof(double) * cap.size(), hipMemcpyHostToDevice, s) ==
                      hipSuccess &&
                  hipMemcpyAsync(ws + pl.o_capp, cap.data(), sizeof(double) * cap.size(), hipMemcpyHostToDevice,
                                 s) == hipSuccess &&
                  hipMemcpyAsync(ws + pl.o_eta, c->eta0.data(), sizeof(double) * B, hipMemcpyHostToDevice, s) ==
                      hipSuccess &&
                  hipMemsetAsync(ws + pl.o_tick, 0, sizeof(uint32_t) * B, s) == hipSuccess &&
                  hipMemsetAsync(ws + pl.o_flags, 0, sizeof(int32_t) * B, s) == hipSuccess &&
                  hipMemsetAsync(ws + pl.o_iters, 0, sizeof(int32_t) * B, s) == hipSuccess &&
                  hipMemsetAsync(ws + pl.o_sync, 0, sizeof(uint32_t) * B * kSyncSlots * kSyncStride, s) == hipSuccess &&
                  hipMemsetAsync(ws + pl.o_conv, 0, sizeof(int32_t) * B, s) == hipSuccess &&
                  hipMemcpyAsync(ws + pl.o_swc, swc.data(), sizeof(double) * B, hipMemcpyHostToDevice, s) ==
                      hipSuccess &&
                  hipMemsetAsync(ws + pl.o_status, 0, sizeof(int32_t), s) == hipSuccess &&
                  hipMemcpyAsync(ws + pl.o_offs, off.data(), sizeof(int64_t) * off.size(), hipMemcpyHostToDevice,
                                 s) == hipSuccess &&
                  hipMemsetAsync(ws + pl.o_inc, 0, sizeof(uint64_t) * static_cast<size_t>(B) * N, s) == hipSuccess;
        if (ok && !dir.empty())
            ok = hipMemcpyAsync(ws + pl.o_dir, dir.data(), sizeof(uint32_t) * dir.size(), hipMemcpyHostToDevice,
                                s) == hipSuccess;
        if (ok && pl.csr)
            ok = hipMemcpyAsync(ws + pl.o_meta, meta.data(), sizeof(TileMeta) * meta.size(), hipMemcpyHostToDevice,
                                s) == hipSuccess &&
                 hipMemcpyAsync(ws + pl.o_jobs, jobs.data(), sizeof(JobSlot) * jobs.size(), hipMemcpyHostToDevice,
                                s) == hipSuccess;
        if (!ok || hipStreamSynchronize(s) != hipSuccess) return fail(ESP_ERR_DEVICE);
        pp.pending[0] = pp.pending[1] = false;
    }

    c->off = std::move(off);
    c->slot_of = std::move(slot_of);
    KArgs &k = c->base;
    k.table = reinterpret_cast<const float *>(ws + pl.o_table);
    k.cluster_stride = pl.columns() * pl.col_len;
    k.has_pen = pl.pen ? 1 : 0;
    k.switch_cost = reinterpret_cast<const double *>(ws + pl.o_swc);
    k.col_len = pl.col_len;
    k.meta = pl.csr ? reinterpret_cast<const TileMeta *>(ws + pl.o_meta) : nullptr;
    k.jobs = pl.csr ? reinterpret_cast<const JobSlot *>(ws + pl.o_jobs) : nullptr;
    k.N = N;
    k.K = pl.csr ? 0 : pl.K;
    k.tiles = pl.tiles;
    k.nblk = pl.nblk;
    k.cap = reinterpret_cast<const double *>(ws + pl.o_cap);
    k.eta0 = reinterpret_cast<const double *>(ws + pl.o_eta);
    k.rule = c->rule == ESP_STEP_INV_SQRT ? 1 : 0;
    k.t = 1;
    k.shift = reinterpret_cast<const int32_t *>(ws + pl.o_shift);
    k.partials = reinterpret_cast<uint64_t *>(ws + pl.o_part);
    k.tickets = reinterpret_cast<uint32_t *>(ws + pl.o_tick);
    k.flags = reinterpret_cast<int32_t *>(ws + pl.o_flags);
    k.status = reinterpret_cast<int32_t *>(ws + pl.o_status);
    k.skip_mask = kFlagError;
    k.acc128 = need_bits > 63 ? 1 : 0;
    k.n_iters = 1;
    k.B = B;
    k.sync = reinterpret_cast<uint32_t *>(ws + pl.o_sync);
    k.lam_ws = reinterpret_cast<double *>(ws + pl.o_lamws);
    k.conv_at = reinterpret_cast<int32_t *>(ws + pl.o_conv);
    k.sweep_alt = c->sweep == 0 ? 1 : 0;
    k.limbs = limbs;
    k.xch_stride = R * limbs;
    k.xch = reinterpret_cast<uint64_t *>(ws + pl.o_xch);
    k.xch_clear = 0;
    c->resident_ok = resident_ok;
    *out = c;
    return ESP_OK;
}

esp_status esp_score_select(esp_ctx *c, const double *prices, int32_t *choice, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (prices == nullptr || choice == nullptr) return ESP_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    KArgs p = c->base;
    p.iters_done = nullptr;
    if ((st = dev(launch_prepare(c->pl.R, p, prices, nullptr, c->pl.B, s))) != ESP_OK) return st;
    KArgs a = c->base;
    a.lam_in = prices;
    a.choice = choice;
    a.reduce = 0;
    a.skip_mask = kFlagError;
    return dev(launch_select(c, a, s));
}

esp_status esp_reduce_demand(esp_ctx *c, const int32_t *choice, double *demand, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (choice == nullptr || demand == nullptr) return ESP_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    KArgs a = c->base;
    a.choice_in = choice;
    a.demand_out = demand;
    a.skip_mask = 0;
    a.reduce = 1;
    return dev(launch_gather(c->pl.R, a, c->pl.B, s));
}

esp_status esp_update_prices(esp_ctx *c, const double *demand, int32_t t, double *prices, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (demand == nullptr || prices == nullptr || t < 1) return ESP_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    KArgs a = c->base;
    a.t = t;
    a.lam_in = prices;
    a.lam_out = prices;
    return dev(launch_update(c->pl.R, a, demand, c->pl.B, s));
}

esp_status esp_solve(esp_ctx *c, double *prices, int32_t iters, int32_t t_start, double tol, int32_t *choice,
                     double *demand, const esp_trace *trace, int32_t *iters_done, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    return solve_with(c, c->base, reinterpret_cast<int32_t *>(c->ws + c->pl.o_iters), prices, iters, t_start, tol,
                      choice, demand, trace, iters_done, stream);
}

esp_status esp_solve_noalloc(esp_ctx *c, double *prices, int32_t iters, int32_t t_start, double tol,
                             int32_t *choice, double *demand, const esp_trace *trace, int32_t *iters_done,
                             void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    const ScratchLayout L = scratch_layout(c->pl);
    if (L.total > ESP_NOALLOC_SCRATCH_BYTES) return ESP_ERR_WORKSPACE;
    if (c->scratch == nullptr) return ESP_ERR_DEVICE;
    KArgs k = c->base;
    k.partials = reinterpret_cast<uint64_t *>(c->scratch + L.part);
    k.tickets = reinterpret_cast<uint32_t *>(c->scratch + L.tick);
    k.sync = reinterpret_cast<uint32_t *>(c->scratch + L.sync);
    k.lam_ws = reinterpret_cast<double *>(c->scratch + L.lamws);
    k.conv_at = reinterpret_cast<int32_t *>(c->scratch + L.conv);
    k.xch = reinterpret_cast<uint64_t *>(c->scratch + L.xch);
    return solve_with(c, k, reinterpret_cast<int32_t *>(c->scratch + L.iters), prices, iters, t_start, tol, choice,
                      demand, trace, iters_done, stream);
}

esp_status esp_set_penalties(esp_ctx *c, const int32_t *current, const double *switch_cost, const float *penalty,
                             void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (!c->pl.pen) return ESP_ERR_STATE;
    const Plan &pl = c->pl;
    if ((st = validate_penalties(pl.B, pl.N, pl.nnz, c->off, current, switch_cost, penalty)) != ESP_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    float *h = nullptr;
    if (hipHostMalloc(reinterpret_cast<void **>(&h), sizeof(float) * pl.col_len) != hipSuccess) return ESP_ERR_DEVICE;
    const size_t ncol = pl.columns();
    for (int b = 0; b < pl.B && st == ESP_OK; ++b) {
        // the previous copy out of h must be done before h is refilled
        if (hipStreamSynchronize(s) != hipSuccess) { st = ESP_ERR_DEVICE; break; }
        fill_penalty_column(h, pl.col_len, b, pl.N, pl.nnz, c->off, c->slot_of, current, penalty);
        float *dcol = reinterpret_cast<float *>(c->ws + pl.o_table) + (static_cast<size_t>(b) * ncol + pl.R + 1) * pl.col_len;
        if (hipMemcpyAsync(dcol, h, sizeof(float) * pl.col_len, hipMemcpyHostToDevice, s) != hipSuccess)
            st = ESP_ERR_DEVICE;
    }
    std::vector<double> swc(pl.B, 0.0);
    if (switch_cost) swc.assign(switch_cost, switch_cost + pl.B);
    if (st == ESP_OK &&
        (hipMemcpyAsync(c->ws + pl.o_swc, swc.data(), sizeof(double) * pl.B, hipMemcpyHostToDevice, s) != hipSuccess ||
         hipStreamSynchronize(s) != hipSuccess))
        st = ESP_ERR_DEVICE;
    (void)hipHostFree(h);
    return st;
}

esp_status esp_device_status(esp_ctx *c, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (hipStreamSynchronize(s) != hipSuccess) return ESP_ERR_DEVICE;
    int32_t v = 0, zero = 0;
    int32_t *d = reinterpret_cast<int32_t *>(c->ws + c->pl.o_status);
    if (hipMemcpy(&v, d, sizeof(v), hipMemcpyDeviceToHost) != hipSuccess) return ESP_ERR_DEVICE;
    if (hipMemcpy(d, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess) return ESP_ERR_DEVICE;
    return static_cast<esp_status>(v);
}

esp_status esp_set_capacity(esp_ctx *c, const double *capacity, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (capacity == nullptr) return ESP_ERR_INVALID_ARG;
    const size_t n = static_cast<size_t>(c->pl.B) * c->pl.R;
    for (size_t i = 0; i < n; ++i) {
        if (!std::isfinite(capacity[i])) return ESP_ERR_NONFINITE;
        if (std::fabs(capacity[i]) > 0x1p200) return ESP_ERR_RANGE;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    // Stage through the pinned buffer (B * kMaxR doubles).
    if ((st = stage_wait(c)) != ESP_OK) return st;
    std::memcpy(c->h_stage, capacity, sizeof(double) * n);
    if (hipMemcpyAsync(c->ws + c->pl.o_capp, c->h_stage, sizeof(double) * n, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipMemcpyAsync(c->ws + c->pl.o_cap, c->ws + c->pl.o_capp, sizeof(double) * n, hipMemcpyDeviceToDevice, s) !=
            hipSuccess ||
        hipEventRecord(c->stage_ev, s) != hipSuccess)
        return ESP_ERR_DEVICE;
    c->stage_pending = true;
    return ESP_OK;
}

esp_status esp_effective_capacity(esp_ctx *c, esp_ctx *queue, const uint8_t *queued, double gamma,
                                  double *capacity_eff, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (queue != nullptr && (st = check_ctx(queue)) != ESP_OK) return st;
    if (!(gamma >= 0.0 && gamma <= 1.0)) return ESP_ERR_INVALID_ARG;     // also rejects NaN
    if (queue != nullptr && (queue->pl.B != c->pl.B || queue->pl.R != c->pl.R)) return ESP_ERR_SHAPE;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int B = c->pl.B, R = c->pl.R;
    double *cap = reinterpret_cast<double *>(c->ws + c->pl.o_cap);
    const double *capp = reinterpret_cast<const double *>(c->ws + c->pl.o_capp);
    if (queue == nullptr) {
        // No pending jobs: C_eff = C.
        const size_t bytes = sizeof(double) * B * R;
        if (hipMemcpyAsync(cap, capp, bytes, hipMemcpyDeviceToDevice, s) != hipSuccess) return ESP_ERR_DEVICE;
        if (capacity_eff && hipMemcpyAsync(capacity_eff, capp, bytes, hipMemcpyDeviceToDevice, s) != hipSuccess)
            return ESP_ERR_DEVICE;
        return ESP_OK;
    }
    ReserveArgs ra;
    ra.queued = queued;
    ra.cap_phys = capp;
    ra.cap_eff = cap;
    ra.out = capacity_eff;
    ra.gamma = gamma;
    return dev(launch_reserve(R, queue->base, ra, B, s));
}

esp_status esp_nearest_profile(esp_ctx *store, int32_t num_queries, const int32_t *family, const float *query,
                               int32_t *nearest, float *estimate, void *stream) {
    esp_status st = check_ctx(store);
    if (st != ESP_OK) return st;
    if (num_queries < 0) return ESP_ERR_INVALID_ARG;
    if (num_queries == 0) return ESP_OK;
    if (family == nullptr || query == nullptr || nearest == nullptr) return ESP_ERR_INVALID_ARG;
    NearestArgs na;
    na.family = family;
    na.query = query;
    na.nearest = nearest;
    na.estimate = estimate;
    na.total = static_cast<int64_t>(store->pl.B) * num_queries;
    na.Q = num_queries;
    const Plan &pl = store->pl;
    na.aos = pl.aos_stride > 0 ? reinterpret_cast<const float *>(store->ws + pl.o_aos) : nullptr;
    na.dir = reinterpret_cast<const uint32_t *>(store->ws + pl.o_dir);
    na.aos_lines = pl.aos_lines;
    na.aos_stride = pl.aos_stride;
    return dev(launch_nearest(store->pl.R, store->base, na, static_cast<hipStream_t>(stream)));
}

esp_status esp_schedule(esp_ctx *c, const esp_iac_model *m, int32_t max_rounds, int32_t iters, double tol,
                        double *prices, int32_t *choice, int32_t *gpu_jobs, int32_t *rounds_used, int32_t *violations,
                        void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (!c->pl.pen) return ESP_ERR_STATE;                 // needs the penalty column
    if (m == nullptr || m->gpus == nullptr || m->sensitivity == nullptr || m->pressure == nullptr ||
        m->tau_base == nullptr || prices == nullptr || choice == nullptr || gpu_jobs == nullptr ||
        rounds_used == nullptr || violations == nullptr)
        return ESP_ERR_INVALID_ARG;
    const int B = c->pl.B, R = c->pl.R;
    if (max_rounds < 1 || iters < 0) return ESP_ERR_INVALID_ARG;
    if (m->r_gpus < 0 || m->r_gpus >= R || m->r_mem < 0 || m->r_mem >= R || m->r_sm < 0 || m->r_sm >= R)
        return ESP_ERR_INVALID_ARG;
    const double vals[] = {m->gpu_memory, m->gpu_compute, m->beta, m->beta_max, m->u_target, m->kappa};
    for (double v : vals)
        if (!std::isfinite(v)) return ESP_ERR_NONFINITE;
    if (m->gpu_memory < 0.0 || m->gpu_compute < 0.0 || !(m->u_target > 0.0) || m->kappa < 0.0)
        return ESP_ERR_INVALID_ARG;
    int gmax = 0;
    for (int b = 0; b < B; ++b) {
        if (m->gpus[b] < 1 || m->gpus[b] > ESP_MAX_GPUS) return ESP_ERR_INVALID_ARG;
        gmax = std::max(gmax, m->gpus[b]);
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    // The pinned staging buffer carries the GPU counts and reads back the
    // violation counts between rounds (B * kMaxR doubles >= B int32).
    if ((st = stage_wait(c)) != ESP_OK) return st;
    int32_t *h32 = reinterpret_cast<int32_t *>(c->h_stage);
    std::memcpy(h32, m->gpus, sizeof(int32_t) * B);
    int32_t *d_gpus = reinterpret_cast<int32_t *>(c->ws + c->pl.o_gpus);
    if (hipMemcpyAsync(d_gpus, h32, sizeof(int32_t) * B, hipMemcpyHostToDevice, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
        return ESP_ERR_DEVICE;
    IacArgs ia;
    ia.choice = choice;
    ia.offsets = reinterpret_cast<const int64_t *>(c->ws + c->pl.o_offs);
    ia.nnz = c->pl.nnz;
    ia.gpus = d_gpus;
    ia.gpu_memory = m->gpu_memory;
    ia.gpu_compute = m->gpu_compute;
    ia.r_gpus = m->r_gpus;
    ia.r_mem = m->r_mem;
    ia.r_sm = m->r_sm;
    ia.sensitivity = m->sensitivity;
    ia.pressure = m->pressure;
    ia.tau_base = m->tau_base;
    ia.beta = m->beta;
    ia.beta_max = m->beta_max;
    ia.u_target = m->u_target;
    ia.kappa = m->kappa;
    ia.inc = reinterpret_cast<uint64_t *>(c->ws + c->pl.o_inc);
    ia.gpu_jobs = gpu_jobs;
    ia.gmax = gmax;
    ia.rounds_used = rounds_used;
    ia.violations = violations;
    // Alg. 1: Gamma <- 0, no cluster frozen
    if ((st = dev(launch_iac_reset(R, c->base, B, 1, s))) != ESP_OK) return st;
    for (int32_t r = 1; r <= max_rounds; ++r) {
        if ((st = esp_solve(c, prices, iters, 1, tol, choice, nullptr, nullptr, nullptr, stream)) != ESP_OK) break;
        ia.round = r;
        if ((st = dev(launch_pack_iac(R, c->base, ia, B, s))) != ESP_OK) break;
        if (r == max_rounds) break;
        // stop early once every cluster is free of violations
        if (hipMemcpyAsync(h32, violations, sizeof(int32_t) * B, hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess) {
            st = ESP_ERR_DEVICE;
            break;
        }
        bool any = false;
        for (int b = 0; b < B; ++b) any = any || h32[b] != 0;
        if (!any) break;
    }
    const esp_status st2 = dev(launch_iac_reset(R, c->base, B, 0, s));
    return st != ESP_OK ? st : st2;
}

esp_status esp_read_penalties(esp_ctx *c, float *penalty, void *stream) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (!c->pl.pen) return ESP_ERR_STATE;
    if (penalty == nullptr) return ESP_ERR_INVALID_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const size_t col_len = c->pl.col_len, ncol = c->pl.columns();
    std::vector<float> h(col_len);
    const int B = c->pl.B, N = c->pl.N;
    const int64_t nnz = c->pl.nnz;
    for (int b = 0; b < B; ++b) {
        const float *d = reinterpret_cast<const float *>(c->ws + c->pl.o_table) +
                         (static_cast<size_t>(b) * ncol + c->pl.R + 1) * col_len;
        if (hipMemcpyAsync(h.data(), d, sizeof(float) * col_len, hipMemcpyDeviceToHost, s) != hipSuccess ||
            hipStreamSynchronize(s) != hipSuccess)
            return ESP_ERR_DEVICE;
        for (int j = 0; j < N; ++j)
            for (int64_t i = 0; i < c->off[j + 1] - c->off[j]; ++i)
                penalty[static_cast<size_t>(b) * nnz + c->off[j] + i] = std::fabs(h[c->slot_of[j] + i]);
    }
    return ESP_OK;
}

esp_status esp_loop_driver(const esp_ctx *c, int32_t *mode) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (mode == nullptr) return ESP_ERR_INVALID_ARG;
    if (c->mode == ESP_MODE_STREAM || c->fell_back) *mode = ESP_MODE_STREAM;
    else if (c->mode == ESP_MODE_RESIDENT || (c->auto_mode && c->resident_ok)) *mode = ESP_MODE_RESIDENT;
    else *mode = ESP_MODE_PERSISTENT;
    return ESP_OK;
}

esp_status esp_destroy(esp_ctx *c) {
    esp_status st = check_ctx(c);
    if (st != ESP_OK) return st;
    if (c->stage_pending) (void)hipEventSynchronize(c->stage_ev);
    if (c->stage_ev) (void)hipEventDestroy(c->stage_ev);
    if (c->h_stage) (void)hipHostFree(c->h_stage);
    c->magic = 0;
    delete c;
    return ESP_OK;
}

}  // extern "C"
