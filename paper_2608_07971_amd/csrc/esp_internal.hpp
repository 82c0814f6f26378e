// Internal definitions shared by the host driver and the gfx950 kernels of the
// Elastic Shadow Pricing library.  Not part of the public ABI (include/esp.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace esp {

// A tile is what one wavefront scores per step: 64 lanes x 4 table entries,
// read with one 128-bit load per lane per column.
constexpr int kTileEntries = 256;
constexpr int kWaveSize = 64;
constexpr int kBlockThreads = 256;                  // 4 wavefronts per workgroup
constexpr int kBlockWaves = kBlockThreads / kWaveSize;
constexpr int kMaxR = 8;
constexpr int kMaxFamily = 256;                     // configurations per job
constexpr int kLaunchChunk = 1024;                  // iterations per persistent launch
constexpr int kColumnPadTiles = 7;                  // unused tiles at the end of every column
// Barrier words of a cluster in a persistent deferred launch, each in its own
// 256-byte line: arrival counters of kSyncGroups groups of workgroups (blk mod
// kSyncGroups), the count of complete groups, and one release word per group.
constexpr int kSyncGroups = 8;
constexpr int kSyncSlots = 2 * kSyncGroups + 1;
constexpr int kSyncStride = 64;                     // uint32 words between barrier words
// Buffers of per-workgroup sums: 0 and 1 hold the sums of solve iterations by
// iteration parity (deferred completion), 2 those of in-launch completion.
constexpr int kPartialBuffers = 3;
constexpr int kInLaunchBuffer = 2;
// Resident launches with several workgroups per cluster exchange their sums
// as limbs of 48 bits (at most 3 for 127-bit sums) in tagged 64-bit words;
// each thread of a workgroup reads at most kXchPerThread words per round.
constexpr int kMaxLimbs = 3;
constexpr int kXchPerThread = 8;

// Flags per cluster (device int32).
constexpr int kFlagStopped = 1;                     // converged under tol: skip further updates
constexpr int kFlagError = 2;                       // invalid prices: skip everything
constexpr int kFlagFrozen = 8;                      // outer rounds: the cluster's schedule is final

// Device status codes (mirror esp_status values).
constexpr int kStatusNonfinite = 3;
constexpr int kStatusInvalid = 1;
constexpr int kStatusRange = 7;

// Tile metadata of the CSR layout: bit i of `head` is set when table slot i of
// the tile starts a job; `first_job` is the job owning slot 0.
struct TileMeta {
    uint32_t head[8];
    uint32_t first_job;
    uint32_t pad[7];
};
static_assert(sizeof(TileMeta) == 64, "tile metadata is one 64-byte line");

// Where job j's family starts in its cluster's columns, and its size.
struct JobSlot {
    uint32_t slot;
    uint32_t size;
};

// Arguments of the select/demand/update kernels (passed by value).
struct KArgs {
    const float *table;            // SoA image: cluster b, column a (0 = utility, 1+r = demand r)
                                   // starts at table + b * cluster_stride + a * col_len
    size_t cluster_stride;         // floats between clusters = (R + 1) * col_len
    size_t col_len;                // floats per column = tiles * 256
    const TileMeta *meta;          // CSR only: [tiles]
    const JobSlot *jobs;           // [N] slot of each family (used by the gather kernel)
    int32_t N;                     // jobs per cluster
    int32_t K;                     // dense family size (0 for CSR)
    int32_t tiles;                 // tiles per cluster
    int32_t nblk;                  // workgroups per cluster
    const double *lam_in;          // [B][R] prices at which to select
    double *lam_out;               // [B][R] updated prices, or NULL (no update)
    const double *cap;             // [B][R] capacities
    const double *eta0;            // [B] step-size scale eta0 of Eq. 8
    int32_t rule;                  // 0: eta_t = eta0, 1: eta_t = eta0 / sqrt(t)
    int32_t t;                     // step index t (1-based) of the launch's first iteration
    const int32_t *shift;          // [B][R] fixed-point window (lowest bit exponent) per column
    uint64_t *partials;            // [kPartialBuffers][B][nblk][R][2] per-workgroup 128-bit sums
    uint32_t *tickets;             // [B] arrival counters (0 between launches)
    int32_t *flags;                // [B] per-cluster run flags
    int32_t skip_mask;             // skip a cluster when (flags[b] & skip_mask) != 0
    int32_t *status;               // first device-detected error
    int32_t *choice;               // [B][N] output, or NULL
    const int32_t *choice_in;      // [B][N] input of the gather kernel
    double *demand_out;            // [B][R] output U, or NULL
    double *tr_lam;                // [B][R] trace row for lambda^{t+1}, or NULL
    double *tr_U;                  // [B][R] trace row for U^t, or NULL
    int32_t *iters_done;           // [B] or NULL
    int32_t iter_no;               // updates made including this one (1-based)
    double tol;                    // > 0 enables the stop test
    int32_t reduce;                // 0: select only (no demand, no ticket)
    int32_t reverse;               // sweep tiles back to front (iteration 0 of the launch)
    int32_t acc128;                // demand accumulators are 128-bit (else 64-bit)
    // Persistent launches run n_iters iterations; t, rows of the traces and the
    // per-iteration choice advance by B, B*R and B*N per iteration, and the
    // sweep direction alternates.
    int32_t n_iters;               // 1 for a single-iteration launch
    int32_t B;                     // clusters
    uint32_t *sync;                // [B][kSyncSlots][kSyncStride] barrier words of persistent
                                   // deferred launches (reset per solve)
    int32_t sweep_alt;             // alternate the sweep direction between iterations
    // Penalty of the ESP score (Eq. 7): column R + 1 of each cluster holds
    // |penalty| per entry, its sign bit set when the entry is not the job's
    // current configuration (the switching cost switch_cost[b] applies).
    int32_t has_pen;
    const double *switch_cost;     // [B]
    // Deferred completion of solve iterations (several workgroups per
    // cluster).  Iteration m (1-based within the solve: iter_no) publishes the
    // workgroup sums into partials buffer m & 1 and ends there.  U_m,
    // lambda_{m+1} and the stop test are computed by every workgroup of the
    // cluster from those sums when iteration m + 1 (or the closing launch)
    // starts.  The sums are integers, so every workgroup obtains the same
    // bits; workgroup 0 writes the outputs.
    int32_t defer;                 // this launch's iterations publish their sums only
    int32_t pend_m;                // > 0: first complete iteration pend_m of the solve
    int32_t pend_t;                // its step index t
    double *lam_ws;                // [2][B][R] lambda_m of iteration m at index m & 1
    double *lam_dst;               // [B][R] the caller's prices: receives every lambda_{m+1}
    int32_t *conv_at;              // [B] iteration whose completion met tol, 0 while none has
    double *trace_lam;             // [iters][B][R]: row m - 1 receives lambda_{m+1}, or NULL
    double *trace_U;               // [iters][B][R]: row m - 1 receives U_m, or NULL
    // Resident launches (tiles held in registers, every iteration completed
    // in the launch): tagged exchange words [2][B][nblk][xch_stride].
    uint64_t *xch;
    int32_t xch_stride;            // words per workgroup = R * limbs
    int32_t limbs;                 // 48-bit limbs per workgroup sum
    size_t xch_clear;              // words k_prepare sets to 0 before a resident solve (0: none)
};

constexpr int kStatusTimeout = 8;  // a persistent wait exceeded its bound

// Host-side launchers (esp_kernels.hip).
hipError_t launch_dense(int R, int lpj, const KArgs &a, int B, hipStream_t s);
// Cooperative launch (all workgroups co-resident) of a multi-iteration dense
// launch.  A grid the device cannot hold co-resident is refused on the host
// (hipErrorCooperativeLaunchTooLarge) before anything is enqueued.
hipError_t launch_dense_persistent(int R, int lpj, const KArgs &a, int B, hipStream_t s);
hipError_t launch_csr(int R, const KArgs &a, int B, hipStream_t s);
hipError_t launch_csr_persistent(int R, const KArgs &a, int B, hipStream_t s);
// Multi-iteration launches over register-resident tiles (at most two per
// wavefront), each iteration completed in the launch (see kResident).
hipError_t launch_dense_resident(int R, int lpj, const KArgs &a, int B, hipStream_t s);
hipError_t launch_csr_resident(int R, const KArgs &a, int B, hipStream_t s);
hipError_t launch_gather(int R, const KArgs &a, int B, hipStream_t s);
hipError_t launch_update(int R, const KArgs &a, const double *demand_in, int B, hipStream_t s);
// Validates prices `lam`; `canon` (NULL or the same buffer, writable) receives
// +0.0 in place of -0.0.
hipError_t launch_prepare(int R, const KArgs &a, const double *lam, double *canon, int B, hipStream_t s);
// Closing launch of a deferred solve: completes its last iteration (no selection).
hipError_t launch_finish(int R, const KArgs &a, int B, hipStream_t s);

}  // namespace esp
