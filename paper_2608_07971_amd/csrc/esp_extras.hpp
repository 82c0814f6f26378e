// Kernels beyond the price loop (Sec. 3.1.2, 3.4): effective capacity,
// outer ESP-IAC rounds, nearest-profile fallback.  Argument blocks and
// host-side launchers (esp_extras.hip).
#pragma once

#include "esp_internal.hpp"

namespace esp {

// Extra arguments of the effective-capacity kernel (Eq. 12): the KArgs of the
// pending jobs' context supply the table, the fixed-point windows and the
// cross-workgroup sum buffers.
struct ReserveArgs {
    const uint8_t *queued;         // [B][N] nonzero = pending, or NULL (all pending)
    const double *cap_phys;        // [B][R] physical capacity C
    double *cap_eff;               // [B][R] receives C - gamma * S (the active context's capacity)
    double *out;                   // [B][R] copy for the caller, or NULL
    double gamma;                  // reservation aggressiveness in [0, 1]
};

// Arguments of the nearest-profile kernel (RST fallback): queries against
// the families of a store context (its KArgs supply the table).
struct NearestArgs {
    const int32_t *family;         // [B][Q] job type (family index) of each query
    const float *query;            // [B][Q][R] resource vectors
    int32_t *nearest;              // [B][Q] index within the family, -1 on error
    float *estimate;               // [B][Q] utility (throughput) of the nearest entry, or NULL
    int64_t total;                 // B * Q
    int32_t Q;                     // queries per cluster
    int64_t chunk;                 // queries per workgroup (set by the launcher)
    // Entry-major copy of the store (ESP_OPT_PROFILE_STORE), or NULL.  Each
    // family is a run of slots of aos_stride floats (utility first, then the
    // R demands; slot k = configuration k of the family) that starts on a
    // kStoreLine-byte line; the slots after the family's last configuration,
    // up to the end of its last line, hold masked entries (utility -inf, zero
    // demands).  Cluster b's copy starts aos_lines lines after cluster b-1's.
    const float *aos;
    // Directory of the runs, shared by all clusters: one record of kDirWords
    // words per kDirFamilies consecutive families.  Word 0 is the first line
    // of the record's first family; family kDirFamilies g + i stores its size
    // minus one at byte i of words 1..15 (byte i % 4 of word 1 + i / 4); its
    // run takes ceil(size * 4 (1 + R) / kStoreLine) lines.
    const uint32_t *dir;
    int64_t aos_lines;             // lines per cluster
    int32_t aos_stride;            // floats per entry: 1 + R
};

constexpr int kStoreLine = 128;                     // bytes: the L2 line of gfx950
constexpr int kDirWords = 16;                       // one 64-byte record
constexpr int kDirFamilies = 4 * (kDirWords - 1);   // 60 sizes of one byte
static_assert(kMaxFamily <= 256, "family sizes minus one fit a byte");

// Outer ESP-IAC rounds (Alg. 1): one wavefront per cluster packs the
// selection onto GPUs (first fit), evaluates co-located pairs and raises the
// penalties of offending configurations.
constexpr int kMaxGpus = 2048;                      // GPUs per cluster (LDS-resident residuals)
constexpr int kMaxPerGpu = 4;                       // jobs sharing one GPU
constexpr int kMaxShards = 8;                       // GPUs of one job

struct IacArgs {
    const int32_t *choice;         // [B][N] selection of this round
    const int64_t *offsets;        // [N+1] entry offsets of the caller's [B][nnz] arrays
    int64_t nnz;
    const int32_t *gpus;           // [B] GPUs per cluster
    double gpu_memory;             // per-GPU capacity of resource r_mem
    double gpu_compute;            // per-GPU capacity of resource r_sm
    int32_t r_gpus, r_mem, r_sm;
    const float *sensitivity;      // [B][nnz]
    const float *pressure;         // [B][nnz]
    const double *tau_base;        // [B][N]
    double beta, beta_max, u_target, kappa;
    uint64_t *inc;                 // [B][N] scratch, zero between rounds (bits of doubles >= 0)
    int32_t *gpu_jobs;             // [B][gmax][kMaxPerGpu] out
    int32_t gmax;
    int32_t *rounds_used;          // [B] out
    int32_t *violations;           // [B] out
    int32_t round;                 // 1-based
};


hipError_t launch_nearest(int R, const KArgs &a, const NearestArgs &na, hipStream_t s);
hipError_t launch_pack_iac(int R, const KArgs &a, const IacArgs &m, int B, hipStream_t s);
// Gamma <- 0 (interference penalties; the switching-cost marks stay) when
// zero_gamma, and clear the frozen flags.
hipError_t launch_iac_reset(int R, const KArgs &a, int B, int zero_gamma, hipStream_t s);
hipError_t launch_reserve(int R, const KArgs &a, const ReserveArgs &ra, int B, hipStream_t s);

}  // namespace esp
