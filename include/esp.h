/*
 * esp.h -- C-ABI of the MI355X (gfx950) Elastic Shadow Pricing library.
 *
 * Elastic Shadow Pricing (paper Sec. 3.2) relaxes the per-resource capacity
 * constraint (Eq. 3) of the job-configuration integer program (Eq. 1-5) with
 * prices lambda_r >= 0 (Eq. 6).  For fixed prices every job j independently
 * takes the configuration maximising u_jk - sum_r lambda_r d_jkr (Sec. 3.2.2);
 * the prices then take the projected subgradient step of Eq. 8,
 *     lambda_r <- max(0, lambda_r + eta_t (U_r - C_r)),  U_r = sum_j d_{j,c_j,r},
 * with eta_t = eta0 (fixed) or eta0 / sqrt(t), and the loop repeats
 * (Sec. 3.2.3; Alg. 1 "EspTatonnement" followed by a re-selection at the
 * final prices).  Around that loop: the penalty Gamma of the ESP score
 * (Eq. 7), the effective capacity of Eq. 12, the outer ESP-IAC rounds of
 * Alg. 1 (esp_schedule) and RST's nearest-profile fallback (Sec. 3.1.2).
 *
 * Conventions for every entry point:
 *   - Every function returns an esp_status; nothing aborts or throws.
 *   - "host" pointers are read during the call only; "device" pointers are
 *     caller-owned device memory (any hipMalloc'ed or torch-allocated buffer)
 *     that must stay valid until the work queued on the stream has finished.
 *   - `stream` is a hipStream_t (NULL = the null stream).  Calls other than
 *     esp_create, esp_device_status, esp_read_penalties, esp_schedule (these
 *     wait for the GPU, as their descriptions say), esp_loop_driver (host
 *     only) and esp_destroy only enqueue work: they return before the GPU
 *     has run it.
 *   - A context is not thread-safe; distinct contexts are independent.
 *   - Arithmetic: scores in binary64 in a fixed order without fused
 *     multiply-add: rent = d_0*l_0, rent = rent + d_r*l_r (r = 1..R-1),
 *     s = u - rent, with the fp32 table values widened exactly.  The choice
 *     is the lowest configuration index among equal best scores.  U_r is the
 *     exact sum of the chosen fp32 demands rounded once to binary64
 *     (round-to-nearest-even), so results do not depend on launch geometry.
 *     Step sizes eta0 / sqrt(t) are one IEEE division and one correctly
 *     rounded square root in binary64 (computed on the device from t, so a
 *     solve holds no host-side state and can be captured in a graph).
 *   - Errors found by the GPU (bad prices, bad choice indices) are recorded
 *     in the context and reported by esp_device_status.
 */
#ifndef ESP_H
#define ESP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ESP_OK = 0,
    ESP_ERR_INVALID_ARG = 1,      /* NULL where required, bad enum, bad scalar */
    ESP_ERR_SHAPE = 2,            /* sizes or CSR offsets inconsistent or out of range */
    ESP_ERR_NONFINITE = 3,        /* NaN or +-Inf in utility, demand, capacity, eta0 or prices */
    ESP_ERR_NEGATIVE_DEMAND = 4,  /* a demand entry below zero (Eq. 3 resources are >= 0) */
    ESP_ERR_EMPTY_FAMILY = 5,     /* a job with no allowed configuration (Eq. 2 unsatisfiable) */
    ESP_ERR_WORKSPACE = 6,        /* workspace NULL, not 256-byte aligned, or too small */
    ESP_ERR_RANGE = 7,            /* magnitudes beyond what exact accumulation / fp64 can hold */
    ESP_ERR_DEVICE = 8,           /* a HIP runtime call failed */
    ESP_ERR_STATE = 9             /* NULL or destroyed context */
} esp_status;

/* Step rules of Eq. 8. */
enum { ESP_STEP_CONST = 0, ESP_STEP_INV_SQRT = 1 };

/* Loop drivers of esp_solve (results are identical in every mode). */
enum {
    ESP_MODE_AUTO = 0,        /* resident (below) when the table fits; else persistent for
                                 short passes (packed table of at most
                                 ESP_AUTO_PERSISTENT_BYTES), where launch latency would dominate,
                                 and for solves with tol > 0 (the loop ends on the device once
                                 every cluster has converged); one launch per iteration
                                 otherwise, where the two drivers run at about the same speed; falls
                                 back to one launch per iteration when the device cannot hold
                                 the grid co-resident */
    ESP_MODE_STREAM = 1,      /* one fused launch per iteration */
    ESP_MODE_PERSISTENT = 2,  /* one cooperative launch runs all iterations, streaming the table
                                 from memory every iteration; the workgroups of a cluster meet at
                                 a barrier after each iteration (ESP_ERR_DEVICE when the grid
                                 cannot be co-resident) */
    ESP_MODE_RESIDENT = 3     /* one launch runs all iterations over tiles held in registers
                                 (every wavefront of the grid holds at most two 256-entry tiles:
                                 tables of up to about 2,000 tiles per cluster); each iteration
                                 is completed inside the launch, the workgroups of a cluster
                                 exchanging their exact sums through tagged words (cooperative
                                 launch; ESP_ERR_DEVICE when the grid cannot be co-resident).
                                 esp_create returns ESP_ERR_SHAPE when the table does not fit.
                                 ESP_MODE_AUTO takes this driver whenever the table fits. */
};

#define ESP_AUTO_PERSISTENT_BYTES (64u << 20)

/* Opaque context: packed table + launch plan, created by esp_create. */
typedef struct esp_ctx esp_ctx;

/*
 * The logical problem (Sec. 3.2.1): B independent clusters that share one
 * job/family layout.  Entry e of the job x configuration table belongs to
 * job j when offsets[j] <= e < offsets[j+1]; its configuration index within
 * the family is k = e - offsets[j].  All pointers are HOST pointers read
 * during esp_workspace_size / esp_create only.
 */
typedef struct {
    int32_t num_clusters;            /* B >= 1 */
    int32_t num_jobs;                /* N >= 1 jobs per cluster */
    int32_t num_resources;           /* R in [1, 8] */
    int32_t configs_per_job;         /* dense layout: K in [1, 256]; ignored when family_offsets != NULL */
    const int64_t *family_offsets;   /* CSR [N+1], offsets[0] = 0, strictly increasing, family sizes
                                        in [1, 256]; NULL selects the dense layout offsets[j] = j*K */
    const float *utility;            /* [B][nnz]: u_jk, the value maximised (w_j T_j(c) of Eq. 1/6, or
                                        T_j(c)/T_j(c_max) - Gamma_j(c) for the Eq. 7 form); finite */
    const float *demand;             /* [B][nnz][R]: R_j(c)[r] of Eq. 3; finite and >= 0 */
    const double *capacity;          /* [B][R]: C_r (or C_eff of Eq. 12); finite, |C_r| <= 2^200 */
    const uint8_t *feasible;         /* optional [B][nnz]: 0 marks a configuration that violates the
                                        performance floor of Eq. 4 (never selected); NULL = all allowed */
    /* Optional penalty Gamma_j(c) of the ESP score (Eq. 7), subtracted after
     * the rent: s = (u - rent) - gamma_0 [k != current_j] - penalty_jk.
     * Give current + switch_cost, penalty, or both; all NULL = no penalty
     * (then esp_set_penalties cannot be used on the context). */
    const int32_t *current;          /* [B][N]: the job's current configuration index, -1 = none */
    const double *switch_cost;       /* [B]: gamma_0, finite, 0 <= gamma_0 <= 2^100 (with current) */
    const float *penalty;            /* [B][nnz]: interference penalty, finite and >= 0 */
} esp_problem;

typedef struct {
    int32_t rule;                    /* ESP_STEP_CONST or ESP_STEP_INV_SQRT */
    const double *eta0;              /* host [B]: finite, 0 < eta0 <= 2^100 */
} esp_step_rule;

typedef struct {
    int32_t blocks_per_cluster;      /* workgroups per cluster; 0 = one per compute unit over the device */
    int32_t sweep_order;             /* 0 = alternate the table sweep direction every iteration (reuses
                                        the memory-side cache), 1 = always front to back; results are
                                        identical either way */
    int32_t mode;                    /* ESP_MODE_* loop driver of esp_solve */
    int32_t flags;                   /* 0 or ESP_OPT_PROFILE_STORE */
    int32_t reserved[4];             /* must be zero */
} esp_options;

/* esp_options.flags: also keep an entry-major copy of the table for
 * esp_nearest_profile, which then reads each job type's family as one
 * contiguous run instead of a piece of each of the 1 + R columns.  Each
 * configuration takes 4 (1 + R) bytes (its utility, then its R demands); each
 * family's run starts on a 128-byte line, found through a directory of 64
 * bytes per 60 job types.  More workspace: B * sum_j ceil(4 (1 + R) K_j / 128)
 * * 128 bytes (about B * nnz * 4 (1 + R) plus 64 bytes per family) and
 * 64 * ceil(N / 60) bytes. */
#define ESP_OPT_PROFILE_STORE 1

/* Optional per-iteration record of esp_solve (device pointers, iteration-major;
 * row i describes iteration t = t_start + i).  Any field may be NULL. */
typedef struct {
    double *prices;                  /* [T][B][R]: lambda^{t+1} after the update of iteration t */
    double *demand;                  /* [T][B][R]: U^t at the selection made at lambda^t */
    int32_t *choice;                 /* [T][B][N]: c^t */
} esp_trace;

/*
 * esp_workspace_size: device workspace bytes esp_create needs for `problem`
 * (only its shapes and offsets are read).  `options` may be NULL.
 * Errors: ESP_ERR_INVALID_ARG (NULL problem/bytes, unknown flags or reserved
 * options nonzero),
 * ESP_ERR_SHAPE.
 */
esp_status esp_workspace_size(const esp_problem *problem, const esp_options *options, size_t *bytes);

/*
 * esp_create: validate the problem, pack the table into the structure-of-
 * arrays device image inside `workspace` and return a context.  The workspace
 * is caller-owned device memory of at least esp_workspace_size bytes,
 * 256-byte aligned, which must outlive the context; its contents are
 * overwritten.  Host arrays may be freed when the call returns (it waits for
 * its own copies on `stream`).
 * Errors: ESP_ERR_INVALID_ARG, ESP_ERR_SHAPE, ESP_ERR_NONFINITE,
 * ESP_ERR_NEGATIVE_DEMAND, ESP_ERR_EMPTY_FAMILY, ESP_ERR_WORKSPACE,
 * ESP_ERR_RANGE (a demand column whose exact sum does not fit the 128-bit
 * accumulator: its nonzero values span too many binary orders of magnitude),
 * ESP_ERR_DEVICE.  On error *out is set to NULL.
 */
esp_status esp_create(const esp_problem *problem, const esp_step_rule *step, const esp_options *options,
                      void *workspace, size_t workspace_bytes, void *stream, esp_ctx **out);

/*
 * esp_score_select (Sec. 3.2.2): for prices `prices` (device [B][R], finite,
 * >= 0) write every job's best configuration index to `choice` (device
 * [B][N] int32).  Errors: ESP_ERR_STATE, ESP_ERR_INVALID_ARG, ESP_ERR_DEVICE.
 */
esp_status esp_score_select(esp_ctx *ctx, const double *prices, int32_t *choice, void *stream);

/*
 * esp_reduce_demand (Sec. 3.2.3, U_r under Eq. 8): demand (device [B][R]) =
 * exact per-resource sum of the demands of the configurations in `choice`
 * (device [B][N]).  An index outside a job's family makes that cluster's
 * demand NaN and is reported by esp_device_status.
 * Errors: ESP_ERR_STATE, ESP_ERR_INVALID_ARG, ESP_ERR_DEVICE.
 */
esp_status esp_reduce_demand(esp_ctx *ctx, const int32_t *choice, double *demand, void *stream);

/*
 * esp_update_prices (Eq. 8): prices (device [B][R], in lambda^t, out
 * lambda^{t+1}) <- max(0, lambda + eta_t (demand - C)); t >= 1 selects
 * eta_t.  Errors: ESP_ERR_STATE, ESP_ERR_INVALID_ARG, ESP_ERR_DEVICE.
 */
esp_status esp_update_prices(esp_ctx *ctx, const double *demand, int32_t t, double *prices, void *stream);

/*
 * esp_solve: `iters` iterations t = t_start .. t_start+iters-1 of
 * select -> demand -> update, one fused kernel pass per iteration (the passes
 * run as one launch each or inside one persistent launch, see ESP_MODE_*;
 * with several workgroups per cluster the update of iteration t is computed
 * at the start of the next pass, or of a closing launch after the last one),
 * then a re-selection at the final prices (Alg. 1).
 *   prices      device [B][R], in lambda^{t_start} (finite, >= 0; a -0.0 entry is stored
 *               back as +0.0 before the first iteration, so no price the call
 *               returns is -0.0), out the final prices
 *   iters       T >= 0;  t_start >= 1 (a warm start continues a previous solve)
 * Graph capture: while `stream` is being captured, the iterations are
 * recorded as one launch each (ESP_MODE_AUTO falls back to it;
 * ESP_MODE_PERSISTENT and ESP_MODE_RESIDENT return ESP_ERR_INVALID_ARG); a
 * replay recomputes the same iterations on the buffers given at capture.
 *   tol         0 = run all T iterations; > 0 = a cluster stops after the first
 *               update with |lambda^{t+1}_r - lambda^t_r| <= tol * max(1, lambda^t_r)
 *               for every r (its later iterations do nothing)
 *   choice      device [B][N] or NULL: selection at the final prices
 *   demand      device [B][R] or NULL: U at that selection
 *   trace       NULL or per-iteration records (see esp_trace)
 *   iters_done  device [B] int32 or NULL: updates made per cluster
 * Errors: ESP_ERR_STATE, ESP_ERR_INVALID_ARG (also: ESP_MODE_PERSISTENT or
 * ESP_MODE_RESIDENT while `stream` is being captured; nothing is enqueued or
 * recorded then), ESP_ERR_DEVICE (a HIP call failed, or ESP_MODE_PERSISTENT /
 * ESP_MODE_RESIDENT with a grid the device cannot hold co-resident: refused
 * on the host before the first iteration is launched).
 */
esp_status esp_solve(esp_ctx *ctx, double *prices, int32_t iters, int32_t t_start, double tol,
                     int32_t *choice, double *demand, const esp_trace *trace, int32_t *iters_done,
                     void *stream);

/*
 * esp_solve_noalloc: esp_solve for callers that cannot allocate memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  Same arguments, results and errors as esp_solve (bit for bit
 * the same outputs), but the call allocates nothing and its per-solve scratch
 * -- per-workgroup partial sums, arrival tickets, barrier words, the prices of
 * the iteration being completed, the stop iteration and the update counts --
 * lives in one static device array of the library, ESP_NOALLOC_SCRATCH_BYTES
 * on each GPU, held until the process ends, instead of the context's
 * workspace (whose read-only parts -- the packed table, capacities, step
 * scales -- it still reads, and whose status word and run flags it still
 * uses).  Every call on one GPU shares that GPU's array, whatever the context:
 * calls that overlap on one GPU race and must be serialized by the caller
 * (one stream, or events).  The array keeps the last call's contents; what
 * must start at zero is cleared by each call's first kernel.  The context
 * must have been created with the GPU current that later calls run on.
 * Errors: those of esp_solve, and ESP_ERR_WORKSPACE when the context's
 * scratch (3 B nblk R 16 + B 4352 + 2 B R 8 bytes and alignment, nblk the
 * workgroups per cluster) exceeds ESP_NOALLOC_SCRATCH_BYTES (B up to about
 * 400 clusters at R = 8), ESP_ERR_DEVICE when the array's address could not
 * be resolved at esp_create.
 */
#define ESP_NOALLOC_SCRATCH_BYTES (2u << 20)
esp_status esp_solve_noalloc(esp_ctx *ctx, double *prices, int32_t iters, int32_t t_start, double tol,
                             int32_t *choice, double *demand, const esp_trace *trace, int32_t *iters_done,
                             void *stream);

/*
 * esp_device_status: wait for `stream`, then return (and clear) the first
 * error the GPU recorded since the last call: ESP_ERR_NONFINITE or
 * ESP_ERR_INVALID_ARG for prices that were NaN, infinite or negative (the
 * affected calls left prices and outputs unchanged), ESP_ERR_INVALID_ARG for
 * a choice index outside its family, the query errors of
 * esp_nearest_profile, or a persistent launch whose workgroups waited too
 * long for each other (ESP_ERR_DEVICE); ESP_OK otherwise.
 */
esp_status esp_device_status(esp_ctx *ctx, void *stream);

/*
 * esp_set_capacity (Sec. 3.2.1, C of Eq. 3): replace the physical capacity
 * C (host [B][R], finite) of a context; the capacity used by later price
 * updates becomes C (any effective capacity installed before is dropped).
 * Stream-ordered after earlier work on `stream`; `capacity` may be freed when
 * the call returns.
 * Errors: ESP_ERR_STATE, ESP_ERR_INVALID_ARG (NULL capacity),
 * ESP_ERR_NONFINITE, ESP_ERR_RANGE (|C| > 2^200), ESP_ERR_DEVICE.
 */
esp_status esp_set_capacity(esp_ctx *ctx, const double *capacity, void *stream);

/*
 * esp_effective_capacity (Sec. 3.4, Eq. 12; first step of Alg. 1): reserve
 * capacity for pending jobs at their smallest footprint,
 *     C_eff_r = C_r - gamma * S_r,
 *     S_r = sum over pending jobs j of min over j's allowed configurations
 *           of d_jkr   (componentwise: each resource takes its own minimum),
 * S_r exact and rounded once to binary64, then one rounded product and one
 * rounded difference.  C is ctx's physical capacity (from esp_create or
 * esp_set_capacity).  C_eff becomes the capacity of ctx's later price
 * updates (esp_solve, esp_update_prices); a later call recomputes it from C,
 * so epochs do not accumulate reservations.
 *   queue         context packed (esp_create) from the pending jobs' profile
 *                 families, same num_clusters and num_resources as ctx; only
 *                 its demand table and feasibility mask are read (its
 *                 utility, capacity and step rule do not enter Eq. 12).  It
 *                 must not run other work concurrently (its cross-workgroup
 *                 sum buffers are used).  NULL = no pending job: C_eff = C.
 *   queued        device [B][N_queue] uint8, nonzero = pending, or NULL (every
 *                 job of `queue` is pending).
 *   gamma         reservation aggressiveness in [0, 1].
 *   capacity_eff  device [B][R] receives C_eff as well, or NULL.
 * Stream-ordered and asynchronous.  C_eff may be negative (a queue that
 * cannot fit); the price update then raises that resource's price.
 * Errors: ESP_ERR_STATE (NULL ctx or invalid queue), ESP_ERR_INVALID_ARG
 * (gamma outside [0, 1] or NaN), ESP_ERR_SHAPE (B or R differ),
 * ESP_ERR_DEVICE.
 */
esp_status esp_effective_capacity(esp_ctx *ctx, esp_ctx *queue, const uint8_t *queued, double gamma,
                                  double *capacity_eff, void *stream);

/*
 * Outer ESP-IAC rounds (Sec. 3.4, Alg. 1).  GPU-level cluster model for the
 * BinPack step and the inputs of the predicted slowdown of a co-located
 * pair, S_x|y = 1 + a_x b_y (a: sensitivity, b: pressure of each job's
 * chosen configuration), a stand-in for the trained predictor of Sec. 3.3.2,
 * with the adaptive thresholds of Eq. 11.
 */
#define ESP_MAX_GPUS 2048      /* GPUs per cluster */
#define ESP_MAX_PER_GPU 4      /* jobs sharing one GPU */
typedef struct {
    const int32_t *gpus;       /* host [B]: GPUs of each cluster, 1..ESP_MAX_GPUS */
    double gpu_memory;         /* per-GPU capacity of resource r_mem (>= 0) */
    double gpu_compute;        /* per-GPU capacity of resource r_sm (>= 0) */
    int32_t r_gpus;            /* resource holding a configuration's GPU count (1..8 whole GPUs;
                                  other values: the job is not placeable) */
    int32_t r_mem;             /* resource split evenly over the job's GPUs: memory */
    int32_t r_sm;              /* resource split evenly over the job's GPUs: compute share */
    const float *sensitivity;  /* device [B][nnz] a per configuration (entry order of esp_problem) */
    const float *pressure;     /* device [B][nnz] b per configuration */
    const double *tau_base;    /* device [B][N] baseline tolerance of each job */
    double beta;               /* Eq. 11 sensitivity to utilisation */
    double beta_max;           /* Eq. 11 clamp of the additive term */
    double u_target;           /* Eq. 11 utilisation target (> 0) */
    double kappa;              /* penalty per unit of excess slowdown (>= 0) */
} esp_iac_model;

/*
 * esp_schedule (Alg. 1): Gamma <- 0 (the interference penalties of the
 * context's penalty column; switching costs stay), then rounds m = 1..
 * max_rounds, per cluster:
 *   1. the tatonnement: esp_solve from `prices` (t = 1.., `iters`, `tol`),
 *      the selection c* at the prices reached written to `choice`;
 *   2. BinPack (first fit; the paper names no algorithm): jobs in index
 *      order; job j needs g = d_j[r_gpus] GPUs and d_j[r_mem] / g memory and
 *      d_j[r_sm] / g compute on each; it takes the g lowest-index GPUs with
 *      room for one share and fewer than ESP_MAX_PER_GPU jobs, all or
 *      nothing (binary64 residuals, updated in job order);
 *   3. IacPredict on every pair (x, y) sharing a GPU: the pair violates when
 *      S_x|y > tau_x or S_y|x > tau_y, tau_x = tau_base_x + min(beta (U /
 *      u_target - 1), beta_max), U = busy GPUs / G;
 *   4. no violation: the cluster's schedule is final (later rounds leave it
 *      alone); otherwise each violating job's chosen configuration has its
 *      penalty raised by kappa times its largest excess S - tau (binary64,
 *      rounded once to fp32), and the next round starts from the prices
 *      reached.
 * Outputs (device): prices [B][R] of each cluster's last round; choice
 * [B][N]; gpu_jobs [B][max gpus][ESP_MAX_PER_GPU], GPU h's jobs in placement
 * order, -1 for an empty slot; rounds_used [B]; violations [B], the
 * violating pairs of the last round.  The context's penalty column keeps the
 * final Gamma.  The context must have been created with penalty inputs
 * (esp_problem.current / switch_cost / penalty).  Synchronises `stream` once
 * per round (to stop when every cluster is free of violations).
 * Errors: ESP_ERR_STATE (NULL context or no penalty column),
 * ESP_ERR_INVALID_ARG (NULL pointers, max_rounds < 1, iters < 0, a resource
 * index outside [0, R), a GPU count outside 1..ESP_MAX_GPUS, negative
 * capacities or kappa, u_target <= 0), ESP_ERR_NONFINITE, and the errors of
 * esp_solve.
 */
esp_status esp_schedule(esp_ctx *ctx, const esp_iac_model *model, int32_t max_rounds, int32_t iters, double tol,
                        double *prices, int32_t *choice, int32_t *gpu_jobs, int32_t *rounds_used,
                        int32_t *violations, void *stream);

/*
 * esp_read_penalties (Eq. 7): copy the context's current interference
 * penalties Gamma (e.g. after esp_schedule) to `penalty`, host [B][nnz] in
 * the entry order of esp_problem.  Waits for `stream`.
 * Errors: ESP_ERR_STATE (NULL context or no penalty column),
 * ESP_ERR_INVALID_ARG, ESP_ERR_DEVICE.
 */
esp_status esp_read_penalties(esp_ctx *ctx, float *penalty, void *stream);

/*
 * esp_nearest_profile (RST's profile fallback, Sec. 3.1.2 and Sec. 4.1): a
 * configuration with no profile takes the throughput of the profile-store
 * entry of its job type whose resource vector is closest in l2 distance.
 * `store` is a context packed (esp_create) from the profile store: family f
 * = job type f, utility = profiled throughput T_j(c), demand = resource
 * vector R_j(c); masked entries (feasible = 0) are not candidates.  For each
 * of the B x num_queries queries (cluster b's queries search cluster b's
 * store):
 *   family    device [B][num_queries] int32, job type of the query;
 *   query     device [B][num_queries][R] float, the configuration's resource
 *             vector (finite);
 *   nearest   device [B][num_queries] int32 out: index within the family of
 *             the nearest entry (squared distance in binary64, order
 *             e_0 = q_0 - d_0, acc = e_0 e_0, acc = acc + e_r e_r for
 *             r = 1..R-1, lowest index among equal distances);
 *   estimate  device [B][num_queries] float out, or NULL: that entry's
 *             utility (the provisional throughput).
 * A family index out of [0, N) or a non-finite query component gives
 * nearest = -1 and estimate NaN for that query and is reported by
 * esp_device_status (ESP_ERR_INVALID_ARG / ESP_ERR_NONFINITE).
 * Stream-ordered and asynchronous; the store may serve any number of calls.
 * Errors: ESP_ERR_STATE, ESP_ERR_INVALID_ARG (negative count, NULL family,
 * query or nearest), ESP_ERR_DEVICE.
 */
esp_status esp_nearest_profile(esp_ctx *store, int32_t num_queries, const int32_t *family, const float *query,
                               int32_t *nearest, float *estimate, void *stream);

/*
 * esp_loop_driver: the loop driver esp_solve uses for this context's solves
 * with tol = 0, ESP_MODE_STREAM, ESP_MODE_PERSISTENT or ESP_MODE_RESIDENT
 * (ESP_MODE_AUTO resolved against the table size, and against the device
 * once a solve has run).  Host-only.
 * Errors: ESP_ERR_STATE (NULL context), ESP_ERR_INVALID_ARG (mode NULL).
 */
esp_status esp_loop_driver(const esp_ctx *ctx, int32_t *mode);

/*
 * esp_set_penalties (Eq. 7): replace the penalty inputs of a context that was
 * created with them (e.g. between the ESP-IAC rounds of Alg. 1).  Same
 * meaning and layout as the esp_problem fields (host pointers; current and
 * switch_cost may be NULL for "no switching cost", penalty NULL for zero
 * penalties).  Stream-ordered after earlier work on `stream`; host arrays may
 * be freed when the call returns.
 * Errors: ESP_ERR_STATE (NULL context, or one created without penalties),
 * ESP_ERR_INVALID_ARG (current out of range, negative penalty or switching
 * cost), ESP_ERR_NONFINITE, ESP_ERR_RANGE, ESP_ERR_DEVICE.
 */
esp_status esp_set_penalties(esp_ctx *ctx, const int32_t *current, const double *switch_cost, const float *penalty,
                             void *stream);

/* esp_destroy: free the host-side context (the workspace stays the caller's).
 * Waits for nothing: the caller must not destroy a context with work in flight. */
esp_status esp_destroy(esp_ctx *ctx);

/* Static, NUL-terminated description of a status code. */
const char *esp_status_string(esp_status status);

#ifdef __cplusplus
}
#endif
#endif /* ESP_H */
