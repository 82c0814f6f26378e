/*
 * CPU oracle for Elastic Shadow Pricing (ESP) -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the bench's CPU-baseline leg may load
 * this file's library.  The product path (the HIP library) never calls it and
 * shares no code with it.
 *
 * Plain, slow, single-threaded C, fp64 arithmetic, built with
 * -O2 -ffp-contract=off -fno-fast-math on x86-64 (SSE2, no x87, no FMA), so
 * every + - * / sqrt below is one correctly rounded IEEE-754 binary64 operation
 * in the order written.
 *
 * What it computes (paper Sec. 3.2, "Elastic Shadow Pricing"):
 *   - the per-job subproblem of the Lagrangian decomposition (Sec. 3.2.2,
 *     Eq. 6): for fixed prices lambda, job j picks
 *         c_j = argmax_k [ u_jk - sum_r lambda_r d_jkr ]
 *     by enumerating its family, lowest index winning ties;
 *   - optionally with the penalty Gamma_j(k) of the ESP score (Eq. 7,
 *     Sec. 3.2.3), subtracted after the rent: a switching cost gamma_0 for
 *     every configuration other than the job's current one, and a given
 *     interference penalty per configuration;
 *   - the aggregate demand U_r = sum_j d_{j,c_j,r} of the current selection
 *     (Sec. 3.2.3, definition under Eq. 8), as the exact real sum rounded once
 *     to binary64 (round-to-nearest-even);
 *   - the projected-subgradient price update of Eq. 8,
 *         lambda_r <- max(0, lambda_r + eta_t (U_r - C_r)),
 *     eta_t = eta0 (fixed) or eta0 / sqrt(t) (diminishing), t = 1, 2, ...;
 *   - the loop of the tatonnement (Sec. 3.2.2/3.2.3; Alg. 1 "EspTatonnement"
 *     followed by the per-job re-selection at the final prices);
 *   - the effective capacity of Eq. 12 (Sec. 3.4): the physical capacity
 *     minus gamma times the exact sum, over the pending jobs, of each job's
 *     componentwise smallest demand vector over its family;
 *   - the outer rounds of Alg. 1 (Sec. 3.4): first-fit BinPack of the
 *     selection onto GPUs, the co-located pairs' predicted slowdowns against
 *     the thresholds of Eq. 11, and penalty updates for the offending
 *     configurations, repeated until no pair violates;
 *   - RST's nearest-profile fallback (Sec. 3.1.2, Sec. 4.1): within a job
 *     type's profile family, the entry whose resource vector is closest in
 *     l2 distance to an unprofiled configuration's vector, and its
 *     throughput as the provisional estimate;
 *   - for the pins only: the Lagrangian dual value g(lambda) of Eq. 6 at the
 *     selected configurations and the primal value sum_j u_{j,c_j} (Eq. 1).
 *
 * Readings where the paper is silent (each listed in the design notes):
 *   score    rent = d0*l0; rent = rent + d_r*l_r (r = 1..R-1); s = u - rent,
 *            table values widened exactly from fp32 to fp64; with Eq. 7's
 *            penalty: s = s - gamma_0 (k != current, current >= 0), then
 *            s = s - penalty_jk;
 *   ties     the lowest configuration index wins (strict '>' scan);
 *   t        1-based within one solve; a warm start passes t_start;
 *   project  x > 0 ? x : +0.0 (a stored price is never -0.0);
 *   Eq. 4    configurations with feasible[e] == 0 are never selected;
 *   stop     optional: after the update of iteration t, stop when every r has
 *            |lambda^{t+1}_r - lambda^t_r| <= tol * max(1, lambda^t_r).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "esp_oracle.h"

/* ------------------------------------------------------------------------ */
/* Exact sum of non-negative binary32 values, rounded once to binary64.       */
/* ------------------------------------------------------------------------ */

/*
 * Every finite binary32 value v >= 0 is an integer multiple of 2^-149, and
 * v * 2^(149+24) is an integer below 2^(128+173) = 2^301.  The accumulator
 * holds that integer for the running sum in 32-bit digits, each kept in a
 * 64-bit word so that digits can absorb up to 2^31 additions before carries
 * are propagated.  ORC_WORDS * 32 = 384 bits >= 301 + 31 bits of growth.
 */
#define ORC_WORDS 12
#define ORC_BIAS 173   /* integer = value * 2^ORC_BIAS */

typedef struct { uint64_t w[ORC_WORDS]; } orc_acc;

static void acc_clear(orc_acc *a) { memset(a, 0, sizeof(*a)); }

static void acc_add_f32(orc_acc *a, float v)
{
    int e;
    float f;
    uint64_t mant, chunk;
    int pos;
    if (v == 0.0f) return;                 /* +0 and -0 add nothing */
    f = frexpf(v, &e);                     /* v = f * 2^e, 0.5 <= f < 1 */
    mant = (uint64_t)ldexpf(f, 24);        /* exact: f has <= 24 significant bits */
    pos = e - 24 + ORC_BIAS;               /* v * 2^BIAS = mant * 2^pos, pos >= 0 */
    chunk = mant << (pos % 32);            /* <= 24 + 31 = 55 bits */
    a->w[pos / 32] += chunk & 0xffffffffu;
    a->w[pos / 32 + 1] += chunk >> 32;
}

static void acc_normalize(orc_acc *a)
{
    int i;
    for (i = 0; i + 1 < ORC_WORDS; i++) {
        a->w[i + 1] += a->w[i] >> 32;
        a->w[i] &= 0xffffffffu;
    }
}

static int acc_bit(const orc_acc *a, int i) { return (int)((a->w[i / 32] >> (i % 32)) & 1u); }

/* Round the accumulated integer * 2^-BIAS to the nearest binary64, ties to even. */
static double acc_to_double(orc_acc *a)
{
    int top = -1, i;
    uint64_t m = 0;
    int guard, sticky = 0;
    acc_normalize(a);
    for (i = ORC_WORDS * 32 - 1; i >= 0; i--)
        if (acc_bit(a, i)) { top = i; break; }
    if (top < 0) return 0.0;
    if (top <= 52) {                       /* fits in 53 bits: exact */
        for (i = top; i >= 0; i--) m = (m << 1) | (uint64_t)acc_bit(a, i);
        return ldexp((double)m, -ORC_BIAS);
    }
    for (i = top; i >= top - 52; i--) m = (m << 1) | (uint64_t)acc_bit(a, i);
    guard = acc_bit(a, top - 53);
    for (i = top - 54; i >= 0; i--) sticky |= acc_bit(a, i);
    if (guard && (sticky || (m & 1u))) m += 1;   /* m may become 2^53: still exact */
    return ldexp((double)m, top - 52 - ORC_BIAS);
}

double orc_exact_sum_f32(const float *v, int64_t n)
{
    orc_acc a;
    int64_t i;
    acc_clear(&a);
    for (i = 0; i < n; i++) acc_add_f32(&a, v[i]);
    return acc_to_double(&a);
}

/* ------------------------------------------------------------------------ */
/* The method.                                                               */
/* ------------------------------------------------------------------------ */

static const float *util_of(const orc_problem *p, int b) { return p->utility + (int64_t)b * p->nnz; }
static const float *dem_of(const orc_problem *p, int b) { return p->demand + (int64_t)b * p->nnz * p->R; }

/* Score of configuration k of job j at prices lam (Sec. 3.2.2, the bracket
 * of Eq. 6), minus the penalty Gamma of Eq. 7 when one is given. */
double orc_score(const orc_problem *p, int b, int64_t j, int32_t k, const double *lam)
{
    const int64_t e = p->offsets[j] + k;
    const float *d = dem_of(p, b) + e * p->R;
    double rent = (double)d[0] * lam[0];
    double s;
    int r;
    for (r = 1; r < p->R; r++) rent = rent + (double)d[r] * lam[r];
    s = (double)util_of(p, b)[e] - rent;
    if (p->current != NULL) {
        const int32_t cur = p->current[(int64_t)b * p->N + j];
        if (cur >= 0 && k != cur) s = s - p->switch_cost[b];
    }
    if (p->penalty != NULL) s = s - (double)p->penalty[(int64_t)b * p->nnz + e];
    return s;
}

/* The objective each job maximises at zero prices (Eq. 1 with Eq. 7's penalty):
 * u_jk - gamma_0 [k != current] - penalty_jk. */
static double penalized_utility(const orc_problem *p, int b, int64_t j, int32_t k)
{
    const int64_t e = p->offsets[j] + k;
    double v = (double)util_of(p, b)[e];
    if (p->current != NULL) {
        const int32_t cur = p->current[(int64_t)b * p->N + j];
        if (cur >= 0 && k != cur) v = v - p->switch_cost[b];
    }
    if (p->penalty != NULL) v = v - (double)p->penalty[(int64_t)b * p->nnz + e];
    return v;
}

static int entry_allowed(const orc_problem *p, int b, int64_t e)
{
    return p->feasible == NULL || p->feasible[(int64_t)b * p->nnz + e] != 0;
}

/* Per-job argmax (Sec. 3.2.2): choice[j] = family index k, lowest k on ties. */
void orc_select(const orc_problem *p, int b, const double *lam, int32_t *choice)
{
    int64_t j;
    for (j = 0; j < p->N; j++) {
        int64_t lo = p->offsets[j], hi = p->offsets[j + 1], e;
        int32_t best_k = -1;
        double best = 0.0;
        for (e = lo; e < hi; e++) {
            double s;
            if (!entry_allowed(p, b, e)) continue;
            s = orc_score(p, b, j, (int32_t)(e - lo), lam);
            if (best_k < 0 || s > best) { best = s; best_k = (int32_t)(e - lo); }
        }
        choice[j] = best_k;                 /* -1 only for a family with no allowed entry */
    }
}

/* U_r = sum_j d_{j, c_j, r} (Sec. 3.2.3), exact sum rounded once. */
void orc_demand(const orc_problem *p, int b, const int32_t *choice, double *U)
{
    const float *d = dem_of(p, b);
    int r;
    for (r = 0; r < p->R; r++) {
        orc_acc a;
        int64_t j;
        acc_clear(&a);
        for (j = 0; j < p->N; j++) {
            if (choice[j] < 0) continue;
            acc_add_f32(&a, d[(p->offsets[j] + choice[j]) * p->R + r]);
        }
        U[r] = acc_to_double(&a);
    }
}

/* Step size of Eq. 8: fixed eta0, or eta0 / sqrt(t). */
double orc_eta(int rule, double eta0, int64_t t)
{
    if (rule == ORC_STEP_INV_SQRT) return eta0 / sqrt((double)t);
    return eta0;
}

/* Projected subgradient step of Eq. 8, in place. */
void orc_update(int R, const double *U, const double *C, double eta, double *lam)
{
    int r;
    for (r = 0; r < R; r++) {
        double g = U[r] - C[r];
        double x = lam[r] + eta * g;
        lam[r] = (x > 0.0) ? x : 0.0;
    }
}

/* Lagrangian (Eq. 6) at the selection: sum_j s_{j,c_j} + sum_r lam_r C_r. */
double orc_dual_value(const orc_problem *p, int b, const double *lam, const int32_t *choice)
{
    double v = 0.0;
    int64_t j;
    int r;
    for (j = 0; j < p->N; j++)
        if (choice[j] >= 0) v = v + orc_score(p, b, j, choice[j], lam);
    for (r = 0; r < p->R; r++) v = v + lam[r] * p->capacity[(int64_t)b * p->R + r];
    return v;
}

/* Objective of Eq. 1 at the selection: sum_j u_{j,c_j} (less Eq. 7's penalty
 * when one is given). */
double orc_primal_value(const orc_problem *p, int b, const int32_t *choice)
{
    double v = 0.0;
    int64_t j;
    for (j = 0; j < p->N; j++)
        if (choice[j] >= 0) v = v + penalized_utility(p, b, j, choice[j]);
    return v;
}

/*
 * The tatonnement for every cluster b (independently):
 *   for t = t_start .. t_start+T-1:
 *       select at lambda^t, sum demand U^t, update to lambda^{t+1} (Eq. 8)
 *   then re-select at the final prices (Alg. 1 after EspTatonnement).
 * lam [B][R] holds lambda^{t_start} on entry and the final prices on exit.
 * Optional outputs (NULL to skip), iteration-major:
 *   tr_lam [T][B][R] lambda^{t+1};  tr_U [T][B][R] U^t;
 *   tr_choice [T][B][N] c^t;  tr_dual [T][B] g at (lambda^t, c^t);
 *   tr_primal [T][B] Eq. 1 value of c^t;
 *   choice_out [B][N], U_out [B][R] at the final prices;
 *   iters_done [B] number of updates made (< T only with tol > 0).
 * Returns 0, or -1 when a family has no allowed entry.
 */
int orc_solve(const orc_problem *p, double *lam, int32_t T, int32_t t_start, double tol,
              double *tr_lam, double *tr_U, int32_t *tr_choice, double *tr_dual,
              double *tr_primal, int32_t *choice_out, double *U_out, int32_t *iters_done)
{
    int R = p->R, b, r;
    int32_t *ch = (int32_t *)malloc(sizeof(int32_t) * (size_t)(p->N > 0 ? p->N : 1));
    double U[ORC_MAX_R], prev[ORC_MAX_R];
    int status = 0;
    if (ch == NULL) return -2;
    for (b = 0; b < p->B; b++) {
        double *lb = lam + (int64_t)b * R;
        const double *Cb = p->capacity + (int64_t)b * R;
        int32_t i, done = 0;
        for (i = 0; i < T; i++) {
            int64_t t = (int64_t)t_start + i;
            double eta;
            int conv = 1;
            orc_select(p, b, lb, ch);
            orc_demand(p, b, ch, U);
            if (tr_dual) tr_dual[(int64_t)i * p->B + b] = orc_dual_value(p, b, lb, ch);
            if (tr_primal) tr_primal[(int64_t)i * p->B + b] = orc_primal_value(p, b, ch);
            if (tr_choice) memcpy(tr_choice + ((int64_t)i * p->B + b) * p->N, ch, sizeof(int32_t) * (size_t)p->N);
            eta = orc_eta(p->rule, p->eta0[b], t);
            for (r = 0; r < R; r++) prev[r] = lb[r];
            orc_update(R, U, Cb, eta, lb);
            if (tr_lam) memcpy(tr_lam + ((int64_t)i * p->B + b) * R, lb, sizeof(double) * (size_t)R);
            if (tr_U) memcpy(tr_U + ((int64_t)i * p->B + b) * R, U, sizeof(double) * (size_t)R);
            done = i + 1;
            if (tol > 0.0) {
                for (r = 0; r < R; r++) {
                    double diff = fabs(lb[r] - prev[r]);
                    double scale = prev[r] > 1.0 ? prev[r] : 1.0;
                    if (!(diff <= tol * scale)) conv = 0;
                }
                if (conv) break;
            }
        }
        if (iters_done) iters_done[b] = done;
        orc_select(p, b, lb, ch);
        for (i = 0; i < p->N; i++) if (ch[i] < 0) status = -1;
        if (choice_out) memcpy(choice_out + (int64_t)b * p->N, ch, sizeof(int32_t) * (size_t)p->N);
        if (U_out) orc_demand(p, b, ch, U_out + (int64_t)b * R);
    }
    free(ch);
    return status;
}

/* ------------------------------------------------------------------------ */
/* Effective capacity (Sec. 3.4, Eq. 12).                                    */
/* ------------------------------------------------------------------------ */

/*
 * Capacity held back for the pending jobs Q at their smallest footprint:
 *     Rmin_jr  = min over the allowed configurations k of d_jkr
 *                (componentwise: each resource takes its own minimum),
 *     S_r      = sum_{j in Q} Rmin_jr        (exact, rounded once),
 *     C_eff_r  = C_r - gamma * S_r           (two rounded operations).
 * q describes the pending jobs of cluster b (its utility is not read; the
 * feasible mask, if any, restricts the family as in Eq. 4).  queued[j] != 0
 * marks job j as pending; NULL means every job of q is pending.
 * Returns 0, or -1 when a pending family has no allowed entry.
 */
int orc_effective_capacity(const orc_problem *q, int b, const uint8_t *queued, const double *C,
                           double gamma, double *C_eff)
{
    const float *d = dem_of(q, b);
    int r, status = 0;
    for (r = 0; r < q->R; r++) {
        orc_acc a;
        int64_t j;
        double S, g;
        acc_clear(&a);
        for (j = 0; j < q->N; j++) {
            int64_t e;
            int have = 0;
            float m = 0.0f;
            if (queued != NULL && queued[j] == 0) continue;
            for (e = q->offsets[j]; e < q->offsets[j + 1]; e++) {
                float v;
                if (!entry_allowed(q, b, e)) continue;
                v = d[e * q->R + r];
                if (!have || v < m) { m = v; have = 1; }
            }
            if (!have) { status = -1; continue; }
            acc_add_f32(&a, m);
        }
        S = acc_to_double(&a);
        g = gamma * S;
        C_eff[r] = C[r] - g;
    }
    return status;
}

/* ------------------------------------------------------------------------ */
/* Nearest-profile interpolation (Sec. 3.1.2 profile fallback, Sec. 4.1).   */
/* ------------------------------------------------------------------------ */

/*
 * For an unprofiled configuration of job type f with resource vector q, the
 * profile store's entry of the same family whose resource vector is closest
 * in l2 distance supplies the provisional throughput.  p holds the store
 * (family f = job type f, utility = profiled throughput, demand = resource
 * vector).  Squared distance in binary64 in a fixed order,
 *     e_0 = q_0 - d_0; acc = e_0 * e_0;
 *     for r = 1..R-1: e_r = q_r - d_r; acc = acc + e_r * e_r,
 * compared without the square root (monotone); the lowest index wins among
 * equal distances; entries with feasible == 0 are not candidates.
 * Returns the index within the family, or -1 when f is out of range or the
 * family has no allowed entry; *dist2 receives acc of the winner.
 */
int32_t orc_nearest(const orc_problem *p, int b, int64_t f, const float *q, double *dist2)
{
    const float *d = dem_of(p, b);
    int64_t e;
    int32_t best_k = -1;
    double best = 0.0;
    if (f < 0 || f >= p->N) return -1;
    for (e = p->offsets[f]; e < p->offsets[f + 1]; e++) {
        double acc, x;
        int r;
        if (!entry_allowed(p, b, e)) continue;
        x = (double)q[0] - (double)d[e * p->R];
        acc = x * x;
        for (r = 1; r < p->R; r++) {
            x = (double)q[r] - (double)d[e * p->R + r];
            acc = acc + x * x;
        }
        if (best_k < 0 || acc < best) { best = acc; best_k = (int32_t)(e - p->offsets[f]); }
    }
    if (dist2) *dist2 = best;
    return best_k;
}

/* A batch of queries of cluster b: family[i], q[i][R] -> k[i] and the
 * throughput estimate est[i] = utility of the nearest entry (NaN when k < 0). */
void orc_nearest_batch(const orc_problem *p, int b, int64_t nq, const int32_t *family, const float *q,
                       int32_t *k, float *est)
{
    int64_t i;
    for (i = 0; i < nq; i++) {
        int32_t c = orc_nearest(p, b, family[i], q + i * p->R, NULL);
        k[i] = c;
        if (est) est[i] = c < 0 ? NAN : util_of(p, b)[p->offsets[family[i]] + c];
    }
}

/* ------------------------------------------------------------------------ */
/* Outer ESP-IAC rounds (Sec. 3.4, Alg. 1; thresholds of Eq. 11).           */
/* ------------------------------------------------------------------------ */

/*
 * BinPack (not specified by the paper; first fit): jobs in index order; job j
 * at its chosen configuration needs g = d_j[r_gpus] GPUs (a whole number in
 * 1..ORC_MAX_SHARDS, otherwise the job is not placeable) and on each of them
 * d_j[r_mem] / g memory and d_j[r_sm] / g compute share.  It takes the g
 * lowest-index GPUs that have room for one share (memory and compute left,
 * fewer than ORC_MAX_PER_GPU jobs), all or nothing, and their residuals drop
 * by one share each.  occ[h * ORC_MAX_PER_GPU + i] lists GPU h's jobs in
 * placement order (-1 = empty slot).  Returns the number of shares placed.
 */
int64_t orc_binpack(const orc_problem *p, int b, const orc_iac *m, const int32_t *choice, int32_t *occ)
{
    const float *d = dem_of(p, b);
    double *mem = (double *)malloc(sizeof(double) * (size_t)m->G);
    double *sm = (double *)malloc(sizeof(double) * (size_t)m->G);
    int *cnt = (int *)calloc((size_t)m->G, sizeof(int));
    int64_t placed = 0, j;
    int h;
    if (mem == NULL || sm == NULL || cnt == NULL) { free(mem); free(sm); free(cnt); return -1; }
    for (h = 0; h < m->G; h++) { mem[h] = m->gpu_memory; sm[h] = m->gpu_compute; }
    for (h = 0; h < m->G * ORC_MAX_PER_GPU; h++) occ[h] = -1;
    for (j = 0; j < p->N; j++) {
        int64_t e;
        double gv, need_m, need_s;
        int g, sel[ORC_MAX_SHARDS], found = 0, i;
        if (choice[j] < 0) continue;
        e = p->offsets[j] + choice[j];
        gv = (double)d[e * p->R + m->r_gpus];
        if (!(gv >= 1.0 && gv <= ORC_MAX_SHARDS && gv == floor(gv))) continue;
        g = (int)gv;
        need_m = (double)d[e * p->R + m->r_mem] / gv;
        need_s = (double)d[e * p->R + m->r_sm] / gv;
        for (h = 0; h < m->G && found < g; h++)
            if (cnt[h] < ORC_MAX_PER_GPU && mem[h] >= need_m && sm[h] >= need_s) sel[found++] = h;
        if (found < g) continue;
        for (i = 0; i < g; i++) {
            h = sel[i];
            mem[h] = mem[h] - need_m;
            sm[h] = sm[h] - need_s;
            occ[h * ORC_MAX_PER_GPU + cnt[h]] = (int32_t)j;
            cnt[h]++;
        }
        placed += g;
    }
    free(mem); free(sm); free(cnt);
    return placed;
}

/*
 * IacPredict over every co-located pair (Alg. 1): on each GPU, every pair of
 * its jobs (x placed before y) with predicted slowdowns
 *     S_x|y = 1 + a_x * b_y,   S_y|x = 1 + a_y * b_x
 * (a = sensitivity, b = pressure of each job's chosen configuration: a
 * synthetic stand-in for the trained predictor of Sec. 3.3.2) against the
 * thresholds of Eq. 11,
 *     tau_x = tau_base_x + min(beta * (U / U_target - 1), beta_max),
 * U = (GPUs holding at least one job) / G, the packing's GPU utilisation.  A pair violates
 * when either slowdown exceeds its threshold; inc[x] receives the largest
 * excess S_x|y - tau_x of job x over all its pairs (0 if none).  Returns the
 * number of violating pairs.
 */
int64_t orc_iac_eval(const orc_problem *p, int b, const orc_iac *m, const int32_t *choice, const int32_t *occ,
                     double *inc)
{
    const float *sa = m->sensitivity + (int64_t)b * p->nnz;
    const float *pb = m->pressure + (int64_t)b * p->nnz;
    const double *tb = m->tau_base + (int64_t)b * p->N;
    double q, w, add;
    int64_t V = 0, j, used = 0;
    int h, x, y;
    for (j = 0; j < p->N; j++) inc[j] = 0.0;
    for (h = 0; h < m->G; h++) used += occ[h * ORC_MAX_PER_GPU] >= 0;
    q = (double)used / (double)m->G;
    q = q / m->u_target;
    w = q - 1.0;
    add = m->beta * w;
    if (add > m->beta_max) add = m->beta_max;
    for (h = 0; h < m->G; h++) {
        const int32_t *o = occ + h * ORC_MAX_PER_GPU;
        for (x = 0; x < ORC_MAX_PER_GPU; x++) {
            if (o[x] < 0) break;
            for (y = x + 1; y < ORC_MAX_PER_GPU; y++) {
                int32_t jx = o[x], jy = o[y];
                int64_t ex, ey;
                double sxy, syx, ox, oy;
                if (jy < 0) break;
                ex = p->offsets[jx] + choice[jx];
                ey = p->offsets[jy] + choice[jy];
                sxy = (double)sa[ex] * (double)pb[ey];
                sxy = 1.0 + sxy;
                syx = (double)sa[ey] * (double)pb[ex];
                syx = 1.0 + syx;
                ox = sxy - (tb[jx] + add);
                oy = syx - (tb[jy] + add);
                if (ox > 0.0 && ox > inc[jx]) inc[jx] = ox;
                if (oy > 0.0 && oy > inc[jy]) inc[jy] = oy;
                if (ox > 0.0 || oy > 0.0) V++;
            }
        }
    }
    return V;
}

/*
 * Alg. 1 for cluster b: Gamma <- 0 (the interference penalties; the switching
 * cost stays), then for rounds m = 1..M: the tatonnement (T iterations from
 * the current prices, t = 1.., stop tolerance tol) and the re-selection at
 * its prices, BinPack, IacPredict over co-located pairs; no violation ends
 * the loop, otherwise each violating job's chosen configuration has its
 * penalty raised by kappa times its largest excess,
 *     Gamma_jc <- (float)(Gamma_jc + kappa * inc_j),
 * and the next round starts from the prices reached.
 * penalty: [nnz] of cluster b, in/out; lam [R] in/out; choice [N] and occ
 * [G * ORC_MAX_PER_GPU] of the last round; *rounds = rounds run, *viol =
 * violating pairs of the last round.  Returns 0, or -1 on a failed solve.
 */
int orc_schedule(const orc_problem *p, int b, const orc_iac *m, int32_t M, int32_t T, double tol, double *lam,
                 float *penalty, int32_t *choice, int32_t *occ, int32_t *rounds, int64_t *viol)
{
    orc_problem v = *p;
    double *inc = (double *)malloc(sizeof(double) * (size_t)(p->N > 0 ? p->N : 1));
    int32_t r;
    int64_t j, e;
    if (inc == NULL) return -2;
    /* a one-cluster view of cluster b whose penalty is the working copy */
    v.B = 1;
    v.utility = p->utility + (int64_t)b * p->nnz;
    v.demand = p->demand + (int64_t)b * p->nnz * p->R;
    v.feasible = p->feasible ? p->feasible + (int64_t)b * p->nnz : NULL;
    v.capacity = p->capacity + (int64_t)b * p->R;
    v.eta0 = p->eta0 + b;
    v.current = p->current ? p->current + (int64_t)b * p->N : NULL;
    v.switch_cost = p->switch_cost ? p->switch_cost + b : NULL;
    v.penalty = penalty;
    for (e = 0; e < p->nnz; e++) penalty[e] = 0.0f;
    *rounds = 0;
    *viol = 0;
    for (r = 1; r <= M; r++) {
        int64_t V;
        if (orc_solve(&v, lam, T, 1, tol, NULL, NULL, NULL, NULL, NULL, choice, NULL, NULL) != 0) {
            free(inc);
            return -1;
        }
        if (orc_binpack(&v, 0, m, choice, occ) < 0) { free(inc); return -2; }
        V = orc_iac_eval(p, b, m, choice, occ, inc);
        *rounds = r;
        *viol = V;
        if (V == 0) break;
        for (j = 0; j < p->N; j++)
            if (inc[j] > 0.0) {
                e = p->offsets[j] + choice[j];
                penalty[e] = (float)((double)penalty[e] + m->kappa * inc[j]);
            }
    }
    free(inc);
    return 0;
}
