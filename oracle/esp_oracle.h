/*
 * CPU oracle for Elastic Shadow Pricing -- TEST INFRASTRUCTURE ONLY.
 * Declarations for esp_oracle.c (paper Sec. 3.2, Eq. 6-8).  Not shared with,
 * and not included by, the HIP library.
 */
#ifndef ESP_ORACLE_H
#define ESP_ORACLE_H
#include <stdint.h>

#define ORC_MAX_R 64
#define ORC_STEP_CONST 0
#define ORC_STEP_INV_SQRT 1

/* A logical problem: B clusters sharing one CSR family layout. */
typedef struct {
    int32_t B, N, R;
    int64_t nnz;
    const int64_t *offsets;   /* [N+1] */
    const float *utility;     /* [B][nnz] */
    const float *demand;      /* [B][nnz][R] */
    const uint8_t *feasible;  /* [B][nnz] or NULL */
    const double *capacity;   /* [B][R] */
    const double *eta0;       /* [B] */
    int32_t rule;
    /* Penalty term Gamma of Eq. 7 (all optional, NULL = absent): */
    const int32_t *current;   /* [B][N] current configuration, -1 = none */
    const double *switch_cost;/* [B] gamma_0, paid by every k != current */
    const float *penalty;     /* [B][nnz] interference penalty per configuration */
} orc_problem;

double orc_exact_sum_f32(const float *v, int64_t n);
double orc_score(const orc_problem *p, int b, int64_t j, int32_t k, const double *lam);
void orc_select(const orc_problem *p, int b, const double *lam, int32_t *choice);
void orc_demand(const orc_problem *p, int b, const int32_t *choice, double *U);
double orc_eta(int rule, double eta0, int64_t t);
void orc_update(int R, const double *U, const double *C, double eta, double *lam);
double orc_dual_value(const orc_problem *p, int b, const double *lam, const int32_t *choice);
double orc_primal_value(const orc_problem *p, int b, const int32_t *choice);
int orc_solve(const orc_problem *p, double *lam, int32_t T, int32_t t_start, double tol,
              double *tr_lam, double *tr_U, int32_t *tr_choice, double *tr_dual,
              double *tr_primal, int32_t *choice_out, double *U_out, int32_t *iters_done);
int orc_effective_capacity(const orc_problem *q, int b, const uint8_t *queued, const double *C,
                           double gamma, double *C_eff);
int32_t orc_nearest(const orc_problem *p, int b, int64_t f, const float *q, double *dist2);
void orc_nearest_batch(const orc_problem *p, int b, int64_t nq, const int32_t *family, const float *q,
                       int32_t *k, float *est);
#endif
