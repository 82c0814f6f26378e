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

/* Alg. 1 outer rounds: cluster model and synthetic interference inputs. */
#define ORC_MAX_PER_GPU 4
#define ORC_MAX_SHARDS 8
typedef struct {
    int32_t G;                /* GPUs of the cluster */
    double gpu_memory;        /* per-GPU capacity of resource r_mem */
    double gpu_compute;       /* per-GPU capacity of resource r_sm */
    int32_t r_gpus, r_mem, r_sm;
    const float *sensitivity; /* [B][nnz] a of each configuration */
    const float *pressure;    /* [B][nnz] b of each configuration */
    const double *tau_base;   /* [B][N] */
    double beta, beta_max, u_target, kappa;
} orc_iac;
int64_t orc_binpack(const orc_problem *p, int b, const orc_iac *m, const int32_t *choice, int32_t *occ);
int64_t orc_iac_eval(const orc_problem *p, int b, const orc_iac *m, const int32_t *choice, const int32_t *occ,
                     double *inc);
int orc_schedule(const orc_problem *p, int b, const orc_iac *m, int32_t M, int32_t T, double tol, double *lam,
                 float *penalty, int32_t *choice, int32_t *occ, int32_t *rounds, int64_t *viol);
#endif
