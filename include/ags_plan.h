/*
 * libags planner: the host-side parallel performance and cost model of Tula
 * (arXiv 2603.18112, Sec. III-A), in the same library as the AGS step.
 * Host code only; no call touches the GPU.
 *
 *   step time, Eq. (2a)-(2c):  t_step = c0 + c_compute * b + c_sync * s(N)
 *       b = B / N the per-node batch, s(N) = N (centralized parameter
 *       server), 1 - 1/N (ring all-reduce) or 0 (none); c0 is an optional
 *       intercept for fixed per-step costs (the paper's terms are
 *       proportional), fitted by least squares on profiled samples: every
 *       profiled configuration (full search) or the extremes (partial
 *       search);
 *   memory bound, Eq. (3):     M_static + m_per_sample * b <= capacity
 *       (parameter, gradient and optimizer memory static; activation and
 *       batch memory linear in b);
 *   time and cost, Eq. (4a), (4b):  T = (E D / B) t_step,  C = T N p
 *       (T in seconds, p per node-hour);
 *   selection (Sec. III-A, configuration selection policy): minimum T,
 *       minimum C, or the knee of the T-B curve found with Kneedle
 *       (Satopaa, Albrecht, Irwin, Raghavan, ICDCS workshops 2011).
 *
 * Conventions: as in ags.h (C linkage, ags_status results, nothing
 * changed on error, ags_last_error(NULL) has the text of the last failed
 * call on this thread).  All arrays are host memory owned by the caller.
 */
#ifndef AGS_PLAN_H
#define AGS_PLAN_H

#include <stdint.h>

#include "ags.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { AGS_SYNC_NONE = 0, AGS_SYNC_RING = 1, AGS_SYNC_PS = 2 } ags_sync_model;

#define AGS_PLAN_INTERCEPT 1u /* c0        */
#define AGS_PLAN_COMPUTE 2u   /* c_compute */
#define AGS_PLAN_SYNC 4u      /* c_sync    */

/* One profiled configuration: N nodes, per-node batch b, seconds per step. */
typedef struct {
    int32_t nodes;      /* >= 1 */
    int32_t reserved;   /* must be 0 */
    double local_batch; /* finite, >= 0 */
    double t_step;      /* finite */
} ags_plan_sample;

typedef struct {
    ags_sync_model sync;
    uint32_t terms;      /* AGS_PLAN_* bits that were fitted */
    double c0, c_compute, c_sync;  /* terms not fitted are 0 */
    double rms_residual; /* sqrt(mean (t - t_model)^2) over the samples */
    int32_t n_samples;
    int32_t reserved;
} ags_plan_model;

/* Least-squares fit of Eq. (2) to n samples (Householder QR in fp64).
 * AGS_E_ARG for a bad sample, an empty or unknown term set, fewer samples
 * than terms, or terms the samples cannot tell apart (rank deficient, e.g.
 * the sync term with AGS_SYNC_NONE or with one cluster size only). */
ags_status ags_plan_fit(const ags_plan_sample *samples, int32_t n, ags_sync_model sync,
                        uint32_t terms, ags_plan_model *out);

/* t_step of Eq. (2) for N nodes and per-node batch b. */
ags_status ags_plan_step_time(const ags_plan_model *m, int32_t nodes, double local_batch,
                              double *t_step);

/* Eq. (4): seconds T and cost C of training E epochs of D samples at
 * global batch B on N nodes priced p per node-hour. */
ags_status ags_plan_time_cost(const ags_plan_model *m, int32_t nodes, double global_batch,
                              double epochs, double dataset_size, double price_per_node_hour,
                              double *T_seconds, double *cost);

/* Eq. (3): the largest integer b with m_static + m_per_sample * b <=
 * capacity (0 when even b = 0 does not fit); m_per_sample > 0. */
ags_status ags_plan_max_local_batch(double capacity, double m_static, double m_per_sample,
                                    int64_t *b_max);

typedef enum {
    AGS_KNEE_CONCAVE_INC = 0,
    AGS_KNEE_CONCAVE_DEC = 1,
    AGS_KNEE_CONVEX_INC = 2,
    AGS_KNEE_CONVEX_DEC = 3 /* e.g. training time over batch size */
} ags_knee_shape;

/* Kneedle on n points, x strictly increasing: both axes normalised to
 * [0, 1], the curve brought to the concave increasing form (y flipped for a
 * convex curve, x flipped for a decreasing concave one, both for an
 * increasing convex one), the difference curve y' - x' formed, and the
 * first local maximum whose difference curve then falls more than
 * sensitivity times the mean normalised x spacing below it, before the next
 * local maximum, is the knee.  *index = its position, or -1 when there is
 * none (also for n < 3 or a constant y).  sensitivity finite, >= 0. */
ags_status ags_plan_knee(const double *x, const double *y, int32_t n, ags_knee_shape shape,
                         double sensitivity, int32_t *index);

typedef enum { AGS_PLAN_MIN_TIME = 0, AGS_PLAN_MIN_COST = 1, AGS_PLAN_KNEE = 2 } ags_plan_objective;

typedef struct {
    int32_t nodes;       /* >= 1 */
    int32_t reserved;    /* must be 0 */
    double global_batch; /* B > 0 */
} ags_plan_candidate;

/* Choose among n candidates (N, B): T and C of Eq. (4) for each into
 * T_out / C_out [n] (may be NULL), +inf for candidates whose per-node batch
 * B / N exceeds max_local_batch (the memory bound); *best = the feasible
 * candidate of least T (AGS_PLAN_MIN_TIME) or least C (AGS_PLAN_MIN_COST),
 * the first on a tie, or the Kneedle knee of T over B among the feasible
 * candidates (AGS_PLAN_KNEE: one cluster size, B strictly increasing, else
 * AGS_E_ARG); -1 when nothing qualifies. */
ags_status ags_plan_select(const ags_plan_model *m, const ags_plan_candidate *cand, int32_t n,
                           double epochs, double dataset_size, double price_per_node_hour,
                           double max_local_batch, ags_plan_objective objective,
                           double sensitivity, int32_t *best, double *T_out, double *C_out);

#ifdef __cplusplus
}
#endif

#endif /* AGS_PLAN_H */
