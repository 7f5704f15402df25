/*
 * ebrl_alloc.h -- the profile-guided elastic resource allocator of Section
 * 4.3.2 ("Elastic Resource Allocation"): Algorithm 1 over stage throughput
 * lookup tables, the end-to-end objective of Eq. (2), and the runtime
 * adaptation trigger.  Host code only: no call here touches a GPU.
 *
 * All rates are in one unit, rollout chunk-steps per second (the unit the
 * paper expresses every stage rate in for Eq. (2)).  Quotas are integer
 * percentages of the GPU's compute units; on one MI355X a quota s is a
 * stream whose CU mask covers s % of the CUs (ebrl.h).
 *
 * Readings of points the paper leaves open (each applied identically by the
 * allocator and by the test oracle):
 *  - c_env*, the "profiled per-environment core count": the candidate whose
 *    simulator rate at the largest profiled quota is highest (ties: the
 *    first candidate), among candidates with floor(N / c_env) >= 1.
 *  - Simulator knee: the smallest profiled simulator quota whose rate is at
 *    least (1 - knee_tol) times the best rate of c_env*'s row.
 *  - Generation and training rates between profiled quotas: linear in the
 *    quota; below the smallest profiled quota, linear from rate 0 at quota 0;
 *    above the largest, the largest quota's rate.  Batch sizes are used only
 *    at their profiled values.
 *  - "Best feasible pair": the (B_g, B_t) with gen_mem + train_mem <= M_gpu
 *    maximising min(T_s, P_gen(s_g, B_g), P_train(s_t, B_t)); ties keep the
 *    first pair in (B_g, B_t) grid order.  Memory does not depend on the
 *    quotas, so no feasible pair at all is reported up front (EBRL_E_OOM).
 *  - Endpoint tie (equal objective at lo and hi): the smaller generation
 *    quota, which leaves the extra compute units to training.
 *
 * Status codes are those of ebrl.h (EBRL_OK, EBRL_E_INVALID, EBRL_E_OOM).
 * Every pointer is host memory owned by the caller and read before return.
 */
#ifndef EBRL_ALLOC_H
#define EBRL_ALLOC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Stage lookup tables P_sim, P_gen, P_train (Section 4.3.2, "Stage
 * performance characterization").  Quota grids strictly ascending. */
typedef struct ebrl_alloc_profiles {
    /* simulator: sim_rate[c * n_ssim + j] is the rate with cenv[c] cores per
       environment, floor(cores / cenv[c]) concurrent environments and a
       simulator quota of ssim[j] percent (0 allowed: a CPU-only simulator) */
    int32_t n_cenv;
    const int32_t* cenv;
    int32_t n_ssim;
    const int32_t* ssim;
    const double* sim_rate;
    /* generation: gen_rate[i * n_bgen + j] at quota sgen[i] (1..100) and
       batch bgen[j]; gen_mem[j] = device bytes generation holds at bgen[j] */
    int32_t n_sgen;
    const int32_t* sgen;
    int32_t n_bgen;
    const int32_t* bgen;
    const double* gen_rate;
    const double* gen_mem;
    /* training: the same layout over strain x btrain */
    int32_t n_strain;
    const int32_t* strain;
    int32_t n_btrain;
    const int32_t* btrain;
    const double* train_rate;
    const double* train_mem;
} ebrl_alloc_profiles;

typedef struct ebrl_alloc_limits {
    int32_t cores;          /* N, CPU cores for simulation */
    double mem_bytes;       /* M_gpu, device memory for generation + training */
    int32_t sgen_min;       /* s_g^min, percent */
    int32_t strain_min;     /* s_t^min, percent */
    double knee_tol;        /* simulator knee tolerance (e.g. 0.05) */
} ebrl_alloc_limits;

typedef struct ebrl_alloc_result {
    int32_t cenv;           /* c_env* */
    int32_t envs;           /* E = floor(N / c_env*) */
    int32_t ssim;           /* s_sim* (percent) */
    int32_t sgen, strain;   /* s_g, s_t = 100 - s_sim* - s_g */
    int32_t bgen, btrain;   /* chosen batch sizes */
    int32_t iterations;     /* bisection steps taken */
    double t_sim;           /* T_s */
    double t_gen;           /* P_gen(s_g, B_g) */
    double t_train;         /* P_train(s_t, B_t) */
    double t_rollout;       /* T_r = min(T_s, P_gen) */
    double theta;           /* Eq. (2): min(T_r, T_train) */
} ebrl_alloc_result;

/* Algorithm 1: simulator first (cores per environment, concurrency, knee
 * quota, capacity T_s), then bisection of the generation quota between
 * s_g^min and 100 - s_sim* - s_t^min, moving toward training while rollout
 * is faster and toward generation otherwise, until the range is one point
 * wide; the better endpoint under Eq. (2) is returned.
 * EBRL_E_INVALID: NULL pointers, empty or unsorted grids, quotas outside
 * [0, 100], negative rates or memory, no c_env with floor(N / c_env) >= 1, or
 * s_g^min + s_t^min + s_sim* > 100.  EBRL_E_OOM: no batch pair fits M_gpu. */
int ebrl_alloc_solve(const ebrl_alloc_profiles* prof, const ebrl_alloc_limits* lim,
                     ebrl_alloc_result* out);

/* Eq. (2) at one configuration: fills t_gen, t_train, t_rollout and theta
 * of *out from the tables (t_sim, sgen, strain, bgen, btrain taken from
 * *out as given).  EBRL_E_INVALID if bgen or btrain is not a profiled batch
 * size or a quota is outside [0, 100]. */
int ebrl_alloc_objective(const ebrl_alloc_profiles* prof, ebrl_alloc_result* out);

/* Runtime adaptation (Section 4.3.2): moving averages of the observed
 * rollout and training rates over the last `window` steps; when their gap
 * exceeds `gap` times the faster of the two for `patience` consecutive
 * steps, observe() reports a trigger (rerun Algorithm 1) and clears its
 * history.  The paper's setting is window 20, gap 0.15, patience 20. */
typedef struct ebrl_alloc_monitor ebrl_alloc_monitor;

int ebrl_alloc_monitor_create(int32_t window, double gap, int32_t patience, ebrl_alloc_monitor** out);
/* *trigger = 1 when this observation completes a run of `patience` steps
 * over the gap, else 0.  Rates must be finite and >= 0. */
int ebrl_alloc_monitor_observe(ebrl_alloc_monitor* m, double rollout_rate, double train_rate,
                               int32_t* trigger);
void ebrl_alloc_monitor_destroy(ebrl_alloc_monitor* m);

/* Table refinement from runtime measurements (Section 4.3.2): the whole
 * generation column of batch cur->bgen is scaled by observed_gen /
 * cur->t_gen, and the training column of cur->btrain by observed_train /
 * cur->t_train, written to gen_rate_out [n_sgen * n_bgen] and
 * train_rate_out [n_strain * n_btrain] (which may alias the profile's
 * tables).  A rate of 0 (observed or predicted) leaves its column as is. */
int ebrl_alloc_refine(const ebrl_alloc_profiles* prof, const ebrl_alloc_result* cur, double observed_gen,
                      double observed_train, double* gen_rate_out, double* train_rate_out);

#ifdef __cplusplus
}
#endif
#endif /* EBRL_ALLOC_H */
