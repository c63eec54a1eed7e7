/*
 * pearl_pd.h -- C ABI of the PD decision engine, the minimal-change orchestration plan and the
 * intra-scale toggle gate (host code; no GPU involved).
 *
 * The paper's controller decides, for each elastic event, whether rollout workers run prefill
 * and decode colocated or disaggregated, and with which prefill/decode split; it turns the
 * decision into a plan that changes as few workers as possible; and it borrows idle training
 * GPUs only when the gain pays for the hand-off (paper, section 4: Design).
 *
 * Models (section 4.3.1), all times in seconds:
 *   colocated (Eq. 1):   T_coloc = S [ (B dL / N) t_prefill + r (A + b B / N) + T_over ] + T_env
 *   decode path (Eq. 2): T_decode = S r (A + b B / (N_D (1 + theta))) (1 + theta)
 *   prefill path (Eq. 3): T_prefill = S ( (B dL / N_P) t_prefill + B dL K / BW )
 *   disaggregated:       T_dis = max(T_prefill, T_decode) + T_env
 * Capacity constraints of a disaggregated split (section 4.2): N_P, N_D >= 1; the decode pool
 * holds the batch's KV cache, B K_seq <= N_D H_max; and the prefill pool keeps pace with the
 * prefill token load lambda_P = B S dL: lambda_P t_prefill / N_P <= u_max * T_decode(N_D).
 * Colocation is always feasible (the fallback).
 *
 * Conventions: every function is pure and re-entrant and allocates nothing.  Functions returning
 * pearl_status validate their arguments (pearl_last_error() names the problem); functions
 * returning double return NaN for invalid arguments.  All arithmetic is IEEE double, evaluated
 * in the order the equations are written (no fused multiply-add contraction).
 */
#ifndef PEARL_PD_H
#define PEARL_PD_H

#include <stdint.h>

#include "pearl_attn.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Workload profile and platform parameters of the makespan models.  Every field is finite;
 * BW > 0, u_max > 0, B > 0, the rest >= 0. */
typedef struct {
  double B;          /* trajectories in the batch */
  double S;          /* interaction turns of the slowest trajectory */
  double dL;         /* prompt tokens added per turn */
  double r;          /* tokens generated per turn */
  double theta;      /* bubble ratio (1 - f) / f, f = fraction of trajectories actively decoding */
  double A;          /* fixed per-iteration decode cost of one worker (weights, dispatch) */
  double b;          /* marginal decode cost per concurrent sequence (mainly KV-cache reads) */
  double t_prefill;  /* per-token prefill time of one worker */
  double T_over;     /* colocated per-turn overhead (prefill/decode switching) */
  double T_env;      /* environment interaction time */
  double K;          /* KV transfer volume per token, bytes */
  double BW;         /* bandwidth between the prefill and decode pools, bytes/s */
  double K_seq;      /* KV-cache bytes per trajectory */
  double H_max;      /* HBM bytes per worker available to the KV cache */
  double u_max;      /* cap on the prefill pool's busy time relative to the decode path */
} pearl_pd_params;

enum { PEARL_PD_COLOC = 0, PEARL_PD_DIS = 1, PEARL_PD_NONE = -1 };

/* A configuration pi = (N_P, N_D, N_C): colocated (n_p = n_d = 0, n_c = N) or disaggregated
 * (n_c = 0, n_p, n_d >= 1), with its predicted makespan. */
typedef struct {
  int32_t mode;      /* PEARL_PD_COLOC, PEARL_PD_DIS, or PEARL_PD_NONE (no such configuration) */
  int32_t n_p, n_d, n_c;
  double makespan;
} pearl_pd_config;

/* Why pearl_pd_decide chose its target. */
enum { PEARL_PD_INITIAL = 0, PEARL_PD_KEEP = 1, PEARL_PD_SWITCH = 2, PEARL_PD_FORCED = 3 };

/* Eq. 1 with N workers; Eq. 2; Eq. 3; T_dis; the capacity constraints (1 feasible, 0 not, -1
 * invalid arguments). */
double pearl_pd_makespan_coloc(const pearl_pd_params* p, int32_t n);
double pearl_pd_decode_path(const pearl_pd_params* p, int32_t n_d);
double pearl_pd_prefill_path(const pearl_pd_params* p, int32_t n_p);
double pearl_pd_makespan_dis(const pearl_pd_params* p, int32_t n_p, int32_t n_d);
int32_t pearl_pd_feasible_dis(const pearl_pd_params* p, int32_t n_p, int32_t n_d);

/*
 * Enumeration (section 4.3.2): every N_P in [1, n-1] with N_D = n - N_P, infeasible splits
 * dropped, the best compared against colocation.  Ties keep colocation; among disaggregated
 * splits the smallest N_P wins.  best receives the optimum; best_dis (nullable) the best
 * feasible disaggregated split or mode PEARL_PD_NONE; t_coloc (nullable) Eq. 1.  n >= 1.
 */
pearl_status pearl_pd_best(const pearl_pd_params* p, int32_t n, pearl_pd_config* best,
                           pearl_pd_config* best_dis, double* t_coloc);

/*
 * Online decision with mode-dependent hysteresis (section 4.3.2).  current (nullable: no
 * configuration yet) gives the mode and, when disaggregated, n_p and n_d.  A disaggregated
 * current configuration whose counts do not add up to n or that violates a capacity constraint
 * forces the optimum.  Otherwise each candidate differing from the current configuration (the
 * best colocated and the best disaggregated) is admitted when its makespan is below the current
 * one's times (1 - delta), delta = delta_mode for a colocation <-> disaggregation switch and
 * delta_ratio for a ratio change; the admitted candidate with the lowest makespan becomes the
 * target, and with none admitted the current configuration is kept.  Thresholds are fractions
 * in [0, 1).  reason receives PEARL_PD_INITIAL / KEEP / SWITCH / FORCED.
 */
pearl_status pearl_pd_decide(const pearl_pd_params* p, int32_t n, const pearl_pd_config* current,
                             double delta_mode, double delta_ratio, pearl_pd_config* target,
                             int32_t* reason);

/* Worker roles in the unified GPU-worker-role table (section 4.4.1, Eq. 4). */
enum { PEARL_ROLE_NONE = 0, PEARL_ROLE_PREFILL = 1, PEARL_ROLE_DECODE = 2, PEARL_ROLE_COLOC = 3 };

/*
 * Minimal-change plan (section 4.4.2, Eqs. 5 and 6).  Slots are stable worker identifiers.
 *   cur_role[w]: role of slot w in the current active set W (PEARL_ROLE_NONE: not active);
 *   target_active[w]: nonzero when slot w is in the target active set W';
 *   n_prefill + n_decode + n_coloc must equal |W'|.
 * new_role[w] receives the role of slot w after the transition (PEARL_ROLE_NONE outside W').
 * Survivors keep their role up to its target count (ascending slots); the remaining deficits,
 * role by role (prefill, decode, colocated), take reassigned survivors first, then added
 * workers, in ascending slot order.  d_worker = |W' \ W| + |W \ W'| and d_role = survivors whose
 * role changes; their sum is the minimum over all assignments.  W_add, W_remove and the role
 * map are read off cur_role / new_role.  Arrays have num_slots entries; caller-owned.
 */
pearl_status pearl_plan_min_change(int32_t num_slots, const int32_t* cur_role, const uint8_t* target_active,
                                   int32_t n_prefill, int32_t n_decode, int32_t n_coloc, int32_t* new_role,
                                   int32_t* d_worker, int32_t* d_role);

/* Benefit-aware toggle gate (section 4.6, Eq. 7): 1 when (R / B)(T_ded - T_full) > T_toggle,
 * 0 otherwise, -1 for invalid arguments (B <= 0 or a non-finite value). */
int32_t pearl_toggle_gate(double R, double B, double T_ded, double T_full, double T_toggle);

/* Eq. 7 with T_ded = the best predicted makespan on the n_ded dedicated workers and T_full = the
 * best on n_ded + n_overlap workers (training GPUs borrowed as overlap workers); R of the B
 * trajectories remain. */
pearl_status pearl_toggle_decide(const pearl_pd_params* p, int32_t n_ded, int32_t n_overlap, double R,
                                 double T_toggle, int32_t* enable, double* T_ded, double* T_full);

/* Runtime refits from telemetry (section 4.3.2; Implementation, runtime statistics):
 * least-squares A and b of iter_time = A + b * concurrency (n >= 2 distinct concurrencies);
 * least-squares t_prefill of time = tokens * t_prefill (n >= 1, some tokens > 0);
 * theta = (1 - f) / f for 0 < f <= 1 (NaN otherwise); one exponential-moving-average step
 * alpha * obs + (1 - alpha) * prev. */
pearl_status pearl_pd_fit_decode_cost(const double* concurrency, const double* iter_time, int32_t n,
                                      double* A, double* b);
pearl_status pearl_pd_fit_prefill_cost(const double* tokens, const double* time, int32_t n, double* t_prefill);
double pearl_pd_bubble_ratio(double f);
double pearl_pd_ema(double prev, double obs, double alpha);

#ifdef __cplusplus
}
#endif

#endif /* PEARL_PD_H */
