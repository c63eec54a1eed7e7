// PD decision engine, minimal-change orchestration plan and intra-scale toggle gate (host code).
// The contract, the models and the tie/hysteresis rules are documented in include/pearl_pd.h.

#include "../../include/pearl_pd.h"
#include "pearl_internal.h"

#include <cmath>
#include <limits>
#include <vector>

// Evaluate every expression exactly as written: no fused multiply-add contraction.
#pragma clang fp contract(off)

namespace pearl {
namespace {

constexpr double kNaN = std::numeric_limits<double>::quiet_NaN();

bool finite_nonneg(double x) { return std::isfinite(x) && x >= 0.0; }

bool params_ok(const pearl_pd_params* p) {
  if (!p) return false;
  const double nonneg[] = {p->S, p->dL, p->r, p->theta, p->A, p->b, p->t_prefill, p->T_over, p->T_env,
                           p->K, p->K_seq, p->H_max};
  for (double x : nonneg)
    if (!finite_nonneg(x)) return false;
  return std::isfinite(p->B) && p->B > 0.0 && std::isfinite(p->BW) && p->BW > 0.0 && std::isfinite(p->u_max) &&
         p->u_max > 0.0;
}

pearl_status bad_params() {
  return set_error(PEARL_ERR_INVALID_ARG,
                   "pd params: need finite values, B > 0, BW > 0, u_max > 0 and every other field >= 0");
}

// Eq. 1
double coloc(const pearl_pd_params& p, int n) {
  const double t_pre_turn = p.B * p.dL / n * p.t_prefill;
  const double t_dec_turn = p.r * (p.A + p.b * p.B / n);
  return p.S * (t_pre_turn + t_dec_turn + p.T_over) + p.T_env;
}

// Eq. 2
double decode_path(const pearl_pd_params& p, int n_d) {
  const double th = p.theta;
  return p.S * p.r * (p.A + p.b * p.B / (n_d * (1.0 + th))) * (1.0 + th);
}

// Eq. 3
double prefill_path(const pearl_pd_params& p, int n_p) {
  return p.S * (p.B * p.dL / n_p * p.t_prefill + p.B * p.dL * p.K / p.BW);
}

double dis(const pearl_pd_params& p, int n_p, int n_d) {
  return std::fmax(prefill_path(p, n_p), decode_path(p, n_d)) + p.T_env;
}

// capacity constraints (section 4.2)
bool feasible(const pearl_pd_params& p, int n_p, int n_d) {
  if (n_p < 1 || n_d < 1) return false;
  const bool holds_kv = p.B * p.K_seq <= n_d * p.H_max;
  const double lam = p.B * p.S * p.dL;
  const bool keeps_pace = lam * p.t_prefill / n_p <= p.u_max * decode_path(p, n_d);
  return holds_kv && keeps_pace;
}

pearl_pd_config make_coloc(int n, double t) { return pearl_pd_config{PEARL_PD_COLOC, 0, 0, n, t}; }
pearl_pd_config make_dis(int n_p, int n_d, double t) { return pearl_pd_config{PEARL_PD_DIS, n_p, n_d, 0, t}; }
pearl_pd_config make_none() { return pearl_pd_config{PEARL_PD_NONE, 0, 0, 0, kNaN}; }

// enumeration over N_P in [1, n-1] (section 4.3.2)
void best_of(const pearl_pd_params& p, int n, pearl_pd_config* best, pearl_pd_config* best_dis, double* t_coloc) {
  const double tc = coloc(p, n);
  pearl_pd_config bd = make_none();
  for (int n_p = 1; n_p < n; ++n_p) {
    const int n_d = n - n_p;
    if (!feasible(p, n_p, n_d)) continue;
    const double t = dis(p, n_p, n_d);
    if (bd.mode == PEARL_PD_NONE || t < bd.makespan) bd = make_dis(n_p, n_d, t);
  }
  *best = (bd.mode == PEARL_PD_DIS && bd.makespan < tc) ? bd : make_coloc(n, tc);
  *best_dis = bd;
  *t_coloc = tc;
}

bool same_config(const pearl_pd_config& a, const pearl_pd_config& b) {
  return a.mode == b.mode && a.n_p == b.n_p && a.n_d == b.n_d && a.n_c == b.n_c;
}

}  // namespace
}  // namespace pearl

using namespace pearl;

extern "C" {

double pearl_pd_makespan_coloc(const pearl_pd_params* p, int32_t n) {
  return params_ok(p) && n >= 1 ? coloc(*p, n) : kNaN;
}

double pearl_pd_decode_path(const pearl_pd_params* p, int32_t n_d) {
  return params_ok(p) && n_d >= 1 ? decode_path(*p, n_d) : kNaN;
}

double pearl_pd_prefill_path(const pearl_pd_params* p, int32_t n_p) {
  return params_ok(p) && n_p >= 1 ? prefill_path(*p, n_p) : kNaN;
}

double pearl_pd_makespan_dis(const pearl_pd_params* p, int32_t n_p, int32_t n_d) {
  return params_ok(p) && n_p >= 1 && n_d >= 1 ? dis(*p, n_p, n_d) : kNaN;
}

int32_t pearl_pd_feasible_dis(const pearl_pd_params* p, int32_t n_p, int32_t n_d) {
  if (!params_ok(p)) return -1;
  return feasible(*p, n_p, n_d) ? 1 : 0;
}

pearl_status pearl_pd_best(const pearl_pd_params* p, int32_t n, pearl_pd_config* best,
                           pearl_pd_config* best_dis, double* t_coloc) {
  clear_error();
  if (!params_ok(p)) return bad_params();
  if (n < 1) return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_best: n must be >= 1");
  if (!best) return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_best: best is NULL");
  pearl_pd_config b, bd;
  double tc;
  best_of(*p, n, &b, &bd, &tc);
  *best = b;
  if (best_dis) *best_dis = bd;
  if (t_coloc) *t_coloc = tc;
  return PEARL_OK;
}

pearl_status pearl_pd_decide(const pearl_pd_params* p, int32_t n, const pearl_pd_config* current,
                             double delta_mode, double delta_ratio, pearl_pd_config* target, int32_t* reason) {
  clear_error();
  if (!params_ok(p)) return bad_params();
  if (n < 1) return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_decide: n must be >= 1");
  if (!target || !reason) return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_decide: target and reason must be non-NULL");
  if (!(delta_mode >= 0.0 && delta_mode < 1.0) || !(delta_ratio >= 0.0 && delta_ratio < 1.0))
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_decide: thresholds must lie in [0, 1)");
  if (current && current->mode != PEARL_PD_COLOC && current->mode != PEARL_PD_DIS)
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_decide: current mode must be PEARL_PD_COLOC or PEARL_PD_DIS");
  pearl_pd_config best, best_dis;
  double tc;
  best_of(*p, n, &best, &best_dis, &tc);
  if (!current) {
    *target = best;
    *reason = PEARL_PD_INITIAL;
    return PEARL_OK;
  }
  if (current->mode == PEARL_PD_DIS &&
      ((int64_t)current->n_p + current->n_d != n || !feasible(*p, current->n_p, current->n_d))) {
    *target = best;
    *reason = PEARL_PD_FORCED;
    return PEARL_OK;
  }
  const pearl_pd_config cur = current->mode == PEARL_PD_COLOC
                                  ? make_coloc(n, tc)
                                  : make_dis(current->n_p, current->n_d, dis(*p, current->n_p, current->n_d));
  const pearl_pd_config cands[2] = {make_coloc(n, tc), best_dis};
  const pearl_pd_config* admitted = nullptr;
  for (const pearl_pd_config& c : cands) {
    if (c.mode == PEARL_PD_NONE || same_config(c, cur)) continue;
    const double delta = c.mode != cur.mode ? delta_mode : delta_ratio;
    if (c.makespan < cur.makespan * (1.0 - delta))
      if (!admitted || c.makespan < admitted->makespan) admitted = &c;
  }
  *target = admitted ? *admitted : cur;
  *reason = admitted ? PEARL_PD_SWITCH : PEARL_PD_KEEP;
  return PEARL_OK;
}

pearl_status pearl_plan_min_change(int32_t num_slots, const int32_t* cur_role, const uint8_t* target_active,
                                   int32_t n_prefill, int32_t n_decode, int32_t n_coloc, int32_t* new_role,
                                   int32_t* d_worker, int32_t* d_role) {
  clear_error();
  if (num_slots < 0) return set_error(PEARL_ERR_INVALID_ARG, "pearl_plan_min_change: num_slots < 0");
  if (num_slots > 0 && (!cur_role || !target_active || !new_role))
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_plan_min_change: NULL array");
  if (!d_worker || !d_role) return set_error(PEARL_ERR_INVALID_ARG, "pearl_plan_min_change: NULL count output");
  if (n_prefill < 0 || n_decode < 0 || n_coloc < 0)
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_plan_min_change: negative target count");
  int64_t n_target = 0;
  for (int w = 0; w < num_slots; ++w) {
    if (cur_role[w] < PEARL_ROLE_NONE || cur_role[w] > PEARL_ROLE_COLOC)
      return set_error(PEARL_ERR_INVALID_ARG, "pearl_plan_min_change: cur_role[%d] = %d is not a role", w, cur_role[w]);
    n_target += target_active[w] != 0;
  }
  if ((int64_t)n_prefill + n_decode + n_coloc != n_target)
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_plan_min_change: target counts add up to %lld, |W'| = %lld",
                     (long long)n_prefill + n_decode + n_coloc, (long long)n_target);
  const int32_t roles[3] = {PEARL_ROLE_PREFILL, PEARL_ROLE_DECODE, PEARL_ROLE_COLOC};
  const int32_t want[4] = {0, n_prefill, n_decode, n_coloc};
  int32_t kept[4] = {0, 0, 0, 0};
  std::vector<int32_t> excess, added;
  int32_t dw = 0;
  for (int w = 0; w < num_slots; ++w) {
    const bool now = cur_role[w] != PEARL_ROLE_NONE, next = target_active[w] != 0;
    new_role[w] = PEARL_ROLE_NONE;
    if (now != next) ++dw;
    if (!next) continue;
    if (!now) {
      added.push_back(w);
    } else if (kept[cur_role[w]] < want[cur_role[w]]) {
      new_role[w] = cur_role[w];            // survivor keeps its role
      ++kept[cur_role[w]];
    } else {
      excess.push_back(w);                  // survivor whose role is over its target count
    }
  }
  size_t i = 0, j = 0;
  for (int32_t r : roles)
    for (int32_t k = kept[r]; k < want[r]; ++k) {
      if (i < excess.size()) new_role[excess[i++]] = r;
      else new_role[added[j++]] = r;
    }
  *d_worker = dw;
  *d_role = (int32_t)excess.size();
  return PEARL_OK;
}

int32_t pearl_toggle_gate(double R, double B, double T_ded, double T_full, double T_toggle) {
  if (!(B > 0.0) || !std::isfinite(B) || !std::isfinite(R) || !std::isfinite(T_ded) || !std::isfinite(T_full) ||
      !std::isfinite(T_toggle))
    return -1;
  return (R / B) * (T_ded - T_full) > T_toggle ? 1 : 0;
}

pearl_status pearl_toggle_decide(const pearl_pd_params* p, int32_t n_ded, int32_t n_overlap, double R,
                                 double T_toggle, int32_t* enable, double* T_ded, double* T_full) {
  clear_error();
  if (!params_ok(p)) return bad_params();
  if (n_ded < 1 || n_overlap < 0 || (int64_t)n_ded + n_overlap > INT32_MAX)
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_toggle_decide: need n_ded >= 1 and n_overlap >= 0");
  if (!enable || !std::isfinite(R) || R < 0.0 || !std::isfinite(T_toggle))
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_toggle_decide: need enable non-NULL, finite R >= 0 and T_toggle");
  pearl_pd_config b, bd;
  double tc;
  best_of(*p, n_ded, &b, &bd, &tc);
  const double t_ded = b.makespan;
  best_of(*p, n_ded + n_overlap, &b, &bd, &tc);
  const double t_full = b.makespan;
  *enable = pearl_toggle_gate(R, p->B, t_ded, t_full, T_toggle) == 1 ? 1 : 0;
  if (T_ded) *T_ded = t_ded;
  if (T_full) *T_full = t_full;
  return PEARL_OK;
}

pearl_status pearl_pd_fit_decode_cost(const double* concurrency, const double* iter_time, int32_t n, double* A,
                                      double* b) {
  clear_error();
  if (n < 2 || !concurrency || !iter_time || !A || !b)
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_fit_decode_cost: need n >= 2 samples and non-NULL pointers");
  double mx = 0.0, my = 0.0;
  for (int i = 0; i < n; ++i) {
    if (!std::isfinite(concurrency[i]) || !std::isfinite(iter_time[i]))
      return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_fit_decode_cost: sample %d is not finite", i);
    mx += concurrency[i];
    my += iter_time[i];
  }
  mx /= n;
  my /= n;
  double sxx = 0.0, sxy = 0.0;
  for (int i = 0; i < n; ++i) {
    sxx += (concurrency[i] - mx) * (concurrency[i] - mx);
    sxy += (concurrency[i] - mx) * (iter_time[i] - my);
  }
  if (!(sxx > 0.0))
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_fit_decode_cost: need two distinct concurrencies");
  *b = sxy / sxx;
  *A = my - *b * mx;
  return PEARL_OK;
}

pearl_status pearl_pd_fit_prefill_cost(const double* tokens, const double* time, int32_t n, double* t_prefill) {
  clear_error();
  if (n < 1 || !tokens || !time || !t_prefill)
    return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_fit_prefill_cost: need n >= 1 samples and non-NULL pointers");
  double sxx = 0.0, sxy = 0.0;
  for (int i = 0; i < n; ++i) {
    if (!std::isfinite(tokens[i]) || !std::isfinite(time[i]))
      return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_fit_prefill_cost: sample %d is not finite", i);
    sxx += tokens[i] * tokens[i];
    sxy += tokens[i] * time[i];
  }
  if (!(sxx > 0.0)) return set_error(PEARL_ERR_INVALID_ARG, "pearl_pd_fit_prefill_cost: every token count is 0");
  *t_prefill = sxy / sxx;
  return PEARL_OK;
}

double pearl_pd_bubble_ratio(double f) { return (f > 0.0 && f <= 1.0) ? (1.0 - f) / f : kNaN; }

double pearl_pd_ema(double prev, double obs, double alpha) { return alpha * obs + (1.0 - alpha) * prev; }

}  // extern "C"
