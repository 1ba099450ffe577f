/*
 * Host controller of LASER (Section 4): EMA load signal, load-aware exit threshold
 * (Eq. 5), budget pre-allocation (Eq. 6-8) and the per-ATP decision of Algorithm 1.
 * Pure C, no device access; every call is O(1) (Section 4.4).
 */
#include <math.h>

#include "laser.h"
#include "laser_error.h"

void laser_params_default(laser_params* p) {
  if (!p) return;
  /* Section 5.1 */
  p->lambda_base = 0.95;
  p->L_target = 10.0;
  p->beta = 0.04;
  p->gamma = 1.0;
  p->alpha = 0.3;
  p->B_base = 10;
  p->lambda_min = 0.88;
  p->lambda_max = 0.97;
  p->B_min = 2;
  /* Section 4.3 */
  p->f_min = 0.6;
  p->f_max = 1.5;
  p->p_min = 50;
  p->p_max = 275;
}

static int check_threshold_params(const laser_params* p) {
  if (!p) return laser_fail(LASER_ERR_INVALID_ARG, "params is NULL");
  if (!(p->L_target > 0.0)) return laser_fail(LASER_ERR_INVALID_ARG, "L_target must be > 0");
  if (!(p->lambda_min <= p->lambda_max)) return laser_fail(LASER_ERR_INVALID_ARG, "lambda_min > lambda_max");
  return LASER_OK;
}

laser_status laser_ema_update(const laser_params* p, laser_load_state* state, int active_requests) {
  if (!p || !state) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (active_requests < 0) return laser_fail(LASER_ERR_INVALID_ARG, "active_requests < 0");
  if (!(p->alpha >= 0.0 && p->alpha <= 1.0)) return laser_fail(LASER_ERR_INVALID_ARG, "alpha outside [0,1]");
  /* Section 4.2: L_bar(t) = alpha * L(t) + (1 - alpha) * L_bar(t-1) */
  state->L_bar = p->alpha * (double)active_requests + (1.0 - p->alpha) * state->L_bar;
  return LASER_OK;
}

static double threshold_of(const laser_params* p, double L_bar) {
  /* Eq. 5, then the [lambda_min, lambda_max] constraint of Eq. 4 */
  double lam = p->lambda_base - p->beta * tanh(p->gamma * (L_bar - p->L_target) / p->L_target);
  if (lam < p->lambda_min) lam = p->lambda_min;
  if (lam > p->lambda_max) lam = p->lambda_max;
  return lam;
}

laser_status laser_threshold(const laser_params* p, double L_bar, double* lambda_out) {
  int st = check_threshold_params(p);
  if (st != LASER_OK) return (laser_status)st;
  if (!lambda_out) return laser_fail(LASER_ERR_INVALID_ARG, "lambda_out is NULL");
  if (isnan(L_bar)) return laser_fail(LASER_ERR_INVALID_ARG, "L_bar is NaN");
  *lambda_out = threshold_of(p, L_bar);
  return LASER_OK;
}

laser_status laser_budget(const laser_params* p, int prompt_len, int active_requests, int* B_out) {
  if (!p || !B_out) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (prompt_len < 0 || active_requests < 0) return laser_fail(LASER_ERR_INVALID_ARG, "negative length or load");
  if (p->p_max <= p->p_min) return laser_fail(LASER_ERR_INVALID_ARG, "p_max must exceed p_min");
  if (p->B_min < 1) return laser_fail(LASER_ERR_INVALID_ARG, "B_min must be >= 1");
  if (!(p->f_min <= p->f_max)) return laser_fail(LASER_ERR_INVALID_ARG, "f_min > f_max");
  /* Eq. 7: linear in the prompt length, clipped to [f_min, f_max] */
  double f_diff = p->f_min + (double)(prompt_len - p->p_min) / (double)(p->p_max - p->p_min) * (p->f_max - p->f_min);
  if (f_diff < p->f_min) f_diff = p->f_min;
  if (f_diff > p->f_max) f_diff = p->f_max;
  /* Eq. 8 */
  int L = active_requests > 1 ? active_requests : 1;
  double f_load = p->L_target / (double)L;
  if (f_load > 1.0) f_load = 1.0;
  /* Eq. 6: floor of the exact product; the guard absorbs the representation error of
   * decimal parameters (an exact non-integer value sits at least ~1e-7 from an integer
   * for the parameter ranges this is used with). */
  double val = (double)p->B_base * f_diff * f_load;
  double fl = floor(val + 1e-9);
  int B = (int)fl;
  if (B < p->B_min) B = p->B_min;
  *B_out = B;
  return LASER_OK;
}

laser_status laser_exit_decision(const laser_params* p, laser_load_state* state, float confidence,
                                 int active_requests, int k_done, int B_i, int* decision_out,
                                 double* lambda_out) {
  int st = check_threshold_params(p);
  if (st != LASER_OK) return (laser_status)st;
  if (!state || !decision_out) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument");
  if (isnan(confidence)) return laser_fail(LASER_ERR_INVALID_ARG, "confidence is NaN");
  if (k_done < 0 || B_i < 1 || k_done >= B_i)
    return laser_fail(LASER_ERR_INVALID_ARG, "need 0 <= k_done < B_i");
  if (active_requests < 0) return laser_fail(LASER_ERR_INVALID_ARG, "active_requests < 0");
  if (!(p->alpha >= 0.0 && p->alpha <= 1.0)) return laser_fail(LASER_ERR_INVALID_ARG, "alpha outside [0,1]");
  /* Algorithm 1: update L_bar, recompute the threshold, compare, count the failed probe */
  state->L_bar = p->alpha * (double)active_requests + (1.0 - p->alpha) * state->L_bar;
  double lam = threshold_of(p, state->L_bar);
  if (lambda_out) *lambda_out = lam;
  if ((double)confidence > lam) {
    *decision_out = LASER_EARLY_EXIT;
  } else if (k_done + 1 >= B_i) {
    *decision_out = LASER_BUDGET_EXHAUSTED;
  } else {
    *decision_out = LASER_CONTINUE;
  }
  return LASER_OK;
}
