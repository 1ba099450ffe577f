/*
 * Serving simulation of Section 5.1: one server, first come first served, per-request
 * inference time from Eq. 2 and the request's reasoning trace, LASER's decisions at the
 * ATPs (Algorithm 1, Eq. 5-8).  Host only.
 *
 * With one FIFO server every request before i has finished when i starts, so the number
 * of requests in the system at a time t inside i's service is the number of requests
 * j >= i that have arrived by t.  Arrivals are sorted, so one cursor over them serves
 * every query of the run.
 */
#include <float.h>
#include <limits.h>
#include <math.h>
#include <stdlib.h>

#include "laser.h"
#include "laser_error.h"

/* requests j in [i, n) with arrival_s <= t; *cur is the first index not yet counted */
static int in_system(const laser_sim_request* req, int n, int i, int* cur, double t) {
  if (*cur < i) *cur = i;
  while (*cur < n && req[*cur].arrival_s <= t) ++*cur;
  return *cur - i;
}

/* milliseconds to decode n tokens starting at context c: sum over j < n of a + b (c + j) */
static double decode_cost_ms(const laser_sim_config* cfg, double c, double n) {
  return n * cfg->decode_ms + cfg->decode_ms_per_ctx * (n * c + n * (n - 1.0) / 2.0);
}

static int cmp_double(const void* a, const void* b) {
  const double x = *(const double*)a, y = *(const double*)b;
  return (x > y) - (x < y);
}

static laser_status validate(const laser_params* p, const laser_sim_config* cfg, int n, const laser_sim_request* req,
                             const int32_t* chunk_tokens, const float* confidence, const uint8_t* correct) {
  if (!p || !cfg || n < 0 || (n > 0 && !req)) return laser_fail(LASER_ERR_INVALID_ARG, "NULL argument or n < 0");
  if (cfg->method < LASER_SIM_VANILLA || cfg->method > LASER_SIM_NOTHINKING)
    return laser_fail(LASER_ERR_INVALID_ARG, "unknown method %d", cfg->method);
  if (!(cfg->prefill_ms >= 0 && cfg->prefill_ms_per_token >= 0 && cfg->decode_ms >= 0 &&
        cfg->decode_ms_per_ctx >= 0 && cfg->probe_ms >= 0 && cfg->probe_ms_per_ctx >= 0 && cfg->slo_s >= 0))
    return laser_fail(LASER_ERR_INVALID_ARG, "negative or NaN cost");
  if (cfg->max_probes < 0 || cfg->max_think_tokens < 0)
    return laser_fail(LASER_ERR_INVALID_ARG, "negative max_probes or max_think_tokens");
  if (isnan(cfg->fixed_lambda)) return laser_fail(LASER_ERR_INVALID_ARG, "fixed_lambda is NaN");
  if (!(p->L_target > 0.0) || !(p->lambda_min <= p->lambda_max) || p->p_max <= p->p_min || p->B_min < 1 ||
      !(p->f_min <= p->f_max) || !(p->alpha >= 0.0 && p->alpha <= 1.0))
    return laser_fail(LASER_ERR_INVALID_ARG, "invalid params");
  const int thinks = cfg->method != LASER_SIM_NOTHINKING;
  long long total = 0;
  for (int i = 0; i < n; ++i) {
    if (isnan(req[i].arrival_s) || (i > 0 && req[i].arrival_s < req[i - 1].arrival_s))
      return laser_fail(LASER_ERR_INVALID_ARG, "arrivals must be non-decreasing (request %d)", i);
    if (req[i].prompt_len < 0 || req[i].conclusion_tokens < 0)
      return laser_fail(LASER_ERR_INVALID_ARG, "negative prompt or conclusion length (request %d)", i);
    if (thinks && req[i].n_chunks < 1) return laser_fail(LASER_ERR_INVALID_ARG, "n_chunks < 1 (request %d)", i);
    if (req[i].n_chunks > 0) total += req[i].n_chunks;
  }
  if (thinks && total > 0) {
    if (!chunk_tokens || !confidence || !correct) return laser_fail(LASER_ERR_INVALID_ARG, "NULL chunk arrays");
    for (long long c = 0; c < total; ++c) {
      if (chunk_tokens[c] < 1) return laser_fail(LASER_ERR_INVALID_ARG, "chunk_tokens < 1 at %lld", c);
      if (isnan(confidence[c])) return laser_fail(LASER_ERR_INVALID_ARG, "NaN confidence at %lld", c);
    }
  }
  return LASER_OK;
}

laser_status laser_simulate(const laser_params* p, const laser_sim_config* cfg, int n, const laser_sim_request* req,
                            const int32_t* chunk_tokens, const float* confidence, const uint8_t* correct,
                            laser_sim_result* out, laser_sim_summary* summary) {
  laser_status st = validate(p, cfg, n, req, chunk_tokens, confidence, correct);
  if (st != LASER_OK) return st;
  const int method = cfg->method;
  const int probes_at_atp = method != LASER_SIM_VANILLA && method != LASER_SIM_NOTHINKING;
  const int adaptive = method == LASER_SIM_LASER || method == LASER_SIM_THRESHOLD_ONLY;
  const int budgeted = method == LASER_SIM_LASER || method == LASER_SIM_BUDGET_ONLY;
  double* lat = n > 0 ? (double*)malloc(sizeof(double) * (size_t)n) : NULL;
  if (n > 0 && !lat) return laser_fail(LASER_ERR_INVALID_ARG, "out of host memory");

  laser_load_state load = {0.0}; /* Algorithm 1: L_bar starts at 0 */
  int cursor = 0;
  long long c0 = 0; /* first chunk of the current request */
  double free_at = -DBL_MAX, sum_lat = 0, sum_tok = 0;
  int n_slo = 0, n_correct = 0, n_exit = 0;
  for (int i = 0; i < n; ++i) {
    const laser_sim_request* r = &req[i];
    laser_sim_result res;
    res.start_s = r->arrival_s > free_at ? r->arrival_s : free_at;
    res.lambda_last = NAN;
    res.budget = 0;
    res.chunks = res.probes = res.think_tokens = 0;
    double t = res.start_s;
    int B = INT_MAX;
    if (budgeted) {
      /* Algorithm 1: the budget is set before inference, from the load at that moment */
      const int L = in_system(req, n, i, &cursor, t);
      laser_budget(p, r->prompt_len, L, &B);
      res.budget = B;
    } else if (cfg->max_probes > 0) {
      B = cfg->max_probes;
    }
    t += (cfg->prefill_ms + cfg->prefill_ms_per_token * r->prompt_len) / 1000.0;
    double ctx = (double)r->prompt_len;
    int outcome = LASER_SIM_SKIPPED, answer = -1; /* answer: chunk whose answer is scored */
    if (method != LASER_SIM_NOTHINKING) {
      outcome = LASER_SIM_FINISHED;
      for (int k = 0; k < r->n_chunks; ++k) {
        const long long c = c0 + k;
        int ntok = chunk_tokens[c];
        int cut = 0; /* the token cap ends thinking here (unless it coincides with the end) */
        if (cfg->max_think_tokens > 0 && res.think_tokens + ntok >= cfg->max_think_tokens) {
          cut = res.think_tokens + ntok > cfg->max_think_tokens || k + 1 < r->n_chunks;
          ntok = cfg->max_think_tokens - res.think_tokens;
        }
        t += decode_cost_ms(cfg, ctx, (double)ntok) / 1000.0;
        ctx += ntok;
        res.think_tokens += ntok;
        res.chunks += 1;
        answer = (int)k;
        if (cut) {
          outcome = LASER_SIM_CAPPED;
          break;
        }
        if (k + 1 == r->n_chunks) break; /* the thinking phase ended by itself */
        if (!probes_at_atp) continue;
        /* the ATP after chunk k: trial answer and its confidence */
        t += (cfg->probe_ms + cfg->probe_ms_per_ctx * ctx) / 1000.0;
        res.probes += 1;
        const int L = in_system(req, n, i, &cursor, t);
        int decision;
        if (adaptive) {
          double lam;
          laser_exit_decision(p, &load, confidence[c], L, res.probes - 1, B, &decision, &lam);
          res.lambda_last = lam;
        } else {
          laser_ema_update(p, &load, L);
          res.lambda_last = cfg->fixed_lambda;
          if ((double)confidence[c] > cfg->fixed_lambda)
            decision = LASER_EARLY_EXIT;
          else
            decision = res.probes >= B ? LASER_BUDGET_EXHAUSTED : LASER_CONTINUE;
        }
        if (decision == LASER_EARLY_EXIT) {
          outcome = LASER_SIM_EXITED;
          break;
        }
        if (decision == LASER_BUDGET_EXHAUSTED) {
          outcome = LASER_SIM_EXHAUSTED;
          break;
        }
      }
    }
    t += decode_cost_ms(cfg, ctx, (double)r->conclusion_tokens) / 1000.0;
    res.finish_s = t;
    res.latency_s = t - r->arrival_s;
    res.outcome = outcome;
    res.correct = answer < 0 ? (r->nothink_correct != 0) : (correct[c0 + answer] != 0);
    if (r->n_chunks > 0) c0 += r->n_chunks;
    free_at = t;
    lat[i] = res.latency_s;
    sum_lat += res.latency_s;
    sum_tok += (double)res.think_tokens + (double)r->conclusion_tokens;
    n_slo += res.latency_s <= cfg->slo_s;
    n_correct += res.correct;
    n_exit += outcome == LASER_SIM_EXITED;
    if (out) out[i] = res;
  }
  if (summary) {
    laser_sim_summary s = {0};
    s.n = n;
    if (n > 0) {
      s.mean_latency_s = sum_lat / n;
      qsort(lat, (size_t)n, sizeof(double), cmp_double);
      const int rank = (int)ceil(0.95 * n); /* nearest rank, 1-based */
      s.p95_latency_s = lat[(rank < 1 ? 1 : rank) - 1];
      const double span = free_at - req[0].arrival_s;
      s.throughput_qps = span > 0 ? n / span : 0.0;
      s.slo_rate = (double)n_slo / n;
      s.accuracy = (double)n_correct / n;
      s.mean_tokens = sum_tok / n;
      s.early_exit_rate = (double)n_exit / n;
    }
    *summary = s;
  }
  free(lat);
  return LASER_OK;
}
