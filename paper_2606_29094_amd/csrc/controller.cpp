// Confidence-threshold controller (host library, libdlmctl.so): SLO-aware
// threshold choice and adaptive load control over a measured latency profile.
// The algorithms and the conventions are stated in include/dlm_ctl.h.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "../../include/dlm_ctl.h"

namespace {

thread_local std::string g_err;

dlm_status fail(const char* fmt, ...) {
  char buf[256];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return DLM_EINVAL;
}

dlm_status check_curve(const dlm_ctl_curve* c, bool may_be_empty) {
  if (!c) return fail("curve is NULL");
  if (c->n == 0 && may_be_empty) return DLM_OK;
  if (c->n < 1 || !c->tokens || !c->latency_s) return fail("curve has no points");
  for (int i = 0; i < c->n; ++i) {
    if (!(c->tokens[i] > 0.0) || !(c->latency_s[i] > 0.0) || !std::isfinite(c->latency_s[i]))
      return fail("curve point %d: tokens %g latency %g", i, c->tokens[i], c->latency_s[i]);
    if (i > 0 && !(c->tokens[i] > c->tokens[i - 1]))
      return fail("curve tokens not strictly ascending at point %d", i);
  }
  return DLM_OK;
}

dlm_status check_params(const dlm_ctl_params* p) {
  if (!p) return fail("params is NULL");
  if (p->n_gamma < 1 || p->n_gamma > DLM_CTL_MAX_GAMMA || !p->gamma)
    return fail("n_gamma %d outside [1, %d]", p->n_gamma, (int)DLM_CTL_MAX_GAMMA);
  for (int i = 1; i < p->n_gamma; ++i)
    if (!(p->gamma[i] > p->gamma[i - 1])) return fail("thresholds not strictly ascending");
  if (p->cache_block < 0) return fail("cache_block %d < 0", p->cache_block);
  if (p->max_seqs_per_batch < 1) return fail("max_seqs_per_batch %d < 1", p->max_seqs_per_batch);
  if (!(p->slo_s > 0.0)) return fail("slo_s %g is not positive", p->slo_s);
  return DLM_OK;
}

dlm_status check_req(const dlm_ctl_params* p, const dlm_ctl_req* r) {
  if (!r || !r->pred_steps_left) return fail("request or its step predictions are NULL");
  for (int i = 0; i < p->n_gamma; ++i)
    if (!(r->pred_steps_left[i] >= 0.0)) return fail("negative or NaN predicted steps");
  if (!(r->num_tokens >= 0.0) || !(r->recomp_steps_left >= 0.0))
    return fail("negative token count or recompute steps");
  return DLM_OK;
}

dlm_status check_instance(const dlm_ctl_instance* in) {
  if (!in || !in->profile) return fail("instance or its profile is NULL");
  dlm_status s = check_curve(&in->profile->recompute, false);
  if (s != DLM_OK) return s;
  s = check_curve(&in->profile->cache, true);
  if (s != DLM_OK) return s;
  if (in->num_reqs < 0 || !(in->num_tokens >= 0.0)) return fail("negative instance load");
  return DLM_OK;
}

double lat(const dlm_ctl_curve& c, double x) {
  const int n = c.n;
  if (n == 1 || x <= c.tokens[0]) return c.latency_s[0];
  int i = 1;
  while (i < n - 1 && x > c.tokens[i]) ++i;     // segment [i-1, i]; the last one extends
  const double w = (x - c.tokens[i - 1]) / (c.tokens[i] - c.tokens[i - 1]);
  return c.latency_s[i - 1] + w * (c.latency_s[i] - c.latency_s[i - 1]);
}

const dlm_ctl_curve& cache_curve(const dlm_ctl_profile& pr) {
  return pr.cache.n > 0 ? pr.cache : pr.recompute;
}

double time_left(const dlm_ctl_params& p, const dlm_ctl_instance& in, const dlm_ctl_req& r,
                 int gi) {
  const double steps = r.pred_steps_left[gi];
  const double recomp_lat = lat(in.profile->recompute, in.num_tokens);
  if (p.cache_block == 0) return steps * recomp_lat;
  const double cache_lat = lat(cache_curve(*in.profile), (double)p.cache_block * in.num_reqs);
  return (steps - r.recomp_steps_left) * cache_lat + r.recomp_steps_left * recomp_lat;
}

double load(const dlm_ctl_params& p, const dlm_ctl_req& r, int gi) {
  const double steps = r.pred_steps_left[gi];
  if (p.cache_block == 0) return steps * r.num_tokens;
  return (steps - r.recomp_steps_left) * p.cache_block + r.recomp_steps_left * r.num_tokens;
}

}  // namespace

extern "C" {

dlm_status dlm_ctl_latency(const dlm_ctl_curve* curve, double tokens, double* out_s) {
  g_err.clear();
  dlm_status s = check_curve(curve, false);
  if (s != DLM_OK) return s;
  if (!out_s) return fail("output is NULL");
  *out_s = lat(*curve, tokens);
  return DLM_OK;
}

dlm_status dlm_ctl_predicted_time_left(const dlm_ctl_params* p, const dlm_ctl_instance* inst,
                                       const dlm_ctl_req* req, int32_t gi, double* out_s) {
  g_err.clear();
  dlm_status s = check_params(p);
  if (s == DLM_OK) s = check_instance(inst);
  if (s == DLM_OK) s = check_req(p, req);
  if (s != DLM_OK) return s;
  if (gi < 0 || gi >= p->n_gamma) return fail("candidate %d out of range", gi);
  if (!out_s) return fail("output is NULL");
  *out_s = time_left(*p, *inst, *req, gi);
  return DLM_OK;
}

dlm_status dlm_ctl_update_threshold(const dlm_ctl_params* p, const dlm_ctl_instance* inst,
                                    dlm_ctl_req* req) {
  g_err.clear();
  dlm_status s = check_params(p);
  if (s == DLM_OK) s = check_instance(inst);
  if (s == DLM_OK) s = check_req(p, req);
  if (s != DLM_OK) return s;
  const uint32_t all = p->n_gamma == 32 ? 0xffffffffu : ((1u << p->n_gamma) - 1u);
  if ((req->allowed & all) == 0) return fail("request has no allowed threshold");
  // the highest allowed candidate that fits the remaining budget, else the
  // lowest allowed one
  int fit = -1, lowest = -1;
  for (int gi = 0; gi < p->n_gamma; ++gi) {
    if (!((req->allowed >> gi) & 1u)) continue;
    if (lowest < 0) lowest = gi;
    if (time_left(*p, *inst, *req, gi) <= req->slo_left_s) fit = gi;
  }
  req->gamma_idx = fit >= 0 ? fit : lowest;
  return DLM_OK;
}

dlm_status dlm_ctl_req_load(const dlm_ctl_params* p, const dlm_ctl_req* req, int32_t gi,
                            double* out) {
  g_err.clear();
  dlm_status s = check_params(p);
  if (s == DLM_OK) s = check_req(p, req);
  if (s != DLM_OK) return s;
  if (gi < 0 || gi >= p->n_gamma) return fail("candidate %d out of range", gi);
  if (!out) return fail("output is NULL");
  *out = load(*p, *req, gi);
  return DLM_OK;
}

dlm_status dlm_ctl_capacity(const dlm_ctl_params* p, const dlm_ctl_profile* profiles,
                            int32_t n_profiles, double tokens_per_req, double* out) {
  g_err.clear();
  dlm_status s = check_params(p);
  if (s != DLM_OK) return s;
  if (n_profiles < 0 || (n_profiles > 0 && !profiles)) return fail("profiles are NULL");
  if (!out) return fail("output is NULL");
  for (int i = 0; i < n_profiles; ++i) {
    s = check_curve(&profiles[i].recompute, false);
    if (s == DLM_OK) s = check_curve(&profiles[i].cache, true);
    if (s != DLM_OK) return s;
  }
  if (p->cache_block > 0 && !(tokens_per_req > 0.0)) return fail("tokens_per_req must be > 0");
  double total = 0.0;
  for (int i = 0; i < n_profiles; ++i) {
    const dlm_ctl_profile& pr = profiles[i];
    if (p->cache_block == 0) {
      double best = 0.0;
      for (int j = 0; j < pr.recompute.n; ++j)
        best = std::max(best, pr.recompute.tokens[j] / pr.recompute.latency_s[j]);
      total += best * p->slo_s;
    } else {
      const double step_load = (double)p->cache_block * p->max_seqs_per_batch;
      const double cache_lat = lat(cache_curve(pr), step_load);
      const double recomp_lat = lat(pr.recompute, tokens_per_req);
      const double nb = p->cache_block - 1;
      total += (step_load * nb + tokens_per_req) / (cache_lat * nb + recomp_lat) * p->slo_s;
    }
  }
  *out = total;
  return DLM_OK;
}

dlm_status dlm_ctl_update_allowed(const dlm_ctl_params* p, dlm_ctl_req* reqs, int32_t n,
                                  double capacity) {
  g_err.clear();
  dlm_status s = check_params(p);
  if (s != DLM_OK) return s;
  if (n < 0 || (n > 0 && !reqs)) return fail("requests are NULL");
  for (int i = 0; i < n; ++i) {
    s = check_req(p, &reqs[i]);
    if (s != DLM_OK) return s;
  }
  if (std::isnan(capacity)) return fail("capacity is NaN");
  // Worst case for request i: every earlier request at the maximum it was
  // given (`given`), request i at a candidate, every later request at the
  // lowest candidate. later[i] is that last sum; request i's maximum is the
  // largest candidate that keeps the worst case within capacity (the lowest
  // candidate when none does), and its allowed set every candidate up to it.
  std::vector<double> later(n > 0 ? n : 1, 0.0);
  double acc = 0.0;
  for (int i = n - 1; i >= 0; --i) {
    later[i] = acc;
    acc += load(*p, reqs[i], 0);
  }
  double given = 0.0;
  for (int i = 0; i < n; ++i) {
    int top = 0;
    for (int gi = 1; gi < p->n_gamma; ++gi)
      if (given + load(*p, reqs[i], gi) + later[i] <= capacity) top = gi;
    given += load(*p, reqs[i], top);
    reqs[i].allowed = top == 31 ? 0xffffffffu : ((2u << top) - 1u);
  }
  return DLM_OK;
}

const char* dlm_ctl_last_error(void) { return g_err.c_str(); }

}  // extern "C"
