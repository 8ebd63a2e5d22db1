/*
 * dlm_ctl.h - C ABI of the confidence-threshold controller, libdlmctl.so (host
 * code only, no GPU).
 *
 * The controller picks, per request, the confidence threshold its next
 * denoising steps use (paper, "Dynamic Confidence Threshold Adjustment and
 * Scheduling"):
 *  - dlm_ctl_update_threshold: the highest allowed candidate whose predicted
 *    remaining time fits the request's remaining SLO budget, else the lowest
 *    allowed one ("SLO-aware Confidence Threshold Adjustment", Algorithm 1;
 *    with KV caching the remaining time prices cache and recompute steps
 *    separately, appendix Algorithm 6);
 *  - dlm_ctl_update_allowed: adaptive load control - for requests in arrival
 *    order, the widest prefix of candidates whose worst-case aggregate load
 *    (committed load + this request + every later request at the lowest
 *    candidate) fits the cluster capacity ("Adaptive Load Control",
 *    Algorithm 2; loads and capacity with KV caching, appendix Algorithm 5).
 * Per-step latencies come from a latency profile measured on the GPU (step
 * latency over batch sizes in tokens); between measured points the latency
 * is linear in tokens, flat below the first point and linear along the last
 * segment beyond the last point.
 *
 * Conventions: all pointers are host pointers owned by the caller; nothing
 * is retained after a call returns. Candidate thresholds are indexed
 * 0..n_gamma-1 in ascending order. Every argument is validated first: on a
 * non-OK status no output is written and dlm_ctl_last_error() (thread-local)
 * holds the reason. Functions are reentrant.
 */
#ifndef DLM_CTL_H
#define DLM_CTL_H

#include <stdint.h>

#include "dlm.h"

#ifdef __cplusplus
extern "C" {
#endif

enum { DLM_CTL_MAX_GAMMA = 32 };

typedef struct dlm_ctl_curve {
  int32_t n;                  /* measured points (>= 1 for a used curve, 0 = absent)    */
  const double* tokens;       /* [n], strictly ascending, > 0                           */
  const double* latency_s;    /* [n], > 0                                               */
} dlm_ctl_curve;

typedef struct dlm_ctl_profile {
  dlm_ctl_curve recompute;    /* recompute / no-cache steps                             */
  dlm_ctl_curve cache;        /* cache steps; n = 0: the recompute curve is used        */
} dlm_ctl_profile;

typedef struct dlm_ctl_params {
  int32_t n_gamma;            /* 1..DLM_CTL_MAX_GAMMA                                   */
  const double* gamma;        /* [n_gamma], strictly ascending                          */
  int32_t cache_block;        /* KV-cache block size; 0 = no caching                    */
  int32_t max_seqs_per_batch; /* requests per batch (capacity with caching), >= 1       */
  double slo_s;               /* latency SLO: the capacity window, > 0                  */
} dlm_ctl_params;

typedef struct dlm_ctl_req {
  double num_tokens;          /* prompt + output length                                 */
  double recomp_steps_left;   /* remaining recompute steps (caching only)               */
  const double* pred_steps_left; /* [n_gamma] predicted remaining steps per candidate   */
  double slo_left_s;          /* remaining latency budget                               */
  uint32_t allowed;           /* bit i: candidate i allowed (dlm_ctl_update_allowed)    */
  int32_t gamma_idx;          /* chosen candidate (dlm_ctl_update_threshold)            */
} dlm_ctl_req;

typedef struct dlm_ctl_instance {
  const dlm_ctl_profile* profile;
  double num_tokens;          /* tokens of the batch the instance runs                  */
  int32_t num_reqs;           /* requests resident on it                                */
} dlm_ctl_instance;

/* Per-step latency at a batch of `tokens` tokens. */
dlm_status dlm_ctl_latency(const dlm_ctl_curve* curve, double tokens, double* out_s);

/* Predicted remaining time of req on inst under candidate gi (Alg. 1 / Alg. 6). */
dlm_status dlm_ctl_predicted_time_left(const dlm_ctl_params* p, const dlm_ctl_instance* inst,
                                       const dlm_ctl_req* req, int32_t gi, double* out_s);

/* Alg. 1: sets req->gamma_idx among the bits of req->allowed (which must be
 * non-empty): the highest one meeting req->slo_left_s, else the lowest. */
dlm_status dlm_ctl_update_threshold(const dlm_ctl_params* p, const dlm_ctl_instance* inst,
                                    dlm_ctl_req* req);

/* Load of req under candidate gi, in token-steps (Alg. 2 / Alg. 5). */
dlm_status dlm_ctl_req_load(const dlm_ctl_params* p, const dlm_ctl_req* req, int32_t gi,
                            double* out);

/* Capacity over the SLO window of instances with the given profiles, in
 * token-steps (Alg. 2 / Alg. 5; tokens_per_req is the average request length,
 * used with caching). */
dlm_status dlm_ctl_capacity(const dlm_ctl_params* p, const dlm_ctl_profile* profiles,
                            int32_t n_profiles, double tokens_per_req, double* out);

/* Alg. 2: sets reqs[i].allowed for n requests in arrival order. */
dlm_status dlm_ctl_update_allowed(const dlm_ctl_params* p, dlm_ctl_req* reqs, int32_t n,
                                  double capacity);

/* Message for the last non-OK status on this thread ("" if none). */
const char* dlm_ctl_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* DLM_CTL_H */
