/*
 * specrouter_sched.h -- C ABI of the model-chain scheduler (SpecRouter,
 * arXiv 2505.07680, Section 4.2 and Algorithm 1).
 *
 * Host code only: every pointer here is a HOST pointer, nothing touches the
 * GPU. The scheduler keeps, per model M_i, a smoothed per-token time T_i and,
 * per ordered pair (draft M_i, verifier M_j), a smoothed total variation
 * distance E[DTV] (Eq. 5, Eq. 6), fed by the `tv` output of
 * specrouter_accept_and_diverge. It predicts each candidate chain's effective
 * time per target token (Eq. 7) and picks the fastest (Algorithm 1).
 *
 * The paper fixes the structure but not every term; this library takes:
 *   - EMA: x <- w * measured + (1 - w) * x, where the first observation of an
 *     unset metric sets it (w = ema_time for T_i, ema_sim for E[DTV]).
 *   - SimScore(i, j) = 1 - E[DTV(i, j)] (Eq. 6).
 *   - alpha_ij = f(SimScore) = sigmoid(A * logit(s) + B), s clamped to
 *     [1e-6, 1 - 1e-6]. (A, B) = (1, 0) until calibrated, which makes
 *     alpha = SimScore: exact speculative sampling accepts a draft from q
 *     with probability sum_x min(p(x), q(x)) = 1 - DTV(p, q).
 *   - Calibration (specrouter_sched_calibrate): (A, B) maximise the
 *     likelihood of the observed accept/reject outcomes plus a Gaussian prior
 *     prior_weight/2 * ((A-1)^2 + B^2) (Platt scaling), solved by Newton's
 *     method. Each observed step of a pair adds (s = 1 - that step's mean DTV,
 *     successes = sum_b k_b, failures = sum_b [k_b < gamma_b]); the last
 *     SPECROUTER_SCHED_MAX_OBS such steps are kept.
 *   - Eq. 7 for a chain [M_1 .. M_N] (N >= 2) with window W and
 *     alpha_l = alpha(M_l, M_l+1):
 *       latency = W T_1 + sum_{j=2..N} W T_j reach_j,
 *       reach_2 = 1, reach_j = prod_{l<=j-2} alpha_l (level j runs only when a
 *       drafted token survived every earlier verifier),
 *       tokens  = reach_N + sum_{k=1..W} (prod_l alpha_l)^k,
 *       T_eff   = latency / tokens;
 *     the target-only chain [M_t] has T_eff = T_t. A chain that uses an unset
 *     T_i or SimScore has T_eff = +infinity.
 *   - Candidates (Algorithm 1, step 1): models sorted by capability
 *     ascending (ties by index); every subset of the models sorted before
 *     M_t, kept in that order and followed by M_t, of at most max_levels
 *     models; enumerated by length, then lexicographically by sorted
 *     position, so [M_t] is first. The result is the first candidate with
 *     the strictly smallest T_eff (default [M_t]).
 *
 * Return values are the SR_* codes of specrouter.h. On an error, nothing in
 * the scheduler changes. A handle is not thread-safe: calls on one handle
 * must not overlap. Separate handles are independent.
 */
#ifndef SPECROUTER_SCHED_H
#define SPECROUTER_SCHED_H

#include <stdint.h>

#include "specrouter.h"

#ifdef __cplusplus
extern "C" {
#endif

#define SPECROUTER_SCHED_MAX_MODELS 16
#define SPECROUTER_SCHED_MAX_OBS 4096

typedef struct specrouter_sched specrouter_sched;

/* Create a scheduler for n_models models (1..SPECROUTER_SCHED_MAX_MODELS).
 * capability  [n_models] finite numbers, larger = more capable (e.g. parameter
 *             count); copied
 * target      index of the target model M_t
 * window      W, the draft window (1..SPECROUTER_MAX_GAMMA)
 * max_levels  longest chain considered (1..n_models)
 * ema_time    EMA weight of T_i, in (0, 1]
 * ema_sim     EMA weight of E[DTV], in (0, 1]
 * prior_weight  weight of the calibration prior, > 0
 * *out        receives the handle (free it with specrouter_sched_destroy).
 * Every T_i and SimScore starts unset. SR_EINVAL on a bad argument. */
int specrouter_sched_create(int n_models, const double* capability, int target, int window,
                            int max_levels, double ema_time, double ema_sim, double prior_weight,
                            specrouter_sched** out);

/* Free a handle (NULL is ignored). */
void specrouter_sched_destroy(specrouter_sched* s);

/* One measured per-token time of model `model` (seconds, finite, >= 0):
 * the T_i update of Section 4.2. */
int specrouter_sched_observe_time(specrouter_sched* s, int model, double seconds_per_token);

/* Seed SimScore(draft, verifier) in [0, 1] (for instance from prefill
 * logits), replacing the smoothed value. draft != verifier. */
int specrouter_sched_set_similarity(specrouter_sched* s, int draft, int verifier, double simscore);

/* One verify step of the pair (draft, verifier), read from the outputs of
 * specrouter_accept_and_diverge copied to the host:
 * gamma [B], accept_len [B] (k_b, or -1 for a sequence with bad data, which is
 * skipped) and tv [B][gamma_max] (Eq. 5 per drafted position).
 * The step's mean DTV over the positions j < gamma_b of valid sequences
 * (each clamped to [0, 1]) updates E[DTV(draft, verifier)] (Eq. 6) and, with
 * the step's accept/reject counts, adds one calibration observation. A step
 * with no drafted position changes nothing. SR_EINVAL when gamma_b lies
 * outside [0, gamma_max], k_b outside [-1, gamma_b], or a counted tv entry is
 * NaN. */
int specrouter_sched_observe_step(specrouter_sched* s, int draft, int verifier, int B, int gamma_max,
                                  const int32_t* gamma, const int32_t* accept_len, const float* tv);

/* Fit (A, B) of f to the kept observations and use them from now on.
 * A_out and B_out may be NULL. With no observation the fit is (1, 0). */
int specrouter_sched_calibrate(specrouter_sched* s, double* A_out, double* B_out);

/* Read the metrics: T [n_models] (NaN = unset), simscore [n_models *
 * n_models] row-major by (draft, verifier) (NaN = unset), calib [2] = (A, B),
 * n_obs [1] = observations kept. Any pointer may be NULL. */
int specrouter_sched_metrics(const specrouter_sched* s, double* T, double* simscore, double* calib,
                             int* n_obs);

/* Eq. 7 for one chain of `len` distinct models listed in increasing
 * capability order (ties by index) and ending with the target; SR_EINVAL
 * otherwise. *t_eff may be +infinity (an unset metric). */
int specrouter_sched_effective_time(const specrouter_sched* s, const int32_t* chain, int len,
                                    double* t_eff);

/* Algorithm 1. chain [n_models] receives the optimal chain, *len its length,
 * *t_eff its predicted time (+infinity when nothing is measured, the chain then
 * being [M_t]). n_candidates, if not NULL, receives the number of candidates. */
int specrouter_sched_optimal_chain(const specrouter_sched* s, int32_t* chain, int* len, double* t_eff,
                                   int* n_candidates);

#ifdef __cplusplus
}
#endif

#endif /* SPECROUTER_SCHED_H */
