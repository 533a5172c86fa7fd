// Model-chain scheduler: smoothed metrics, calibrated acceptance map, Eq. 7
// prediction and Algorithm 1's chain selection (Section 4.2). Host code.

#include <algorithm>
#include <cmath>
#include <limits>
#include <new>
#include <vector>

#include "specrouter_sched.h"

namespace {

constexpr double kClamp = 1e-6;  // SimScore clamp before the logit
constexpr double kInf = std::numeric_limits<double>::infinity();
constexpr double kNaN = std::numeric_limits<double>::quiet_NaN();

struct Obs {
  double x;  // logit of the step's SimScore
  double a;  // accepted drafts
  double r;  // rejections
};

double logit(double s) {
  s = std::min(std::max(s, kClamp), 1.0 - kClamp);
  return std::log(s) - std::log1p(-s);
}

double sigmoid(double z) {
  if (z >= 0) return 1.0 / (1.0 + std::exp(-z));
  const double e = std::exp(z);
  return e / (1.0 + e);
}

// log(1 + e^t) without overflow.
double softplus(double t) { return std::max(t, 0.0) + std::log1p(std::exp(-std::fabs(t))); }

double ema(double old, double measured, double w) {
  return std::isnan(old) ? measured : w * measured + (1.0 - w) * old;
}

}  // namespace

struct specrouter_sched {
  int n, target, window, max_levels;
  double ema_time, ema_sim, prior;
  std::vector<double> capability;
  std::vector<int> order;  // model indices by capability ascending, ties by index
  std::vector<int> rank;   // position of each model in `order`
  std::vector<double> T;   // smoothed per-token time (NaN = unset)
  std::vector<double> dtv; // smoothed DTV, [draft * n + verifier] (NaN = unset)
  double A = 1.0, B = 0.0;
  std::vector<Obs> obs;  // ring of the latest observations
  int obs_head = 0;

  double alpha(int i, int j) const {
    const double d = dtv[(size_t)i * n + j];
    if (std::isnan(d)) return kNaN;
    return sigmoid(A * logit(1.0 - d) + B);
  }

  // Eq. 7 for a validated chain.
  double effective_time(const int* c, int len) const {
    if (len == 1) return std::isnan(T[c[0]]) ? kInf : T[c[0]];
    double al[SPECROUTER_SCHED_MAX_MODELS];
    for (int l = 0; l < len; ++l)
      if (std::isnan(T[c[l]])) return kInf;
    for (int l = 0; l + 1 < len; ++l) {
      al[l] = alpha(c[l], c[l + 1]);
      if (std::isnan(al[l])) return kInf;
    }
    const double W = window;
    double latency = W * T[c[0]];
    double reach = 1.0;  // probability that level l + 2 runs
    double reach_target = 1.0;
    for (int l = 0; l + 1 < len; ++l) {
      latency += W * T[c[l + 1]] * reach;
      reach_target = reach;
      reach *= al[l];
    }
    double prod = 1.0;
    for (int l = 0; l + 1 < len; ++l) prod *= al[l];
    double tokens = 0.0, pk = 1.0;
    for (int k = 1; k <= window; ++k) {
      pk *= prod;
      tokens += pk;
    }
    return latency / (reach_target + tokens);
  }
};

namespace {

bool valid_model(const specrouter_sched* s, int m) { return s && m >= 0 && m < s->n; }

// Penalised negative log-likelihood of (A, B) over the kept observations.
double calib_objective(const specrouter_sched* s, double A, double B) {
  double f = 0.5 * s->prior * ((A - 1.0) * (A - 1.0) + B * B);
  for (const Obs& o : s->obs) {
    const double z = A * o.x + B;
    f += o.a * softplus(-z) + o.r * softplus(z);
  }
  return f;
}

}  // namespace

extern "C" {

int specrouter_sched_create(int n_models, const double* capability, int target, int window,
                            int max_levels, double ema_time, double ema_sim, double prior_weight,
                            specrouter_sched** out) {
  if (!out || !capability || n_models < 1 || n_models > SPECROUTER_SCHED_MAX_MODELS) return SR_EINVAL;
  if (target < 0 || target >= n_models || window < 1 || window > SPECROUTER_MAX_GAMMA) return SR_EINVAL;
  if (max_levels < 1 || max_levels > n_models) return SR_EINVAL;
  if (!(ema_time > 0.0 && ema_time <= 1.0) || !(ema_sim > 0.0 && ema_sim <= 1.0)) return SR_EINVAL;
  if (!(prior_weight > 0.0 && std::isfinite(prior_weight))) return SR_EINVAL;
  for (int i = 0; i < n_models; ++i)
    if (!std::isfinite(capability[i])) return SR_EINVAL;
  specrouter_sched* s = new (std::nothrow) specrouter_sched();
  if (!s) return SR_EINVAL;
  s->n = n_models;
  s->target = target;
  s->window = window;
  s->max_levels = max_levels;
  s->ema_time = ema_time;
  s->ema_sim = ema_sim;
  s->prior = prior_weight;
  s->capability.assign(capability, capability + n_models);
  s->order.resize(n_models);
  for (int i = 0; i < n_models; ++i) s->order[i] = i;
  std::sort(s->order.begin(), s->order.end(), [s](int a, int b) {
    return s->capability[a] != s->capability[b] ? s->capability[a] < s->capability[b] : a < b;
  });
  s->rank.resize(n_models);
  for (int i = 0; i < n_models; ++i) s->rank[s->order[i]] = i;
  s->T.assign(n_models, kNaN);
  s->dtv.assign((size_t)n_models * n_models, kNaN);
  s->obs.reserve(SPECROUTER_SCHED_MAX_OBS);
  *out = s;
  return SR_OK;
}

void specrouter_sched_destroy(specrouter_sched* s) { delete s; }

int specrouter_sched_observe_time(specrouter_sched* s, int model, double seconds_per_token) {
  if (!valid_model(s, model) || !std::isfinite(seconds_per_token) || seconds_per_token < 0.0) return SR_EINVAL;
  s->T[model] = ema(s->T[model], seconds_per_token, s->ema_time);
  return SR_OK;
}

int specrouter_sched_set_similarity(specrouter_sched* s, int draft, int verifier, double simscore) {
  if (!valid_model(s, draft) || !valid_model(s, verifier) || draft == verifier) return SR_EINVAL;
  if (!(simscore >= 0.0 && simscore <= 1.0)) return SR_EINVAL;
  s->dtv[(size_t)draft * s->n + verifier] = 1.0 - simscore;
  return SR_OK;
}

int specrouter_sched_observe_step(specrouter_sched* s, int draft, int verifier, int B, int gamma_max,
                                  const int32_t* gamma, const int32_t* accept_len, const float* tv) {
  if (!valid_model(s, draft) || !valid_model(s, verifier) || draft == verifier) return SR_EINVAL;
  if (B < 0 || gamma_max < 0 || gamma_max > SPECROUTER_MAX_GAMMA) return SR_EINVAL;
  if (B > 0 && (!gamma || !accept_len || (gamma_max > 0 && !tv))) return SR_EINVAL;
  // Validate everything before changing anything.
  double sum = 0.0, acc = 0.0, rej = 0.0;
  long n = 0;
  for (int b = 0; b < B; ++b) {
    const int g = gamma[b], k = accept_len[b];
    if (g < 0 || g > gamma_max || k < -1 || k > g) return SR_EINVAL;
    if (k < 0) continue;
    for (int j = 0; j < g; ++j) {
      const double t = tv[(size_t)b * gamma_max + j];
      if (std::isnan(t)) return SR_EINVAL;
      sum += std::min(std::max(t, 0.0), 1.0);
      ++n;
    }
    acc += k;
    rej += k < g ? 1.0 : 0.0;
  }
  if (n == 0) return SR_OK;
  const double mean = sum / (double)n;
  double& d = s->dtv[(size_t)draft * s->n + verifier];
  d = ema(d, mean, s->ema_sim);
  const Obs o{logit(1.0 - mean), acc, rej};
  if ((int)s->obs.size() < SPECROUTER_SCHED_MAX_OBS) {
    s->obs.push_back(o);
  } else {
    s->obs[s->obs_head] = o;
    s->obs_head = (s->obs_head + 1) % SPECROUTER_SCHED_MAX_OBS;
  }
  return SR_OK;
}

int specrouter_sched_calibrate(specrouter_sched* s, double* A_out, double* B_out) {
  if (!s) return SR_EINVAL;
  // Newton's method with backtracking on a strictly convex objective, from
  // the prior's centre.
  double A = 1.0, B = 0.0;
  double f = calib_objective(s, A, B);
  for (int it = 0; it < 200; ++it) {
    double gA = s->prior * (A - 1.0), gB = s->prior * B;
    double hAA = s->prior, hAB = 0.0, hBB = s->prior;
    for (const Obs& o : s->obs) {
      const double sg = sigmoid(A * o.x + B);
      const double nt = o.a + o.r;
      const double e = nt * sg - o.a;  // d/dz of the observation's term
      gA += e * o.x;
      gB += e;
      const double w = nt * sg * (1.0 - sg);
      hAA += w * o.x * o.x;
      hAB += w * o.x;
      hBB += w;
    }
    const double det = hAA * hBB - hAB * hAB;
    if (!(det > 0.0)) break;
    const double dA = -(hBB * gA - hAB * gB) / det;
    const double dB = -(hAA * gB - hAB * gA) / det;
    const double dec = -(gA * dA + gB * dB);  // Newton decrement squared
    if (!(dec > 1e-24 * std::max(1.0, std::fabs(f)))) break;
    double t = 1.0;
    double fn = calib_objective(s, A + t * dA, B + t * dB);
    while (fn > f - 0.25 * t * dec && t > 1e-12) {
      t *= 0.5;
      fn = calib_objective(s, A + t * dA, B + t * dB);
    }
    if (!(fn <= f)) break;
    A += t * dA;
    B += t * dB;
    f = fn;
  }
  s->A = A;
  s->B = B;
  if (A_out) *A_out = A;
  if (B_out) *B_out = B;
  return SR_OK;
}

int specrouter_sched_metrics(const specrouter_sched* s, double* T, double* simscore, double* calib,
                             int* n_obs) {
  if (!s) return SR_EINVAL;
  if (T) std::copy(s->T.begin(), s->T.end(), T);
  if (simscore)
    for (size_t i = 0; i < s->dtv.size(); ++i) simscore[i] = 1.0 - s->dtv[i];
  if (calib) {
    calib[0] = s->A;
    calib[1] = s->B;
  }
  if (n_obs) *n_obs = (int)s->obs.size();
  return SR_OK;
}

int specrouter_sched_effective_time(const specrouter_sched* s, const int32_t* chain, int len,
                                    double* t_eff) {
  if (!s || !chain || !t_eff || len < 1 || len > s->n) return SR_EINVAL;
  int c[SPECROUTER_SCHED_MAX_MODELS];
  for (int l = 0; l < len; ++l) {
    if (!valid_model(s, chain[l])) return SR_EINVAL;
    if (l > 0 && s->rank[chain[l - 1]] >= s->rank[chain[l]]) return SR_EINVAL;
    c[l] = chain[l];
  }
  if (c[len - 1] != s->target) return SR_EINVAL;
  *t_eff = s->effective_time(c, len);
  return SR_OK;
}

int specrouter_sched_optimal_chain(const specrouter_sched* s, int32_t* chain, int* len, double* t_eff,
                                   int* n_candidates) {
  if (!s || !chain || !len || !t_eff) return SR_EINVAL;
  const int nb = s->rank[s->target];  // models sorted before the target: order[0 .. nb)
  const int rmax = std::min(s->max_levels - 1, nb);
  int best[SPECROUTER_SCHED_MAX_MODELS], best_len = 1;
  best[0] = s->target;
  double t_best = kInf;
  int count = 0;
  int pos[SPECROUTER_SCHED_MAX_MODELS];  // chosen sorted positions, increasing
  int c[SPECROUTER_SCHED_MAX_MODELS];
  for (int r = 0; r <= rmax; ++r) {
    for (int i = 0; i < r; ++i) pos[i] = i;
    while (true) {
      for (int i = 0; i < r; ++i) c[i] = s->order[pos[i]];
      c[r] = s->target;
      const double t = s->effective_time(c, r + 1);
      ++count;
      if (t < t_best) {
        t_best = t;
        best_len = r + 1;
        std::copy(c, c + r + 1, best);
      }
      // next combination of r positions out of nb, lexicographic
      int i = r - 1;
      while (i >= 0 && pos[i] == nb - r + i) --i;
      if (i < 0) break;
      ++pos[i];
      for (int k = i + 1; k < r; ++k) pos[k] = pos[k - 1] + 1;
    }
  }
  std::copy(best, best + best_len, chain);
  *len = best_len;
  *t_eff = t_best;
  if (n_candidates) *n_candidates = count;
  return SR_OK;
}

}  // extern "C"
