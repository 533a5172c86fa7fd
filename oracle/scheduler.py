"""Chain-scheduler reference (Section 4.2) -- TEST INFRASTRUCTURE ONLY.

Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import or run this module; the product path never does.

Plain fp64 Python written from Section 4.2 of the paper (arXiv 2505.07680):

  * ema                 -- the exponential moving average that smooths every
                           scheduler metric (the T_i update of Section 4.2 and
                           the smoothed DTV of Eq. 6);
  * step_mean_tv        -- the per-step average of Eq. 5's total variation
                           distance over the drafted positions of a batch;
  * simscore            -- Eq. 6, one minus the smoothed DTV;
  * acceptance          -- alpha_ij = f(SimScore), f a calibrated sigmoid;
  * calibrate           -- the calibration of f from observed accept/reject
                           outcomes;
  * effective_time      -- Eq. 7, predicted time per target token of a chain;
  * candidate_chains    -- Algorithm 1, step 1;
  * optimal_chain       -- Algorithm 1, steps 2-3.

The paper leaves f, the EMA weights, the initial values and the exact terms
of Eq. 7 open. The readings taken here:

  R1  A metric with no observation yet is "unset" (NaN); its first
      observation sets it, later ones are blended with the EMA weight.
  R2  A step's DTV observation for the pair (draft i, verifier j) is the mean
      of the per-position distances over every drafted position j < gamma_b of
      every valid sequence (accept_len_b >= 0); a step with no drafted
      position leaves the EMA unchanged.
  R3  f(s) = sigmoid(A * logit(s) + B), with s clamped to [1e-6, 1 - 1e-6].
      With A = 1, B = 0 (the default), f(s) = s: for exact speculative
      sampling the probability that a drafted token is accepted is
      sum_x min(p(x), q(x)) = 1 - DTV(p, q), so SimScore is already the
      acceptance rate and calibration only corrects for drift, for the
      smoothing and for position effects. (A, B) are fitted by maximum
      likelihood on observed outcomes (Platt scaling) with a Gaussian prior
      of weight lam centred on (1, 0).
  R4  A step of a pair contributes one calibration observation:
      x = logit(1 - step mean DTV), successes = sum_b k_b, failures =
      sum_b [k_b < gamma_b] (each drafted token is a Bernoulli trial up to the
      first rejection; the likelihood of a prefix of k accepts ended by a
      rejection is alpha^k (1 - alpha)).
  R5  Eq. 7 for C = [M_1 .. M_N], N >= 2, window W, alpha_l = f(S(M_l, M_l+1)):
        latency = W T_1 + sum_{j=2..N} W T_j reach_j,
        reach_2 = 1, reach_j = prod_{l=1..j-2} alpha_l (level j is reached
        when at least one drafted token survived every earlier verifier),
        tokens  = reach_N + sum_{k=1..W} (prod_l alpha_l)^k (the expected
        surviving prefix plus the target's own correction or bonus token,
        which it emits whenever it runs),
        T_eff   = latency / tokens.
      For the target-only chain [M_t] one pass yields one token: T_eff = T_t.
      A chain with an unset T or SimScore has T_eff = +inf.
  R6  SortModelsByCapability orders by capability ascending, ties by model
      index. GenerateCandidateChains yields every chain made of a subset of
      the models that sort before M_t, in that order, followed by M_t, with
      at most max_levels models: by length ascending, then lexicographically
      by sorted position (so [M_t] comes first). The optimum is the first
      candidate with the strictly smallest T_eff (Algorithm 1 keeps the
      default [M_t] unless a chain is strictly faster).
"""

from __future__ import annotations

import itertools
import math

import numpy as np
from scipy import optimize

S_CLAMP = 1e-6


def ema(old: float, measured: float, weight: float) -> float:
    """T_new = weight * T_measured + (1 - weight) * T_old; an unset old value
    (NaN) takes the measurement (R1)."""
    if math.isnan(old):
        return float(measured)
    return weight * float(measured) + (1.0 - weight) * old


def step_mean_tv(tv, gamma, accept_len):
    """Mean per-position DTV over drafted positions j < gamma_b of valid
    sequences (R2). Returns (mean, count); mean is NaN when count is 0."""
    tot = 0.0
    n = 0
    for b in range(len(gamma)):
        if int(accept_len[b]) < 0:
            continue
        for j in range(int(gamma[b])):
            tot += min(max(float(tv[b][j]), 0.0), 1.0)
            n += 1
    return (tot / n if n else float("nan")), n


def step_outcomes(gamma, accept_len):
    """(successes, failures) of one step's accept/reject trials (R4)."""
    a = r = 0
    for b in range(len(gamma)):
        k = int(accept_len[b])
        if k < 0:
            continue
        a += k
        r += 1 if k < int(gamma[b]) else 0
    return a, r


def simscore(dtv_smoothed: float) -> float:
    """Eq. 6: SimScore = 1 - E[DTV]."""
    return 1.0 - dtv_smoothed


def _logit(s: float) -> float:
    s = min(max(s, S_CLAMP), 1.0 - S_CLAMP)
    return math.log(s) - math.log1p(-s)


def _sigmoid(z: float) -> float:
    if z >= 0:
        return 1.0 / (1.0 + math.exp(-z))
    e = math.exp(z)
    return e / (1.0 + e)


def acceptance(s: float, A: float = 1.0, B: float = 0.0) -> float:
    """alpha = f(SimScore) = sigmoid(A logit(s) + B) (R3)."""
    if math.isnan(s):
        return float("nan")
    return _sigmoid(A * _logit(s) + B)


def calibration_objective(params, obs, lam: float) -> float:
    """Negative penalised log-likelihood of (A, B) over observations
    (simscore, successes, failures) (R3, R4)."""
    A, B = params
    tot = 0.5 * lam * ((A - 1.0) ** 2 + B ** 2)
    for s, a, r in obs:
        z = A * _logit(s) + B
        # log sigmoid(z) and log(1 - sigmoid(z)) written stably
        log_p = -math.log1p(math.exp(-z)) if z >= 0 else z - math.log1p(math.exp(z))
        log_np = -z + log_p
        tot -= a * log_p + r * log_np
    return tot


def calibration_gradient(params, obs, lam: float):
    """Gradient of calibration_objective: with z = A x + B and n = a + r
    trials, d/dz of an observation's term is n sigmoid(z) - a."""
    A, B = params
    gA, gB = lam * (A - 1.0), lam * B
    for s, a, r in obs:
        x = _logit(s)
        e = (a + r) * _sigmoid(A * x + B) - a
        gA += e * x
        gB += e
    return np.array([gA, gB])


def calibrate(obs, lam: float = 1.0):
    """(A, B) minimising calibration_objective (R3). The objective is
    strictly convex (lam > 0), so the minimiser is unique."""
    obs = list(obs)
    res = optimize.minimize(calibration_objective, x0=np.array([1.0, 0.0]), args=(obs, lam),
                            jac=calibration_gradient, method="BFGS", options={"gtol": 1e-10, "maxiter": 10000})
    return float(res.x[0]), float(res.x[1])


def effective_time(chain, T, S, W: int, A: float = 1.0, B: float = 0.0) -> float:
    """Eq. 7 under reading R5. T: per-model times (NaN = unset); S: dict or
    matrix of SimScore[i][j] (NaN = unset)."""
    if len(chain) == 1:
        t = T[chain[0]]
        return float("inf") if math.isnan(t) else float(t)
    for m in chain:
        if math.isnan(T[m]):
            return float("inf")
    alphas = []
    for i, j in zip(chain[:-1], chain[1:]):
        s = S[i][j]
        if math.isnan(s):
            return float("inf")
        alphas.append(acceptance(s, A, B))
    latency = W * T[chain[0]]
    for jj in range(1, len(chain)):  # levels 2..N
        reach = 1.0
        for l in range(jj - 1):
            reach *= alphas[l]
        latency += W * T[chain[jj]] * reach
    prod = 1.0
    for a in alphas:
        prod *= a
    reach_target = 1.0
    for a in alphas[:-1]:
        reach_target *= a
    tokens = reach_target + sum(prod ** k for k in range(1, W + 1))
    return latency / tokens


def sort_by_capability(capability):
    """Model indices ordered by capability ascending, ties by index (R6)."""
    return sorted(range(len(capability)), key=lambda m: (capability[m], m))


def candidate_chains(capability, target: int, max_levels: int):
    """Algorithm 1 step 1 under reading R6."""
    order = sort_by_capability(capability)
    below = order[:order.index(target)]
    out = []
    for r in range(0, min(max_levels - 1, len(below)) + 1):
        for sub in itertools.combinations(below, r):
            out.append(list(sub) + [target])
    return out


def optimal_chain(capability, target: int, T, S, W: int, max_levels: int, A: float = 1.0, B: float = 0.0):
    """Algorithm 1: the candidate with the strictly smallest Eq. 7 time,
    default [M_t]. Returns (chain, t_eff, all (chain, t_eff) pairs)."""
    best, t_best = [target], float("inf")
    scored = []
    for c in candidate_chains(capability, target, max_levels):
        t = effective_time(c, T, S, W, A, B)
        scored.append((c, t))
        if t < t_best:
            best, t_best = c, t
    return best, t_best, scored
