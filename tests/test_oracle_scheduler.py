"""Pins of the chain-scheduler reference (Section 4.2; Eq. 5-7; Algorithm 1).

Each test checks the reference against something other than itself: a closed
form, a brute-force enumeration, an independent library routine, or the
speculative-sampling identity P(accept) = 1 - DTV(p, q).
"""

import itertools
import math

import numpy as np
import pytest

import oracle
from oracle import scheduler as sch


# ---------------------------------------------------------------- EMA (Section 4.2, T_i update; Eq. 6)

def test_ema_matches_explicit_weights():
    rng = np.random.default_rng(0)
    for w in (0.05, 0.3, 1.0):
        m = rng.uniform(1e-3, 5e-2, size=9)
        v = float("nan")
        for x in m:
            v = sch.ema(v, x, w)
        n = len(m)
        # closed form: the first sample keeps (1-w)^(n-1), sample k>=2 gets w (1-w)^(n-k)
        want = (1 - w) ** (n - 1) * m[0] + sum(w * (1 - w) ** (n - k) * m[k - 1] for k in range(2, n + 1))
        assert v == pytest.approx(want, rel=1e-13)


def test_ema_constant_input_is_fixed_point():
    v = float("nan")
    for _ in range(20):
        v = sch.ema(v, 0.125, 0.37)
    assert v == 0.125


# ---------------------------------------------------------------- step statistics (Eq. 5 average, R2, R4)

def test_step_mean_tv_and_outcomes_by_mask():
    rng = np.random.default_rng(1)
    B, gmax = 11, 5
    gamma = rng.integers(0, gmax + 1, size=B)
    acc = np.array([rng.integers(-1, g + 1) for g in gamma])
    tv = rng.uniform(0, 1, size=(B, gmax))
    tv[:, :] = np.where(np.arange(gmax)[None, :] < gamma[:, None], tv, np.nan)  # unused rows hold NaN
    mask = (np.arange(gmax)[None, :] < gamma[:, None]) & (acc[:, None] >= 0)
    mean, n = sch.step_mean_tv(tv, gamma, acc)
    assert n == mask.sum()
    assert mean == pytest.approx(tv[mask].mean(), rel=1e-14)
    a, r = sch.step_outcomes(gamma, acc)
    valid = acc >= 0
    assert a == acc[valid].sum()
    assert r == int((acc[valid] < gamma[valid]).sum())


def test_step_mean_tv_empty_is_nan():
    mean, n = sch.step_mean_tv(np.zeros((3, 2)), [0, 0, 2], [0, 0, -1])
    assert n == 0 and math.isnan(mean)


# ---------------------------------------------------------------- f(SimScore) (Eq. 6, R3)

def _dists(rng, V):
    p = rng.dirichlet(np.full(V, 0.3))
    q = rng.dirichlet(np.full(V, 0.3))
    return p, q


def test_default_f_is_the_speculative_acceptance_rate():
    """Accepting x ~ q with probability min(1, p(x)/q(x)) succeeds with
    probability sum_x min(p(x), q(x)) = 1 - DTV(p, q); with the default
    calibration alpha = f(1 - DTV) must equal it."""
    rng = np.random.default_rng(2)
    for V in (2, 5, 40):
        p, q = _dists(rng, V)
        brute = sum(q[x] * min(1.0, p[x] / q[x]) for x in range(V) if q[x] > 0)
        dtv = 0.5 * np.abs(p - q).sum()
        assert sch.acceptance(sch.simscore(dtv)) == pytest.approx(brute, rel=1e-9, abs=1e-12)


def test_default_f_matches_monte_carlo_of_the_accept_rule():
    """Empirical acceptance of single drafts through the accept reference
    agrees with f(1 - TV) for the TV that reference reports."""
    rng = np.random.default_rng(3)
    V, N = 6, 40000
    lp = rng.normal(size=V)
    lq = rng.normal(size=V)
    q = np.exp(lq - lq.max())
    q /= q.sum()
    drafts = rng.choice(V, size=N, p=q)
    P = np.broadcast_to(np.stack([lp, lp])[None], (N, 2, V)).astype(np.float32)
    Q = np.broadcast_to(lq[None, None], (N, 1, V)).astype(np.float32)
    res = oracle.accept_and_diverge(P, Q, drafts[:, None], np.ones(N, np.int32),
                                    rng.uniform(0, 1, (N, 1)).astype(np.float32),
                                    rng.uniform(0, 1, (N, 2)).astype(np.float32))
    rate = res["accept_len"].mean()
    alpha = sch.acceptance(sch.simscore(res["tv"][0, 0]))
    assert abs(rate - alpha) < 4 * math.sqrt(alpha * (1 - alpha) / N)


def test_f_is_monotone_and_maps_into_unit_interval():
    s = np.linspace(0, 1, 101)
    for A, B in ((1.0, 0.0), (2.5, -0.7), (0.4, 1.2)):
        a = np.array([sch.acceptance(x, A, B) for x in s])
        assert (np.diff(a) >= 0).all() and (a > 0).all() and (a < 1).all()


def test_calibration_keeps_identity_on_consistent_data():
    """When observed rates equal the SimScores the likelihood gradient at
    (A, B) = (1, 0) is zero, so the prior's centre is the exact optimum."""
    obs = [(0.5, 50, 50), (0.8, 80, 20), (0.25, 25, 75), (0.9, 900, 100)]
    A, B = sch.calibrate(obs, lam=1.0)
    assert A == pytest.approx(1.0, abs=1e-7) and B == pytest.approx(0.0, abs=1e-7)


def test_calibration_matches_unpenalised_logistic_regression():
    from sklearn.linear_model import LogisticRegression

    rng = np.random.default_rng(4)
    s = rng.uniform(0.2, 0.95, size=30)
    true_A, true_B = 1.6, -0.4
    n = rng.integers(5, 60, size=30)
    a = np.array([rng.binomial(k, sch.acceptance(x, true_A, true_B)) for x, k in zip(s, n)])
    obs = list(zip(s, a, n - a))
    A, B = sch.calibrate(obs, lam=1e-10)
    X = np.concatenate([np.log(s / (1 - s)), np.log(s / (1 - s))])[:, None]
    y = np.concatenate([np.ones(30), np.zeros(30)])
    wts = np.concatenate([a, n - a]).astype(float)
    lr = LogisticRegression(penalty=None, tol=1e-12, max_iter=10000).fit(X, y, sample_weight=wts)
    assert A == pytest.approx(lr.coef_[0, 0], rel=1e-4)
    assert B == pytest.approx(lr.intercept_[0], abs=1e-4)


# ---------------------------------------------------------------- Eq. 7 (R5)

def _brute_eq7(chain, T, alphas, W):
    """E[latency] / E[tokens] by enumerating every accept/reject pattern of
    the W drafted tokens at every verifier level (independent trials)."""
    N = len(chain)
    lat = tok = 0.0
    for bits in itertools.product((0, 1), repeat=W * (N - 1)):
        prob = 1.0
        for l in range(N - 1):
            for k in range(W):
                a = alphas[l]
                prob *= a if bits[l * W + k] else 1 - a
        if prob == 0:
            continue
        surv = W  # drafted tokens still alive: a prefix of the draft
        latency = W * T[chain[0]]
        ran = True
        for l in range(N - 1):
            ran = l == 0 or surv > 0  # level l + 2 runs only if something survived
            if ran:
                latency += W * T[chain[l + 1]]
            pref = 0
            while pref < W and bits[l * W + pref]:
                pref += 1
            surv = min(surv, pref)
        lat += prob * latency
        tok += prob * (surv + (1 if ran else 0))  # the target adds one token when it runs
    return lat / tok


def test_eq7_target_only_is_its_own_time():
    assert sch.effective_time([2], [0.1, 0.2, 0.7], None, 4) == 0.7


def test_eq7_two_levels_closed_form():
    """Two models: expected tokens per cycle (1 - a^(W+1)) / (1 - a)."""
    T = [0.01, 0.2]
    for a in (0.05, 0.3, 0.77, 0.999):  # away from the [1e-6, 1 - 1e-6] clamp
        for W in (1, 3, 8):
            S = [[np.nan, a], [np.nan, np.nan]]
            want = (W * T[0] + W * T[1]) * (1 - a) / (1 - a ** (W + 1))
            assert sch.effective_time([0, 1], T, S, W) == pytest.approx(want, rel=1e-12)


@pytest.mark.parametrize("N,W", [(3, 1), (3, 3), (4, 2)])
def test_eq7_matches_enumeration(N, W):
    rng = np.random.default_rng(N * 10 + W)
    T = list(rng.uniform(0.001, 0.1, size=N))
    chain = list(range(N))
    alphas = list(rng.uniform(0.1, 0.95, size=N - 1))
    S = np.full((N, N), np.nan)
    for l in range(N - 1):
        S[l, l + 1] = alphas[l]  # default f is the identity
    assert sch.effective_time(chain, T, S, W) == pytest.approx(_brute_eq7(chain, T, alphas, W), rel=1e-12)


def test_eq7_unset_metrics_give_infinity():
    S = [[np.nan, 0.7], [np.nan, np.nan]]
    assert sch.effective_time([0, 1], [np.nan, 0.1], S, 4) == math.inf
    assert sch.effective_time([0, 1], [0.01, 0.1], [[np.nan] * 2] * 2, 4) == math.inf


# ---------------------------------------------------------------- Algorithm 1 (R6)

def _brute_candidates(capability, target, max_levels):
    order = sorted(range(len(capability)), key=lambda m: (capability[m], m))
    rank = {m: i for i, m in enumerate(order)}
    out = set()
    others = [m for m in range(len(capability)) if m != target]
    for r in range(0, max_levels):
        for perm in itertools.permutations(others, r):
            c = list(perm) + [target]
            if all(rank[x] < rank[y] for x, y in zip(c[:-1], c[1:])):
                out.add(tuple(c))
    return out


def test_candidates_are_every_capability_ordered_chain():
    cap = [7.0, 1.0, 3.0, 3.0, 70.0, 0.5]
    for target in (4, 2, 5):
        for ml in (1, 2, 3, 6):
            got = sch.candidate_chains(cap, target, ml)
            assert len(got) == len({tuple(c) for c in got})
            assert {tuple(c) for c in got} == _brute_candidates(cap, target, ml)
            assert got[0] == [target]


def test_optimal_chain_is_the_brute_force_minimum():
    rng = np.random.default_rng(5)
    n = 6
    cap = list(rng.uniform(1, 100, size=n))
    target = int(np.argmax(cap))
    T = list(np.array(cap) * 1e-4)
    S = rng.uniform(0.3, 0.95, size=(n, n))
    best, t_best, scored = sch.optimal_chain(cap, target, T, S, 4, n)
    brute = min(sch.effective_time(list(c), T, S, 4) for c in _brute_candidates(cap, target, n))
    assert t_best == brute
    assert sch.effective_time(best, T, S, 4) == t_best


def test_optimal_chain_special_cases():
    cap = [1.0, 8.0, 70.0]
    T = [0.001, 0.01, 0.05]
    S = np.full((3, 3), np.nan)
    # drafts never accepted: target alone
    S[0, 2] = S[1, 2] = S[0, 1] = 1e-9
    best, t, _ = sch.optimal_chain(cap, 2, T, S, 4, 3)
    assert best == [2] and t == 0.05
    # a perfect, almost free draft: W + 1 tokens per cycle
    S[0, 2] = 1.0 - 1e-12
    best, t, _ = sch.optimal_chain(cap, 2, T, S, 4, 3)
    assert best == [0, 2]
    assert t == pytest.approx(4 * (0.001 + 0.05) / 5, rel=1e-5)
    # unset similarities exclude chains; the default survives
    best, t, _ = sch.optimal_chain(cap, 2, T, np.full((3, 3), np.nan), 4, 3)
    assert best == [2] and t == 0.05
    # nothing measured at all: default [M_t] with infinite time
    best, t, _ = sch.optimal_chain(cap, 2, [np.nan] * 3, np.full((3, 3), np.nan), 4, 3)
    assert best == [2] and t == math.inf


def test_calibration_gradient_matches_finite_differences():
    rng = np.random.default_rng(6)
    obs = [(float(s), int(rng.integers(0, 30)), int(rng.integers(0, 5))) for s in rng.uniform(0.05, 0.98, 25)]
    for A, B in ((1.0, 0.0), (1.7, -0.3), (0.6, 0.8)):
        g = sch.calibration_gradient((A, B), obs, 0.7)
        h = 1e-6
        fd = [(sch.calibration_objective((A + h, B), obs, 0.7) - sch.calibration_objective((A - h, B), obs, 0.7)) / (2 * h),
              (sch.calibration_objective((A, B + h), obs, 0.7) - sch.calibration_objective((A, B - h), obs, 0.7)) / (2 * h)]
        np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-6)
