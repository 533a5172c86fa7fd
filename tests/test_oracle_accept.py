"""Pins for the accept/divergence reference (CPU only).

What fixes the reference here, independently of its own formulas:
  * exact enumeration on tiny vocabularies: the first emitted token is
    distributed exactly as p, and two consecutive tokens (across verify steps)
    as p(y1) p(y2 | y1) -- the losslessness of speculative sampling (Section 2.2,
    probabilistic acceptance; Section 3.1 'preserving the output quality');
  * hand-worked acceptance probabilities and residuals (golden fixture);
  * Eq. 3 / Eq. 4's expected token count under i.i.d. rows (golden fixture);
  * the identity P(accept) = sum_x q(x) min(1, p(x)/q(x)) = 1 - TV (Eq. 2 with x ~ q);
  * KL and TV against scipy's independent routines, Gibbs and Pinsker bounds;
  * q == p accepts every draft; gamma = 0 reduces to inverse-CDF sampling from p.
"""

import json
import math
import os
from fractions import Fraction as F
from itertools import product

import numpy as np
import pytest
from scipy.spatial.distance import cityblock
from scipy.special import rel_entr

from oracle.accept import accept_and_diverge, accept_sequence, inverse_cdf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _frac_list(xs):
    return [F(x) for x in xs]


def _logits(dist):
    return np.array([math.log(float(x)) if x > 0 else -np.inf for x in dist])


# ---------------------------------------------------------------- exact enumeration

class TableModel:
    """Tiny 'models': p(. | prefix) and q(. | prefix) as exact rationals."""

    def __init__(self, V, seed, iid=None):
        self.V = V
        self.rng = np.random.default_rng(seed)
        self.cache = {}
        self.iid = iid

    def _dist(self, key):
        if key not in self.cache:
            w = self.rng.integers(1, 7, size=self.V)
            if self.rng.random() < 0.3:
                w[self.rng.integers(self.V)] = 0 if key[0] == "q" else w[0]
            if w.sum() == 0:
                w[0] = 1
            tot = int(w.sum())
            self.cache[key] = [F(int(x), tot) for x in w]
        return self.cache[key]

    def p(self, prefix):
        return self.iid[0] if self.iid else self._dist(("p",) + tuple(prefix))

    def q(self, prefix):
        if self.iid:
            return self.iid[1]
        d = self._dist(("q",) + tuple(prefix))
        if all(x == 0 for x in d):  # pragma: no cover
            d = [F(1, self.V)] * self.V
        return d


def _cdf_intervals(w):
    """Exact [lo, hi) u-intervals of CDF inversion over weights w (Fractions)."""
    W = sum(w)
    acc = F(0)
    out = []
    for x, wx in enumerate(w):
        if wx > 0:
            out.append((x, acc / W, (acc + wx) / W))
        acc += wx
    return out


def step_outcomes(model, prefix, gamma):
    """Enumerate one verify step exactly.

    Yields (probability, emitted token tuple). The reference is evaluated at
    interior points of every region of (drafts, u_acc, u_res) space on which
    its outcome is constant; the regions come from exact rational
    thresholds computed here, not by the reference.
    """
    V = model.V
    for drafts in product(range(V), repeat=gamma):
        prob_d = F(1)
        ok = True
        for j in range(gamma):
            qj = model.q(list(prefix) + list(drafts[:j]))[drafts[j]]
            prob_d *= qj
            if qj == 0:
                ok = False
        if not ok:
            continue
        P = np.stack([_logits(model.p(list(prefix) + list(drafts[:j]))) for j in range(gamma + 1)])
        Q = np.stack([_logits(model.q(list(prefix) + list(drafts[:j]))) for j in range(gamma)]) if gamma else np.zeros((0, V))
        a = []
        for j in range(gamma):
            pj = model.p(list(prefix) + list(drafts[:j]))[drafts[j]]
            qj = model.q(list(prefix) + list(drafts[:j]))[drafts[j]]
            a.append(min(F(1), pj / qj))
        for k in range(gamma + 1):
            reach = F(1)
            for j in range(k):
                reach *= a[j]
            if k < gamma:
                reach *= 1 - a[k]
            if reach == 0:
                continue
            u_acc = np.zeros(max(gamma, 1))
            for j in range(k):
                u_acc[j] = float(a[j]) / 2
            if k < gamma:
                u_acc[k] = (float(a[k]) + 1) / 2
            pk = model.p(list(prefix) + list(drafts[:k]))
            if k < gamma:
                qk = model.q(list(prefix) + list(drafts[:k]))
                w = [max(F(0), x - y) for x, y in zip(pk, qk)]
                if sum(w) == 0:
                    w = pk
            else:
                w = pk
            for _, lo, hi in _cdf_intervals(w):
                u_res = np.zeros(gamma + 1)
                u_res[k] = float((lo + hi) / 2)
                r = accept_sequence(P, Q, np.array(drafts, dtype=np.int64), gamma, u_acc, u_res, gamma, V)
                assert r["status"] == 0
                assert r["accept_len"] == k
                toks = tuple(int(t) for t in r["tokens"][: k + 1])
                yield prob_d * reach * (hi - lo), toks


def first_token_dist(model, prefix, gamma):
    d = [F(0)] * model.V
    total = F(0)
    for pr, toks in step_outcomes(model, prefix, gamma):
        d[toks[0]] += pr
        total += pr
    assert total == 1
    return d


@pytest.mark.parametrize("V,gamma,seed", [(3, 1, 0), (3, 2, 1), (4, 2, 2), (2, 3, 3), (4, 1, 4)])
def test_first_token_is_distributed_as_p(V, gamma, seed):
    model = TableModel(V, seed)
    d = first_token_dist(model, [], gamma)
    p0 = model.p([])
    for x in range(V):
        assert abs(float(d[x]) - float(p0[x])) < 1e-12


@pytest.mark.parametrize("V,gamma,seed", [(3, 1, 10), (3, 2, 11), (2, 2, 12)])
def test_two_tokens_across_steps_are_distributed_as_p(V, gamma, seed):
    """P(y1, y2) = p(y1) p(y2 | y1): exercises the bonus token from p_gamma."""
    model = TableModel(V, seed)
    joint = np.zeros((V, V))
    for pr, toks in step_outcomes(model, [], gamma):
        if len(toks) >= 2:
            joint[toks[0], toks[1]] += float(pr)
        else:
            nxt = first_token_dist(model, [toks[0]], gamma)
            for y in range(V):
                joint[toks[0], y] += float(pr * nxt[y])
    for y1 in range(V):
        for y2 in range(V):
            want = float(model.p([])[y1] * model.p([y1])[y2])
            assert abs(joint[y1, y2] - want) < 1e-12


def test_residual_sign_matters():
    """A plausible slip (sampling from max(0, q - p)) would break losslessness.

    This pins the direction of the residual through the exact distribution,
    not through the formula: with p=(1/2,1/3,1/6), q=(1/6,1/3,1/2) the only
    possible token after a rejection is 0.
    """
    g = json.load(open(os.path.join(GOLDEN, "accept_rule_v3.json")))
    p, q = _frac_list(g["p"]), _frac_list(g["q"])
    model = TableModel(3, 0, iid=(p, q))
    for pr, toks in step_outcomes(model, [], 1):
        if len(toks) == 1:
            assert toks[0] == g["residual"].index("1")


def test_golden_acceptance_probabilities_and_tv():
    g = json.load(open(os.path.join(GOLDEN, "accept_rule_v3.json")))
    p, q = _frac_list(g["p"]), _frac_list(g["q"])
    P, Q = _logits(p)[None, :], _logits(q)[None, :]
    for x, want in enumerate(_frac_list(g["accept_prob_by_draft"])):
        r = accept_and_diverge(
            np.concatenate([P, P])[None], Q[None], np.array([[x]]), np.array([1]),
            np.array([[0.5]], dtype=np.float32), np.array([[0.5, 0.5]], dtype=np.float32),
        )
        assert abs(r["accept_prob"][0, 0] - float(want)) < 1e-12
        assert abs(r["tv"][0, 0] - float(F(g["tv"]))) < 1e-12
        assert abs(r["p_tok"][0, 0] - float(p[x])) < 1e-12
        assert abs(r["q_tok"][0, 0] - float(q[x])) < 1e-12


def test_eq3_expected_emitted_tokens():
    g = json.load(open(os.path.join(GOLDEN, "eq3_expected_tokens.json")))
    for case in g["cases"]:
        p, q = _frac_list(case["p"]), _frac_list(case["q"])
        model = TableModel(len(p), 0, iid=(p, q))
        e = sum(pr * len(toks) for pr, toks in step_outcomes(model, [], case["gamma"]))
        assert e == F(case["expected_emitted"])
        alpha = F(case["alpha"])
        assert alpha == sum(min(a, b) for a, b in zip(p, q))


# ---------------------------------------------------------------- identities

def _rand_pair(rng, V, sigma=3.0, noise=1.0):
    zp = rng.normal(0, sigma, V)
    zq = zp + rng.normal(0, noise, V)
    return zp, zq


def _softmax(z):
    e = np.exp(z - z.max())
    return e / e.sum()


@pytest.mark.parametrize("V,seed", [(5, 0), (50, 1), (1000, 2)])
def test_acceptance_rate_equals_one_minus_tv(V, seed):
    """Eq. 2 holds exactly per position when the draft is drawn from q."""
    rng = np.random.default_rng(seed)
    zp, zq = _rand_pair(rng, V)
    q = _softmax(zq)
    P = np.stack([zp, zp])[None]
    Q = zq[None, None]
    rate = 0.0
    tv = None
    for x in range(V):
        r = accept_and_diverge(P, Q, np.array([[x]]), np.array([1]),
                               np.array([[0.0]], np.float32), np.array([[0.0, 0.0]], np.float32))
        rate += q[x] * r["accept_prob"][0, 0]
        tv = r["tv"][0, 0]
    assert abs(rate - (1.0 - tv)) < 1e-12


@pytest.mark.parametrize("seed", range(5))
def test_kl_tv_against_scipy(seed):
    rng = np.random.default_rng(seed)
    V = 777
    zp, zq = _rand_pair(rng, V, noise=0.5 + seed)
    p, q = _softmax(zp), _softmax(zq)
    r = accept_and_diverge(np.stack([zp, zp])[None], zq[None, None], np.array([[3]]), np.array([1]),
                           np.array([[0.1]], np.float32), np.array([[0.2, 0.3]], np.float32))
    kl, tv = r["kl"][0, 0], r["tv"][0, 0]
    assert abs(kl - rel_entr(p, q).sum()) <= 1e-12 * max(1.0, kl)
    assert abs(tv - 0.5 * cityblock(p, q)) <= 1e-12
    assert kl >= 0.0
    assert 0.0 <= tv <= 1.0
    assert tv <= math.sqrt(kl / 2.0) + 1e-15  # Pinsker


def test_tv_symmetric_and_zero_on_equal_rows():
    rng = np.random.default_rng(7)
    zp, zq = _rand_pair(rng, 300)
    kw = dict(drafts=np.array([[1]]), gamma=np.array([1]),
              u_acc=np.array([[0.5]], np.float32), u_res=np.array([[0.5, 0.5]], np.float32))
    a = accept_and_diverge(np.stack([zp, zp])[None], zq[None, None], **kw)
    b = accept_and_diverge(np.stack([zq, zq])[None], zp[None, None], **kw)
    assert abs(a["tv"][0, 0] - b["tv"][0, 0]) < 1e-14
    c = accept_and_diverge(np.stack([zp, zp])[None], zp[None, None], **kw)
    assert c["tv"][0, 0] == 0.0 and c["kl"][0, 0] == 0.0


def test_kl_closed_form_two_point():
    """KL between Bernoulli(a) and Bernoulli(b) written out by hand."""
    a, b = 0.8, 0.3
    zp = np.log([a, 1 - a])
    zq = np.log([b, 1 - b])
    r = accept_and_diverge(np.stack([zp, zp])[None], zq[None, None], np.array([[0]]), np.array([1]),
                           np.array([[0.5]], np.float32), np.array([[0.5, 0.5]], np.float32))
    want = a * math.log(a / b) + (1 - a) * math.log((1 - a) / (1 - b))
    assert abs(r["kl"][0, 0] - want) < 1e-14
    assert abs(r["tv"][0, 0] - abs(a - b)) < 1e-14


@pytest.mark.parametrize("seed", range(4))
def test_draft_equal_to_verifier_accepts_everything(seed):
    rng = np.random.default_rng(seed)
    V, g = 200, 6
    z = rng.normal(0, 3, (g + 1, V))
    drafts = rng.integers(0, V, g)
    u_acc = rng.random(g).astype(np.float32)
    u_res = rng.random(g + 1).astype(np.float32)
    r = accept_and_diverge(z[None], z[None, :g], drafts[None], np.array([g]), u_acc[None], u_res[None],
                           kv_len=np.array([100]))
    assert r["accept_len"][0] == g
    assert (r["accept_prob"][0] == 1.0).all()
    assert (r["kl"][0] == 0).all() and (r["tv"][0] == 0).all()
    assert r["new_len"][0] == 100
    # the bonus token comes from p_gamma
    cdf = np.cumsum(_softmax(z[g]))
    assert r["out_tokens"][0, g] == int(np.searchsorted(cdf, u_res[g], side="right"))


@pytest.mark.parametrize("seed", range(3))
def test_gamma_zero_is_plain_sampling(seed):
    rng = np.random.default_rng(seed)
    V = 1000
    z = rng.normal(0, 3, (1, V))
    for u in rng.random(20).astype(np.float32):
        r = accept_and_diverge(z[None], np.zeros((1, 0, V)), np.zeros((1, 0), np.int64), np.array([0]),
                               np.zeros((1, 0), np.float32), np.array([[u]], np.float32))
        cdf = np.cumsum(_softmax(z[0]))
        assert r["accept_len"][0] == 0
        assert r["out_tokens"][0, 0] == int(np.searchsorted(cdf, u, side="right"))


def test_acceptance_length_statistics():
    """P(k >= i) = prod_{j<i} (1 - TV_j) (Monte Carlo, rows differ)."""
    rng = np.random.default_rng(11)
    V, g, N = 40, 3, 4000
    zp = rng.normal(0, 2, (g + 1, V))
    zq = zp[:g] + rng.normal(0, 1.0, (g, V))
    qs = [_softmax(zq[j]) for j in range(g)]
    counts = np.zeros(g + 2)
    tv = None
    for _ in range(N):
        drafts = np.array([rng.choice(V, p=qs[j]) for j in range(g)])
        r = accept_and_diverge(zp[None], zq[None], drafts[None], np.array([g]),
                               rng.random((1, g)).astype(np.float32), rng.random((1, g + 1)).astype(np.float32))
        counts[r["accept_len"][0]] += 1
        tv = r["tv"][0]
    surv = 1.0
    for i in range(1, g + 1):
        surv *= 1.0 - tv[i - 1]
        emp = counts[i:].sum() / N
        sd = math.sqrt(surv * (1 - surv) / N)
        assert abs(emp - surv) < 5 * sd + 1e-3


def test_inverse_cdf_worked_example():
    """Uniform weights over 4 tokens, u = 0.6: C = (.25, .5, .75, 1), so the
    smallest x with C(x) > 0.6 is 2, at distance 0.1 from both brackets."""
    t, m = inverse_cdf(np.full(4, 0.25), 0.6)
    assert t == 2 and abs(m - 0.1) < 1e-12
    t, _ = inverse_cdf(np.array([0.0, 1.0, 0.0]), 0.0)
    assert t == 1


def test_data_errors_set_status():
    V = 10
    z = np.zeros((1, 3, V))
    ok = dict(p_logits=z, q_logits=z[:, :2], drafts=np.array([[1, 2]]), gamma=np.array([2]),
              u_acc=np.array([[0.1, 0.2]], np.float32), u_res=np.array([[0.1, 0.2, 0.3]], np.float32))
    assert accept_and_diverge(**ok)["status"] == 0
    bad = dict(ok, gamma=np.array([3]))
    r = accept_and_diverge(**bad)
    assert r["status"] == 1 and r["accept_len"][0] == -1
    bad = dict(ok, drafts=np.array([[1, 10]]))
    assert accept_and_diverge(**bad)["status"] == 4
    bad = dict(ok, u_res=np.array([[0.1, 0.2, 1.0]], np.float32))
    r = accept_and_diverge(**bad)
    assert r["status"] == 8 and np.isnan(r["kl"][0]).all()
    r = accept_and_diverge(**ok, kv_len=np.array([2]))
    assert r["status"] == 2 and r["new_len"][0] == 2


def test_boundary_margin_reports_near_threshold_uniforms():
    V = 3
    zp = np.log([0.5, 0.25, 0.25])
    zq = np.log([0.25, 0.25, 0.5])
    # draft 2 has a = 0.5; a uniform 1e-8 above it is a boundary case
    r = accept_and_diverge(np.stack([zp, zp])[None], zq[None, None], np.array([[2]]), np.array([1]),
                           np.array([[0.5 + 1e-8]]), np.array([[0.3, 0.3]]))
    assert r["accept_len"][0] == 0 and r["boundary"][0]
    r = accept_and_diverge(np.stack([zp, zp])[None], zq[None, None], np.array([[2]]), np.array([1]),
                           np.array([[0.7]]), np.array([[0.3, 0.3]]))
    assert not r["boundary"][0]
