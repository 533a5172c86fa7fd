"""Pins for the sampling variants of the accept reference (CPU only).

  * Greedy decoding: speculative generation with any draft model emits exactly
    the tokens of greedy decoding with the target alone -- the paper's own
    correctness check (Section 5.1, output quality) -- on tiny table models
    whose integer logits tie often, so the lowest-index rule is exercised.
  * Temperature: with T = 1/2 the tempered distributions of rational p and q
    are p^2 / sum p^2 and q^2 / sum q^2, again rational, so exact enumeration
    over every (draft, uniform) region shows that the first emitted token is
    distributed exactly as the tempered target distribution.
  * T = 1 is the untempered rule; greedy divergences match the argmax
    agreement of the two rows.
"""

import math
from fractions import Fraction as F
from itertools import product

import numpy as np
import pytest

from oracle.accept import accept_and_diverge, accept_sequence, accept_sequence_greedy


# ---------------------------------------------------------------- greedy identity with the target alone

class IntTable:
    """Deterministic logits z(. | last two tokens) with small integers (many ties)."""

    def __init__(self, V, seed, spread):
        self.V, self.rng, self.spread, self.cache = V, np.random.default_rng(seed), spread, {}

    def logits(self, prefix):
        key = tuple(prefix[-2:])
        if key not in self.cache:
            self.cache[key] = self.rng.integers(0, self.spread, size=self.V).astype(np.float64)
        return self.cache[key]


def _argmax_lowest(z):
    best = 0
    for i in range(1, len(z)):
        if z[i] > z[best]:
            best = i
    return best


def _target_only(target, prompt, n):
    out = list(prompt)
    while len(out) < len(prompt) + n:
        out.append(_argmax_lowest(target.logits(out)))
    return out[len(prompt):]


def _speculative(target, draft, prompt, n, gamma):
    out = list(prompt)
    while len(out) < len(prompt) + n:
        drafts = []
        ctx = list(out)
        for _ in range(gamma):  # the draft model decodes greedily
            x = _argmax_lowest(draft.logits(ctx))
            drafts.append(x)
            ctx.append(x)
        P = np.stack([target.logits(out + drafts[:j]) for j in range(gamma + 1)])
        Q = np.stack([draft.logits(out + drafts[:j]) for j in range(gamma)]) if gamma else np.zeros((0, target.V))
        r = accept_sequence_greedy(P, Q, np.array(drafts, dtype=np.int64), gamma, gamma, target.V)
        assert r["status"] == 0
        k = r["accept_len"]
        out.extend(int(t) for t in r["tokens"][: k + 1])
    return out[len(prompt): len(prompt) + n]


@pytest.mark.parametrize("V,spread,gamma,seed", [(5, 3, 1, 0), (7, 4, 3, 1), (4, 2, 5, 2), (9, 6, 4, 3), (6, 3, 0, 4)])
def test_greedy_speculation_reproduces_target_only_decoding(V, spread, gamma, seed):
    target = IntTable(V, seed, spread)
    for dseed, dspread in ((100 + seed, spread), (200 + seed, 2)):
        draft = IntTable(V, dseed, dspread)
        for prompt in ([0], [1, 2], [V - 1, 0, 3 % V]):
            assert _speculative(target, draft, prompt, 40, gamma) == _target_only(target, prompt, 40)


def test_greedy_draft_equal_to_target_accepts_everything():
    t = IntTable(6, 7, 3)
    P = np.stack([t.logits([j]) for j in range(4)])
    drafts = np.array([_argmax_lowest(P[j]) for j in range(3)])
    r = accept_sequence_greedy(P, P[:3], drafts, 3, 3, 6)
    assert r["accept_len"] == 3 and list(r["tokens"]) == list(drafts) + [_argmax_lowest(P[3])]
    assert (r["tv"] == 0).all() and (r["kl"] == 0).all() and (r["accept_prob"] == 1).all()


def test_greedy_divergences_are_argmax_agreement():
    P = np.array([[0.0, 2.0, 2.0], [5.0, 1.0, 0.0], [1.0, 1.0, 1.0]])
    Q = np.array([[0.0, 2.0, 3.0], [5.0, 5.0, 0.0]])
    r = accept_sequence_greedy(P, Q, np.array([2, 0]), 2, 2, 3)
    # row 0: argmax p = 1 (tie with 2 -> lowest), argmax q = 2: disagree; draft 2 rejected
    assert r["tv"][0] == 1.0 and r["kl"][0] == math.inf
    assert r["p_tok"][0] == 0.0 and r["q_tok"][0] == 1.0 and r["accept_prob"][0] == 0.0
    # row 1: argmax p = 0, argmax q = 0 (tie with 1 -> lowest): agree
    assert r["tv"][1] == 0.0 and r["kl"][1] == 0.0
    assert r["accept_len"] == 0 and list(r["tokens"]) == [1, -1, -1]


def test_greedy_needs_no_uniforms_and_flags_bad_tokens():
    P = np.zeros((1, 3, 4), np.float32)
    Q = np.zeros((1, 2, 4), np.float32)
    nan = np.full((1, 3), np.nan, np.float32)
    r = accept_and_diverge(P, Q, np.array([[0, 0]]), np.array([2]), nan[:, :2], nan, temperature=0)
    assert r["status"] == 0 and r["accept_len"][0] == 2
    r = accept_and_diverge(P, Q, np.array([[0, 9]]), np.array([2]), nan[:, :2], nan, temperature=0)
    assert r["status"] == 4 and r["accept_len"][0] == -1


# ---------------------------------------------------------------- temperature

def _rat_dist(rng, V):
    w = rng.integers(1, 6, size=V)
    return [F(int(x), int(w.sum())) for x in w]


def _tempered_half(d):
    """softmax(log d / (1/2)) = d^2 / sum d^2, exactly."""
    sq = [x * x for x in d]
    tot = sum(sq)
    return [x / tot for x in sq]


def _cdf_intervals(w):
    W = sum(w)
    acc, out = F(0), []
    for x, wx in enumerate(w):
        if wx > 0:
            out.append((x, acc / W, (acc + wx) / W))
        acc += wx
    return out


def _logits(d):
    return np.array([math.log(float(x)) for x in d])


@pytest.mark.parametrize("V,gamma,seed", [(3, 1, 0), (3, 2, 1), (4, 2, 2), (2, 3, 3)])
def test_temperature_half_first_token_is_tempered_p(V, gamma, seed):
    rng = np.random.default_rng(seed)
    cache = {}

    def dist(kind, prefix):
        key = (kind,) + tuple(prefix)
        if key not in cache:
            cache[key] = _rat_dist(rng, V)
        return cache[key]

    T = 0.5
    first = [F(0)] * V
    total = F(0)
    for drafts in product(range(V), repeat=gamma):
        # drafts are drawn from the tempered draft distribution
        pd = F(1)
        for j in range(gamma):
            pd *= _tempered_half(dist("q", drafts[:j]))[drafts[j]]
        P = np.stack([_logits(dist("p", drafts[:j])) for j in range(gamma + 1)])
        Q = np.stack([_logits(dist("q", drafts[:j])) for j in range(gamma)])
        a = []
        for j in range(gamma):
            pj = _tempered_half(dist("p", drafts[:j]))[drafts[j]]
            qj = _tempered_half(dist("q", drafts[:j]))[drafts[j]]
            a.append(min(F(1), pj / qj))
        for k in range(gamma + 1):
            reach = F(1)
            for j in range(k):
                reach *= a[j]
            if k < gamma:
                reach *= 1 - a[k]
            if reach == 0:
                continue
            u_acc = np.zeros(gamma)
            for j in range(k):
                u_acc[j] = float(a[j]) / 2
            if k < gamma:
                u_acc[k] = (float(a[k]) + 1) / 2
            pk = _tempered_half(dist("p", drafts[:k]))
            if k < gamma:
                qk = _tempered_half(dist("q", drafts[:k]))
                w = [max(F(0), x - y) for x, y in zip(pk, qk)]
                if sum(w) == 0:
                    w = pk
            else:
                w = pk
            for _, lo, hi in _cdf_intervals(w):
                u_res = np.zeros(gamma + 1)
                u_res[k] = float((lo + hi) / 2)
                r = accept_sequence(P, Q, np.array(drafts, dtype=np.int64), gamma, u_acc, u_res, gamma, V,
                                    temperature=T)
                assert r["status"] == 0 and r["accept_len"] == k
                pr = pd * reach * (hi - lo)
                first[int(r["tokens"][0])] += pr
                total += pr
    assert total == 1
    want = _tempered_half(dist("p", ()))
    for x in range(V):
        assert abs(float(first[x]) - float(want[x])) < 1e-12


def test_temperature_one_is_the_plain_rule():
    rng = np.random.default_rng(5)
    B, g, V = 3, 4, 50
    P = rng.normal(0, 3, (B, g + 1, V)).astype(np.float32)
    Q = (P[:, :g] + rng.normal(0, 1, (B, g, V))).astype(np.float32)
    d = rng.integers(0, V, (B, g))
    ua = rng.random((B, g)).astype(np.float32)
    ur = rng.random((B, g + 1)).astype(np.float32)
    a = accept_and_diverge(P, Q, d, np.full(B, g), ua, ur)
    b = accept_and_diverge(P, Q, d, np.full(B, g), ua, ur, temperature=1.0)
    for key in ("accept_len", "out_tokens", "tv", "kl", "accept_prob"):
        np.testing.assert_array_equal(a[key], b[key])


def test_tempered_divergences_against_scipy():
    from scipy.special import log_softmax, rel_entr

    rng = np.random.default_rng(6)
    V = 40
    zp = rng.normal(0, 3, V)
    zq = zp + rng.normal(0, 1, V)
    for T in (0.3, 0.7, 1.8):
        r = accept_sequence(np.stack([zp, zp]), zq[None], np.array([3]), 1, np.array([0.5]), np.array([0.5, 0.5]),
                            1, V, temperature=T)
        p, q = np.exp(log_softmax(zp / T)), np.exp(log_softmax(zq / T))
        assert r["tv"][0] == pytest.approx(0.5 * np.abs(p - q).sum(), rel=1e-12)
        assert r["kl"][0] == pytest.approx(rel_entr(p, q).sum(), rel=1e-10)
        assert r["p_tok"][0] == pytest.approx(p[3], rel=1e-12)
