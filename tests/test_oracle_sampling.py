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
  * Top-k / top-p: the filter against its definition written entry by entry
    (strictly larger count < k; strictly larger mass < p, ties included),
    against the ascending cumulative rule for distinct logits, top-k then
    top-p composition and the extremes (k = 1 and tiny p keep the maximum
    only); top-k = 1 with argmax drafts is greedy decoding; and exact
    enumeration shows the first emitted token is distributed as the filtered
    target row when the drafts come from the filtered draft rows.
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


# ---------------------------------------------------------------- top-k / top-p

from oracle.accept import filter_logits  # noqa: E402


def _kept(z):
    return np.isfinite(z)


@pytest.mark.parametrize("seed", range(6))
def test_top_k_keeps_entries_with_fewer_than_k_strictly_larger(seed):
    rng = np.random.default_rng(seed)
    V = 23
    z = rng.integers(0, 6, V).astype(np.float64)  # many ties
    for k in range(1, V):
        got, _ = filter_logits(z, top_k=k)
        greater = np.array([(z > z[i]).sum() for i in range(V)])  # the definition, entry by entry
        np.testing.assert_array_equal(_kept(got), greater < k)
        np.testing.assert_array_equal(got[_kept(got)], z[greater < k])  # kept logits unchanged
    for k in (0, V, V + 5):  # off
        np.testing.assert_array_equal(filter_logits(z, top_k=k)[0], z)


@pytest.mark.parametrize("seed", range(6))
def test_top_p_keeps_entries_whose_larger_mass_is_below_p(seed):
    rng = np.random.default_rng(100 + seed)
    V = 17
    z = np.round(rng.normal(0, 1.5, V), 1)  # rounded: ties
    r = np.exp(z - z.max())
    r /= r.sum()
    for p in (0.05, 0.3, 0.5, 0.77, 0.9, 0.999):
        got, margin = filter_logits(z, top_p=p)
        above = np.array([r[z > z[i]].sum() for i in range(V)])  # the definition, entry by entry
        np.testing.assert_array_equal(_kept(got), above < p)
        assert _kept(got)[np.argmax(z)]  # the largest logit always stays
        assert margin == pytest.approx(np.min(np.abs(np.unique(above) - p)), abs=1e-15)
    np.testing.assert_array_equal(filter_logits(z, top_p=1.0)[0], z)


def test_top_p_is_the_ascending_cumulative_rule_for_distinct_logits():
    rng = np.random.default_rng(7)
    for _ in range(20):
        V = 40
        z = rng.normal(0, 2, V)
        p = float(rng.uniform(0.05, 0.95))
        r = np.exp(z - z.max())
        r /= r.sum()
        order = np.argsort(z)  # ascending, as the usual rule sorts
        cum = np.cumsum(r[order])
        removed = np.zeros(V, bool)
        removed[order[cum <= 1 - p]] = True
        got, _ = filter_logits(z, top_p=p)
        np.testing.assert_array_equal(_kept(got), ~removed)


def test_top_k_then_top_p_and_the_extremes():
    rng = np.random.default_rng(8)
    z = rng.normal(0, 2, 30)
    zk, _ = filter_logits(z, top_k=6)
    both, _ = filter_logits(z, top_k=6, top_p=0.6)
    np.testing.assert_array_equal(both, filter_logits(zk, top_p=0.6)[0])  # top-p acts on the top-k result
    assert _kept(both).sum() <= 6
    top1 = np.flatnonzero(z == z.max())
    np.testing.assert_array_equal(np.flatnonzero(_kept(filter_logits(z, top_k=1)[0])), top1)
    np.testing.assert_array_equal(np.flatnonzero(_kept(filter_logits(z, top_p=1e-9)[0])), top1)


def test_top_k_one_with_argmax_drafts_is_greedy():
    rng = np.random.default_rng(9)
    g, V = 4, 60
    for _ in range(10):
        P = rng.normal(0, 3, (g + 1, V))
        Q = P[:g] + rng.normal(0, 1.5, (g, V))
        d = np.argmax(Q, axis=1)  # what the filtered draft distribution (one-hot) emits
        ua, ur = rng.random(g), rng.random(g + 1)
        r = accept_sequence(P, Q, d, g, ua, ur, g, V, temperature=0.8, top_k=1)
        gr = accept_sequence_greedy(P, Q, d, g, g, V)
        assert r["accept_len"] == gr["accept_len"]
        np.testing.assert_array_equal(r["tokens"], gr["tokens"])
        np.testing.assert_array_equal(r["tv"], gr["tv"])


def _filtered_exact(d, top_k, top_p):
    """Top-k / top-p of a rational distribution d (distinct values), exactly."""
    V = len(d)
    keep = [sum(1 for y in d if y > x) < top_k for x in d] if 0 < top_k < V else [True] * V
    kept = [x if k else F(0) for x, k in zip(d, keep)]
    tot = sum(kept)
    r = [x / tot for x in kept]
    if top_p < 1:
        keep2 = [k and sum(y for y in r if y > x) < F(top_p) for x, k in zip(r, keep)]
        kept = [x if k else F(0) for x, k in zip(r, keep2)]
        tot = sum(kept)
        r = [x / tot for x in kept]
    return r


@pytest.mark.parametrize("V,gamma,top_k,top_p,seed", [(4, 1, 2, 1.0, 0), (4, 2, 3, 1.0, 1), (5, 2, 0, 0.6, 2),
                                                      (5, 1, 4, 0.75, 3), (3, 3, 2, 0.9, 4)])
def test_filtered_first_token_is_the_filtered_target(V, gamma, top_k, top_p, seed):
    """Exact enumeration: drafts drawn from the filtered draft rows, the
    accept rule on the filtered rows; the first emitted token is distributed
    exactly as the filtered target row."""
    rng = np.random.default_rng(seed)
    cache = {}

    def dist(kind, prefix):
        key = (kind,) + tuple(prefix)
        if key not in cache:
            w = rng.permutation(np.arange(1, V + 1)) * 7 + rng.integers(0, 3, V)  # distinct weights
            cache[key] = [F(int(x), int(w.sum())) for x in w]
        return cache[key]

    def filt(kind, prefix):
        return _filtered_exact(dist(kind, prefix), top_k, top_p)

    first = [F(0)] * V
    total = F(0)
    for drafts in product(range(V), repeat=gamma):
        pd = F(1)
        for j in range(gamma):
            pd *= filt("q", drafts[:j])[drafts[j]]
        if pd == 0:
            continue
        P = np.stack([_logits(dist("p", drafts[:j])) for j in range(gamma + 1)])
        Q = np.stack([_logits(dist("q", drafts[:j])) for j in range(gamma)])
        a = []
        for j in range(gamma):
            pj, qj = filt("p", drafts[:j])[drafts[j]], filt("q", drafts[:j])[drafts[j]]
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
            pk = filt("p", drafts[:k])
            if k < gamma:
                w = [max(F(0), x - y) for x, y in zip(pk, filt("q", drafts[:k]))]
                if sum(w) == 0:
                    w = pk
            else:
                w = pk
            for _, lo, hi in _cdf_intervals(w):
                u_res = np.zeros(gamma + 1)
                u_res[k] = float((lo + hi) / 2)
                r = accept_sequence(P, Q, np.array(drafts, dtype=np.int64), gamma, u_acc, u_res, gamma, V,
                                    top_k=top_k, top_p=top_p)
                assert r["status"] == 0 and r["accept_len"] == k
                pr = pd * reach * (hi - lo)
                first[int(r["tokens"][0])] += pr
                total += pr
    assert total == 1
    want = filt("p", ())
    for x in range(V):
        assert abs(float(first[x]) - float(want[x])) < 1e-12
