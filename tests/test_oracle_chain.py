"""Pins of the three-level chain reading (multi-level verification, Section
3.1 and Section 4.3; the reading is stated in oracle/chain.py).

Exact enumeration over three tiny table models -- draft M1, intermediate M2,
target M3 with rational conditionals -- of one chain step: M1 drafts gamma2
tokens, M2 verifies them (accept/reject, residual or bonus), the target
verifies the first min(k2 + 1, gamma_cap) tokens M2 emitted with M2's rows as
its draft distribution, and emits its own correction or bonus token. Every
discrete choice and every region of the uniforms on which the references'
outcome is constant is enumerated with exact rational thresholds computed
here (not by the reference); the reference is evaluated at an interior point
of each region. The emitted tokens must follow the target's distribution:
the first exactly, and the first two (continuing with the target alone when
the step emitted one token) as p3(y1) p3(y2 | y1).
"""

from fractions import Fraction as F
from itertools import product
import math

import numpy as np
import pytest

from oracle import chain
from oracle.accept import accept_sequence


class Tables:
    """p1, p2, p3 (. | prefix) as exact rationals with occasional zeros."""

    def __init__(self, V, seed):
        self.V, self.rng, self.cache = V, np.random.default_rng(seed), {}

    def dist(self, level, prefix):
        key = (level,) + tuple(prefix)
        if key not in self.cache:
            w = self.rng.integers(0, 6, size=self.V)
            if w.sum() == 0:
                w[self.rng.integers(self.V)] = 1
            tot = int(w.sum())
            self.cache[key] = [F(int(x), tot) for x in w]
        return self.cache[key]


def _logits(d):
    return np.array([math.log(float(x)) if x > 0 else -np.inf for x in d])


def _cdf_intervals(w):
    W = sum(w)
    acc, out = F(0), []
    for x, wx in enumerate(w):
        if wx > 0:
            out.append((x, acc / W, (acc + wx) / W))
        acc += wx
    return out


def verify_outcomes(m, prefix, drafts, p_level, q_level):
    """Every outcome of one verify step of `drafts` (from q_level) by p_level:
    (probability given the drafts, accept_len, emitted tokens), with the
    reference evaluated at an interior point of each uniform region."""
    g = len(drafts)
    V = m.V
    rows_p = [m.dist(p_level, list(prefix) + list(drafts[:j])) for j in range(g + 1)]
    rows_q = [m.dist(q_level, list(prefix) + list(drafts[:j])) for j in range(g)]
    P = np.stack([_logits(r) for r in rows_p])
    Q = np.stack([_logits(r) for r in rows_q]) if g else np.zeros((0, V))
    a = [min(F(1), rows_p[j][drafts[j]] / rows_q[j][drafts[j]]) for j in range(g)]
    for k in range(g + 1):
        reach = F(1)
        for j in range(k):
            reach *= a[j]
        if k < g:
            reach *= 1 - a[k]
        if reach == 0:
            continue
        u_acc = np.zeros(g)
        for j in range(k):
            u_acc[j] = float(a[j]) / 2
        if k < g:
            u_acc[k] = (float(a[k]) + 1) / 2
        if k < g:
            w = [max(F(0), x - y) for x, y in zip(rows_p[k], rows_q[k])]
            if sum(w) == 0:
                w = rows_p[k]
        else:
            w = rows_p[k]
        for _, lo, hi in _cdf_intervals(w):
            u_res = np.zeros(g + 1)
            u_res[k] = float((lo + hi) / 2)
            r = accept_sequence(P, Q, np.array(drafts, dtype=np.int64), g, u_acc, u_res, g, V)
            assert r["status"] == 0 and r["accept_len"] == k
            yield reach * (hi - lo), k, [int(t) for t in r["tokens"][: k + 1]]


def chain_outcomes(m, prefix, gamma2, gamma_cap):
    """(probability, tokens the chain step emits) over every outcome."""
    V = m.V
    for x in product(range(V), repeat=gamma2):
        px = F(1)
        for j in range(gamma2):
            px *= m.dist(1, list(prefix) + list(x[:j]))[x[j]]
        if px == 0:
            continue
        for p2, k2, e2 in verify_outcomes(m, prefix, list(x), 2, 1):
            out2 = np.full((1, gamma2 + 1), -1)
            out2[0, : k2 + 1] = e2
            g3, d3 = chain.window([k2], out2, gamma_cap)
            drafts3 = [int(t) for t in d3[0, : int(g3[0])]]
            for p3, k3, e3 in verify_outcomes(m, prefix, drafts3, 3, 2):
                out3 = np.full((1, gamma_cap + 1), -1)
                out3[0, : k3 + 1] = e3
                up, lo, pend, npend, st = chain.consensus([len(prefix)], [k2], [k3], out2, out3)
                assert st == 0
                # the emitted sequence and the rows each level keeps
                assert e3[:k3] == e2[:k3]
                assert up[0] == len(prefix) + 1 + k3 and lo[0] == len(prefix) + 1 + min(k2, k3)
                assert list(pend[0, : npend[0]]) == e3[min(k2, k3):]
                yield px * p2 * p3, e3


@pytest.mark.parametrize("V,gamma2,cap,seed", [(2, 2, 2, 0), (3, 2, 2, 1), (3, 1, 2, 2), (2, 3, 2, 3), (3, 2, 3, 4)])
def test_chain_first_token_is_distributed_as_target(V, gamma2, cap, seed):
    m = Tables(V, seed)
    d = [F(0)] * V
    total = F(0)
    for pr, toks in chain_outcomes(m, [], gamma2, cap):
        d[toks[0]] += pr
        total += pr
    assert total == 1
    assert d == m.dist(3, [])


@pytest.mark.parametrize("V,gamma2,cap,seed", [(2, 2, 2, 5), (3, 2, 2, 6)])
def test_chain_two_tokens_are_distributed_as_target(V, gamma2, cap, seed):
    m = Tables(V, seed)
    joint = {}
    for pr, toks in chain_outcomes(m, [], gamma2, cap):
        if len(toks) >= 2:
            joint[(toks[0], toks[1])] = joint.get((toks[0], toks[1]), F(0)) + pr
        else:
            for y, p in enumerate(m.dist(3, [toks[0]])):
                joint[(toks[0], y)] = joint.get((toks[0], y), F(0)) + pr * p
    for y1 in range(V):
        for y2 in range(V):
            assert joint.get((y1, y2), F(0)) == m.dist(3, [])[y1] * m.dist(3, [y1])[y2]


def test_a_wrong_target_draft_distribution_breaks_losslessness():
    """Verifying M2's emitted tokens against M1's rows (a plausible slip)
    does not give the target distribution: the enumeration can tell."""
    m = Tables(3, 1)
    V, gamma2, cap = 3, 2, 2
    d = [F(0)] * V
    for x in product(range(V), repeat=gamma2):
        px = F(1)
        for j in range(gamma2):
            px *= m.dist(1, list(x[:j]))[x[j]]
        if px == 0:
            continue
        for p2, k2, e2 in verify_outcomes(m, [], list(x), 2, 1):
            drafts3 = e2[: min(k2 + 1, cap)]
            if any(m.dist(1, drafts3[:j])[drafts3[j]] == 0 for j in range(len(drafts3))):
                continue
            for p3, k3, e3 in verify_outcomes(m, [], drafts3, 3, 1):
                d[e3[0]] += px * p2 * p3
    assert d != m.dist(3, [])


def test_window_and_consensus_edge_cases():
    g, d = chain.window([0, 4, 9, -1], [[7, -1, -1, -1, -1], [1, 2, 3, 4, 5], [1, 2, 3, 4, 5], [0] * 5], 4)
    assert list(g) == [1, 4, -1, -1]  # k = 9 cannot come from 5 emitted slots
    assert list(d[0]) == [7, 0, 0, 0] and list(d[3]) == [0, 0, 0, 0]
    up, lo, pend, n, st = chain.consensus([5, 5, 5, 5], [0, 3, 2, 1], [1, 0, -1, 3],
                                          [[8, -1, -1, -1]] + [[1, 2, 3, 4]] * 3,
                                          [[8, 9, -1, -1]] + [[6, -1, -1, -1]] * 3)
    assert list(up) == [7, 6, 5, 5] and list(lo) == [6, 6, 5, 5]
    assert st == chain.ST_CHAIN and n[3] == 0  # k_upper = 3 > k_lower + 1: not one chain step
    assert list(pend[0]) == [8, 9] and n[0] == 2          # the target accepted M2's correction token
    assert list(pend[1]) == [6, -1] and n[1] == 1
    assert n[2] == 0                                       # flagged upstream: nothing kept, nothing pending
