"""Accept/reject, resampling and divergences, fp64 reference (test infrastructure only).

Follows Section 2.2 (basic speculative decoding, steps 3-4, probabilistic
acceptance, Eq. 2) and Section 4.2 (total variation distance, Eq. 5).

Per sequence b with gamma = gamma_b drafted tokens x_0 .. x_{gamma-1}:

  1. p_j = softmax(P[b, j]) for j = 0..gamma (the verifier's gamma + 1
     conditionals) and q_j = softmax(Q[b, j]) for j < gamma (the drafter's).
  2. TV_j = 1/2 sum_v |p_j(v) - q_j(v)|            (Eq. 5)
     KL_j = sum_{v: p_j(v) > 0} p_j(v) log(p_j(v) / q_j(v))   (nats)
  3. a_j = min(1, p_j(x_j) / q_j(x_j)); a draft with q_j(x_j) = 0 gets a_j = 1.
  4. k = the first j < gamma whose draft is rejected, i.e. NOT (u_acc[b, j] < a_j);
     k = gamma if all are accepted.
  5. One more token t: if k < gamma it is drawn from the residual
     max(0, p_k - q_k) (renormalised); if every draft was accepted it is
     drawn from p_gamma. A residual that is identically zero falls back to p_k.
  6. Drawing from weights w: C(x) = sum_{y <= x} w_y in ascending vocabulary
     order, W = C(V - 1), and t = the smallest x with C(x) > u_res[b, k] * W
     (the largest x with w_x > 0 if rounding leaves none).
  7. Outputs: accept_len = k, tokens = (x_0 .. x_{k-1}, t) padded with -1,
     new_len = kv_len_b - gamma + k.

Readings where the paper is loose: the verifier gives gamma + 1 rows (the
extra row feeds the bonus token); after a rejection the extra token comes from
the residual rather than from p itself (the cited probabilistic-acceptance
rule, which is what makes the output distribution equal p); acceptance is the
strict test u < a with u in [0, 1); KL is KL(p_verifier || q_draft); TV and KL
are reported for every j < gamma_b whether or not row j was reached; one
uniform is spent per decision (u_acc per draft, u_res per possible stop row).

Each sequence also gets a decision margin: the smallest distance, over the
decisions actually taken, between a uniform and the threshold it was compared
against (|u_acc - a_j|, and the distance of u_res * W to the two CDF values
bracketing t, divided by W). A margin below 1e-6 marks a boundary case whose
discrete outcome may legitimately differ under fp32 arithmetic.

Sampling variants (the paper's "chosen sampling rule": greedy or
probabilistic acceptance, with the sampling parameters of the logits
processors). Temperature T > 0 replaces every distribution above by
softmax(z / T) -- p, q, the divergences, the acceptance test, the residual and
the bonus draw alike -- so T = 1 is the rule above. T = 0 is greedy decoding:
p and q become one-hot at their argmax (lowest vocabulary index on ties), a
draft is accepted iff it is argmax p_j (no uniform is used), the extra token is
argmax p_k, a_j, p(x) and q(x) are 1 or 0, TV_j is 0 when the two argmaxes
agree and 1 otherwise, and KL_j is 0 or +infinity likewise.

Top-k / top-p (the remaining logits processors, applied after the
temperature, in that order, to every verifier row p_j and every draft row
q_j alike -- the drafter samples from its filtered distribution and the
verifier judges with its own; the rule above then runs on the filtered
distributions unchanged, so its output is distributed as the filtered p):
  top-k (1 <= k < V; 0 or k >= V is off): keep the entries whose logit is at
    least the k-th largest logit; entries tied with it are all kept.
  top-p (0 < p < 1; 1 is off): with r the softmax of the top-k result, keep
    entry v iff the r-mass of the entries with a strictly larger logit is
    below p. Equal logits are kept or removed together, the largest is always
    kept. For distinct logits this is the usual rule (sort ascending, drop the
    entries whose cumulative mass is at most 1 - p).
A row's top-p margin is the smallest |mass above - p| over its distinct
logits; a sequence with a margin below 1e-5 on any of its rows is marked as
a boundary case (its filtered sets may legitimately differ under fp32 sums).
Greedy decoding (T = 0) is unaffected (the largest logit is always kept).

Data errors (status bits, same meaning as the library's): 1 gamma_b outside
[0, gamma_max]; 2 kv_len_b < gamma_b + 1 (only when kv_len is given);
4 a draft outside [0, V); 8 a needed uniform outside [0, 1). Such a sequence
gets accept_len = -1, tokens -1, NaN float outputs and new_len = kv_len_b.
"""

from __future__ import annotations

import numpy as np

ST_GAMMA = 1
ST_KVLEN = 2
ST_TOKEN = 4
ST_UNIFORM = 8

BOUNDARY = 1e-6
FILTER_BOUNDARY = 1e-5


def decode_logits(x) -> np.ndarray:
    """fp32 logits or bf16 bit patterns (uint16) -> fp64 values."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return (x.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def log_softmax(z) -> np.ndarray:
    """Max-subtracted log-softmax in fp64 (so underflowing probabilities keep a log)."""
    z = np.asarray(z, dtype=np.float64)
    m = np.max(z)
    return z - (m + np.log(np.sum(np.exp(z - m))))


def filter_logits(z, top_k=0, top_p=1.0):
    """Top-k then top-p on one row of (temperature-scaled) logits; removed
    entries become -inf. Returns (filtered logits, top-p margin)."""
    z = np.array(z, dtype=np.float64)
    V = z.shape[0]
    if 0 < top_k < V:
        kth = np.sort(z)[V - top_k]  # the k-th largest value
        z = np.where(z >= kth, z, -np.inf)
    margin = np.inf
    if top_p < 1.0:
        r = np.exp(log_softmax(z))
        vals, group = np.unique(z, return_inverse=True)  # ascending distinct values
        mass = np.bincount(group, weights=r, minlength=vals.shape[0])
        above = np.cumsum(mass[::-1])[::-1] - mass       # mass of the strictly larger values
        keep = above < top_p
        live = np.isfinite(vals)
        if live.any():
            margin = float(np.min(np.abs(above[live] - top_p)))
        z = np.where(keep[group], z, -np.inf)
    return z, margin


def total_variation(p, q) -> float:
    """Eq. 5: half the L1 distance between two distributions."""
    return 0.5 * float(np.sum(np.abs(p - q)))


def kl_divergence(lp, lq) -> float:
    """KL(p || q) in nats from log-probabilities; terms with p = 0 contribute 0."""
    p = np.exp(lp)
    live = p > 0
    diff = lp[live] - lq[live]
    return float(np.sum(p[live] * diff))


def acceptance_probability(lp_x: float, lq_x: float) -> float:
    """min(1, p(x)/q(x)) evaluated from log-probabilities; q(x) = 0 gives 1."""
    if lq_x == -np.inf or lp_x >= lq_x:
        return 1.0
    return float(np.exp(lp_x - lq_x))


def inverse_cdf(w, u: float):
    """Draw from weights w by CDF inversion with uniform u in [0, 1).

    Returns (token, margin): token = smallest x with C(x) > u * W, W = C(V-1);
    margin = distance of u * W to the bracketing CDF values, over W.
    """
    C = np.cumsum(w)
    W = float(C[-1])
    target = u * W
    t = int(np.searchsorted(C, target, side="right"))
    if t >= C.shape[0]:
        t = int(np.flatnonzero(w > 0)[-1])
    lo = float(C[t - 1]) if t > 0 else 0.0
    hi = float(C[t])
    margin = min(abs(target - lo), abs(hi - target)) / W if W > 0 else 0.0
    return t, margin


def accept_sequence_greedy(P, Q, drafts, gamma, gmax, V):
    """One sequence under greedy decoding (temperature 0). Uniforms are not used."""
    res = dict(
        accept_len=-1, tokens=np.full(gmax + 1, -1, dtype=np.int64),
        accept_prob=np.full(gmax, np.nan), p_tok=np.full(gmax, np.nan),
        q_tok=np.full(gmax, np.nan), kl=np.full(gmax, np.nan), tv=np.full(gmax, np.nan),
        lse_p=np.full(gmax + 1, np.nan), lse_q=np.full(gmax, np.nan),
        margin=np.inf, status=0,
    )
    g = int(gamma)
    if not (0 <= g <= gmax):
        res["status"] = ST_GAMMA
        return res
    if any(not (0 <= int(drafts[j]) < V) for j in range(g)):
        res["status"] = ST_TOKEN
        return res
    ap = [int(np.argmax(P[j])) for j in range(g + 1)]  # first occurrence: lowest index on ties
    aq = [int(np.argmax(Q[j])) for j in range(g)]
    k = g
    for j in range(g):
        x = int(drafts[j])
        same = ap[j] == aq[j]
        res["tv"][j] = 0.0 if same else 1.0
        res["kl"][j] = 0.0 if same else np.inf
        res["p_tok"][j] = 1.0 if x == ap[j] else 0.0
        res["q_tok"][j] = 1.0 if x == aq[j] else 0.0
        res["accept_prob"][j] = res["p_tok"][j]
        if k == g and x != ap[j]:
            k = j
    res["accept_len"] = k
    res["tokens"][:k] = np.asarray(drafts[:k], dtype=np.int64)
    res["tokens"][k] = ap[k]
    return res


def accept_sequence(P, Q, drafts, gamma, u_acc, u_res, gmax, V, temperature=1.0, top_k=0, top_p=1.0):
    """One sequence. P [>= gamma+1, V], Q [>= gamma, V] fp64 logits; every
    distribution is softmax(logits / temperature) (temperature > 0), after
    top-k / top-p filtering of each row."""
    if temperature != 1.0:
        P = np.asarray(P, dtype=np.float64) / temperature
        Q = np.asarray(Q, dtype=np.float64) / temperature
    filter_margin = np.inf
    if (0 < top_k < V) or top_p < 1.0:
        P = np.array(P, dtype=np.float64)
        Q = np.array(Q, dtype=np.float64)
        for rows in (P, Q):
            for j in range(rows.shape[0]):
                rows[j], m = filter_logits(rows[j], top_k, top_p)
                filter_margin = min(filter_margin, m)
    res = dict(
        accept_len=-1, tokens=np.full(gmax + 1, -1, dtype=np.int64),
        accept_prob=np.full(gmax, np.nan), p_tok=np.full(gmax, np.nan),
        q_tok=np.full(gmax, np.nan), kl=np.full(gmax, np.nan), tv=np.full(gmax, np.nan),
        lse_p=np.full(gmax + 1, np.nan), lse_q=np.full(gmax, np.nan),
        margin=np.inf, filter_margin=filter_margin, status=0,
    )
    g = int(gamma)
    if not (0 <= g <= gmax):
        res["status"] = ST_GAMMA
        return res
    if any(not (0 <= int(drafts[j]) < V) for j in range(g)):
        res["status"] = ST_TOKEN
        return res
    us = [float(u_acc[j]) for j in range(g)] + [float(u_res[j]) for j in range(g + 1)]
    if any(not (0.0 <= u < 1.0) for u in us):
        res["status"] = ST_UNIFORM
        return res

    lp = [log_softmax(P[j]) for j in range(g + 1)]
    lq = [log_softmax(Q[j]) for j in range(g)]
    a = np.empty(g)
    for j in range(g):
        p, q = np.exp(lp[j]), np.exp(lq[j])
        res["tv"][j] = total_variation(p, q)
        res["kl"][j] = kl_divergence(lp[j], lq[j])
        x = int(drafts[j])
        res["p_tok"][j] = p[x]
        res["q_tok"][j] = q[x]
        a[j] = acceptance_probability(lp[j][x], lq[j][x])
        res["accept_prob"][j] = a[j]
    for j in range(g + 1):
        zmax = float(np.max(P[j]))
        res["lse_p"][j] = zmax + np.log(np.sum(np.exp(np.asarray(P[j], np.float64) - zmax)))
    for j in range(g):
        zmax = float(np.max(Q[j]))
        res["lse_q"][j] = zmax + np.log(np.sum(np.exp(np.asarray(Q[j], np.float64) - zmax)))

    k = g
    for j in range(g):
        if not (u_acc[j] < a[j]):
            k = j
            break
    margin = np.inf
    for j in range(min(k + 1, g)):
        margin = min(margin, abs(float(u_acc[j]) - a[j]))

    if k < g:
        w = np.maximum(0.0, np.exp(lp[k]) - np.exp(lq[k]))
        if not np.any(w > 0):
            w = np.exp(lp[k])
    else:
        w = np.exp(lp[g])
    t, m2 = inverse_cdf(w, float(u_res[k]))
    margin = min(margin, m2)

    res["accept_len"] = k
    res["tokens"][:k] = np.asarray(drafts[:k], dtype=np.int64)
    res["tokens"][k] = t
    res["margin"] = margin
    return res


def accept_and_diverge(p_logits, q_logits, drafts, gamma, u_acc, u_res, kv_len=None, seqs=None, temperature=1.0,
                       top_k=0, top_p=1.0):
    """Reference accept-and-diverge pass over a batch (temperature 0: greedy;
    top_k / top_p: the logits processors, off by default).

    p_logits [B, gmax+1, V] and q_logits [B, gmax, V]: fp32, fp64, or bf16 bit
    patterns (uint16). drafts [B, gmax] int; gamma [B]; u_acc [B, gmax];
    u_res [B, gmax+1] (fp32 values in [0, 1)); kv_len [B] or None.
    seqs: optional subset of sequences to evaluate (others keep their padding).

    Returns a dict of numpy arrays: accept_len [B], out_tokens [B, gmax+1],
    new_len [B] (or None), accept_prob/p_tok/q_tok/kl/tv [B, gmax],
    lse_p [B, gmax+1], lse_q [B, gmax], margin [B], boundary [B] (bool) and
    the OR of the status bits.
    """
    B, gmax1, V = p_logits.shape
    gmax = gmax1 - 1
    out = dict(
        accept_len=np.full(B, -1, dtype=np.int64),
        out_tokens=np.full((B, gmax1), -1, dtype=np.int64),
        new_len=None if kv_len is None else np.asarray(kv_len, dtype=np.int64).copy(),
        accept_prob=np.full((B, gmax), np.nan), p_tok=np.full((B, gmax), np.nan),
        q_tok=np.full((B, gmax), np.nan), kl=np.full((B, gmax), np.nan),
        tv=np.full((B, gmax), np.nan), lse_p=np.full((B, gmax1), np.nan),
        lse_q=np.full((B, gmax), np.nan), margin=np.full(B, np.inf),
        boundary=np.zeros(B, dtype=bool), filter_boundary=np.zeros(B, dtype=bool), status=0,
    )
    for b in (range(B) if seqs is None else seqs):
        g = int(gamma[b])
        if kv_len is not None and 0 <= g <= gmax and int(kv_len[b]) < g + 1:
            out["status"] |= ST_KVLEN
            continue
        gg = max(0, min(g, gmax))
        P = decode_logits(p_logits[b, : gg + 1])
        Q = decode_logits(q_logits[b, :gg])
        if temperature == 0:
            r = accept_sequence_greedy(P, Q, drafts[b], g, gmax, V)
        else:
            r = accept_sequence(P, Q, drafts[b], g, u_acc[b], u_res[b], gmax, V, temperature, top_k, top_p)
        out["status"] |= r["status"]
        if r["status"]:
            continue
        out["accept_len"][b] = r["accept_len"]
        out["out_tokens"][b] = r["tokens"]
        for key in ("accept_prob", "p_tok", "q_tok", "kl", "tv", "lse_q"):
            out[key][b] = r[key]
        out["lse_p"][b] = r["lse_p"]
        out["margin"][b] = r["margin"]
        out["filter_boundary"][b] = r.get("filter_margin", np.inf) < FILTER_BOUNDARY
        out["boundary"][b] = r["margin"] < BOUNDARY or out["filter_boundary"][b]
        if kv_len is not None:
            out["new_len"][b] = int(kv_len[b]) - g + r["accept_len"]
    return out
