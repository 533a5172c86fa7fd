"""Glue of the three-level chain, reference (test infrastructure only).

The paper has intermediate models verify drafts before the target does
(Section 4.3, VerifyProcessor, repeated for each verification level) and then
rolls every model's cache back to a consensus length (RollbackProcessor). It
does not spell out what the next level verifies or the consensus rule; the
reading taken here:

  * the target level verifies the first gamma3_b = min(k2_b + 1, gamma_tgt)
    tokens the intermediate level emitted (its accepted drafts plus its
    correction or bonus token), with the intermediate level's verifier rows
    0 .. gamma3_b - 1 serving as the target level's draft distribution;
  * each level's cache holds ctx context rows plus one row per token it ran
    this step, the first being the previous step's pending token;
  * rollback targets: target level ctx + 1 + k3; intermediate and draft
    levels ctx + 1 + min(k2, k3) (rows past the last token every level agrees
    on are invalid);
  * pending tokens: what a level must run at the start of the next step,
    i.e. the emitted tokens it has not cached (the target's correction or
    bonus token for every level, preceded, for the lower levels, by the
    intermediate level's own correction token when the target accepted it).

Losslessness of this reading: the tokens the intermediate level emits are an
exact sample path of its own distribution p2 (speculative sampling), and
whether position j exists for the target level (k2 >= j) is decided before
token j is drawn, so verifying them with q = p2 yields samples of p3. The
test suite checks this by exact enumeration over three tiny table models.
"""

from __future__ import annotations

import numpy as np

ST_CHAIN = 64  # accept lengths that one chain step cannot produce


def window(accept_len, out_tokens, gamma_cap: int):
    """Next verifier level's window and drafts from the level below:
    gamma_next_b = min(k_b + 1, gamma_cap), and -1 for a sequence the level
    below flagged (k_b < 0) or an accept length its emitted tokens [B, gmax+1]
    cannot hold (k_b > gmax); drafts_next_b = its first gamma_next_b emitted
    tokens, padded with 0 to gamma_cap."""
    k = np.asarray(accept_len, dtype=np.int64)
    B = k.shape[0]
    width = len(out_tokens[0]) if B else 0
    g = np.where((k >= 0) & (k < width), np.minimum(k + 1, gamma_cap), -1).astype(np.int32)
    d = np.zeros((B, gamma_cap), dtype=np.int32)
    for b in range(B):
        n = int(g[b])
        if n > 0:
            d[b, :n] = np.asarray(out_tokens[b][:n])
    return g, d


def consensus(ctx_len, k_lower, k_upper, out_lower, out_upper):
    """Consensus after a two-level verify (reading above): the upper level
    keeps ctx + 1 + k_upper rows, the lower levels ctx + 1 + min(k_lower,
    k_upper); the tokens emitted but not cached by the lower levels are
    pending for the next step: the lower level's own correction token when the
    upper level accepted it (k_upper = k_lower + 1), then the upper level's
    correction or bonus token. A sequence either level flagged (k < 0) keeps
    ctx rows everywhere and gets no pending token; so does one whose lengths
    cannot come from one chain step (k_upper > k_lower + 1, or an accept
    length past its level's window), which also sets status bit ST_CHAIN.
    Returns (len_upper, len_lower, pending [B, 2] padded with -1, n_pending,
    status)."""
    ctx = np.asarray(ctx_len, dtype=np.int64)
    kl = np.asarray(k_lower, dtype=np.int64)
    ku = np.asarray(k_upper, dtype=np.int64)
    B = ctx.shape[0]
    up = np.empty(B, dtype=np.int32)
    lo = np.empty(B, dtype=np.int32)
    pend = np.full((B, 2), -1, dtype=np.int32)
    npend = np.zeros(B, dtype=np.int32)
    status = 0
    wl, wu = (len(out_lower[0]), len(out_upper[0])) if B else (0, 0)
    for b in range(B):
        if kl[b] < 0 or ku[b] < 0:
            up[b] = lo[b] = ctx[b]
            continue
        if ku[b] > kl[b] + 1 or kl[b] >= wl or ku[b] >= wu:
            up[b] = lo[b] = ctx[b]
            status |= ST_CHAIN
            continue
        up[b] = ctx[b] + 1 + ku[b]
        lo[b] = ctx[b] + 1 + min(kl[b], ku[b])
        toks = []
        if ku[b] == kl[b] + 1:
            toks.append(int(out_lower[b][kl[b]]))
        toks.append(int(out_upper[b][ku[b]]))
        pend[b, : len(toks)] = toks
        npend[b] = len(toks)
    return up, lo, pend, npend, status


def target_window(accept_len_int, gamma_tgt: int) -> np.ndarray:
    """gamma3_b = min(k2_b + 1, gamma_tgt)."""
    return np.minimum(np.asarray(accept_len_int, dtype=np.int64) + 1, gamma_tgt).astype(np.int32)


def target_drafts(out_tokens_int, gamma3, gamma_tgt: int) -> np.ndarray:
    """First gamma3_b tokens emitted by the intermediate level, padded with 0."""
    B = out_tokens_int.shape[0]
    d = np.zeros((B, gamma_tgt), dtype=np.int32)
    for b in range(B):
        n = int(gamma3[b])
        d[b, :n] = out_tokens_int[b, :n]
    return d


def rollback_targets(ctx: int, k_int, k_tgt):
    """(target, intermediate, draft) new lengths after the step."""
    k_int = np.asarray(k_int, dtype=np.int64)
    k_tgt = np.asarray(k_tgt, dtype=np.int64)
    tgt = ctx + 1 + k_tgt
    agree = ctx + 1 + np.minimum(k_int, k_tgt)
    return tgt.astype(np.int32), agree.astype(np.int32), agree.astype(np.int32)
