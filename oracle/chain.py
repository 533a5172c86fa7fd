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
    on are invalid).
"""

from __future__ import annotations

import numpy as np


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
