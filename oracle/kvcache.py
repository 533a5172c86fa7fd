"""KV-cache state reference (Section 4.4, StateManager) -- TEST INFRASTRUCTURE ONLY.

Plain numpy on the cache layout of the verify step: K and V [B][Hkv][L_cap][D]
(bf16 bit patterns, moved verbatim), validity mask [B][L_cap] in {0, 1},
per-sequence lengths kv_len [B].

  * append  -- a step's new K/V rows (gamma_b + 1 per sequence, the pending
               token and the drafts, laid out [B][gamma_max+1][Hkv][D]) are
               written at the sequence's write cursor and marked valid. The
               cursor is the sequence's own length, or, in the paper's layout,
               one physical length L shared by the batch: then a sequence
               that rolled back further than the others keeps the masked
               holes between its last valid row and L (Eq. 8's mask decides
               what attention sees).
  * compact -- optional: every sequence's valid rows moved to the front in
               order, the mask set to exactly those rows and kv_len to their
               count (the holes reclaimed, which Eq. 9 only does for the
               common tail).
  * physical_truncation -- Eq. 9: with a shared length L and rollbacks r_b,
               the common tail r_min = min_b r_b can be cut.

Data errors: a sequence whose cursor + gamma_b + 1 exceeds L_cap, whose gamma
is outside [0, gamma_max] or whose kv_len is outside [0, L_cap] is left
untouched and reported with status bits 2 (lengths) or 1 (gamma).
"""

from __future__ import annotations

import numpy as np

ST_GAMMA = 1
ST_KVLEN = 2


def append(k_cache, v_cache, mask, kv_len, k_new, v_new, gamma, phys_len=None):
    """Returns (k_cache, v_cache, mask, kv_len, status) as new arrays."""
    k = np.array(k_cache, copy=True)
    v = np.array(v_cache, copy=True)
    m = None if mask is None else np.array(mask, copy=True)
    kl = np.array(kv_len, dtype=np.int64, copy=True)
    B, Hkv, L_cap, D = k.shape
    gmax = k_new.shape[1] - 1
    status = 0
    for b in range(B):
        g = int(gamma[b])
        if not (0 <= g <= gmax):
            status |= ST_GAMMA
            continue
        if not (0 <= kl[b] <= L_cap):
            status |= ST_KVLEN
            continue
        cur = int(kl[b]) if phys_len is None else int(phys_len)
        if cur < 0 or cur + g + 1 > L_cap:
            status |= ST_KVLEN
            continue
        for i in range(g + 1):
            for h in range(Hkv):
                k[b, h, cur + i] = k_new[b, i, h]
                v[b, h, cur + i] = v_new[b, i, h]
            if m is not None:
                m[b, cur + i] = 1
        kl[b] = cur + g + 1
    return k, v, m, kl.astype(np.int32), status


def compact(k_cache, v_cache, mask, kv_len):
    """Valid rows of [0, kv_len_b) moved to the front in order. Returns
    (k_cache, v_cache, mask, kv_len, status); rows past the new length keep
    whatever they held (they are masked)."""
    k = np.array(k_cache, copy=True)
    v = np.array(v_cache, copy=True)
    m = np.array(mask, copy=True)
    kl = np.array(kv_len, dtype=np.int64, copy=True)
    B, Hkv, L_cap, D = k.shape
    status = 0
    for b in range(B):
        L = int(kl[b])
        if not (0 <= L <= L_cap):
            status |= ST_KVLEN
            continue
        keep = [j for j in range(L) if m[b, j] != 0]
        n = len(keep)
        k[b][:, :n] = np.asarray(k_cache[b])[:, keep]
        v[b][:, :n] = np.asarray(v_cache[b])[:, keep]
        m[b, :n] = 1
        m[b, n:L] = 0
        kl[b] = n
    return k, v, m, kl.astype(np.int32), status


def physical_truncation(L: int, rollback):
    """Eq. 9: the common tail r_min = min_b r_b of a shared length L can be
    cut; returns (new physical length L - r_min, r_min)."""
    r_min = int(min(rollback)) if len(rollback) else 0
    r_min = max(r_min, 0)
    return L - r_min, r_min
