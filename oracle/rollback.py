"""Per-sequence KV rollback, reference (test infrastructure only).

Follows Section 4.4 (rollback mechanism, Eq. 9): a sequence that must drop its
last r_b cache entries has those entries' logical validity bits cleared
("logical rollback", no data movement), and the common physical length can
shrink by r_min = min_b r_b.

Reading: the call takes the absolute new logical length L'_b (new_len) rather
than r_b, which makes it idempotent. Per sequence:

    n = min(kv_len_b, new_len_b);  mask[b, n : kv_len_b) = 0;  kv_len_b = n.

phys_len = max_b kv_len_b after the update; when every sequence started at
the same physical length L this equals L - r_min (Eq. 9). K/V data and the
token ids are never touched.

Status bits: 2 = kv_len_b outside [0, cap] or new_len_b < 0 (sequence left
unchanged); 16 = new_len_b > kv_len_b (a grow request, treated as a no-op).
"""

from __future__ import annotations

import numpy as np

ST_KVLEN = 2
ST_ROLLBACK_GROW = 16


def rollback(kv_len, mask, new_len, cap=None):
    """Returns (kv_len' int64 [B], mask' (copy) or None, phys_len, status)."""
    kv = np.asarray(kv_len, dtype=np.int64).copy()
    nl = np.asarray(new_len, dtype=np.int64)
    m = None if mask is None else np.asarray(mask).copy()
    if cap is None:
        cap = m.shape[1] if m is not None else np.iinfo(np.int64).max
    status = 0
    for b in range(kv.shape[0]):
        old = int(kv[b])
        want = int(nl[b])
        if not (0 <= old <= cap) or want < 0:
            status |= ST_KVLEN
            continue
        if want > old:
            status |= ST_ROLLBACK_GROW
        n = min(old, want)
        if m is not None:
            m[b, n:old] = 0
        kv[b] = n
    phys = int(kv.max()) if kv.shape[0] else 0
    return kv, m, phys, status
