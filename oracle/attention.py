"""Verification attention, fp64 reference (test infrastructure only).

Follows the paper's verify pass: the verifier runs one forward pass over the
context plus the gamma drafted tokens (Section 2.2, basic speculative decoding,
step 2), and attention ignores every cache entry whose logical validity bit is
0 even if data is stored there (Section 4.4, the logical validity mask and
Eq. 8).

Reading used where the paper is silent (GenerateAttentionMask in Eq. 8 is not
spelled out): key j is visible to query row i of sequence b iff j <= pos_i and
mask[b, j] = 1, where pos_i = kv_len_b - (gamma_b + 1) + i is the row's own
position (causal among the new rows). Query head h reads kv-head h // (Hq/Hkv)
(grouped-query attention). Scores are scale * q.k; an empty key set gives a
zero output row, and rows i > gamma_b are zero.

Status bits (same meaning as the library's): 1 = gamma_b outside
[0, gamma_max]; 2 = kv_len_b outside [gamma_b + 1, cap]. Such a sequence's
output is all zero.
"""

from __future__ import annotations

import numpy as np

ST_GAMMA = 1
ST_KVLEN = 2


def decode_bf16(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> the exact values they encode, as fp64."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def _as_f64(x) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return decode_bf16(x)
    return x.astype(np.float64)


def attend_rows(q_rows, k_rows, v_rows, visible, scale):
    """softmax(scale * q k^T over visible keys) v for a block of query rows.

    q_rows [R, D]; k_rows, v_rows [L, D]; visible [R, L] bool.
    """
    q_rows = np.asarray(q_rows, dtype=np.float64)
    out = np.zeros((q_rows.shape[0], v_rows.shape[1]), dtype=np.float64)
    s = scale * (q_rows @ k_rows.T)
    for r in range(q_rows.shape[0]):
        vis = visible[r]
        if not vis.any():
            continue
        sr = s[r, vis]
        w = np.exp(sr - sr.max())
        w /= w.sum()
        out[r] = w @ v_rows[vis]
    return out


def sequence_status(kv_len_b: int, gamma_b: int, gmax: int, cap: int) -> int:
    if not (0 <= gamma_b <= gmax):
        return ST_GAMMA
    if not (gamma_b + 1 <= kv_len_b <= cap):
        return ST_KVLEN
    return 0


def attend_sequence(q_b, k_b, v_b, kv_len_b, gamma_b, scale, mask_b=None):
    """One sequence: q_b [gmax+1, Hq, D]; k_b, v_b [Hkv, cap, D] -> [gmax+1, Hq, D]."""
    gmax1, Hq, D = q_b.shape
    Hkv, cap, _ = k_b.shape
    G = Hq // Hkv
    out = np.zeros((gmax1, Hq, D), dtype=np.float64)
    if sequence_status(kv_len_b, gamma_b, gmax1 - 1, cap):
        return out
    L = int(kv_len_b)
    n_new = int(gamma_b) + 1
    keys = np.arange(L)
    valid = np.ones(L, dtype=bool) if mask_b is None else (np.asarray(mask_b[:L]) != 0)
    pos = L - n_new + np.arange(n_new)
    vis_i = (keys[None, :] <= pos[:, None]) & valid[None, :]  # [n_new, L]
    for g in range(Hkv):
        K = _as_f64(k_b[g, :L])
        Vv = _as_f64(v_b[g, :L])
        heads = slice(g * G, (g + 1) * G)
        Q = _as_f64(q_b[:n_new, heads]).reshape(n_new * G, D)
        vis = np.repeat(vis_i, G, axis=0)
        out[:n_new, heads] = attend_rows(Q, K, Vv, vis, scale).reshape(n_new, G, D)
    return out


def verify_attention(q, k_cache, v_cache, kv_len, gamma, scale, mask=None, seqs=None):
    """Reference verification attention.

    q        [B, gmax+1, Hq, D]  bf16 bits (uint16) or float
    k_cache  [B, Hkv, cap, D]    bf16 bits or float
    v_cache  [B, Hkv, cap, D]
    kv_len   [B] int; gamma [B] int; mask [B, cap] (0/1) or None
    seqs     optional iterable of sequence indices to compute (others stay 0)

    Returns (out [B, gmax+1, Hq, D] fp64, status bits).
    """
    q = np.asarray(q)
    B, gmax1, Hq, D = q.shape
    cap = k_cache.shape[2]
    out = np.zeros((B, gmax1, Hq, D), dtype=np.float64)
    status = 0
    for b in (range(B) if seqs is None else seqs):
        st = sequence_status(int(kv_len[b]), int(gamma[b]), gmax1 - 1, cap)
        status |= st
        if st:
            continue
        out[b] = attend_sequence(
            q[b], k_cache[b], v_cache[b], int(kv_len[b]), int(gamma[b]), scale,
            None if mask is None else mask[b],
        )
    return out, status
