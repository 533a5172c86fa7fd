"""Pins for the verification-attention reference (CPU only).

Fixed independently of the reference's own code by:
  * a scalar brute force written here with the math module (tiny shapes);
  * torch's scaled_dot_product_attention on the CPU in fp64 with an explicit
    boolean mask (an independent library routine);
  * special cases with closed forms: one visible key returns that key's V
    row; Q = 0 returns the mean of the visible V rows;
  * the masking rule of Section 4.4: data under mask = 0 or beyond kv_len
    never changes the output (Eq. 8).
"""

import math

import numpy as np
import pytest
import torch

from oracle.attention import decode_bf16, verify_attention
from workloads import bf16_bits_from_f32


def _rand_bits(rng, shape, scale=1.0):
    return bf16_bits_from_f32((rng.standard_normal(shape) * scale).astype(np.float32))


def _case(seed, B=2, Hq=4, Hkv=2, D=8, cap=12, gmax=3, masked=True):
    rng = np.random.default_rng(seed)
    q = _rand_bits(rng, (B, gmax + 1, Hq, D))
    k = _rand_bits(rng, (B, Hkv, cap, D))
    v = _rand_bits(rng, (B, Hkv, cap, D))
    gamma = rng.integers(0, gmax + 1, B)
    kv_len = np.array([rng.integers(g + 1, cap + 1) for g in gamma])
    mask = (rng.random((B, cap)) < 0.8).astype(np.uint8) if masked else None
    return q, k, v, kv_len, gamma, mask


def _brute(q, k, v, kv_len, gamma, mask, scale):
    """Scalar triple loop, fsum accumulation, no numpy arithmetic."""
    B, G1, Hq, D = q.shape
    Hkv = k.shape[1]
    qf, kf, vf = decode_bf16(q), decode_bf16(k), decode_bf16(v)
    out = np.zeros(q.shape)
    for b in range(B):
        L, g = int(kv_len[b]), int(gamma[b])
        for i in range(g + 1):
            pos = L - (g + 1) + i
            for h in range(Hq):
                kh = h // (Hq // Hkv)
                keys = [j for j in range(pos + 1) if mask is None or mask[b, j]]
                if not keys:
                    continue
                s = [scale * math.fsum(float(qf[b, i, h, c]) * float(kf[b, kh, j, c]) for c in range(D)) for j in keys]
                m = max(s)
                e = [math.exp(x - m) for x in s]
                z = math.fsum(e)
                for c in range(D):
                    out[b, i, h, c] = math.fsum(e[t] * float(vf[b, kh, j, c]) for t, j in enumerate(keys)) / z
    return out


@pytest.mark.parametrize("seed", range(6))
def test_matches_scalar_brute_force(seed):
    q, k, v, kv_len, gamma, mask = _case(seed, masked=seed % 2 == 0)
    scale = 1 / math.sqrt(q.shape[-1])
    got, st = verify_attention(q, k, v, kv_len, gamma, scale, mask)
    assert st == 0
    want = _brute(q, k, v, kv_len, gamma, mask, scale)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed,G", [(0, 1), (1, 4), (2, 8)])
def test_matches_torch_sdpa(seed, G):
    rng = np.random.default_rng(seed)
    B, Hkv, D, cap, gmax = 3, 2, 64, 300, 6
    Hq = G * Hkv
    q = _rand_bits(rng, (B, gmax + 1, Hq, D))
    k = _rand_bits(rng, (B, Hkv, cap, D))
    v = _rand_bits(rng, (B, Hkv, cap, D))
    gamma = np.array([0, 3, 6])
    kv_len = np.array([1, 150, 300])
    mask = (rng.random((B, cap)) < 0.9).astype(np.uint8)
    scale = 0.11
    got, _ = verify_attention(q, k, v, kv_len, gamma, scale, mask)
    for b in range(B):
        L, g = int(kv_len[b]), int(gamma[b])
        Q = torch.from_numpy(decode_bf16(q[b, : g + 1])).permute(1, 0, 2)  # [Hq, n, D]
        K = torch.from_numpy(decode_bf16(k[b, :, :L])).repeat_interleave(G, dim=0)
        Vv = torch.from_numpy(decode_bf16(v[b, :, :L])).repeat_interleave(G, dim=0)
        pos = L - (g + 1) + torch.arange(g + 1)
        allowed = (torch.arange(L)[None, :] <= pos[:, None]) & torch.from_numpy(mask[b, :L].astype(bool))[None, :]
        empty = ~allowed.any(dim=1)
        allowed[empty, 0] = True  # keep SDPA finite; such rows must come out zero
        ref = torch.nn.functional.scaled_dot_product_attention(Q, K, Vv, attn_mask=allowed, scale=scale)
        ref = ref.permute(1, 0, 2).numpy()
        live = ~empty.numpy()
        np.testing.assert_allclose(got[b, : g + 1][live], ref[live], rtol=1e-10, atol=1e-12)
        assert (got[b, : g + 1][~live] == 0).all()
        assert (got[b, g + 1:] == 0).all()


def test_single_visible_key_returns_its_value_row():
    rng = np.random.default_rng(3)
    q, k, v, _, _, _ = _case(3, B=1, Hq=2, Hkv=1, D=16, cap=10, gmax=0, masked=False)
    mask = np.zeros((1, 10), np.uint8)
    mask[0, 4] = 1
    got, _ = verify_attention(q, k, v, np.array([8]), np.array([0]), 0.7, mask)
    for h in range(2):
        np.testing.assert_array_equal(got[0, 0, h], decode_bf16(v[0, 0, 4]))


def test_zero_query_gives_mean_of_visible_values():
    rng = np.random.default_rng(4)
    _, k, v, _, _, _ = _case(4, B=1, Hq=2, Hkv=1, D=16, cap=20, gmax=2, masked=False)
    q = np.zeros((1, 3, 2, 16), np.uint16)  # bf16 +0.0
    mask = (rng.random((1, 20)) < 0.6).astype(np.uint8)
    L, g = 15, 2
    got, _ = verify_attention(q, k, v, np.array([L]), np.array([g]), 1.0, mask)
    for i in range(g + 1):
        pos = L - (g + 1) + i
        keys = [j for j in range(pos + 1) if mask[0, j]]
        want = decode_bf16(v[0, 0, keys]).mean(axis=0)
        np.testing.assert_allclose(got[0, i, 0], want, rtol=1e-13, atol=1e-14)


def test_data_under_mask_and_beyond_length_is_ignored():
    q, k, v, kv_len, gamma, mask = _case(5, B=2, cap=16)
    base, _ = verify_attention(q, k, v, kv_len, gamma, 0.3, mask)
    k2, v2 = k.copy(), v.copy()
    for b in range(2):
        dead = np.flatnonzero(mask[b] == 0).tolist() + list(range(int(kv_len[b]), 16))
        k2[b, :, dead] = 0x7FC0  # NaN
        v2[b, :, dead] = 0x7F80  # +inf
    got, _ = verify_attention(q, k2, v2, kv_len, gamma, 0.3, mask)
    np.testing.assert_array_equal(got, base)


def test_fully_masked_row_is_zero_and_padding_rows_are_zero():
    q, k, v, _, _, _ = _case(6, B=1, cap=8, gmax=3, masked=False)
    mask = np.zeros((1, 8), np.uint8)
    got, st = verify_attention(q, k, v, np.array([8]), np.array([1]), 1.0, mask)
    assert st == 0 and (got == 0).all()


def test_invalid_lengths_set_status_and_zero_output():
    q, k, v, kv_len, gamma, mask = _case(7, B=2, cap=12, gmax=3)
    got, st = verify_attention(q, k, v, np.array([3, 13]), np.array([4, 0]), 1.0, mask)
    assert st == 1 | 2 and (got == 0).all()


def test_sharp_softmax_is_stable():
    """Scores in the thousands: the result must stay finite and match the
    max-subtracted brute force (a softmax without the shift overflows)."""
    q, k, v, kv_len, gamma, mask = _case(8, masked=False)
    scale = 500.0
    got, _ = verify_attention(q, k, v, kv_len, gamma, scale, mask)
    assert np.isfinite(got).all()
    np.testing.assert_allclose(got, _brute(q, k, v, kv_len, gamma, mask, scale), rtol=1e-10, atol=1e-12)
