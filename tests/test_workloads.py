"""Input generator checks (CPU only): determinism, bf16 rounding, value
distributions, ragged parameter ranges, and that drafts are samples of q."""

import numpy as np
import pytest

from workloads import CONFIGS, bf16_bits_from_f32, kv_slab, level_inputs, small_shape
from workloads.gen import _gumbel_argmax, f32_from_bf16_bits, ragged_params


def test_bf16_round_to_nearest_even_bit_patterns():
    cases = {
        1.0: 0x3F80,
        -2.0: 0xC000,
        1.0 + 2.0 ** -8: 0x3F80,        # exact tie -> even (down)
        1.0 + 3 * 2.0 ** -8: 0x3F82,    # tie between 0x3F81 and 0x3F82 -> even (up)
        1.0 + 2.0 ** -8 + 2.0 ** -20: 0x3F81,  # just above the tie -> up
        3.140625: 0x4049,
        1e4: 0x461C,
        0.0: 0x0000,
    }
    for x, bits in cases.items():
        assert int(bf16_bits_from_f32(np.array([x], np.float32))[0]) == bits, x
    assert f32_from_bf16_bits(np.array([0x3F80], np.uint16))[0] == 1.0


def test_deterministic_and_slab_regeneration():
    s = small_shape(B=2, Hq=4, Hkv=2, D=64, V=500)
    a = level_inputs(s)
    b = level_inputs(s)
    for name in ("q", "k", "v", "kv_len", "gamma", "p_logits", "q_logits", "drafts", "u_acc", "u_res"):
        x, y = getattr(a, name), getattr(b, name)
        assert np.array_equal(x, y, equal_nan=True) if x.dtype.kind == "f" else np.array_equal(x, y)
    slab = kv_slab(s.seed, 1, 1, "v", int(a.kv_len[1]), s.cap, s.D)
    np.testing.assert_array_equal(slab, a.v[1, 1])


def test_value_distributions():
    s = small_shape(B=2, Hq=8, Hkv=2, D=128, V=20000, gamma=(5, 5), ctx=(1000, 1000), noise=(1.5, 1.5))
    x = level_inputs(s)
    kv = f32_from_bf16_bits(x.k[0, 0, : x.kv_len[0]])
    assert abs(kv.mean()) < 0.02 and abs(kv.std() - 1) < 0.02
    zp = x.p_logits[:, :6].astype(np.float64)
    zq = x.q_logits[:, :5].astype(np.float64)
    assert abs(zp.std() - 3.0) < 0.02
    assert abs((zq - zp[:, :5]).std() - 1.5) < 0.02
    assert x.u_acc.dtype == np.float32 and (x.u_acc >= 0).all() and (x.u_acc < 1).all()
    # padding: cache tail is finite +-1e4, logits padding is NaN
    tail = f32_from_bf16_bits(x.k[0, 0, x.kv_len[0]:])
    assert np.isin(tail, [9984.0, -9984.0]).all()  # bf16(1e4) = 9984


def test_ragged_parameters_in_range():
    s = CONFIGS[5]
    ctx, gam, sig = ragged_params(s)
    assert ctx.min() >= 256 and ctx.max() <= 8192
    assert gam.min() >= 1 and gam.max() <= 8 and len(set(gam.tolist())) == 8
    assert sig.min() >= 0.5 and sig.max() <= 3.0
    assert (ctx + gam + 1).max() <= s.cap


def test_drafts_are_samples_of_q():
    rng = np.random.default_rng(0)
    z = rng.normal(0, 1.0, 6).astype(np.float32)
    p = np.exp(z - z.max())
    p /= p.sum()
    N = 20000
    counts = np.bincount([_gumbel_argmax(5, 5, b, 0, z) for b in range(N)], minlength=6)
    chi2 = (((counts - N * p) ** 2) / (N * p)).sum()
    assert chi2 < 25.0  # 5 dof, p ~ 1e-4


def test_config_shapes():
    c2 = CONFIGS[2]
    assert (c2.B, c2.Hq, c2.Hkv, c2.D, c2.V, c2.gmax) == (16, 32, 8, 128, 128256, 5)
    assert c2.cap >= 2048 + 6
    c4 = CONFIGS[4]
    assert c4.cap >= 32768 + 9
