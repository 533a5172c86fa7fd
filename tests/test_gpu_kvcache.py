"""GPU parity of the KV-cache calls (specrouter_kv_append, specrouter_kv_compact)
against the reference, byte for byte, and the paper's shared-length layout
end to end on the device: append at the shared length, attention over the
holed mask, rollback to each sequence's accepted prefix (Eq. 9's physical
length), compaction, with a paper-shaped model (32 heads MHA, D = 128,
V = 32000)."""

import numpy as np
import pytest
import torch

import oracle
from oracle import kvcache
from workloads import level_inputs, small_shape

from gpu_util import check_accept, check_attention, dev, host, run_accept

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _library():
    import paper_2505_07680_amd as sr

    sr.load()
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def _bits(rng, shape):
    return rng.integers(0, 1 << 15, shape).astype(np.uint16)


def _bf16(rng, shape, sigma=1.0):
    x = rng.normal(0, sigma, shape).astype(np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


@pytest.mark.parametrize("shared", [False, True])
@pytest.mark.parametrize("D", [64, 128])
def test_append_matches_reference(shared, D):
    import paper_2505_07680_amd as sr

    rng = np.random.default_rng(D + shared)
    B, Hkv, L_cap, gmax = 9, 3, 300, 5
    k, v = _bits(rng, (B, Hkv, L_cap, D)), _bits(rng, (B, Hkv, L_cap, D))
    mask = (rng.random((B, L_cap)) < 0.8).astype(np.uint8)
    kv_len = rng.integers(0, 290, B).astype(np.int32)
    gamma = rng.integers(0, gmax + 1, B).astype(np.int32)
    gamma[3] = gmax + 2          # bad gamma
    kv_len[5] = L_cap - 1        # overflows at its own cursor unless gamma is 0
    gamma[5] = 2
    kv_len[6] = L_cap + 5        # a length outside [0, L_cap]: flagged in both layouts
    phys = 250
    kn, vn = _bits(rng, (B, gmax + 1, Hkv, D)), _bits(rng, (B, gmax + 1, Hkv, D))
    kd, vd, md, ld = dev(k), dev(v), dev(mask), dev(kv_len)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    sl = torch.tensor([phys], dtype=torch.int32, device="cuda") if shared else None
    say(f"kv append D={D} shared={shared}")
    sr.specrouter_kv_append(dev(kn), dev(vn), dev(gamma), kd, vd, md, ld, shared_len=sl, status=st)
    rk, rv, rm, rl, rst = kvcache.append(k, v, mask, kv_len, kn, vn, gamma, phys_len=phys if shared else None)
    assert int(host(st)[0]) == rst and rst & kvcache.ST_GAMMA and rst & kvcache.ST_KVLEN
    np.testing.assert_array_equal(host(ld), rl)
    np.testing.assert_array_equal(host(md), rm)
    np.testing.assert_array_equal(host(kd).view(np.uint16), rk)
    np.testing.assert_array_equal(host(vd).view(np.uint16), rv)


@pytest.mark.parametrize("D", [64, 128])
def test_compact_matches_reference(D):
    import paper_2505_07680_amd as sr

    rng = np.random.default_rng(20 + D)
    B, Hkv, L_cap = 7, 4, 1000
    k, v = _bits(rng, (B, Hkv, L_cap, D)), _bits(rng, (B, Hkv, L_cap, D))
    kv_len = np.array([0, 1, 64, 200, 999, 1000, 517], np.int32)
    mask = np.zeros((B, L_cap), np.uint8)
    for b, frac in enumerate([0.5, 1.0, 1.0, 0.3, 0.9, 0.99, 0.0]):
        mask[b] = rng.random(L_cap) < frac
    mask[3, :100] = 1  # a long valid prefix stays in place
    kd, vd, md, ld = dev(k), dev(v), dev(mask), dev(kv_len)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    say(f"kv compact D={D}")
    sr.specrouter_kv_compact(kd, vd, md, ld, st)
    rk, rv, rm, rl, rst = kvcache.compact(k, v, mask, kv_len)
    assert int(host(st)[0]) == rst == 0
    np.testing.assert_array_equal(host(ld), rl)
    np.testing.assert_array_equal(host(md), rm)
    np.testing.assert_array_equal(host(kd).view(np.uint16), rk)
    np.testing.assert_array_equal(host(vd).view(np.uint16), rv)


def test_paper_layout_cycle_on_device():
    """Shared physical length, paper-shaped attention (MHA, 32 heads)."""
    import paper_2505_07680_amd as sr

    rng = np.random.default_rng(7)
    B, H, D, L_cap, g = 4, 32, 128, 700, 5
    L = 480
    k = _bf16(rng, (B, H, L_cap, D))
    v = _bf16(rng, (B, H, L_cap, D))
    mask = np.zeros((B, L_cap), np.uint8)
    mask[:, :L] = 1
    kd, vd, md = dev(k), dev(v), dev(mask)
    kvl = dev(np.full(B, L, np.int32))
    shared = torch.tensor([L], dtype=torch.int32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    gamma = np.full(B, g, np.int32)
    gd = dev(gamma)
    scale = 1.0 / np.sqrt(D)
    for step in range(4):
        kn, vn = _bf16(rng, (B, g + 1, H, D)), _bf16(rng, (B, g + 1, H, D))
        sr.specrouter_kv_append(dev(kn), dev(vn), gd, kd, vd, md, kvl, shared_len=shared, status=st)
        q = _bf16(rng, (B, g + 1, H, D))
        out = torch.empty((B, g + 1, H, D), dtype=torch.float32, device="cuda")
        sr.specrouter_verify_attention(dev(q), kd, vd, md, kvl, gd, out, scale,
                                       sr.attention_workspace(B, g, H, H, D, L_cap), st)
        torch.cuda.synchronize()
        kl_h, m_h = host(kvl), host(md)
        ref, _ = oracle.verify_attention(q, host(kd).view(np.uint16), host(vd).view(np.uint16), kl_h, gamma, scale,
                                         m_h)
        check_attention(host(out), ref)
        # each sequence keeps a different accepted prefix: holes below the shared length
        keep = rng.integers(1, g + 2, B).astype(np.int32)
        new_len = (kl_h - (g + 1) + keep).astype(np.int32)
        phys = torch.zeros(1, dtype=torch.int32, device="cuda")
        sr.specrouter_rollback(kvl, md, dev(new_len), phys, st)
        torch.cuda.synchronize()
        assert int(host(phys)[0]) == int(new_len.max())  # Eq. 9: L - r_min
        shared.copy_(phys)
        kvl.fill_(int(new_len.max()))  # the paper's layout: one physical length
        say(f"paper layout step {step}: physical length {int(new_len.max())}, holes "
            f"{int((host(md)[:, : int(new_len.max())] == 0).sum())}")
    assert int(host(st)[0]) == 0
    # compaction keeps attention unchanged
    q = _bf16(rng, (B, 1, H, D))
    g0 = torch.zeros(B, dtype=torch.int32, device="cuda")
    out_h = torch.empty((B, 1, H, D), dtype=torch.float32, device="cuda")
    sr.specrouter_verify_attention(dev(q), kd, vd, md, kvl, g0, out_h, scale,
                                   sr.attention_workspace(B, 0, H, H, D, L_cap), st)
    torch.cuda.synchronize()
    holed = (host(kd).view(np.uint16), host(vd).view(np.uint16), host(md), host(kvl))
    sr.specrouter_kv_compact(kd, vd, md, kvl, st)
    out_c = torch.empty_like(out_h)
    sr.specrouter_verify_attention(dev(q), kd, vd, md, kvl, g0, out_c, scale,
                                   sr.attention_workspace(B, 0, H, H, D, L_cap), st)
    torch.cuda.synchronize()
    assert int(host(st)[0]) == 0
    zero = np.zeros(B, np.int32)
    ref_h, _ = oracle.verify_attention(q, holed[0], holed[1], holed[3], zero, scale, holed[2])
    ref_c, _ = oracle.verify_attention(q, host(kd).view(np.uint16), host(vd).view(np.uint16), host(kvl), zero, scale,
                                       host(md))
    np.testing.assert_allclose(ref_c, ref_h, rtol=1e-12, atol=1e-12)  # Eq. 8: the holes are invisible
    check_attention(host(out_h), ref_h)
    check_attention(host(out_c), ref_c)
    assert (host(md)[:, : int(host(kvl).min())] == 1).all()


@pytest.mark.parametrize("logits", ["f32", "bf16"])
def test_paper_vocabulary_accept(logits):
    shape = small_shape(name=f"v32000-{logits}", B=6, V=32000, gamma=(3, 5), seed=31, logits=logits)
    inp = level_inputs(shape, kv=False)
    got = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res)
    ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res)
    assert got["status"] == ref["status"] == 0
    check_accept(got, ref)
