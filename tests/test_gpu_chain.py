"""GPU parity of the chain glue (specrouter_chain_window and
specrouter_chain_consensus) against the reference, and a whole three-level
chain step on the device: intermediate verify, window, target verify with the
intermediate rows as its draft distribution, consensus, and one rollback per
level -- every step through the C ABI, no host round trip in between."""

import numpy as np
import pytest
import torch

import oracle
from oracle import chain
from workloads import CONFIGS

from gpu_util import check_accept, check_attention, dev, host, run_rollback

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


def _i32(shape):
    return torch.full(shape if isinstance(shape, tuple) else (shape,), -7, dtype=torch.int32, device="cuda")


def test_window_and_consensus_match_reference():
    import paper_2505_07680_amd as sr

    rng = np.random.default_rng(3)
    B, gl, gu = 700, 8, 4
    k_lo = rng.integers(-1, gl + 1, B).astype(np.int32)
    out_lo = rng.integers(0, 128256, (B, gl + 1)).astype(np.int32)
    ctx = rng.integers(0, 4000, B).astype(np.int32)
    say("chain window")
    g, d, kvn = _i32(B), _i32((B, gu)), _i32(B)
    sr.specrouter_chain_window(dev(k_lo), dev(out_lo), gu, g, d, ctx_len=dev(ctx), kv_len_next=kvn)
    rg, rd = chain.window(k_lo, out_lo, gu)
    np.testing.assert_array_equal(host(g), rg)
    np.testing.assert_array_equal(host(d), rd)
    np.testing.assert_array_equal(host(kvn), ctx + 1 + np.maximum(rg, 0))
    # upper level: any accept length up to its window, plus a few impossible ones
    k_up = np.array([rng.integers(-1, max(int(x), 0) + 1) if x >= 0 else rng.integers(-1, 2) for x in rg], np.int32)
    k_up[::97] = gu  # often more than k_lower + 1
    out_up = rng.integers(0, 128256, (B, gu + 1)).astype(np.int32)
    say("chain consensus")
    up, lo, pend, npend = _i32(B), _i32(B), _i32((B, 2)), _i32(B)
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    sr.specrouter_chain_consensus(dev(ctx), dev(k_lo), dev(out_lo), dev(k_up), dev(out_up), up, lo, pend, npend, st)
    r_up, r_lo, r_pend, r_n, r_st = chain.consensus(ctx, k_lo, k_up, out_lo, out_up)
    np.testing.assert_array_equal(host(up), r_up)
    np.testing.assert_array_equal(host(lo), r_lo)
    np.testing.assert_array_equal(host(pend), r_pend)
    np.testing.assert_array_equal(host(npend), r_n)
    assert int(host(st)[0]) == r_st == chain.ST_CHAIN


def test_config3_chain_step_on_device():
    import paper_2505_07680_amd as sr
    from workloads import chain_inputs

    shape = CONFIGS[3]
    say("config3: generating chain inputs")
    ci = chain_inputs(shape)
    B, ctx, gi, gt = shape.B, shape.ctx, shape.gamma_int, shape.gamma_tgt
    inter, t = ci["inter"], ci["target"]
    z1, z2, z3 = ci["z"]
    V = inter.p_logits.shape[2]
    seqs = list(range(0, B, 4))

    # ---- intermediate level: attention + accept, all on the device
    Hq_i, D_i = inter.q.shape[2], inter.q.shape[3]
    Hkv_i, cap = inter.k.shape[1], inter.k.shape[2]
    q_i, k_i, v_i = dev(inter.q), dev(inter.k), dev(inter.v)
    kv_i, g_i = dev(inter.kv_len), dev(inter.gamma)
    out_i = torch.empty((B, gi + 1, Hq_i, D_i), dtype=torch.float32, device="cuda")
    st = torch.zeros(1, dtype=torch.int32, device="cuda")
    sr.specrouter_verify_attention(q_i, k_i, v_i, None, kv_i, g_i, out_i, inter.scale,
                                   sr.attention_workspace(B, gi, Hq_i, Hkv_i, D_i, cap), st)
    p2 = dev(z2)
    ab_i = sr.AcceptBuffers(B, gi, V, sr.SR_F32)
    sr.specrouter_accept_and_diverge(p2, dev(z1), dev(inter.drafts), g_i, dev(inter.u_acc), dev(inter.u_res), kv_i,
                                     ab_i.accept_len, ab_i.out_tokens, ab_i.new_len, ab_i.accept_prob, ab_i.p_tok,
                                     ab_i.q_tok, ab_i.kl, ab_i.tv, ab_i.workspace, st)
    # ---- window of the target level, on the device
    g3, d3 = _i32(B), _i32((B, gt))
    ctx_t = torch.full((B,), ctx, dtype=torch.int32, device="cuda")
    kv3 = _i32(B)
    sr.specrouter_chain_window(ab_i.accept_len, ab_i.out_tokens, gt, g3, d3, ctx_len=ctx_t, kv_len_next=kv3)
    # ---- target level: attention over its window, accept with q = the intermediate rows
    Hq_t, D_t = t["q"].shape[2], t["q"].shape[3]
    Hkv_t = t["k"].shape[1]
    out_t = torch.empty((B, gt + 1, Hq_t, D_t), dtype=torch.float32, device="cuda")
    kv3_w = kv3.clone()
    sr.specrouter_verify_attention(dev(t["q"]), dev(t["k"]), dev(t["v"]), None, kv3_w, g3, out_t, t["scale"],
                                   sr.attention_workspace(B, gt, Hq_t, Hkv_t, D_t, cap), st)
    ab_t = sr.AcceptBuffers(B, gt, V, sr.SR_F32)
    sr.specrouter_accept_and_diverge(dev(t["p_logits"]), p2[:, :gt], d3, g3, dev(t["u_acc"]), dev(t["u_res"]), kv3,
                                     ab_t.accept_len, ab_t.out_tokens, ab_t.new_len, ab_t.accept_prob, ab_t.p_tok,
                                     ab_t.q_tok, ab_t.kl, ab_t.tv, ab_t.workspace, st)
    # ---- consensus and the rollbacks
    up, lo, pend, npend = _i32(B), _i32(B), _i32((B, 2)), _i32(B)
    sr.specrouter_chain_consensus(ctx_t, ab_i.accept_len, ab_i.out_tokens, ab_t.accept_len, ab_t.out_tokens,
                                  up, lo, pend, npend, st)
    sr.specrouter_rollback(kv3_w, None, up, None, st, L_cap=cap)
    kv_i_w = kv_i.clone()
    sr.specrouter_rollback(kv_i_w, None, lo, None, st, L_cap=cap)
    torch.cuda.synchronize()
    assert int(host(st)[0]) == 0
    say(f"config3 device chain: mean k2 {host(ab_i.accept_len).mean():.2f}, mean k3 {host(ab_t.accept_len).mean():.2f}")

    # ---- the reference, step by step on the device's own intermediate outcome
    k2, e2 = host(ab_i.accept_len), host(ab_i.out_tokens)
    rg3, rd3 = chain.window(k2, e2, gt)
    np.testing.assert_array_equal(host(g3), rg3)
    np.testing.assert_array_equal(host(d3), rd3)
    np.testing.assert_array_equal(host(kv3), ctx + 1 + rg3)
    ref_att, _ = oracle.verify_attention(t["q"], t["k"], t["v"], ctx + 1 + rg3, rg3, t["scale"], seqs=seqs)
    check_attention(host(out_t), ref_att, seqs=seqs)
    aref = oracle.accept_and_diverge(t["p_logits"], z2[:, :gt], rd3, rg3, t["u_acc"], t["u_res"],
                                     kv_len=ctx + 1 + rg3, seqs=seqs)
    got_t = {k: host(getattr(ab_t, k)) for k in ("accept_len", "out_tokens", "new_len", "accept_prob", "p_tok",
                                                 "q_tok", "kl", "tv")}
    check_accept(got_t, aref, seqs=seqs)
    k3, e3 = host(ab_t.accept_len), host(ab_t.out_tokens)
    r_up, r_lo, r_pend, r_n, r_st = chain.consensus(np.full(B, ctx), k2, k3, e2, e3)
    assert r_st == 0
    np.testing.assert_array_equal(host(up), r_up)
    np.testing.assert_array_equal(host(lo), r_lo)
    np.testing.assert_array_equal(host(pend), r_pend)
    np.testing.assert_array_equal(host(npend), r_n)
    np.testing.assert_array_equal(host(kv3_w), np.minimum(ctx + 1 + rg3, r_up))
    np.testing.assert_array_equal(host(kv_i_w), np.minimum(inter.kv_len, r_lo))
    # the target's own new length agrees with the consensus
    np.testing.assert_array_equal(host(ab_t.new_len), r_up)
