"""GPU parity of specrouter_accept_and_rollback: one call must give, bit for bit,
what specrouter_accept_and_diverge_sampled followed by specrouter_rollback
gives (the accept outputs, the rolled-back lengths and mask, the physical
length and the status bits), and the rollback part must match the
reference's rollback of the accept's new lengths (Section 4.4, Eq. 9)."""

import numpy as np
import pytest
import torch

import paper_2505_07680_amd as sr
import oracle
from workloads import level_inputs, small_shape

from gpu_util import dev, host

pytestmark = pytest.mark.gpu

OUTS = ("accept_len", "out_tokens", "new_len", "accept_prob", "p_tok", "q_tok", "kl", "tv")


@pytest.fixture(scope="module", autouse=True)
def _library():
    sr.load()
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()


def say(msg):
    print(f"[gpu-test] {msg}", flush=True)


def _cache_state(inp, cap, rng, holes=0.2):
    B = inp.gamma.shape[0]
    kv = np.asarray(inp.kv_len, np.int32).copy()
    mask = np.zeros((B, cap), np.uint8)
    for b in range(B):
        mask[b, : max(int(kv[b]), 0)] = rng.random(max(int(kv[b]), 0)) >= holes
    return kv, mask


def _both(inp, cache_kv, mask, cap, temperature, calls=1, top_k=0, top_p=1.0):
    """Runs the separate pair and the fused call `calls` times on the same
    inputs (fresh cache state each time, shared workspaces) and returns the
    results of the last call of each."""
    B, G1, V = inp.p_logits.shape
    code = sr.SR_BF16 if inp.p_logits.dtype == np.uint16 else sr.SR_F32
    p, q = dev(inp.p_logits), dev(inp.q_logits)
    d, g = dev(np.asarray(inp.drafts, np.int32)), dev(np.asarray(inp.gamma, np.int32))
    ua, ur = dev(np.asarray(inp.u_acc, np.float32)), dev(np.asarray(inp.u_res, np.float32))
    kv_in = dev(np.asarray(inp.kv_len, np.int32))
    bufs = {k: sr.AcceptBuffers(B, G1 - 1, V, code) for k in ("sep", "fused")}
    res = {}
    for _ in range(calls):
        for k, a in bufs.items():
            a.status.zero_()
            kvc, mk = dev(cache_kv), dev(mask)
            phys = torch.full((1,), -9, dtype=torch.int32, device="cuda")
            args = (p, q, d, g, ua, ur, kv_in, a.accept_len, a.out_tokens, a.new_len, a.accept_prob, a.p_tok,
                    a.q_tok, a.kl, a.tv)
            if k == "sep":
                sr.specrouter_accept_and_diverge_sampled(*args, a.workspace, a.status, temperature=temperature,
                                                         top_k=top_k, top_p=top_p)
                sr.specrouter_rollback(kvc, mk, a.new_len, phys, a.status)
            else:
                sr.specrouter_accept_and_rollback(*args, kvc, mk, phys, a.workspace, a.status,
                                                  temperature=temperature, top_k=top_k, top_p=top_p)
            torch.cuda.synchronize()
            r = {n: host(getattr(a, n)) for n in OUTS}
            r.update(kv=host(kvc), mask=host(mk), phys=int(host(phys)[0]), status=int(host(a.status)[0]))
            res[k] = r
    return res["sep"], res["fused"]


def _same(sep, fused):
    for n in sep:
        if isinstance(sep[n], np.ndarray):
            np.testing.assert_array_equal(fused[n].view(np.uint8), sep[n].view(np.uint8), err_msg=n)
        else:
            assert fused[n] == sep[n], n


@pytest.mark.parametrize("temperature", [1.0, 0.0, 0.6])
@pytest.mark.parametrize("logits", ["f32", "bf16"])
def test_fused_equals_accept_then_rollback(temperature, logits):
    rng = np.random.default_rng(11)
    shape = small_shape(name=f"ar-{logits}", B=12, V=20000, gamma=(0, 6), seed=61, logits=logits)
    inp = level_inputs(shape, kv=False)
    cap = int(inp.kv_len.max()) + 8
    cache_kv, mask = _cache_state(inp, cap, rng)
    say(f"accept+rollback {logits} T={temperature}: B={inp.gamma.shape[0]} gammas {inp.gamma.tolist()}")
    sep, fused = _both(inp, cache_kv, mask, cap, temperature, calls=2)  # the second call after the reset
    assert sep["status"] == 0
    _same(sep, fused)
    ref_kv, ref_mask, ref_phys, ref_st = oracle.rollback(cache_kv, mask, sep["new_len"], cap)
    np.testing.assert_array_equal(fused["kv"], ref_kv)
    np.testing.assert_array_equal(fused["mask"], ref_mask)
    assert fused["phys"] == ref_phys and ref_st == 0


@pytest.mark.parametrize("top_k,top_p", [(20, 1.0), (0, 0.85), (50, 0.9)])
def test_fused_with_top_k_top_p(top_k, top_p):
    """The filtered sampling rule through the fused call: the same bits as the
    filtered accept call followed by the rollback."""
    rng = np.random.default_rng(14)
    inp = level_inputs(small_shape(name="ar-filt", B=10, V=12288, gamma=(0, 6), seed=64), kv=False)
    cap = int(inp.kv_len.max()) + 8
    cache_kv, mask = _cache_state(inp, cap, rng)
    say(f"accept+rollback top_k={top_k} top_p={top_p}")
    sep, fused = _both(inp, cache_kv, mask, cap, 0.8, calls=2, top_k=top_k, top_p=top_p)
    assert sep["status"] == 0
    _same(sep, fused)


def test_fused_data_errors_match():
    """Bad cache lengths, a rollback that would grow, an invalid gamma and an
    out-of-vocabulary draft: the same outputs, lengths, mask and status."""
    rng = np.random.default_rng(12)
    inp = level_inputs(small_shape(name="ar-bad", B=10, V=5000, gamma=(1, 5), seed=62), kv=False)
    cap = int(inp.kv_len.max()) + 4
    cache_kv, mask = _cache_state(inp, cap, rng)
    cache_kv[1] = -1                 # length outside [0, L_cap]
    cache_kv[2] = cap + 3
    cache_kv[3] = 1                  # shorter than the accepted length: the rollback would grow it
    inp.gamma[4] = inp.drafts.shape[1] + 1  # gamma above gamma_max
    inp.gamma[5] = -1                # invalid gamma
    inp.drafts[6, 0] = 5000          # a draft token outside the vocabulary
    sep, fused = _both(inp, cache_kv, mask, cap, 1.0)
    assert sep["status"] != 0
    say(f"data errors: status {sep['status']:#x}")
    _same(sep, fused)


def test_fused_over_several_launches():
    """More sequences than one sweep launch takes: the physical length still
    covers all of them, and the workspace is reset for the next call."""
    rng = np.random.default_rng(13)
    inp = level_inputs(small_shape(name="ar-many", B=4100, V=256, gamma=(0, 2), ctx=(8, 64), seed=63),
                       kv=False)
    cap = int(inp.kv_len.max()) + 2
    cache_kv, mask = _cache_state(inp, cap, rng, holes=0.0)
    say(f"accept+rollback over {inp.gamma.shape[0]} sequences")
    sep, fused = _both(inp, cache_kv, mask, cap, 1.0, calls=2)
    assert sep["status"] == 0
    _same(sep, fused)
