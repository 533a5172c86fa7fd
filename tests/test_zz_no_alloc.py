"""specrouter_accept_and_rollback_noalloc (the library's own fixed device array
as the workspace) against specrouter_accept_and_rollback with a caller
workspace: bit-identical outputs, lengths, mask, physical length and status,
on two calls in a row, the second with a smaller problem than the first (the
array keeps the first call's state in between), at T = 1, under top-k/top-p
and greedily; the first call's accept also against the reference."""

import numpy as np
import pytest
import torch

import oracle
import paper_2505_07680_amd as sr
from workloads import level_inputs, small_shape

from gpu_util import check_accept, dev, host

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


def _run(inp, noalloc, cap, temperature=1.0, top_k=0, top_p=1.0):
    B, G1, V = inp.p_logits.shape
    code = sr.SR_BF16 if inp.p_logits.dtype == np.uint16 else sr.SR_F32
    a = sr.AcceptBuffers(B, G1 - 1, V, code)
    p, q = dev(inp.p_logits), dev(inp.q_logits)
    d, g = dev(np.asarray(inp.drafts, np.int32)), dev(np.asarray(inp.gamma, np.int32))
    ua, ur = dev(np.asarray(inp.u_acc, np.float32)), dev(np.asarray(inp.u_res, np.float32))
    kv_in = dev(np.asarray(inp.kv_len, np.int32))
    kvc = dev(np.asarray(inp.kv_len, np.int32))
    mask = np.ones((B, cap), np.uint8)
    mk = dev(mask)
    phys = torch.full((1,), -9, dtype=torch.int32, device="cuda")
    args = (p, q, d, g, ua, ur, kv_in, a.accept_len, a.out_tokens, a.new_len, a.accept_prob, a.p_tok, a.q_tok,
            a.kl, a.tv)
    if noalloc:
        sr.specrouter_accept_and_rollback_noalloc(*args, kvc, mk, phys, a.status, temperature=temperature,
                                                  top_k=top_k, top_p=top_p)
    else:
        sr.specrouter_accept_and_rollback(*args, kvc, mk, phys, a.workspace, a.status, temperature=temperature,
                                          top_k=top_k, top_p=top_p)
    torch.cuda.synchronize()
    r = {n: host(getattr(a, n)) for n in OUTS}
    r.update(kv=host(kvc), mask=host(mk), phys=int(host(phys)[0]), status=int(host(a.status)[0]))
    return r


def _same(want, got):
    for n, w in want.items():
        if isinstance(w, np.ndarray):
            np.testing.assert_array_equal(got[n].view(np.uint8), w.view(np.uint8), err_msg=n)
        else:
            assert got[n] == w, n


CASES = [
    # (label, first shape, second (smaller) shape, sampling)
    ("f32-T1", dict(B=24, V=20000, gamma=(1, 8), seed=71), dict(B=5, V=3000, gamma=(0, 4), seed=72), {}),
    ("bf16-T1", dict(B=40, V=33000, gamma=(2, 8), logits="bf16", seed=73),
     dict(B=3, V=1000, gamma=(1, 3), logits="bf16", seed=74), {}),
    ("f32-topk-topp", dict(B=12, V=16000, gamma=(1, 6), seed=75), dict(B=2, V=4096, gamma=(2, 2), seed=76),
     dict(temperature=0.7, top_k=40, top_p=0.9)),
    ("bf16-greedy", dict(B=16, V=12000, gamma=(1, 8), logits="bf16", seed=77),
     dict(B=4, V=2056, gamma=(0, 5), logits="bf16", seed=78), dict(temperature=0.0)),
]


@pytest.mark.parametrize("label,big,small,sampling", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_workspace_call(label, big, small, sampling):
    for step, shape in (("first", big), ("second, smaller", small)):
        inp = level_inputs(small_shape(name=f"noalloc-{label}", **shape), kv=False)
        cap = int(inp.kv_len.max()) + 8
        say(f"{label} {step}: B={inp.B} V={inp.p_logits.shape[2]} {sampling}")
        want = _run(inp, False, cap, **sampling)
        got = _run(inp, True, cap, **sampling)
        _same(want, got)
        if step == "first" and not sampling:
            ref = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc,
                                            inp.u_res, kv_len=inp.kv_len)
            check_accept(got, ref)
        assert got["status"] == 0
