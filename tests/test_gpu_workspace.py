"""One accept workspace reused by calls of different shapes and logit types:
every call equals a call with a fresh (zero) workspace, bit for bit, and
leaves the workspace all zero (the next call lays its regions over the same
bytes, and its polls read any non-zero record word as published)."""

import numpy as np
import pytest
import torch

import paper_2505_07680_amd as sr
from workloads import level_inputs, small_shape

from gpu_util import run_accept

pytestmark = pytest.mark.gpu

SEQ = [
    (dict(B=24, V=20000, gamma=(1, 8), seed=81), {}),
    (dict(B=5, V=3000, gamma=(0, 4), seed=82), {}),
    (dict(B=40, V=33000, gamma=(2, 8), logits="bf16", seed=83), {}),
    (dict(B=12, V=16000, gamma=(1, 6), seed=84), dict(temperature=0.7, top_k=40, top_p=0.9)),
    (dict(B=3, V=1000, gamma=(1, 3), logits="bf16", seed=85), {}),
    (dict(B=16, V=12000, gamma=(1, 8), logits="bf16", seed=86), dict(temperature=0.0)),
    (dict(B=9, V=50264, gamma=(3, 5), logits="bf16", seed=87), dict(temperature=0.8, top_p=0.95)),
]


@pytest.fixture(scope="module", autouse=True)
def _library():
    sr.load()
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()


def _bufs(inp, ws=None):
    B, G1, V = inp.p_logits.shape
    code = sr.SR_BF16 if inp.p_logits.dtype == np.uint16 else sr.SR_F32
    b = sr.AcceptBuffers(B, G1 - 1, V, code)
    if ws is not None:
        b.workspace = ws[: b.workspace.numel()]
    return b


def test_workspace_reused_across_shapes():
    inps = [level_inputs(small_shape(name=f"ws-reuse-{i}", **shape), kv=False) for i, (shape, _) in enumerate(SEQ)]
    need = max(_bufs(inp).workspace.numel() for inp in inps)
    shared = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for i, (inp, (shape, kw)) in enumerate(zip(inps, SEQ)):
        print(f"[gpu-test] call {i}: {shape} {kw}", flush=True)
        args = (inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res)
        fresh = run_accept(*args, kv_len=inp.kv_len, bufs=_bufs(inp), **kw)
        reused = run_accept(*args, kv_len=inp.kv_len, bufs=_bufs(inp, shared), **kw)
        for n, w in fresh.items():
            if isinstance(w, np.ndarray):
                np.testing.assert_array_equal(reused[n].view(np.uint8), w.view(np.uint8), err_msg=f"call {i}: {n}")
            else:
                assert reused[n] == w, f"call {i}: {n}"
        assert fresh["status"] == 0
        nz = int((shared != 0).sum().item())
        assert nz == 0, f"call {i} left {nz} workspace bytes non-zero"
