"""The chain scheduler fed by the HIP accept-and-diverge call: the smoothed
SimScore (Eq. 6) and the calibration built from the kernel's `tv` and
`accept_len` outputs agree with the reference fed by the CPU reference's
outputs for the same seeded inputs."""

import numpy as np
import pytest
import torch

import oracle
from oracle import scheduler as ref
from workloads import CONFIGS, level_inputs, small_shape

from gpu_util import DIV_RTOL, run_accept

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _library():
    import paper_2505_07680_amd as sr

    sr.load()
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()


def test_scheduler_consumes_kernel_divergence():
    import paper_2505_07680_amd as sr

    s = sr.ChainScheduler([0.068, 1.1, 7.0], 2, 4, ema_sim=0.3)
    D = float("nan")
    obs = []
    for seed, (i, j) in zip((31, 32, 33), ((0, 2), (0, 2), (1, 2))):
        shape = small_shape(name=f"sched{seed}", B=12, V=3000, gamma=(0, 5), seed=seed)
        inp = level_inputs(shape, kv=False)
        print(f"[gpu-test] scheduler: accept seed {seed}", flush=True)
        got = run_accept(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res)
        want = oracle.accept_and_diverge(inp.p_logits, inp.q_logits, inp.drafts, inp.gamma, inp.u_acc, inp.u_res)
        assert got["status"] == want["status"] == 0
        s.observe_step(i, j, inp.gamma, got["accept_len"], got["tv"])
        mean, n = ref.step_mean_tv(want["tv"], inp.gamma, want["accept_len"])
        assert n > 0
        if (i, j) == (0, 2):
            D = ref.ema(D, mean, 0.3)
        # calibration outcomes use the kernel's accept lengths; the reference
        # decisions agree except at counted boundary cases
        obs.append((1.0 - mean, *ref.step_outcomes(inp.gamma, got["accept_len"])))
    _, S, _, n_obs = s.metrics()
    assert n_obs == 3
    assert S[0, 2] == pytest.approx(1.0 - D, rel=DIV_RTOL)
    A, B = s.calibrate()
    rA, rB = ref.calibrate(obs, lam=1.0)
    assert A == pytest.approx(rA, rel=1e-3, abs=1e-3) and B == pytest.approx(rB, rel=1e-3, abs=1e-3)
    chain, t, _ = s.optimal_chain()
    assert chain == [2]  # no per-token times observed: the default chain
