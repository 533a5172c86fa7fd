"""GPU check of the HBM read-bandwidth probe: it runs over buffers of several
sizes (blocks of unequal length and ragged tails included), leaves the sink alone
(the folded value of these buffers is never the trigger constant) and reads at
a plausible rate."""

import pytest
import torch

import paper_2505_07680_amd as sr

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _library():
    sr.load()
    assert torch.cuda.is_available()
    yield
    torch.cuda.synchronize()


@pytest.mark.parametrize("nbytes", [16, 4096 + 16, (64 << 20) + 48])
def test_probe_runs_and_leaves_the_sink(nbytes):
    buf = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    sink = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    print(f"[gpu-test] probe over {nbytes} bytes", flush=True)
    sr.specrouter_hbm_read_probe(buf, sink)
    torch.cuda.synchronize()
    assert int(sink.item()) == 7


def test_probe_reads_at_a_plausible_rate():
    n = (1 << 30) // 4
    bufs = [torch.ones(n, dtype=torch.float32, device="cuda") for _ in range(3)]
    for b in bufs:
        sr.specrouter_hbm_read_probe(b)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(9):
        sr.specrouter_hbm_read_probe(bufs[i % 3])
    e1.record()
    torch.cuda.synchronize()
    gbs = 9 * n * 4 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    print(f"[gpu-test] probe read {gbs:.0f} GB/s", flush=True)
    assert 1000 < gbs < 8000
