"""The matrix-core rate probe behind the roofline figures: it runs, reports
the operations of a launch (per wave and iteration 8 independent MFMAs of
32768 operations for int8 16x16x64 or 65536 for e4m3 x e2m1 16x16x128, 4
of 65536 for int8 32x32x32) and writes one word per thread, and its rate is a positive finite
number of TOPS below twice the nominal 5 POPS dense peak."""
import pytest

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kind,per", [(0, 8 * 32768), (1, 8 * 65536), (2, 4 * 65536)])
def test_probe_mfma_runs(gpu, kind, per):
    import torch
    import paper_2512_02901_amd as f2
    blocks, iters = 64, 64
    sink = torch.full((blocks * 256,), -7, dtype=torch.int32, device=gpu)
    ops = f2.probe_mfma(kind, blocks, iters, sink)
    assert ops == blocks * 4 * iters * per
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    f2.probe_mfma(kind, blocks, iters, sink)
    e1.record()
    torch.cuda.synchronize()
    tops = ops / (e0.elapsed_time(e1) * 1e-3) / 1e12
    assert 0 < tops < 10000
    # every thread stored its word (the initial pattern -7 is overwritten
    # unless a thread's sum happens to equal it)
    assert int((sink == -7).sum().item()) < sink.numel() // 2
