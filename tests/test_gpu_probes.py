"""The measurement probes (mpa_probe_stream_read, mpa_probe_mfma_bf16): they
run, report the work they do, and measure rates below the MI355X datasheet
peaks (8 TB/s HBM, 2.5 PFLOP/s dense bf16) but within a factor of two of
them, which is what an intact probe of this device reads."""

import pytest

import paper_2609_27085_amd as mpa

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_gpu():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    mpa.lib()
    return torch


def _time(torch, launch, reps=3):
    launch()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        launch()
    b.record()
    b.synchronize()
    return a.elapsed_time(b) / reps * 1e-3


def test_stream_read_rate(torch_gpu):
    torch = torch_gpu
    print("[gpu] probe stream read 1 GiB", flush=True)
    buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    t = _time(torch, lambda: mpa.probe_stream_read(buf, sink))
    gbs = buf.numel() / t / 1e9
    print(f"[gpu] stream read {gbs:.0f} GB/s", flush=True)
    assert 4000 < gbs < 8000
    # a ragged size (not a multiple of the 4 KB run) reads in bounds
    mpa.probe_stream_read(buf[: (1 << 20) + 48], sink)
    torch.cuda.synchronize()


def test_mfma_rate(torch_gpu):
    torch = torch_gpu
    print("[gpu] probe bf16 MFMA", flush=True)
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    flops = []
    t = _time(torch, lambda: flops.append(mpa.probe_mfma_bf16(4000, sink)))
    assert flops[-1] == 2 * 32 * 32 * 16 * 4 * 4000 * 4096
    tf = flops[-1] / t / 1e12
    print(f"[gpu] bf16 MFMA {tf:.0f} TFLOP/s", flush=True)
    assert 1250 < tf < 2500
    assert sink.item() == 0.0  # never written
