"""The step-time model against measured steps on the GPU: the budget sweep
(256 decode rows of 4k-8k context plus a chunk of B = 0, 256, 1024, 4096
tokens on a 4096-token prefix) and the decode-only decode8b step.  Each step
is kv_append then mixed attention on one stream, timed over 10 steps between
two events; the prediction must be within 15 % (box-to-box spread is about
+-4 %) and must order the sweep as the measurement does."""

import numpy as np
import pytest

import paper_2609_27085_amd as mpa
from workloads.configs import config_specs
from workloads.device import device_step

pytestmark = pytest.mark.gpu

CONFIGS = ["budget0", "budget256", "budget1024", "budget4096", "decode8b"]


@pytest.fixture(scope="module")
def torch_gpu():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    mpa.lib()
    return torch


def measure(torch, name, steps=10):
    specs, heads, nb, rng = config_specs(name, 0)
    d = device_step(specs, heads, "bf16", rng, 0, num_blocks=nb)
    ws = mpa.alloc_workspace(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.qsl_host, d.scale)
    out = torch.empty_like(d.q)

    def step():
        mpa.kv_append(d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                      d.seq_lens_host, d.qsl_host)
        mpa.mixed_paged_attention(d.q, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                                  d.seq_lens_host, d.qsl_host, out, workspace=ws, scale=d.scale)

    for _ in range(3):
        step()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    measured_us = e0.elapsed_time(e1) * 1e3 / steps
    shape = mpa.shape_of(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.scale)
    predicted = mpa.predict_step(shape, d.seq_lens_host, d.qsl_host)
    del d, ws, out
    torch.cuda.empty_cache()
    return measured_us, predicted.step_us


def test_predicted_step_time_matches_measured(torch_gpu):
    got = {}
    for name in CONFIGS:
        m, p = measure(torch_gpu, name)
        print(f"[gpu] step model {name}: measured {m:.1f} us, predicted {p:.1f} us ({100 * (p / m - 1):+.1f} %)",
              flush=True)
        got[name] = (m, p)
    for name, (m, p) in got.items():
        assert abs(p / m - 1) <= 0.15, f"{name}: predicted {p:.1f} us, measured {m:.1f} us"
    sweep = ["budget0", "budget256", "budget1024", "budget4096"]
    assert np.argsort([got[n][0] for n in sweep]).tolist() == np.argsort([got[n][1] for n in sweep]).tolist()
