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


# Shapes the library's rates were not fitted to (they were fitted to seed 0
# of the full-head workloads): other seeds of the agentic and lent mixes and
# of the budget sweep, and one GPU's share of a TP4 layout.
HELD_OUT = ([(c, s, 1) for c in ("agentic", "lent") for s in (1, 2, 3, 4)]
            + [(c, s, 1) for c in ("budget256", "budget4096") for s in (1, 2)]
            + [(c, 0, 4) for c in ("agentic", "lent", "budget4096", "budget1024", "decode8b", "longctx")]
            + [(c, 1, 4) for c in ("agentic", "lent")])


def _timed(torch, fn, steps=10):
    for _ in range(3):
        fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / steps


def test_held_out_shapes(torch_gpu):
    """The step model within 12 % on every held-out shape (8.2-8.7 % at most
    and 2.0-3.0 % on average over two boxes when written; the largest error
    is the 58 us TP4 share of decode8b), and the co-execution planner's
    choice never slower than one stream beyond timing noise, and within 15 %
    of the best of the four modes measured (11-13 % at most, 1.9-2.2 % on
    average)."""
    torch = torch_gpu
    errs, regrets = [], []
    for cfg, seed, tp in HELD_OUT:
        specs, heads, nb, rng = config_specs(cfg, seed, tp=tp)
        d = device_step(specs, heads, "bf16", rng, seed, num_blocks=nb)
        ws = mpa.alloc_workspace(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.qsl_host, d.scale)
        out = torch.empty_like(d.q)
        args = (d.q, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc, d.seq_lens_host,
                d.qsl_host, out)

        def step():
            mpa.kv_append(d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                          d.seq_lens_host, d.qsl_host)
            mpa.mixed_paged_attention(*args, workspace=ws, scale=d.scale)

        measured = _timed(torch, step)
        shape = mpa.shape_of(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.scale)
        predicted = mpa.predict_step(shape, d.seq_lens_host, d.qsl_host).step_us
        err = predicted / measured - 1
        errs.append(abs(err))
        line = f"[gpu] held out {cfg} seed {seed} tp{tp}: step {measured:.1f} us, predicted {predicted:.1f} ({100 * err:+.1f} %)"
        q_lens = np.diff(d.qsl_host)
        if (q_lens > 1).any() and (q_lens == 1).any():
            choice, _ = mpa.plan_coexec(shape, d.seq_lens_host, d.qsl_host)
            modes = [_timed(torch, lambda m=m: mpa.coexec_attention(*args, workspace=ws, scale=d.scale, mode=m))
                     for m in range(4)]
            regret = modes[choice] / min(modes) - 1
            regrets.append(regret)
            line += (f"; modes {', '.join(f'{t:.0f}' for t in modes)} us, planner picks {choice} "
                     f"({100 * regret:+.1f} % from the best)")
            assert modes[choice] <= 1.03 * modes[0], f"{cfg} seed {seed} tp{tp}: mode {choice} slower than serial"
            assert regret <= 0.15, f"{cfg} seed {seed} tp{tp}: mode {choice} {100 * regret:.1f} % from the best"
        print(line, flush=True)
        assert abs(err) <= 0.12, f"{cfg} seed {seed} tp{tp}: predicted {predicted:.1f} us, measured {measured:.1f} us"
        del d, ws, out
        torch.cuda.empty_cache()
    print(f"[gpu] held out: step model mean |error| {100 * np.mean(errs):.1f} %, max {100 * max(errs):.1f} %; "
          f"planner mean regret {100 * np.mean(regrets):.1f} %, max {100 * max(regrets):.1f} %", flush=True)
