"""HIP-graph capture of a whole step: mpa_kv_append then
mpa_mixed_paged_attention (or the one mpa_append_attention call) recorded
once into a graph (through torch's graph
capture on the library's stream argument) and replayed.

Every launch takes its plan as kernel arguments and the library enqueues no
memset and no copy, so a captured step is a fixed sequence of kernel nodes.
Replays run with eager work and synchronisations between them, and every
replay must reproduce the eager step bit for bit (outputs, lse and both
caches); the eager step itself is checked against the oracle.
"""

import numpy as np
import pytest

import paper_2609_27085_amd as mpa
from oracle import ref
from workloads import HeadSpec, SeqSpec, make_batch
from workloads.device import to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_gpu():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    mpa.lib()
    return torch


def graph_specs(rng):
    # long decode rows (split-K + merge), short chunks on long prefixes
    # (prefill KV splits + their merge), a chunk with no prefix, q_len 0
    specs = [SeqSpec(int(c), 1) for c in rng.integers(1, 4000, size=6)]
    specs += [SeqSpec(6000, 1), SeqSpec(1500 + 100, 100), SeqSpec(2100 + 37, 37), SeqSpec(300, 300),
              SeqSpec(40, 0)]
    order = rng.permutation(len(specs))
    return [specs[i] for i in order]


@pytest.mark.parametrize("fused", [False, True], ids=["two_calls", "one_call"])
@pytest.mark.parametrize("heads", [(32, 8, 128), (8, 2, 64)], ids=lambda h: f"hq{h[0]}_hkv{h[1]}_d{h[2]}")
def test_graph_replays_equal_eager_step(torch_gpu, heads, fused):
    """The step as mpa_kv_append + mpa_mixed_paged_attention, or as the one
    mpa_append_attention call (whose decode kernel writes the new tokens)."""
    torch = torch_gpu
    rng = np.random.default_rng(60 + heads[2])
    b = make_batch(graph_specs(rng), HeadSpec(*heads, 16), "bf16", rng)
    print(f"[gpu] graph capture: S={b.num_seqs} T={b.total_q} heads={heads} fused={fused}", flush=True)
    d = to_device(b)
    ws = mpa.alloc_workspace(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.qsl_host, d.scale)
    out = torch.full_like(d.q, float("nan"))
    lse = torch.full(d.q.shape[:2], float("nan"), dtype=torch.float32, device="cuda")

    def step():
        if fused:
            mpa.append_attention(d.q, d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens,
                                 d.query_start_loc, d.seq_lens_host, d.qsl_host, out, lse=lse, workspace=ws,
                                 scale=d.scale)
            return
        mpa.kv_append(d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                      d.seq_lens_host, d.qsl_host)
        mpa.mixed_paged_attention(d.q, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                                  d.seq_lens_host, d.qsl_host, out, lse=lse, workspace=ws, scale=d.scale)

    step()  # eager step (also the first use of every kernel on this device)
    torch.cuda.synchronize()
    o_e, l_e = out.clone(), lse.clone()
    k_e, v_e = d.k_cache.clone(), d.v_cache.clone()

    o_ref, l_ref = ref.attention_reference(b.q, b.k_cache, b.v_cache, b.k_new, b.v_new, b.block_tables,
                                           b.seq_lens, b.query_start_loc, b.scale, heads[1], 16, "bf16")
    rows = np.repeat(b.q_lens > 0, b.q_lens)
    err = np.abs(o_e.float().cpu().numpy().astype(np.float64)[rows] - o_ref[rows])
    assert err.max() <= 1e-2 and err.mean() <= 1e-3, f"eager step: max {err.max():.3g} mean {err.mean():.3g}"
    assert np.abs(l_e.cpu().numpy().astype(np.float64)[rows] - l_ref[rows]).max() <= 2e-3  # bf16 P rounding

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    rows_t = torch.from_numpy(rows).cuda()
    for replay in range(3):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out[rows_t].view(torch.int16), o_e[rows_t].view(torch.int16)), f"replay {replay}: out"
        assert torch.equal(lse[rows_t], l_e[rows_t]), f"replay {replay}: lse"
        assert torch.equal(d.k_cache.view(torch.int16), k_e.view(torch.int16)), f"replay {replay}: K cache"
        assert torch.equal(d.v_cache.view(torch.int16), v_e.view(torch.int16)), f"replay {replay}: V cache"
