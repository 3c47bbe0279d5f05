"""Co-execution of the attention halves on CU-partitioned streams
(mpa_plan_coexec, mpa_partition_streams): in every mode the step's outputs are
bit-identical to mpa_mixed_paged_attention on one stream, which the oracle
checks."""

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


@pytest.mark.parametrize("heads", [(32, 8, 128), (8, 2, 64)], ids=lambda h: f"hq{h[0]}_hkv{h[1]}_d{h[2]}")
def test_every_mode_equals_the_mixed_call(torch_gpu, heads):
    torch = torch_gpu
    rng = np.random.default_rng(90 + heads[2])
    specs = [SeqSpec(int(c), 1) for c in rng.integers(1, 5000, size=24)]
    specs += [SeqSpec(3000 + 300, 300), SeqSpec(1500 + 100, 100), SeqSpec(600, 600), SeqSpec(2000 + 37, 37)]
    order = rng.permutation(len(specs))
    b = make_batch([specs[i] for i in order], HeadSpec(*heads, 16), "bf16", rng)
    print(f"[gpu] coexec modes: S={b.num_seqs} T={b.total_q} heads={heads}", flush=True)
    d = to_device(b)
    mpa.kv_append(d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                  d.seq_lens_host, d.qsl_host)
    ws = mpa.alloc_workspace(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.qsl_host, d.scale)
    args = (d.q, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc, d.seq_lens_host, d.qsl_host)
    rows = torch.from_numpy(np.repeat(b.q_lens > 0, b.q_lens)).cuda()

    def run(mode):
        out = torch.full_like(d.q, float("nan"))
        lse = torch.full(d.q.shape[:2], float("nan"), dtype=torch.float32, device="cuda")
        if mode is None:
            mpa.mixed_paged_attention(*args, out, lse=lse, workspace=ws, scale=d.scale)
            used = None
        else:
            used = mpa.coexec_attention(*args, out, lse=lse, workspace=ws, scale=d.scale,
                                        mode=None if mode == "auto" else mode)
        torch.cuda.synchronize()
        return out, lse, used

    o0, l0, _ = run(None)
    o_ref, l_ref = ref.attention_reference(b.q, b.k_cache, b.v_cache, b.k_new, b.v_new, b.block_tables, b.seq_lens,
                                           b.query_start_loc, b.scale, heads[1], 16, "bf16")
    r = np.repeat(b.q_lens > 0, b.q_lens)
    err = np.abs(o0.float().cpu().numpy().astype(np.float64)[r] - o_ref[r])
    assert err.max() <= 1e-2 and err.mean() <= 1e-3
    for mode in (1, 2, 3, "auto"):
        o, l, used = run(mode)
        assert used in (0, 1, 2, 3)
        assert torch.equal(o[rows].view(torch.int16), o0[rows].view(torch.int16)), f"mode {mode}: out"
        assert torch.equal(l[rows], l0[rows]), f"mode {mode}: lse"


def test_partition_streams_are_cached(torch_gpu):
    a = mpa.partition_streams(2)
    b = mpa.partition_streams(2)
    assert a[0].cuda_stream == b[0].cuda_stream and a[1].cuda_stream == b[1].cuda_stream
    assert a[0].cuda_stream != a[1].cuda_stream
