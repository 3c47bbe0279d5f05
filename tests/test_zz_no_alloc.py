"""mpa_append_attention_noalloc (the one-call step with its partial results
in the library's fixed device array) against mpa_append_attention with a
caller workspace, through the C ABI: two calls in a row, the second on a
smaller batch, each giving the same cache bits, out and lse as the
workspace entry point (and the oracle's append and attention within the
bars)."""

import numpy as np
import pytest

import paper_2609_27085_amd as mpa
from oracle import ref
from workloads import HeadSpec, SeqSpec, make_batch
from workloads.device import tensor_to_raw, to_device

pytestmark = pytest.mark.gpu


def _step(torch, d, noalloc):
    out = torch.full_like(d.q, float("nan"))
    lse = torch.full(d.q.shape[:2], float("nan"), dtype=torch.float32, device=d.q.device)
    kw = dict(lse=lse, scale=d.scale, block_tables_host=d.block_tables_host, k_scale=d.k_scale, v_scale=d.v_scale)
    args = (d.q, d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
            d.seq_lens_host, d.qsl_host, out)
    if noalloc:
        mpa.append_attention_noalloc(*args, **kw)
    else:
        ws = mpa.alloc_workspace(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.qsl_host, d.scale)
        mpa.append_attention(*args, workspace=ws, **kw)
    torch.cuda.synchronize()
    return out, lse


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_noalloc_matches_workspace_entry_point(dtype):
    import torch

    assert torch.cuda.is_available()
    mpa.lib()
    rng = np.random.default_rng(400)
    big = [SeqSpec(int(L), 1) for L in rng.integers(1, 9000, size=40)]
    big += [SeqSpec(3000 + 200, 200), SeqSpec(1500 + 100, 100), SeqSpec(40 + 30, 30)]
    small = [SeqSpec(int(L), 1) for L in rng.integers(1, 3000, size=5)] + [SeqSpec(900 + 50, 50)]
    for k, specs in enumerate((big, small)):
        b = make_batch([specs[i] for i in rng.permutation(len(specs))], HeadSpec(32, 8, 128), dtype, rng)
        sh = mpa.make_shape(num_seqs=b.num_seqs, num_q_heads=32, num_kv_heads=8, head_dim=128,
                            num_blocks=b.num_blocks, max_blocks_per_seq=b.block_tables.shape[1],
                            total_q_tokens=b.total_q, scale=b.scale,
                            dtype=mpa.MPA_FP8 if dtype == "fp8" else mpa.MPA_BF16, k_scale=b.k_scale,
                            v_scale=b.v_scale)
        need = mpa.workspace_size(sh, b.seq_lens, b.query_start_loc)
        print(f"[gpu] noalloc call {k}: S={b.num_seqs} T={b.total_q} {dtype}, partials {need} bytes", flush=True)
        assert 0 < need <= mpa.MPA_SCRATCH_BYTES
        d1, d2 = to_device(b), to_device(b)
        o1, l1 = _step(torch, d1, noalloc=False)
        o2, l2 = _step(torch, d2, noalloc=True)
        assert tensor_to_raw(d2.k_cache, dtype).tobytes() == tensor_to_raw(d1.k_cache, dtype).tobytes()
        assert tensor_to_raw(d2.v_cache, dtype).tobytes() == tensor_to_raw(d1.v_cache, dtype).tobytes()
        assert torch.equal(o2.view(torch.int16), o1.view(torch.int16)) and torch.equal(l2, l1)
        # and the oracle's bars
        kc, vc = ref.append_reference(b.k_cache, b.v_cache, b.k_new, b.v_new, b.block_tables, b.seq_lens,
                                      b.query_start_loc, 16, dtype, k_scale=b.k_scale, v_scale=b.v_scale)
        assert tensor_to_raw(d2.k_cache, dtype).tobytes() == kc.tobytes()
        assert tensor_to_raw(d2.v_cache, dtype).tobytes() == vc.tobytes()
        o_ref, l_ref = ref.attention_reference(b.q, b.k_cache, b.v_cache, b.k_new, b.v_new, b.block_tables,
                                               b.seq_lens, b.query_start_loc, b.scale, 8, 16, dtype,
                                               k_scale=b.k_scale, v_scale=b.v_scale)
        err = np.abs(o2.float().cpu().numpy().astype(np.float64) - o_ref)
        assert err.max() <= 1e-2 and err.mean() <= 1e-3, (err.max(), err.mean())
        assert np.abs(l2.cpu().numpy().astype(np.float64) - l_ref).max() <= 2e-3
