"""The benchmark's algorithmic byte / FLOP accounting on a hand-sized batch,
its refusal of more than one GPU, and the tensor-parallel workload share
(CPU only)."""

import subprocess
import sys

import pytest

import bench


def test_algorithmic_work_hand_example():
    # decode row L=20; chunk C=3 on P=5 (L=8); a q_len-0 sequence; Hq=4, Hkv=2, d=8, bf16
    w = bench.algorithmic_work([20, 8, 30], [0, 1, 4, 4], hq=4, hkv=2, d=8, elem_bytes=2)
    # decode: K+V 2*20*2*8*2 = 1280, q+out 2*4*8*2 = 128, block ids 4*2 = 8
    assert w["decode_bytes"] == 1280 + 128 + 8
    # prefill: K+V 2*8*2*8*2 = 512, q+out 2*3*4*8*2 = 384
    assert w["prefill_bytes"] == 512 + 384
    # append: 4 tokens * 4 * Hkv * d * e = 4*4*2*8*2
    assert w["append_bytes"] == 512
    # FLOPs: 4*d*Hq per pair; decode 20 pairs; chunk 3*5 + 3*4/2 = 21 pairs
    assert w["decode_flops"] == 4 * 8 * 4 * 20
    assert w["prefill_flops"] == 4 * 8 * 4 * 21
    assert (w["decode_rows"], w["prefill_chunks"], w["query_tokens"]) == (1, 1, 4)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_tensor_parallel_share_keeps_the_sequences():
    """One GPU's share of a TP layout: the same sequences (same draws) with
    1/tp of both head counts; head counts that do not divide are refused."""
    from workloads.configs import config_specs

    for name in ("decode8b", "agentic", "longctx"):
        s1, h1, nb1, _ = config_specs(name, 3)
        s4, h4, nb4, _ = config_specs(name, 3, tp=4)
        assert s1 == s4 and nb1 == nb4
        assert (h4.num_q_heads * 4, h4.num_kv_heads * 4) == (h1.num_q_heads, h1.num_kv_heads)
        assert (h4.head_dim, h4.block_size) == (h1.head_dim, h1.block_size)
    with pytest.raises(ValueError):
        config_specs("decode8b", 0, tp=16)  # 8 KV heads
    with pytest.raises(ValueError):
        config_specs("tiny", 0, tp=4)  # 2 KV heads
