"""Seeded random mixed batches against the oracle.

Each case draws a head layout (1, 2 or 4 KV heads, groups of 1-16 query
heads, head_dim 64 or 128), 0-4 decode rows of 1-2,499 keys and 1-3 prefill
chunks of 2-299 tokens on prefixes of 0, 1-63 or 64-2,199 keys, in a random
order, a cache type (bf16, fp8, f32) and a KV-split setting for the prefill
chunks (the library's choice, or 1, 2 or 4 splits).  The append is checked bit
for bit over the whole pool.

Half of the bf16 and fp8 cases are drawn as for the stated tolerances
(unit-normal values; max |err| 1e-2, mean 1e-3, lse 2e-3).  In the other half
the queries are scaled by 4 or 12, which concentrates each row's attention on
a few keys.  There the bf16 format itself bounds the error:
- the output's rounding is up to 2^-8 |o|;
- one dominant probability rounded to bf16 moves the output by up to 2^-8
  times the spread of the values;
- that probability moves the log-sum-exp by up to ln(1 + 2^-8).
The test checks those bounds, which a wrong key, mask or scale would exceed
by far.
"""

import os

import numpy as np
import pytest

import paper_2609_27085_amd as mpa
from oracle import ref
from workloads import HeadSpec, SeqSpec, bf16_bits_from_f32, make_batch
from workloads.device import tensor_to_raw, to_device

from test_gpu_parity import as_f64, bf16_to_f32, check_batch, oracle_for, run_step, say

pytestmark = pytest.mark.gpu

N_CASES = 64
V_SPREAD = 6.0  # |v| of the N(0,1) values drawn here stays below 6


@pytest.fixture(scope="module")
def torch_gpu():
    import torch

    assert torch.cuda.is_available(), "GPU tests need a GPU"
    mpa.lib()
    return torch


def draw_case(case):
    rng = np.random.default_rng(10_000 + case)
    hkv = int(rng.choice([1, 2, 4]))
    g = int(rng.choice([1, 2, 3, 4, 5, 6, 7, 8, 12, 16]))
    while hkv * g > 32:
        hkv //= 2
    hkv = max(hkv, 1)
    d = int(rng.choice([64, 128]))
    dtype = str(rng.choice(["bf16", "bf16", "fp8", "f32"]))
    specs = [SeqSpec(int(rng.integers(1, 2500)), 1) for _ in range(int(rng.integers(0, 5)))]
    for _ in range(int(rng.integers(1, 4))):
        c = int(rng.integers(2, 300))
        r = rng.random()
        p = 0 if r < 0.15 else int(rng.integers(1, 64)) if r < 0.3 else int(rng.integers(64, 2200))
        specs.append(SeqSpec(p + c, c))
    specs = [specs[i] for i in rng.permutation(len(specs))]
    splits = str(rng.choice(["auto", "1", "2", "4"]))
    b = make_batch(specs, HeadSpec(hkv * g, hkv, d), dtype, rng)
    qmul = float(rng.choice([1.0, 1.0, 4.0, 12.0])) if dtype != "f32" else 1.0
    if qmul != 1.0:
        q = bf16_to_f32(b.q).astype(np.float64) * qmul
        b.q[...] = bf16_bits_from_f32(q.astype(np.float32))
    return b, splits, qmul, specs


@pytest.mark.parametrize("case", range(N_CASES))
def test_random_batch(torch_gpu, case, monkeypatch):
    b, splits, qmul, specs = draw_case(case)
    if splits != "auto":
        monkeypatch.setenv("MPA_PREFILL_SPLITS", splits)
    else:
        monkeypatch.delenv("MPA_PREFILL_SPLITS", raising=False)
    what = (f"random case {case}: {b.heads} {b.dtype} splits {splits} q x{qmul} "
            f"(prefix, q_len) {[(s.ctx - s.q_len, s.q_len) for s in specs]}")
    if qmul == 1.0:
        check_batch(b, what)
        return
    say(f"[gpu] {what}")
    d = to_device(b)
    out, lse = run_step(d)
    kc, vc = ref.append_reference(b.k_cache, b.v_cache, b.k_new, b.v_new, b.block_tables, b.seq_lens,
                                  b.query_start_loc, b.heads.block_size, b.dtype, k_scale=b.k_scale,
                                  v_scale=b.v_scale)
    assert tensor_to_raw(d.k_cache, b.dtype).tobytes() == kc.tobytes(), f"{what}: K append not bit-exact"
    assert tensor_to_raw(d.v_cache, b.dtype).tobytes() == vc.tobytes(), f"{what}: V append not bit-exact"
    o_ref, l_ref = oracle_for(b)
    rows = np.repeat(b.q_lens > 0, b.q_lens)
    got, exp = as_f64(out)[rows], o_ref[rows]
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    bound = 2.0 ** -8 * (np.abs(exp) + V_SPREAD) + 2e-3
    err = np.abs(got - exp)
    assert (err <= bound).all(), f"{what}: max err {err.max():.4f} beyond the bf16 format bound"
    lerr = np.abs(lse.cpu().numpy().astype(np.float64)[rows] - l_ref[rows]).max()
    assert lerr <= np.log1p(2.0 ** -8) + 2e-4, f"{what}: lse err {lerr:.5f}"
