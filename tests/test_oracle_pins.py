"""Pins for the CPU oracle: each checks it against something other than itself.

* a hand-worked closed-form fixture (tests/golden/hand_worked.txt);
* brute force on tiny inputs, reading the pool through the header's flat
  offset formula and exponentiating without subtracting the maximum;
* closed forms: context length 1 returns V exactly, Q = 0 gives the running
  mean of V, identical keys give the mean of V, a dominant key returns its V;
* invariances: block-table permutation, block size, paged vs contiguous;
* a library special case: torch float64 scaled_dot_product_attention with an
  explicit bottom-right mask and repeat_interleave for grouped heads;
* the split/merge identity of the softmax denominators;
* row independence of a mixed batch;
* the append: new bits land at their slots and nothing else changes.
"""

import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import ref
from workloads import HeadSpec, SeqSpec, make_batch
from workloads.gen import bf16_bits_from_f32, k_cache_shape, v_cache_shape

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked.txt")


def run_oracle(b, seqs=None):
    return ref.attention_reference(
        b.q, b.k_cache, b.v_cache, b.k_new, b.v_new, b.block_tables, b.seq_lens,
        b.query_start_loc, b.scale, b.heads.num_kv_heads, b.heads.block_size, b.dtype, seqs=seqs,
    )


# ----------------------------------------------------------------------------
# hand-worked fixture


def _golden_rows():
    rows = []
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            p = line.split()
            rows.append((p[0], int(p[1]), int(p[2]), [Fraction(x) for x in p[3:7]], int(p[7])))
    return rows


def _f32_pool(nb, hkv, d, bs):
    k = np.full(k_cache_shape(nb, HeadSpec(hkv, hkv, d, bs), "f32"), np.nan, dtype=np.float32)
    v = np.full(v_cache_shape(nb, HeadSpec(hkv, hkv, d, bs), "f32"), np.nan, dtype=np.float32)
    return k, v


def _put_k(kc, b, h, t, vec):
    # header formula: K element (b, h, t, i) at [b][h][i // X][t][i % X], X = 4 for f32
    for i, val in enumerate(vec):
        kc[b, h, i // 4, t, i % 4] = val


def _put_v(vc, b, h, t, vec):
    for i, val in enumerate(vec):
        vc[b, h, i, t] = val


def test_golden_hand_worked():
    d, bs = 4, 2
    e = np.eye(4, dtype=np.float32)
    kvec = [np.array([j, 0, 0, 0], dtype=np.float32) for j in range(4)]
    scale = math.log(2.0)
    got = {}
    # case A: P = 0, chunk of 3, one head; everything arrives as new tokens.
    kc, vc = _f32_pool(2, 1, d, bs)
    q = np.array([[[1, 0, 0, 0]]] * 3, dtype=np.float32)
    kn = np.stack(kvec[:3])[:, None, :]
    vn = e[:3][:, None, :]
    o, lse = ref.attention_reference(
        q, kc, vc, kn, vn, np.array([[0, 1]], np.int32), np.array([3], np.int32),
        np.array([0, 3], np.int32), scale, 1, bs, "f32")
    for r in range(3):
        got[("A", r, 0)] = (o[r, 0], lse[r, 0])
    # case B: P = 2 cached in block 1, chunk of 2 new tokens into block 0, Hq=2, Hkv=1.
    kc, vc = _f32_pool(2, 1, d, bs)
    for j in range(2):
        _put_k(kc, 1, 0, j, kvec[j])
        _put_v(vc, 1, 0, j, e[j])
    q = np.array([[[1, 0, 0, 0], [0, 0, 0, 0]]] * 2, dtype=np.float32)
    kn = np.stack(kvec[2:4])[:, None, :]
    vn = e[2:4][:, None, :]
    o, lse = ref.attention_reference(
        q, kc, vc, kn, vn, np.array([[1, 0]], np.int32), np.array([4], np.int32),
        np.array([0, 2], np.int32), scale, 1, bs, "f32")
    for r in range(2):
        for h in range(2):
            got[("B", r, h)] = (o[r, h], lse[r, h])
    rows = _golden_rows()
    assert len(rows) == 7
    for case, r, h, ofr, lse_arg in rows:
        o_got, lse_got = got[(case, r, h)]
        np.testing.assert_allclose(o_got, [float(x) for x in ofr], rtol=0, atol=1e-14)
        assert abs(lse_got - math.log(lse_arg)) < 1e-13


# ----------------------------------------------------------------------------
# brute force


def _flat_k(b, h, t, i, hkv, d, bs, x):
    return ((((b * hkv + h) * (d // x) + i // x) * bs + t) * x) + i % x


def _flat_v(b, h, t, i, hkv, d, bs):
    return ((b * hkv + h) * d + i) * bs + t


def _brute(b):
    """Double loop; exp without max subtraction; pool read by flat offsets."""
    hq, hkv, d, bs = b.heads.num_q_heads, b.heads.num_kv_heads, b.heads.head_dim, b.heads.block_size
    x = 16 // (2 if b.dtype == "bf16" else 4)
    qv = ref.decode_raw(b.q, b.dtype)
    kn = ref.decode_raw(b.k_new, b.dtype)
    vn = ref.decode_raw(b.v_new, b.dtype)
    kflat = ref.decode_raw(b.k_cache, b.dtype).ravel()
    vflat = ref.decode_raw(b.v_cache, b.dtype).ravel()
    g = hq // hkv
    out = np.zeros(qv.shape)
    lse = np.zeros(qv.shape[:2])
    for s in range(b.num_seqs):
        t0, t1 = int(b.query_start_loc[s]), int(b.query_start_loc[s + 1])
        L = int(b.seq_lens[s])
        P = L - (t1 - t0)
        for i in range(t1 - t0):
            for h in range(hq):
                kh = h // g
                den = 0.0
                num = [0.0] * d
                for j in range(P + i + 1):
                    if j < P:
                        blk = int(b.block_tables[s, j // bs])
                        kj = [kflat[_flat_k(blk, kh, j % bs, c, hkv, d, bs, x)] for c in range(d)]
                        vj = [vflat[_flat_v(blk, kh, j % bs, c, hkv, d, bs)] for c in range(d)]
                    else:
                        kj = list(kn[t0 + j - P, kh])
                        vj = list(vn[t0 + j - P, kh])
                    sc = b.scale * sum(qv[t0 + i, h, c] * kj[c] for c in range(d))
                    w = math.exp(sc)
                    den += w
                    for c in range(d):
                        num[c] += w * vj[c]
                out[t0 + i, h] = [n / den for n in num]
                lse[t0 + i, h] = math.log(den)
    return out, lse


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seed", [0, 1])
def test_brute_force(dtype, seed):
    specs = [SeqSpec(5, 1), SeqSpec(9, 3), SeqSpec(1, 1), SeqSpec(4, 4), SeqSpec(7, 0), SeqSpec(12, 2)]
    b = make_batch(specs, HeadSpec(4, 2, 8, 4), dtype, seed)
    o, lse = run_oracle(b)
    ob, lb = _brute(b)
    np.testing.assert_allclose(o, ob, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lb, rtol=0, atol=1e-12)


# ----------------------------------------------------------------------------
# closed forms


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_context_one_returns_v_exactly(dtype):
    specs = [SeqSpec(1, 1), SeqSpec(1, 1), SeqSpec(1, 1)]
    b = make_batch(specs, HeadSpec(8, 2, 16, 16), dtype, 3)
    o, lse = run_oracle(b)
    v = ref.decode_raw(b.v_new, dtype)
    g = 4
    for h in range(8):
        assert np.array_equal(o[:, h], v[:, h // g])
    # one key: the denominator is exp(score) itself, so lse is the scaled score
    qv = ref.decode_raw(b.q, dtype)
    kv = ref.decode_raw(b.k_new, dtype)
    for h in range(8):
        np.testing.assert_allclose(lse[:, h], b.scale * (qv[:, h] * kv[:, h // g]).sum(-1), rtol=0, atol=1e-14)


def test_zero_query_gives_running_mean():
    specs = [SeqSpec(40, 7), SeqSpec(9, 9), SeqSpec(30, 1)]
    b = make_batch(specs, HeadSpec(4, 4, 16, 8), "f32", 4)
    b.q[:] = 0
    o, lse = run_oracle(b)
    for s in range(3):
        t0, t1 = int(b.query_start_loc[s]), int(b.query_start_loc[s + 1])
        L = int(b.seq_lens[s])
        P = L - (t1 - t0)
        _, vp = ref.gather_kv(b.k_cache, b.v_cache, b.block_tables[s], P, 4, 16, 8, "f32")
        v = np.concatenate([vp, b.v_new[t0:t1].astype(np.float64)])
        cm = np.cumsum(v, axis=0) / np.arange(1, L + 1)[:, None, None]
        np.testing.assert_allclose(o[t0:t1], cm[P:L], rtol=0, atol=1e-13)
        np.testing.assert_allclose(lse[t0:t1], np.log(np.arange(P + 1, L + 1))[:, None] * np.ones(4), atol=1e-13)


def test_identical_keys_give_mean():
    specs = [SeqSpec(33, 1), SeqSpec(20, 5)]
    b = make_batch(specs, HeadSpec(4, 2, 8, 16), "f32", 5, nan_fill=False)
    b.k_cache[:] = 0.5
    b.k_new[:] = 0.5
    o, _ = run_oracle(b)
    for s in range(2):
        t0, t1 = int(b.query_start_loc[s]), int(b.query_start_loc[s + 1])
        L = int(b.seq_lens[s])
        P = L - (t1 - t0)
        _, vp = ref.gather_kv(b.k_cache, b.v_cache, b.block_tables[s], P, 2, 8, 16, "f32")
        v = np.concatenate([vp, b.v_new[t0:t1].astype(np.float64)])
        for i in range(t1 - t0):
            mean = v[: P + i + 1].mean(axis=0)  # [Hkv, d]
            for h in range(4):
                np.testing.assert_allclose(o[t0 + i, h], mean[h // 2], rtol=0, atol=1e-13)


def test_dominant_key_returns_its_value():
    # Orthogonal keys; q = alpha * k_t makes key t's weight 1 - O(L e^{-alpha}).
    d, L, t = 16, 12, 7
    specs = [SeqSpec(L, 1)]
    b = make_batch(specs, HeadSpec(1, 1, d, 4), "f32", 6, scale=1.0)
    keys = np.eye(d, dtype=np.float32)[:L]
    for j in range(L - 1):
        blk = b.block_tables[0, j // 4]
        _put_k(b.k_cache, blk, 0, j % 4, keys[j])
    b.k_new[0, 0] = keys[L - 1]
    for alpha in (20.0, 40.0):
        b.q[0, 0] = alpha * keys[t]
        o, _ = run_oracle(b)
        _, v = ref.gather_kv(b.k_cache, b.v_cache, b.block_tables[0], L - 1, 1, d, 4, "f32")
        assert np.abs(o[0, 0] - v[t, 0]).max() < L * math.exp(-alpha) * 10


# ----------------------------------------------------------------------------
# invariances


def _permute_pool(b, rng):
    """Same logical contents, physical blocks relabelled by a permutation."""
    perm = rng.permutation(b.num_blocks)  # new id of old block i is perm[i]
    inv = np.argsort(perm)
    kc = b.k_cache[inv].copy()
    vc = b.v_cache[inv].copy()
    bt = np.where(b.block_tables >= 0, perm[np.maximum(b.block_tables, 0)], -1).astype(np.int32)
    return kc, vc, bt


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_block_permutation_invariance(dtype):
    specs = [SeqSpec(70, 1), SeqSpec(50, 13), SeqSpec(17, 1), SeqSpec(64, 64)]
    b = make_batch(specs, HeadSpec(4, 2, 16, 16), dtype, 7)
    o1, l1 = run_oracle(b)
    kc, vc, bt = _permute_pool(b, np.random.default_rng(1))
    o2, l2 = ref.attention_reference(b.q, kc, vc, b.k_new, b.v_new, bt, b.seq_lens, b.query_start_loc,
                                     b.scale, 2, 16, dtype)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def _logical_to_pool(kl, vl, bs, dtype, rng):
    """Scatter contiguous per-sequence KV [L, H, d] into a shuffled pool of
    block size bs (test-side writer using the header layout)."""
    hkv, d = kl[0].shape[1], kl[0].shape[2]
    x = 16 // (2 if dtype == "bf16" else 4)
    nbs = [-(-k.shape[0] // bs) for k in kl]
    nb = sum(nbs)
    perm = rng.permutation(nb)
    raw = np.uint16 if dtype == "bf16" else np.float32
    kc = np.zeros((nb, hkv, d // x, bs, x), dtype=raw)
    vc = np.zeros((nb, hkv, d, bs), dtype=raw)
    bt = np.full((len(kl), max(nbs)), -1, np.int32)
    off = 0
    for s, (k, v) in enumerate(zip(kl, vl)):
        for p in range(k.shape[0]):
            blk = perm[off + p // bs]
            bt[s, p // bs] = blk
            kc[blk, :, :, p % bs, :] = k[p].reshape(hkv, d // x, x)
            vc[blk, :, :, p % bs] = v[p]
        off += nbs[s]
    return kc, vc, bt


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_block_size_invariance_and_sdpa(dtype):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(8)
    hq, hkv, d = 8, 2, 16
    ctx = [37, 1, 64, 29]
    qlen = [5, 1, 64, 1]
    raw = np.uint16 if dtype == "bf16" else np.float32

    def draw(shape):
        v = rng.standard_normal(shape, dtype=np.float32)
        return bf16_bits_from_f32(v) if dtype == "bf16" else v

    kl = [draw((c, hkv, d)) for c in ctx]
    vl = [draw((c, hkv, d)) for c in ctx]
    q = draw((sum(qlen), hq, d))
    qsl = np.concatenate([[0], np.cumsum(qlen)]).astype(np.int32)
    seq_lens = np.array(ctx, np.int32)
    k_new = np.concatenate([k[c - n:] for k, c, n in zip(kl, ctx, qlen)]).astype(raw)
    v_new = np.concatenate([v[c - n:] for v, c, n in zip(vl, ctx, qlen)]).astype(raw)
    outs = []
    for bs in (1, 8, 16, 32):
        kc, vc, bt = _logical_to_pool(kl, vl, bs, dtype, rng)
        outs.append(ref.attention_reference(q, kc, vc, k_new, v_new, bt, seq_lens, qsl, 0.25, hkv, bs, dtype))
    for o, l in outs[1:]:
        assert np.array_equal(o, outs[0][0]) and np.array_equal(l, outs[0][1])
    # Library special case: per sequence, torch fp64 SDPA on the contiguous
    # arrays with an explicit bottom-right mask and repeat_interleave groups.
    o0 = outs[0][0]
    for s in range(len(ctx)):
        t0, t1 = qsl[s], qsl[s + 1]
        c, n = ctx[s], qlen[s]
        qt = torch.from_numpy(ref.decode_raw(q[t0:t1], dtype)).permute(1, 0, 2)  # [Hq, n, d]
        kt = torch.from_numpy(ref.decode_raw(kl[s], dtype)).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)
        vt = torch.from_numpy(ref.decode_raw(vl[s], dtype)).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)
        mask = torch.arange(c)[None, :] <= (c - n + torch.arange(n))[:, None]
        st = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=0.25)
        np.testing.assert_allclose(o0[t0:t1], st.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)


def test_split_merge_identity():
    rng = np.random.default_rng(9)
    n, L, d = 6, 90, 16
    q = rng.standard_normal((n, d))
    k = rng.standard_normal((L, d))
    v = rng.standard_normal((L, d))
    prefix = L - n
    lim = prefix + np.arange(n)
    keys = np.arange(L)
    full = ref.softmax_attention(q, k, v, 0.3, keys[None] <= lim[:, None])
    for cuts in ([40], [16, 48, 80], [1, 2, 83]):
        edges = [0] + cuts + [L]
        parts = []
        for a, c in zip(edges[:-1], edges[1:]):
            vis = (keys[None] <= lim[:, None]) & (keys[None] >= a) & (keys[None] < c)
            assert vis.any(axis=1).all()
            parts.append(ref.softmax_attention(q, k, v, 0.3, vis))
        o, l = ref.lse_merge(parts)
        np.testing.assert_allclose(o, full[0], rtol=0, atol=1e-12)
        np.testing.assert_allclose(l, full[1], rtol=0, atol=1e-12)


def test_row_independence():
    specs = [SeqSpec(40, 1), SeqSpec(64, 16), SeqSpec(23, 1), SeqSpec(19, 3)]
    b = make_batch(specs, HeadSpec(4, 2, 16, 16), "bf16", 10)
    o, l = run_oracle(b)
    for s in range(len(specs)):
        t0, t1 = b.query_start_loc[s], b.query_start_loc[s + 1]
        os_, ls = ref.attention_reference(
            b.q[t0:t1], b.k_cache, b.v_cache, b.k_new[t0:t1], b.v_new[t0:t1], b.block_tables[s:s + 1],
            b.seq_lens[s:s + 1], np.array([0, t1 - t0], np.int32), b.scale, 2, 16, "bf16")
        assert np.array_equal(os_, o[t0:t1]) and np.array_equal(ls, l[t0:t1])


# ----------------------------------------------------------------------------
# append


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_append_reference(dtype):
    specs = [SeqSpec(70, 1), SeqSpec(50, 13), SeqSpec(17, 0), SeqSpec(64, 64), SeqSpec(33, 2)]
    hq, hkv, d, bs = 4, 2, 16, 16
    b = make_batch(specs, HeadSpec(hq, hkv, d, bs), dtype, 11)
    kc, vc = ref.append_reference(b.k_cache, b.v_cache, b.k_new, b.v_new, b.block_tables, b.seq_lens,
                                  b.query_start_loc, bs, dtype)
    x = 16 // (2 if dtype == "bf16" else 4)
    touched_k = np.zeros(kc.size, bool)
    touched_v = np.zeros(vc.size, bool)
    kflat, vflat = kc.ravel(), vc.ravel()
    for s, sp in enumerate(specs):
        t0 = int(b.query_start_loc[s])
        for i in range(sp.q_len):
            p = sp.ctx - sp.q_len + i
            blk = int(b.block_tables[s, p // bs])
            for h in range(hkv):
                for c in range(d):
                    fk = _flat_k(blk, h, p % bs, c, hkv, d, bs, x)
                    fv = _flat_v(blk, h, p % bs, c, hkv, d, bs)
                    assert kflat[fk].tobytes() == b.k_new[t0 + i, h, c].tobytes()
                    assert vflat[fv].tobytes() == b.v_new[t0 + i, h, c].tobytes()
                    touched_k[fk] = touched_v[fv] = True
    assert kc.ravel()[~touched_k].tobytes() == b.k_cache.ravel()[~touched_k].tobytes()
    assert vc.ravel()[~touched_v].tobytes() == b.v_cache.ravel()[~touched_v].tobytes()
    # Attending over the appended pool with no new tokens gives the same rows.
    o1, l1 = run_oracle(b)
    for s, sp in enumerate(specs):
        if sp.q_len == 0:
            continue
        k, v = ref.gather_kv(kc, vc, b.block_tables[s], sp.ctx, hkv, d, bs, dtype)
        t0 = int(b.query_start_loc[s])
        o2, l2 = ref.sequence_attention(ref.decode_raw(b.q[t0:t0 + sp.q_len], dtype), k, v,
                                        sp.ctx - sp.q_len, b.scale, hkv)
        assert np.array_equal(o2, o1[t0:t0 + sp.q_len]) and np.array_equal(l2, l1[t0:t0 + sp.q_len])


# ----------------------------------------------------------------------------
# bf16 handling (decode in the oracle, round-to-nearest-even in the generator)


def test_bf16_decode_and_rounding():
    bits = np.array([0x3F80, 0xC000, 0x7F80, 0x0001, 0x8000], np.uint16)
    got = ref.decode_raw(bits, "bf16")
    assert list(got[:3]) == [1.0, -2.0, math.inf]
    assert got[3] == 2.0 ** -133 and got[4] == 0.0 and math.copysign(1, got[4]) < 0
    ties = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), np.nan], np.float32)
    r = bf16_bits_from_f32(ties)
    assert list(r[:3]) == [0x3F80, 0x3F82, 0xBF80] and r[3] == 0x7FC0
    torch = pytest.importorskip("torch")
    x = np.random.default_rng(12).standard_normal(100000, dtype=np.float32) * 100
    tb = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf16_bits_from_f32(x), tb)


def test_round_bf16_ties_carries_and_nan():
    """The oracle's float32 -> bf16 rounding (used for the rotary output),
    against values worked out by hand from round-to-nearest-even on the top
    16 bits of the float32 pattern, and against torch's conversion."""
    pat = np.array([
        0x3F808000,  # 1 + 2^-8: a tie, the even pattern 0x3F80 stays
        0x3F818000,  # 1 + 3*2^-8: a tie, up to the even 0x3F82
        0xBF808000,  # -(1 + 2^-8): a tie, the sign kept
        0x3F808008,  # just above the tie of 1 + 2^-8: up
        0x3F807FFF,  # just below it: down
        0x3F7F8000,  # 1 - 2^-9: a tie from the odd 0x3F7F, carries into the exponent (1.0)
        0x3FFFFFFF,  # just under 2: carries into the exponent (2.0)
        0x00008000,  # a subnormal tie: to +0
        0x00018000,  # a subnormal tie from an odd pattern: up to 0x0002
        0x7F7FFFFF,  # the largest float32: past the largest bf16, to +inf
        0xFF800000,  # -inf stays
        0x7F800001,  # a signalling NaN whose payload sits in the low bits only: stays a NaN
        0xFFC00000,  # a negative quiet NaN
    ], np.uint32)
    got = ref.round_bf16(pat.view(np.float32))
    assert got.tolist() == [0x3F80, 0x3F82, 0xBF80, 0x3F81, 0x3F80, 0x3F80, 0x4000, 0x0000, 0x0002, 0x7F80, 0xFF80,
                            0x7FC0, 0xFFC0]
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(13)
    x = (rng.standard_normal(100000) * 100).astype(np.float32)
    ties = (rng.integers(0, 0x7F000000, size=20000, dtype=np.uint32) & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    ties |= (rng.random(20000) < 0.5).astype(np.uint32) << np.uint32(31)
    x = np.concatenate([x, ties.view(np.float32)])
    tb = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ref.round_bf16(x), tb)


# ----------------------------------------------------------------------------
# rotary position embedding (the append step's optional rotation)


def theta_table(max_pos, rope_dim, base=10000.0):
    """The standard rotary angle table, cos/sin of p * base^(-2j/R), in float64
    then stored as float32 (what a caller hands the library)."""
    j = np.arange(rope_dim // 2)
    ang = np.arange(max_pos)[:, None] * base ** (-2.0 * j / rope_dim)[None, :]
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1).astype(np.float32)


def test_rope_hand_worked():
    # d = R = 8, one angle with cos 1/2 and sin 1/4 (both exact in binary):
    # pairs (j, j+4): y_j = x_j/2 - x_{j+4}/4, y_{j+4} = x_{j+4}/2 + x_j/4
    x = np.arange(1, 9, dtype=np.float32).reshape(1, 1, 8)
    cs = np.tile(np.array([0.5, 0.25], np.float32), (1, 4, 1))
    y = ref.rope_reference(x, [0], cs, 8, "f32")
    assert y.ravel().tolist() == [-0.75, -0.5, -0.25, 0.0, 2.75, 3.5, 4.25, 5.0]
    # rope_dim 4 of d 8: pairs (0, 2), (1, 3); dims 4..7 pass through
    y = ref.rope_reference(x, [0], cs[:, :2], 4, "f32")
    assert y.ravel().tolist() == [1 * .5 - 3 * .25, 2 * .5 - 4 * .25, 3 * .5 + 1 * .25, 4 * .5 + 2 * .25,
                                  5, 6, 7, 8]


def test_rope_bf16_rounding_hand_worked():
    """A bf16 rotation whose float32 products, sum and bf16 result all need
    rounding, worked by hand (R = d = 2: one pair, x = (3, 5); the table holds
    float32 0.6 and 0.8):
      c = fl(0.6) = 10066330 * 2^-24, s = fl(0.8) = 13421773 * 2^-24;
      fl(3c) = 15099495 * 2^-23 (exact), fl(5s) = 4 (67108865 * 2^-24 rounded);
      y0 = fl(fl(3c) - 4) = -18454937 * 2^-23, a float32 tie, to -9227468 * 2^-22;
           bf16: 140.8 units of 2^-6, so -141 * 2^-6 = -2.203125 (0xC00D);
      fl(5c) = 3 (50331650 * 2^-24, a tie to even), fl(3s) = 10066330 * 2^-22;
      y1 = 3 + fl(3s) = 11324621 * 2^-21, exact; bf16: 172.8 units of 2^-5,
           so 173 * 2^-5 = 5.40625 (0x40AD).
    And with the table (1 + 2^-8, 2^-9) on x = (1, 1): y0 = 1 + 2^-9 rounds
    down to 1.0 (0x3F80), y1 = 1 + 3 * 2^-9 up to 1 + 2^-7 (0x3F81)."""
    x = np.array([[[0x4040, 0x40A0]], [[0x3F80, 0x3F80]]], np.uint16)
    cs = np.array([[[0.6, 0.8]], [[1 + 2 ** -8, 2 ** -9]]], np.float32)
    y = ref.rope_reference(x, [0, 1], cs, 2, "bf16")
    assert y.reshape(2, 2).tolist() == [[0xC00D, 0x40AD], [0x3F80, 0x3F81]]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_rope_zero_and_quarter_turn(dtype):
    rng = np.random.default_rng(40)
    x32 = rng.standard_normal((5, 3, 64)).astype(np.float32)
    raw = bf16_bits_from_f32(x32) if dtype == "bf16" else x32
    zero = np.tile(np.array([1.0, 0.0], np.float32), (1, 32, 1))
    assert np.array_equal(ref.rope_reference(raw, [0] * 5, zero, 64, dtype), raw)
    quarter = np.tile(np.array([0.0, 1.0], np.float32), (1, 32, 1))
    y = ref.decode_raw(ref.rope_reference(raw, [0] * 5, quarter, 64, dtype), dtype)
    x = ref.decode_raw(raw, dtype)
    assert np.array_equal(y[..., :32], -x[..., 32:]) and np.array_equal(y[..., 32:], x[..., :32])


def test_rope_preserves_pair_norms_and_relative_position():
    rng = np.random.default_rng(41)
    d, rd = 128, 96
    tab = theta_table(4096, rd)
    q = rng.standard_normal((1, 1, d)).astype(np.float32)
    k = rng.standard_normal((1, 1, d)).astype(np.float32)
    yq = ref.rope_reference(q, [777], tab, rd, "f32").astype(np.float64)
    # each rotated pair keeps its length (up to float32 rounding); dims >= R pass
    n0 = q[0, 0, :rd // 2] ** 2 + q[0, 0, rd // 2:rd] ** 2
    n1 = yq[0, 0, :rd // 2] ** 2 + yq[0, 0, rd // 2:rd] ** 2
    assert np.allclose(n1, n0, rtol=1e-6) and np.array_equal(yq[0, 0, rd:], q[0, 0, rd:])
    # q.k after rotation depends on the position difference only
    dots = [float(ref.rope_reference(q, [p], tab, rd, "f32").astype(np.float64).ravel()
                  @ ref.rope_reference(k, [p - 300], tab, rd, "f32").astype(np.float64).ravel())
            for p in (300, 1000, 3000)]
    assert np.allclose(dots, dots[0], rtol=1e-5, atol=1e-5)
    # ... and does change with it
    other = float(ref.rope_reference(q, [1000], tab, rd, "f32").astype(np.float64).ravel()
                  @ ref.rope_reference(k, [1000 - 301], tab, rd, "f32").astype(np.float64).ravel())
    assert abs(other - dots[0]) > 1e-3


def test_rope_positions_of_new_tokens():
    pos = ref.new_token_positions([5, 9, 3], [0, 1, 4, 4])
    assert pos.tolist() == [4, 6, 7, 8]


# ----------------------------------------------------------------------------
# fp8 (OCP E4M3) cache codes


def test_e4m3_table_fixed_points():
    v = ref.e4m3_values()
    # from the format's definition: bias 7, 3 mantissa bits, S.1111.111 NaN
    assert v[0x38] == 1.0 and v[0xB8] == -1.0 and v[0x7E] == 448.0 and v[0xFE] == -448.0
    assert v[0x01] == 2.0 ** -9 and v[0x07] == 7 * 2.0 ** -9 and v[0x08] == 2.0 ** -6
    assert v[0x3C] == 1.5 and v[0x40] == 2.0 and v[0x30] == 0.5
    assert v[0x00] == 0.0 and v[0x80] == 0.0 and math.copysign(1, v[0x80]) < 0
    assert np.isnan(v[0x7F]) and np.isnan(v[0xFF]) and np.isfinite(np.delete(v, [0x7F, 0xFF])).all()


def test_e4m3_quantize_round_trip_ties_and_saturation():
    v = ref.e4m3_values()
    finite = np.array([c for c in range(256) if not np.isnan(v[c])], np.uint8)
    assert np.array_equal(ref.quantize_e4m3(v[finite].astype(np.float32)), finite)  # every code reproduces
    x = np.array([1 + 1 / 16, 1 + 3 / 16, 7.5 * 2 ** -9, 0.5 * 2 ** -9, 1.5 * 2 ** -9, 464, 463.99, 1e6, -1e6,
                  -2 ** -12], np.float32)
    # ties to the even mantissa (also at the subnormal/normal seam and at 0),
    # saturation at +-448, and the sign kept on an underflow to zero
    assert ref.quantize_e4m3(x).tolist() == [0x38, 0x3A, 0x08, 0x00, 0x02, 0x7E, 0x7E, 0x7E, 0xFE, 0x80]
    y = np.sort(np.random.default_rng(50).standard_normal(20000).astype(np.float32) * 100)
    c = ref.quantize_e4m3(y)
    assert np.all(np.diff(v[c]) >= 0)  # monotone


def test_fp8_codes_scale_direction_and_round_trip():
    """fp8_codes stores x * (1 / scale).  Hand-worked: 1.0 at scale 0.5 is
    2.0 = 1.0 * 2^1 (exponent field 8: 0x40); 1.0 at scale 2 is 0.5 (0x30);
    3.0 at scale 0.25 is 12 = 1.5 * 2^3 (0x54); 1.0 at scale fl(0.3) is
    3.3333333, nearer 3.25 = 1.625 * 2 (0x45) than 3.5; -1.0 at scale 0.5 is
    -2.0 (0xC0).  Then every finite code c survives the trip through its
    value times a non-unit scale, rounded to bf16: codes are 2^-4 apart
    relative to their value (2^-9 absolute below 2^-6), far wider than the
    2^-9 relative error of the bf16 rounding."""
    one, three, minus = 0x3F80, 0x4040, 0xBF80
    assert ref.fp8_codes(np.array([one], np.uint16), 0.5).tolist() == [0x40]
    assert ref.fp8_codes(np.array([one], np.uint16), 2.0).tolist() == [0x30]
    assert ref.fp8_codes(np.array([three], np.uint16), 0.25).tolist() == [0x54]
    assert ref.fp8_codes(np.array([one], np.uint16), 0.3).tolist() == [0x45]
    assert ref.fp8_codes(np.array([minus], np.uint16), 0.5).tolist() == [0xC0]
    v = ref.e4m3_values()
    finite = np.array([c for c in range(256) if not np.isnan(v[c])], np.uint8)
    for scale in (0.5, 0.0173, 3.7):
        x = bf16_bits_from_f32((v[finite] * scale).astype(np.float32))
        assert np.array_equal(ref.fp8_codes(x, scale), finite), scale


def test_e4m3_matches_torch_in_range():
    torch = pytest.importorskip("torch")
    if not hasattr(torch, "float8_e4m3fn"):
        pytest.skip("torch without float8_e4m3fn")
    x = np.random.default_rng(51).standard_normal(200000).astype(np.float32) * np.float32(60.0)
    x = x[np.abs(x) < 440]
    t = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(ref.quantize_e4m3(x), t)


def test_fp8_attention_is_attention_on_the_scaled_codes():
    """The fp8 path is ordinary attention on code value * scale, with the new
    tokens entering as the codes the append stores."""
    rng = np.random.default_rng(52)
    hkv, d, bs = 2, 64, 16
    specs = [(70, 1), (40, 5)]
    nb = sum(-(-c // bs) for c, _ in specs)
    qsl = np.concatenate([[0], np.cumsum([ql for _, ql in specs])]).astype(np.int32)
    t = int(qsl[-1])
    q = bf16_bits_from_f32(rng.standard_normal((t, 4, d), dtype=np.float32))
    kn = bf16_bits_from_f32(rng.standard_normal((t, hkv, d), dtype=np.float32))
    vn = bf16_bits_from_f32(rng.standard_normal((t, hkv, d), dtype=np.float32))
    kc = rng.integers(0, 0x7E, size=(nb, hkv, d // 8, bs, 8)).astype(np.uint8)
    vc = rng.integers(0, 0x7E, size=(nb, hkv, d, bs)).astype(np.uint8)
    kc |= (rng.random(kc.shape) < 0.5).astype(np.uint8) << 7
    bt = np.arange(nb, dtype=np.int32).reshape(1, -1).repeat(2, 0)
    bt[1] = np.roll(bt[1], 3)
    sl = np.array([c for c, _ in specs], np.int32)
    ks, vs = 0.0173, 0.0211
    o8, l8 = ref.attention_reference(q, kc, vc, kn, vn, bt, sl, qsl, 0.125, hkv, bs, "fp8", k_scale=ks, v_scale=vs)
    # the same through the f32 path, on the dequantized pool and new rows
    kc32 = (ref.e4m3_values()[kc] * ks).astype(np.float32)
    vc32 = (ref.e4m3_values()[vc] * vs).astype(np.float32)
    kc32 = kc32.reshape(nb, hkv, d // 8, bs, 2, 4).transpose(0, 1, 2, 4, 3, 5).reshape(nb, hkv, d // 4, bs, 4)
    kn32 = (ref.e4m3_values()[ref.fp8_codes(kn, ks)] * ks).astype(np.float32)
    vn32 = (ref.e4m3_values()[ref.fp8_codes(vn, vs)] * vs).astype(np.float32)
    q32 = ref.decode_raw(q, "bf16").astype(np.float32)
    o32, l32 = ref.attention_reference(q32, kc32, vc32, kn32, vn32, bt, sl, qsl, 0.125, hkv, bs, "f32")
    assert np.allclose(o8, o32, atol=1e-6) and np.allclose(l8, l32, atol=1e-6)
    # and the append stores exactly those codes
    kc2, vc2 = ref.append_reference(kc, vc, kn, vn, bt, sl, qsl, bs, "fp8", k_scale=ks, v_scale=vs)
    pos = ref.new_token_positions(sl, qsl)
    seq = np.repeat(np.arange(2), np.diff(qsl))
    blk = bt[seq, pos // bs]
    assert np.array_equal(kc2.reshape(nb, hkv, d // 8, bs, 8)[blk, :, :, pos % bs, :].reshape(t, hkv, d),
                          ref.fp8_codes(kn, ks))
