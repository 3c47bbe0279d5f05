"""CPU oracle for one mixed prefill+decode step over a paged KV cache.

TEST INFRASTRUCTURE ONLY.  The tests, the smoke check and the benchmark's
CPU-baseline leg call this module; the library and its Python binding never
import it, and it imports nothing of theirs.  It is plain, slow numpy in
float64.

What the step computes.  The paper (section 2.1) describes prefill as
materialising the KV cache of the input tokens and decode as producing one
token per running sequence while re-reading an expanding KV cache; section 4.4
has the decode node reuse a resident (radix-cached) prefix and process the
remaining prompt tokens; section 5 co-batches those prefill chunks with the
running decode rows in one mixed batch.  The paper never writes the attention
formula, so the oracle is the textbook definition of scaled dot-product
softmax attention with these readings of what the paper leaves unsaid:

* a sequence with KV length ``L`` (after the append) and ``C`` new tokens has
  a cached prefix ``P = L - C``; new token ``i`` sits at logical position
  ``P + i`` and sees keys ``0 .. P + i`` inclusive (bottom-right causal);
  a decode row is the case ``C = 1``;
* query head ``h`` reads KV head ``h // G`` with ``G = Hq / Hkv`` (contiguous
  groups);
* the softmax scale is a parameter (the tests use ``1 / sqrt(head_dim)``);
* the step appends first and attends second, so the oracle gathers each
  sequence's keys from the pool as it was *before* the append, plus this
  step's ``k_new`` / ``v_new`` rows for positions ``P .. L - 1``.

The step may also rotate the new queries and keys by their positions before
the append (the rotary embedding, ``rope_reference``); the paper describes
neither its models' position encoding nor such a kernel, so that function is
the standard rotate-half definition with the rounding spelled out.

The KV cache may also hold fp8 codes (OCP E4M3 with one scale per tensor,
dtype "fp8"; queries, new rows and outputs stay bf16).  The paper is silent
on cache precision; the reading is that a value x is stored as the E4M3
code nearest to x / scale (ties to even, saturating at 448; ``fp8_codes``)
and read back as code value * scale.  With both (rotation and an fp8
cache), the rows are rotated as bf16 rows and the rotated key is then
stored as any new key is: ``fp8_codes`` of the ``rope_reference`` result.

Cache layout read here (the library header's definition), with
``X = 8`` elements (bf16, fp8) or 4 (f32): K element (block b, head h, slot t, dim i) is at
``[b][h][i // X][t][i % X]``; V element (b, h, t, i) is at ``[b][h][i][t]``.
bf16 values arrive as their 16-bit patterns.
"""

from __future__ import annotations

import numpy as np

ELEM_BYTES = {"bf16": 2, "f32": 4, "fp8": 1}
CHUNK = {"bf16": 8, "f32": 4, "fp8": 8}  # X: elements per K chunk of the cache layout


def e4m3_values() -> np.ndarray:
    """The 256 codes of OCP FP8 E4M3 (e4m3fn) as float64: sign in bit 7, a
    4-bit exponent with bias 7 and a 3-bit mantissa; exponent 0 holds the
    subnormals m * 2^-9; S.1111.111 is NaN and there is no infinity, so the
    largest finite magnitude is 1.75 * 2^8 = 448."""
    codes = np.arange(256)
    e = (codes >> 3) & 0xF
    m = codes & 7
    v = np.where(e == 0, m * 2.0 ** -9, (1 + m / 8.0) * 2.0 ** (e - 7.0))
    v = np.where(codes & 0x80, -v, v)
    v[(codes & 0x7F) == 0x7F] = np.nan
    return v


def quantize_e4m3(y32: np.ndarray) -> np.ndarray:
    """float32 -> E4M3 codes: the nearest finite value, a tie going to the
    code with the even mantissa, magnitudes past 448 to 448 (saturating), NaN
    to the NaN pattern; the sign is kept (so -0 -> 0x80)."""
    y32 = np.asarray(y32, dtype=np.float32)
    vals = e4m3_values()[:0x7F]  # +0 .. 448, increasing
    a = np.abs(y32.astype(np.float64))
    hi = np.clip(np.searchsorted(vals, a), 0, 0x7E)
    lo = np.clip(hi - 1, 0, 0x7E)
    dlo, dhi = a - vals[lo], vals[hi] - a
    pick = np.where(dlo < dhi, lo, np.where(dhi < dlo, hi, np.where(lo % 2 == 0, lo, hi)))
    pick = np.where(a >= 448.0, 0x7E, pick)
    code = pick | np.where(np.signbit(y32), 0x80, 0)
    code = np.where(np.isnan(y32), 0x7F | np.where(np.signbit(y32), 0x80, 0), code)
    return code.astype(np.uint8)


def fp8_codes(x_raw_bf16: np.ndarray, scale: float) -> np.ndarray:
    """The cache codes of bf16 values under a per-tensor scale: x * (1/scale),
    the reciprocal and the product each rounded to float32, then
    quantize_e4m3."""
    inv = np.float32(1.0) / np.float32(scale)
    return quantize_e4m3(decode_raw(x_raw_bf16, "bf16").astype(np.float32) * inv)


def decode_raw(raw: np.ndarray, dtype: str) -> np.ndarray:
    """Raw storage -> float64.  A bf16 pattern is the top half of a float32;
    an fp8 code is an E4M3 value (before its tensor's scale)."""
    if dtype == "fp8":
        return e4m3_values()[np.asarray(raw, dtype=np.uint8)]
    if dtype == "bf16":
        u = np.ascontiguousarray(raw, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(raw, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def _x(dtype: str) -> int:
    return CHUNK[dtype]


def gather_kv(k_cache, v_cache, block_row, n_tokens, num_kv_heads, head_dim, block_size, dtype):
    """Logical positions 0 .. n_tokens-1 of one sequence, as float64
    ``[n_tokens, Hkv, d]`` arrays: position p is slot ``p % bs`` of physical
    block ``block_row[p // bs]``."""
    if n_tokens == 0:
        z = np.zeros((0, num_kv_heads, head_dim))
        return z, z.copy()
    x = _x(dtype)
    nb = -(-n_tokens // block_size)
    blocks = np.asarray(block_row[:nb], dtype=np.int64)
    kb = k_cache.reshape(-1, num_kv_heads, head_dim // x, block_size, x)[blocks]
    vb = v_cache.reshape(-1, num_kv_heads, head_dim, block_size)[blocks]
    # [nb, H, d/X, bs, X] -> [nb, bs, H, d/X, X] -> [nb*bs, H, d]
    k = decode_raw(kb, dtype).transpose(0, 3, 1, 2, 4).reshape(nb * block_size, num_kv_heads, head_dim)
    # [nb, H, d, bs] -> [nb, bs, H, d]
    v = decode_raw(vb, dtype).transpose(0, 3, 1, 2).reshape(nb * block_size, num_kv_heads, head_dim)
    return k[:n_tokens], v[:n_tokens]


def softmax_attention(q, k, v, scale, visible):
    """Scaled dot-product attention for one head.

    q [n, d], k [L, d], v [L, d] float64; ``visible`` [n, L] bool says which
    keys each query row may attend.  Every row must see at least one key.
    Returns (o [n, d], lse [n]) with lse the natural log of the softmax
    denominator of the scaled scores.  The row maximum is subtracted before
    exponentiating; the masked scores are removed by selection."""
    # Contiguous operands, so the result depends on the values only and not
    # on the strides a gather happened to produce.
    q, k, v = (np.ascontiguousarray(a, dtype=np.float64) for a in (q, k, v))
    s = scale * (q @ k.T)
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    l = e.sum(axis=1, keepdims=True)
    o = (e @ v) / l
    return o, (m + np.log(l))[:, 0]


def lse_merge(parts):
    """Combine attention results over disjoint key sets.

    ``parts`` is a list of (o [n, d], lse [n]).  Softmax over the union of the
    key sets re-weights each part by its share of the total denominator,
    exp(lse_j - lse), with lse = log(sum_j exp(lse_j))."""
    lses = np.stack([p[1] for p in parts])  # [J, n]
    top = lses.max(axis=0)
    w = np.exp(lses - top)  # [J, n]
    total = w.sum(axis=0)
    o = sum(w[j][:, None] * parts[j][0] for j in range(len(parts))) / total[:, None]
    return o, top + np.log(total)


def sequence_attention(q_rows, k, v, prefix, scale, num_kv_heads, row_tile=512, rows=None):
    """All query heads of one sequence.

    q_rows [C, Hq, d]; k, v [L, Hkv, d] with L = prefix + C.  Row i sits at
    position prefix + i and sees keys 0 .. prefix + i.  ``rows`` (optional)
    restricts the result to those row indices, in that order."""
    c, hq, d = q_rows.shape
    big_l = k.shape[0]
    g = hq // num_kv_heads
    rows = np.arange(c) if rows is None else np.asarray(rows)
    n = len(rows)
    o = np.empty((n, hq, d))
    lse = np.empty((n, hq))
    keys = np.arange(big_l)
    kh = [np.ascontiguousarray(k[:, j]) for j in range(num_kv_heads)]
    vh = [np.ascontiguousarray(v[:, j]) for j in range(num_kv_heads)]
    for r0 in range(0, n, row_tile):
        r1 = min(n, r0 + row_tile)
        rr = rows[r0:r1]
        visible = keys[None, :] <= (prefix + rr)[:, None]
        for h in range(hq):
            o[r0:r1, h], lse[r0:r1, h] = softmax_attention(q_rows[rr, h], kh[h // g], vh[h // g], scale, visible)
    return o, lse


def attention_reference(
    q,
    k_cache,
    v_cache,
    k_new,
    v_new,
    block_tables,
    seq_lens,
    query_start_loc,
    scale,
    num_kv_heads,
    block_size,
    dtype,
    seqs=None,
    k_scale=1.0,
    v_scale=1.0,
):
    """Outputs of one mixed step.

    Raw inputs in the library's layouts; the caches are the pool *before* the
    step's append.  Returns (out [T, Hq, d], lse [T, Hq]) float64; rows of
    sequences not in ``seqs`` (default: all) are NaN.

    dtype "fp8": q, k_new and v_new are bf16 and the caches hold E4M3 codes
    with per-tensor scales; attention sees code value * scale, for the new
    tokens too (their codes as the append writes them, fp8_codes)."""
    qd = "bf16" if dtype == "fp8" else dtype
    qf = decode_raw(q, qd)
    t, hq, d = qf.shape
    out = np.full((t, hq, d), np.nan)
    lse = np.full((t, hq), np.nan)
    seq_lens = np.asarray(seq_lens)
    qsl = np.asarray(query_start_loc)
    todo = range(len(seq_lens)) if seqs is None else seqs
    for s in todo:
        t0, t1 = int(qsl[s]), int(qsl[s + 1])
        c = t1 - t0
        if c == 0:
            continue
        big_l = int(seq_lens[s])
        prefix = big_l - c
        kp, vp = gather_kv(k_cache, v_cache, block_tables[s], prefix, num_kv_heads, d, block_size, dtype)
        if dtype == "fp8":
            kn = decode_raw(fp8_codes(k_new[t0:t1], k_scale), "fp8")
            vn = decode_raw(fp8_codes(v_new[t0:t1], v_scale), "fp8")
            k = np.concatenate([kp, kn], axis=0) * k_scale
            v = np.concatenate([vp, vn], axis=0) * v_scale
        else:
            k = np.concatenate([kp, decode_raw(k_new[t0:t1], dtype)], axis=0)
            v = np.concatenate([vp, decode_raw(v_new[t0:t1], dtype)], axis=0)
        out[t0:t1], lse[t0:t1] = sequence_attention(qf[t0:t1], k, v, prefix, scale, num_kv_heads)
    return out, lse


def append_reference(k_cache, v_cache, k_new, v_new, block_tables, seq_lens, query_start_loc, block_size, dtype,
                     k_scale=1.0, v_scale=1.0):
    """The pool after the step's append, as raw copies of the inputs.

    Token i of sequence s goes to logical position P_s + i, i.e. slot
    ``(P_s + i) % bs`` of block ``block_tables[s][(P_s + i) // bs]``; its bits
    are copied unchanged (dtype "fp8": its fp8_codes are stored).  Nothing
    else in the pool changes."""
    if dtype == "fp8":
        k_new, v_new = fp8_codes(k_new, k_scale), fp8_codes(v_new, v_scale)
    x = _x(dtype)
    kc = k_cache.copy()
    vc = v_cache.copy()
    t, hkv, d = k_new.shape
    k5 = kc.reshape(-1, hkv, d // x, block_size, x)
    v4 = vc.reshape(-1, hkv, d, block_size)
    qsl = np.asarray(query_start_loc)
    for s in range(len(seq_lens)):
        t0, t1 = int(qsl[s]), int(qsl[s + 1])
        if t1 == t0:
            continue
        pos = int(seq_lens[s]) - (t1 - t0) + np.arange(t1 - t0)
        blk = np.asarray(block_tables[s])[pos // block_size]
        slot = pos % block_size
        k5[blk, :, :, slot, :] = k_new[t0:t1].reshape(t1 - t0, hkv, d // x, x)
        v4[blk, :, :, slot] = v_new[t0:t1]
    return kc, vc


def round_bf16(x32: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest, ties to even; NaN stays
    a (quiet) NaN."""
    x32 = np.ascontiguousarray(x32, dtype=np.float32)
    u = x32.view(np.uint32).astype(np.uint64)
    r = ((u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(x32)
    r[nan] = ((x32.view(np.uint32)[nan] >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16)
    return r


def rope_reference(x_raw, positions, cos_sin, rope_dim, dtype):
    """Rotary position embedding of rows ``x [T, H, d]`` (raw storage), row t
    at position ``positions[t]``, in the rotate-half form over the first
    ``rope_dim`` dimensions.

    The paper describes neither its models' position encoding nor a fused
    kernel; this is the standard rotary embedding, applied where the step
    writes new keys (and to the queries).  With R = rope_dim, for j < R/2 and
    the caller's angle table ``cos_sin[p, j] = (cos, sin)``:

        y[j]       = x[j] * cos - x[j + R/2] * sin
        y[j + R/2] = x[j + R/2] * cos + x[j] * sin

    and ``y[i] = x[i]`` for i >= R.  Every product and the sum are rounded to
    float32 (no fused multiply-add) and the result is rounded to the storage
    type (bf16: nearest even), so that the float32 rounding that decides
    each stored code is the same on both sides.  Returns raw storage."""
    x = decode_raw(x_raw, dtype).astype(np.float32)  # exact: inputs are bf16 or f32
    t, h, d = x.shape
    half = rope_dim // 2
    cs = np.asarray(cos_sin, dtype=np.float32)[np.asarray(positions)]  # [T, R/2, 2]
    c = cs[:, None, :, 0]
    s = cs[:, None, :, 1]
    x1, x2 = x[:, :, :half], x[:, :, half:rope_dim]
    y = x.copy()
    with np.errstate(over="ignore", invalid="ignore"):
        y[:, :, :half] = (x1 * c).astype(np.float32) - (x2 * s).astype(np.float32)
        y[:, :, half:rope_dim] = (x2 * c).astype(np.float32) + (x1 * s).astype(np.float32)
    if dtype == "bf16":
        return round_bf16(y)
    return y


def new_token_positions(seq_lens, query_start_loc):
    """Position P_s + i of every new token (row of q / k_new)."""
    qsl = np.asarray(query_start_loc)
    pos = np.zeros(int(qsl[-1]), dtype=np.int64)
    for s in range(len(seq_lens)):
        t0, t1 = int(qsl[s]), int(qsl[s + 1])
        pos[t0:t1] = int(seq_lens[s]) - (t1 - t0) + np.arange(t1 - t0)
    return pos
