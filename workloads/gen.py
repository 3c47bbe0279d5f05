"""Seeded host-side generator for one mixed prefill+decode step.

A step is a list of sequences.  Sequence ``s`` has a KV length ``ctx`` (after
this step's append) and ``q_len`` new query tokens, which sit at the logical
positions ``ctx - q_len .. ctx - 1``.  ``q_len == 1`` is a decode row;
``q_len > 1`` is a prefill chunk on a cached prefix of ``ctx - q_len`` tokens
(the paper, section 4.4: the decode node reuses the resident prefix and runs
the remaining prompt tokens; section 5: those chunks are co-batched with the
running decode rows).

Draw order for one seed: lengths, prefill parameters (both in ``configs``),
then the block-pool permutation, then values.  Values are i.i.d. N(0, 1)
float32, rounded to bf16 with round-to-nearest-even for bf16 runs.  Every pool
slot that the step must not read before its own append -- unreferenced blocks,
the slots this step appends to, and the slots past ``ctx`` in a sequence's last
block -- holds NaN, so a kernel that reads one shows it in its output.

dtype "fp8" is an fp8 KV cache (OCP E4M3 codes, one scale per tensor) next to
bf16 queries and new rows: the pool's values are N(0, 1) divided by the
tensor's scale and mapped to the nearest code (the sentinel is the NaN code
0x7F).

Cache layout (the one ``include/mpa.h`` defines; the paper is silent on it),
with ``X`` elements per K chunk (8 for bf16 and fp8, 4 for fp32):

* K: ``[num_blocks][num_kv_heads][head_dim / X][block_size][X]``
* V: ``[num_blocks][num_kv_heads][head_dim][block_size]``
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

ELEM_BYTES = {"bf16": 2, "f32": 4, "fp8": 1}
RAW_DTYPE = {"bf16": np.uint16, "f32": np.float32, "fp8": np.uint8}
CHUNK = {"bf16": 8, "f32": 4, "fp8": 8}
BF16_NAN = np.uint16(0x7FC0)
FP8_NAN = np.uint8(0x7F)
# per-tensor scales of the fp8 pools: the largest code (448) covers 6.3 and
# 7.5 standard deviations of the N(0, 1) values
FP8_K_SCALE = 0.0141
FP8_V_SCALE = 0.0167


@dataclass(frozen=True)
class SeqSpec:
    ctx: int  # KV length after this step's append
    q_len: int  # new query tokens this step


@dataclass(frozen=True)
class HeadSpec:
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int = 16


def _x(dtype: str) -> int:
    return CHUNK[dtype]


def k_cache_shape(num_blocks: int, heads: HeadSpec, dtype: str):
    x = _x(dtype)
    return (num_blocks, heads.num_kv_heads, heads.head_dim // x, heads.block_size, x)


def v_cache_shape(num_blocks: int, heads: HeadSpec, dtype: str):
    return (num_blocks, heads.num_kv_heads, heads.head_dim, heads.block_size)


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns, round to nearest even, NaN kept NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    r[np.isnan(x)] = BF16_NAN
    return r


def _fp8_nearest_codes(x: np.ndarray) -> np.ndarray:
    """Input drawing only: the E4M3 code nearest to each value (the sign
    kept, magnitudes clipped to 448); how ties break does not matter here."""
    codes = np.arange(0x7F)
    e, m = codes >> 3, codes & 7
    vals = np.where(e == 0, m * 2.0 ** -9, (1 + m / 8.0) * 2.0 ** (e - 7.0))
    a = np.minimum(np.abs(x.astype(np.float64)), 448.0)
    hi = np.clip(np.searchsorted(vals, a), 0, 0x7E)
    lo = np.clip(hi - 1, 0, 0x7E)
    pick = np.where(a - vals[lo] <= vals[hi] - a, lo, hi)
    return (pick | np.where(x < 0, 0x80, 0)).astype(np.uint8)


def _draw_values(rng: np.random.Generator, shape, dtype: str, fp8_scale: float = 1.0) -> np.ndarray:
    v = rng.standard_normal(size=shape, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_from_f32(v)
    if dtype == "fp8":
        return _fp8_nearest_codes(v / np.float32(fp8_scale))
    return v


@dataclass
class Batch:
    """One step's inputs, in host memory, in the library's layouts."""

    dtype: str
    heads: HeadSpec
    num_blocks: int
    seq_lens: np.ndarray  # int32 [S], KV length after append
    query_start_loc: np.ndarray  # int32 [S+1]
    block_tables: np.ndarray  # int32 [S, max_blocks_per_seq], -1 padded
    q: np.ndarray  # raw [T, Hq, d]
    k_new: np.ndarray  # raw [T, Hkv, d]
    v_new: np.ndarray  # raw [T, Hkv, d]
    k_cache: np.ndarray  # raw, K layout above, contents before the append
    v_cache: np.ndarray  # raw, V layout above, contents before the append
    scale: float
    seed: Optional[int] = None
    k_scale: float = 1.0  # fp8 caches: value = code value * scale
    v_scale: float = 1.0

    @property
    def qdtype(self) -> str:
        """Storage of q, k_new, v_new and the outputs."""
        return "bf16" if self.dtype == "fp8" else self.dtype

    @property
    def num_seqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def total_q(self) -> int:
        return int(self.query_start_loc[-1])

    @property
    def q_lens(self) -> np.ndarray:
        return np.diff(self.query_start_loc)

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_tables.shape[1])


def allocate_blocks(
    specs: Sequence[SeqSpec],
    block_size: int,
    rng: Optional[np.random.Generator],
    num_blocks: Optional[int] = None,
    spare: float = 0.05,
):
    """Hand out physical blocks in sequence order from a (seeded) permutation
    of the pool.  Returns (block_tables [S, MB] int32 padded with -1, num_blocks)."""
    nb = [max(1, -(-s.ctx // block_size)) if s.ctx > 0 else 0 for s in specs]
    need = int(sum(nb))
    if num_blocks is None:
        num_blocks = max(need, int(math.ceil(need * (1.0 + spare))), 1)
    if need > num_blocks:
        raise ValueError(f"pool of {num_blocks} blocks cannot hold {need}")
    perm = rng.permutation(num_blocks) if rng is not None else np.arange(num_blocks)
    mb = max(1, max(nb) if nb else 1)
    bt = np.full((len(specs), mb), -1, dtype=np.int32)
    off = 0
    for i, n in enumerate(nb):
        bt[i, :n] = perm[off : off + n]
        off += n
    return bt, num_blocks


def _nan_fill(k_cache, v_cache, block_tables, specs, heads: HeadSpec, dtype: str):
    bs = heads.block_size
    nan = {"bf16": BF16_NAN, "fp8": FP8_NAN}.get(dtype, np.float32(np.nan))
    used = np.zeros(k_cache.shape[0], dtype=bool)
    for i, s in enumerate(specs):
        n = -(-s.ctx // bs) if s.ctx > 0 else 0
        used[block_tables[i, :n]] = True
        # Slots this step appends to, and slots past ctx in the last block.
        for p in range(s.ctx - s.q_len, n * bs):
            b = block_tables[i, p // bs]
            k_cache[b, :, :, p % bs, :] = nan
            v_cache[b, :, :, p % bs] = nan
    k_cache[~used] = nan
    v_cache[~used] = nan


def make_batch(
    specs: Sequence[SeqSpec],
    heads: HeadSpec,
    dtype: str,
    rng,
    num_blocks: Optional[int] = None,
    spare: float = 0.05,
    scale: Optional[float] = None,
    nan_fill: bool = True,
    shuffle_blocks: bool = True,
) -> Batch:
    """Build one step's host inputs.  ``rng`` is a numpy Generator (or a seed)."""
    if dtype not in ELEM_BYTES:
        raise ValueError(dtype)
    seed = None
    if not isinstance(rng, np.random.Generator):
        seed = int(rng)
        rng = np.random.default_rng(seed)
    for s in specs:
        if not (0 <= s.q_len <= s.ctx):
            raise ValueError(f"bad sequence {s}")
    bt, num_blocks = allocate_blocks(
        specs, heads.block_size, rng if shuffle_blocks else None, num_blocks, spare
    )
    seq_lens = np.array([s.ctx for s in specs], dtype=np.int32)
    qsl = np.zeros(len(specs) + 1, dtype=np.int32)
    qsl[1:] = np.cumsum([s.q_len for s in specs])
    t = int(qsl[-1])
    qd = "bf16" if dtype == "fp8" else dtype
    ks, vs = (FP8_K_SCALE, FP8_V_SCALE) if dtype == "fp8" else (1.0, 1.0)
    q = _draw_values(rng, (t, heads.num_q_heads, heads.head_dim), qd)
    k_new = _draw_values(rng, (t, heads.num_kv_heads, heads.head_dim), qd)
    v_new = _draw_values(rng, (t, heads.num_kv_heads, heads.head_dim), qd)
    k_cache = _draw_values(rng, k_cache_shape(num_blocks, heads, dtype), dtype, ks)
    v_cache = _draw_values(rng, v_cache_shape(num_blocks, heads, dtype), dtype, vs)
    if nan_fill:
        _nan_fill(k_cache, v_cache, bt, specs, heads, dtype)
    if scale is None:
        scale = 1.0 / math.sqrt(heads.head_dim)
    return Batch(
        dtype=dtype,
        heads=heads,
        num_blocks=num_blocks,
        seq_lens=seq_lens,
        query_start_loc=qsl,
        block_tables=bt,
        q=q,
        k_new=k_new,
        v_new=v_new,
        k_cache=k_cache,
        v_cache=v_cache,
        scale=float(scale),
        seed=seed,
        k_scale=ks,
        v_scale=vs,
    )


def random_specs(
    rng: np.random.Generator,
    num_decode: int,
    decode_ctx: tuple,
    prefill: List[tuple],
    interleave: bool = False,
) -> List[SeqSpec]:
    """Decode rows with ctx ~ U{lo..hi} plus prefill chunks given as
    (chunk_len, prefix_len) pairs; optionally shuffled into one order."""
    lo, hi = decode_ctx
    ctx = rng.integers(lo, hi, size=num_decode, endpoint=True) if num_decode else []
    specs = [SeqSpec(int(c), 1) for c in ctx]
    specs += [SeqSpec(int(p + c), int(c)) for c, p in prefill]
    if interleave:
        order = rng.permutation(len(specs))
        specs = [specs[i] for i in order]
    return specs
