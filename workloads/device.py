"""Device copies of a step's inputs, and a device-side generator for the full
sizes (whose KV pools, up to ~11 GB, are too large to draw in host memory).

Still input plumbing only: moving arrays to the GPU, drawing N(0,1) values with
torch's seeded generator on the device, NaN-filling the slots a step must not
read, and copying chosen sequences back into a small host ``Batch`` so that the
oracle can be run on exactly the values the GPU saw.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

from .gen import FP8_K_SCALE, FP8_V_SCALE, Batch, HeadSpec, SeqSpec, allocate_blocks, k_cache_shape, v_cache_shape


def _torch():
    import torch

    return torch


def _tdtype(dtype: str):
    torch = _torch()
    return {"bf16": torch.bfloat16, "fp8": torch.uint8}.get(dtype, torch.float32)


def raw_to_tensor(raw: np.ndarray, dtype: str, device):
    torch = _torch()
    if dtype == "fp8":
        return torch.from_numpy(np.ascontiguousarray(raw, dtype=np.uint8)).to(device)
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(raw).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(raw, dtype=np.float32))
    return t.to(device)


def tensor_to_raw(t, dtype: str) -> np.ndarray:
    torch = _torch()
    t = t.detach().contiguous().cpu()
    if dtype == "fp8":
        return t.view(torch.uint8).numpy().copy()
    if dtype == "bf16":
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().astype(np.float32, copy=True)


@dataclass
class DeviceStep:
    """Device tensors of one step plus the host metadata the library reads."""

    dtype: str
    heads: HeadSpec
    num_blocks: int
    scale: float
    q: object
    k_new: object
    v_new: object
    k_cache: object
    v_cache: object
    block_tables: object
    seq_lens: object
    query_start_loc: object
    block_tables_host: np.ndarray
    seq_lens_host: np.ndarray
    qsl_host: np.ndarray
    k_scale: float = 1.0
    v_scale: float = 1.0

    @property
    def qdtype(self) -> str:
        return "bf16" if self.dtype == "fp8" else self.dtype

    @property
    def total_q(self) -> int:
        return int(self.qsl_host[-1])

    @property
    def num_seqs(self) -> int:
        return int(self.seq_lens_host.shape[0])


def to_device(b: Batch, device="cuda") -> DeviceStep:
    torch = _torch()
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)
    return DeviceStep(
        dtype=b.dtype,
        heads=b.heads,
        num_blocks=b.num_blocks,
        scale=b.scale,
        q=raw_to_tensor(b.q, b.qdtype, device),
        k_new=raw_to_tensor(b.k_new, b.qdtype, device),
        v_new=raw_to_tensor(b.v_new, b.qdtype, device),
        k_cache=raw_to_tensor(b.k_cache, b.dtype, device),
        v_cache=raw_to_tensor(b.v_cache, b.dtype, device),
        block_tables=i32(b.block_tables),
        seq_lens=i32(b.seq_lens),
        query_start_loc=i32(b.query_start_loc),
        block_tables_host=np.ascontiguousarray(b.block_tables, dtype=np.int32),
        seq_lens_host=np.ascontiguousarray(b.seq_lens, dtype=np.int32),
        qsl_host=np.ascontiguousarray(b.query_start_loc, dtype=np.int32),
        k_scale=b.k_scale,
        v_scale=b.v_scale,
    )


def _randn_into(t, gen, chunk_elems: int = 1 << 28, fp8_scale: float = 1.0):
    """Fill a tensor with N(0,1) drawn in float32 and rounded to its dtype (a
    uint8 tensor receives the E4M3 codes of the values over fp8_scale, via
    torch's float8_e4m3fn conversion after clipping to +-448)."""
    torch = _torch()
    flat = t.view(-1)
    for i in range(0, flat.numel(), chunk_elems):
        n = min(chunk_elems, flat.numel() - i)
        x = torch.randn(n, generator=gen, device=t.device, dtype=torch.float32)
        if t.dtype == torch.uint8:
            flat[i : i + n] = (x / fp8_scale).clamp_(-448.0, 448.0).to(torch.float8_e4m3fn).view(torch.uint8)
        else:
            flat[i : i + n] = x.to(t.dtype)


def device_step(
    specs: Sequence[SeqSpec],
    heads: HeadSpec,
    dtype: str,
    rng: np.random.Generator,
    seed: int,
    num_blocks: Optional[int] = None,
    device="cuda",
    scale: Optional[float] = None,
) -> DeviceStep:
    """Full-size step: metadata from ``rng`` (numpy, same draw order as the
    host generator), values from torch's generator seeded with ``seed`` on the
    device, NaN in every slot the step must not read before its append."""
    torch = _torch()
    bt, num_blocks = allocate_blocks(specs, heads.block_size, rng, num_blocks)
    seq_lens = np.array([s.ctx for s in specs], dtype=np.int32)
    qsl = np.zeros(len(specs) + 1, dtype=np.int32)
    qsl[1:] = np.cumsum([s.q_len for s in specs])
    t = int(qsl[-1])
    td = _tdtype(dtype)
    tq = _tdtype("bf16" if dtype == "fp8" else dtype)
    ks, vs = (FP8_K_SCALE, FP8_V_SCALE) if dtype == "fp8" else (1.0, 1.0)
    gen = torch.Generator(device=device)
    gen.manual_seed(int(seed))
    q = torch.empty((t, heads.num_q_heads, heads.head_dim), dtype=tq, device=device)
    k_new = torch.empty((t, heads.num_kv_heads, heads.head_dim), dtype=tq, device=device)
    v_new = torch.empty_like(k_new)
    k_cache = torch.empty(k_cache_shape(num_blocks, heads, dtype), dtype=td, device=device)
    v_cache = torch.empty(v_cache_shape(num_blocks, heads, dtype), dtype=td, device=device)
    for x in (q, k_new, v_new):
        _randn_into(x, gen)
    _randn_into(k_cache, gen, fp8_scale=ks)
    _randn_into(v_cache, gen, fp8_scale=vs)
    # NaN sentinels
    bs = heads.block_size
    used = np.zeros(num_blocks, dtype=bool)
    blk_idx: List[np.ndarray] = []
    slot_idx: List[np.ndarray] = []
    for i, s in enumerate(specs):
        n = -(-s.ctx // bs) if s.ctx > 0 else 0
        used[bt[i, :n]] = True
        pos = np.arange(s.ctx - s.q_len, n * bs)
        blk_idx.append(bt[i, pos // bs])
        slot_idx.append(pos % bs)
    nan = 0x7F if dtype == "fp8" else float("nan")
    unused = torch.from_numpy(np.nonzero(~used)[0]).to(device)
    if unused.numel():
        k_cache[unused] = nan
        v_cache[unused] = nan
    bi = torch.from_numpy(np.concatenate(blk_idx).astype(np.int64)).to(device)
    si = torch.from_numpy(np.concatenate(slot_idx).astype(np.int64)).to(device)
    if bi.numel():
        k_cache[bi, :, :, si, :] = nan
        v_cache[bi, :, :, si] = nan
    i32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(device)
    return DeviceStep(
        dtype=dtype,
        heads=heads,
        num_blocks=num_blocks,
        scale=float(scale if scale is not None else 1.0 / math.sqrt(heads.head_dim)),
        q=q,
        k_new=k_new,
        v_new=v_new,
        k_cache=k_cache,
        v_cache=v_cache,
        block_tables=i32(bt),
        seq_lens=i32(seq_lens),
        query_start_loc=i32(qsl),
        block_tables_host=np.ascontiguousarray(bt, dtype=np.int32),
        seq_lens_host=seq_lens,
        qsl_host=qsl,
        k_scale=ks,
        v_scale=vs,
    )


def host_subbatch(d: DeviceStep, seqs: Sequence[int]) -> Dict:
    """Copy chosen sequences (pre-append pool contents, query rows, new K/V)
    into a compact host ``Batch``.  Returns {"batch": Batch, "rows": original
    query-row index of each row of the sub-batch}."""
    torch = _torch()
    bs = d.heads.block_size
    blocks, bts, lens, qlens, rows = [], [], [], [], []
    nb_total = 0
    for s in seqs:
        L = int(d.seq_lens_host[s])
        n = -(-L // bs)
        blocks.append(d.block_tables_host[s, :n])
        bts.append(np.arange(nb_total, nb_total + n, dtype=np.int32))
        nb_total += n
        lens.append(L)
        t0, t1 = int(d.qsl_host[s]), int(d.qsl_host[s + 1])
        qlens.append(t1 - t0)
        rows.append(np.arange(t0, t1))
    allb = torch.from_numpy(np.concatenate(blocks).astype(np.int64)).to(d.k_cache.device)
    kc = tensor_to_raw(d.k_cache.index_select(0, allb), d.dtype)
    vc = tensor_to_raw(d.v_cache.index_select(0, allb), d.dtype)
    mb = max(len(b) for b in bts)
    bt = np.full((len(seqs), mb), -1, dtype=np.int32)
    for i, b in enumerate(bts):
        bt[i, : len(b)] = b
    rows_all = np.concatenate(rows)
    ridx = torch.from_numpy(rows_all.astype(np.int64)).to(d.q.device)
    qsl = np.zeros(len(seqs) + 1, dtype=np.int32)
    qsl[1:] = np.cumsum(qlens)
    sub = Batch(
        dtype=d.dtype,
        heads=d.heads,
        num_blocks=nb_total,
        seq_lens=np.array(lens, dtype=np.int32),
        query_start_loc=qsl,
        block_tables=bt,
        q=tensor_to_raw(d.q.index_select(0, ridx), d.qdtype),
        k_new=tensor_to_raw(d.k_new.index_select(0, ridx), d.qdtype),
        v_new=tensor_to_raw(d.v_new.index_select(0, ridx), d.qdtype),
        k_cache=kc,
        v_cache=vc,
        scale=d.scale,
        k_scale=d.k_scale,
        v_scale=d.v_scale,
    )
    return {"batch": sub, "rows": rows_all}
