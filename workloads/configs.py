"""The five synthetic step shapes that the parity tests and the bench use.

Each function draws, from one numpy Generator, the decode contexts first and
the prefill parameters second, and returns (specs, heads, num_blocks), where
``num_blocks`` is None for "needed blocks plus 5% spare".  Decode rows come
first in the batch, prefill chunks after them.  "k" means 1024 throughout.

The shapes stand in for the paper's workloads, which are traces that are not
available here: up to 256 running requests and contexts up to 128K tokens on a
decode worker (section 6.1), decode contexts of 65K-98K tokens (section 3.2),
prefill chunks on radix-cached prefixes (section 4.4, section 5), and a
per-step prefill token budget as the lease's compute credit (section 4.2).

* tiny     -- 4 decode rows (ctx 64-256) + one 32-token chunk on a 96-token
              prefix; 4 query / 2 KV heads, head_dim 64; a 64-block pool.
* decode8b -- 64 decode rows, ctx 512-8192; 32/8 heads, head_dim 128.
* lent     -- 128 decode rows (ctx 1k-16k) + two 2048-token chunks on prefixes
              0-8k; 32/8/128.
* agentic  -- 256 decode rows, lognormal ctx (median 6k, sigma 1, cap 32k)
              + 4 chunks of 512-4096 tokens whose prefix covers 50-90% of a
              4k-24k prompt (block-aligned); 64/8/128.
* budget   -- 256 decode rows (ctx 4k-8k) + one chunk of B tokens on a 4k
              prefix, B in {0, 256, 1024, 4096}; 32/8/128.
* longctx  -- 32 decode rows (ctx 32k-128k) + one 8192-token chunk on a 64k
              prefix; 32/8/128.
"""

from __future__ import annotations

import dataclasses
import math

import numpy as np

from .gen import HeadSpec, SeqSpec, make_batch

K = 1024


def tiny(rng):
    heads = HeadSpec(4, 2, 64, 16)
    pool = 64
    while True:
        ctx = rng.integers(64, 256, size=4, endpoint=True)
        specs = [SeqSpec(int(c), 1) for c in ctx] + [SeqSpec(96 + 32, 32)]
        if sum(-(-s.ctx // 16) for s in specs) <= pool:
            return specs, heads, pool


def decode8b(rng):
    ctx = rng.integers(512, 8 * K, size=64, endpoint=True)
    return [SeqSpec(int(c), 1) for c in ctx], HeadSpec(32, 8, 128, 16), None


def lent(rng):
    ctx = rng.integers(1 * K, 16 * K, size=128, endpoint=True)
    prefix = rng.integers(0, 8 * K, size=2, endpoint=True)
    specs = [SeqSpec(int(c), 1) for c in ctx]
    specs += [SeqSpec(int(p) + 2048, 2048) for p in prefix]
    return specs, HeadSpec(32, 8, 128, 16), None


def agentic(rng, sigma: float = 1.0):
    z = rng.standard_normal(256)
    ctx = np.clip(np.rint(np.exp(math.log(6 * K) + sigma * z)), 1, 32 * K).astype(int)
    specs = [SeqSpec(int(c), 1) for c in ctx]
    for _ in range(4):
        lp = int(rng.integers(4 * K, 24 * K, endpoint=True))
        hit = float(rng.uniform(0.5, 0.9))
        p = 16 * int(math.floor(hit * lp / 16))
        c = min(int(rng.integers(512, 4096, endpoint=True)), lp - p)
        specs.append(SeqSpec(p + c, c))
    return specs, HeadSpec(64, 8, 128, 16), None


def budget(rng, b: int = 1024):
    ctx = rng.integers(4 * K, 8 * K, size=256, endpoint=True)
    specs = [SeqSpec(int(c), 1) for c in ctx]
    if b > 0:
        specs.append(SeqSpec(4 * K + b, b))
    return specs, HeadSpec(32, 8, 128, 16), None


def longctx(rng):
    ctx = rng.integers(32 * K, 128 * K, size=32, endpoint=True)
    specs = [SeqSpec(int(c), 1) for c in ctx]
    specs.append(SeqSpec(64 * K + 8 * K, 8 * K))
    return specs, HeadSpec(32, 8, 128, 16), None


CONFIGS = {
    "tiny": tiny,
    "decode8b": decode8b,
    "lent": lent,
    "agentic": agentic,
    "budget0": lambda rng: budget(rng, 0),
    "budget256": lambda rng: budget(rng, 256),
    "budget1024": lambda rng: budget(rng, 1024),
    "budget4096": lambda rng: budget(rng, 4096),
    "longctx": longctx,
}


def config_specs(name: str, seed: int, tp: int = 1):
    """Draw a config's sequence list; returns (specs, heads, num_blocks, rng),
    the rng positioned for the block permutation and the values.

    ``tp`` > 1 gives one GPU's share of a tp-way tensor-parallel layout: the
    same sequences with num_q_heads / tp query heads and num_kv_heads / tp KV
    heads (the paper's decode workers run TP4, section 6.1).  Both head counts
    must divide by tp."""
    rng = np.random.default_rng(seed)
    specs, heads, nb = CONFIGS[name](rng)
    if tp != 1:
        if tp < 1 or heads.num_q_heads % tp or heads.num_kv_heads % tp:
            raise ValueError(f"{name}: {heads.num_q_heads} q / {heads.num_kv_heads} kv heads do not split {tp} ways")
        heads = dataclasses.replace(heads, num_q_heads=heads.num_q_heads // tp,
                                    num_kv_heads=heads.num_kv_heads // tp)
    return specs, heads, nb, rng


def config_batch(name: str, seed: int, dtype: str = "bf16", **kw):
    """Host batch for a config (small configs only: the whole pool is drawn
    in host memory)."""
    specs, heads, nb, rng = config_specs(name, seed)
    return make_batch(specs, heads, dtype, rng, num_blocks=nb, **kw)
