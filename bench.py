#!/usr/bin/env python3
"""Throughput of one mixed prefill+decode attention step on one MI355X.

A step is the whole hot path on one batch: the append of the step's new K/V
rows, the decode rows (split-K + merge) and the prefill chunks (causal MFMA
tiles), all through the C ABI on one stream.  By default the append runs
inside the attention calls (mpa_append_prefill_attention, then
mpa_append_decode_attention, whose decode kernel writes the decode rows' new
tokens); --append separate calls mpa_kv_append first.  Inputs are synthetic and resident in HBM
before timing starts.  Prints one JSON line:

  value          query tokens/s: T / step time, the median step of the timed
                 steps, each preceded by a 512 MB streaming read of device
                 memory (a cache flush) and bracketed by its own two events
                 (--flush-mb 0: wall clock over back-to-back steps)
  roofline       the dominant half's algorithmic bytes (or FLOPs) per launch
                 over its average duration: back-to-back launches of that
                 half's attention call alone (no append), at least --phase-reps
                 and at least 20 ms of them after at least 25 ms of untimed
                 ones, between one event pair on its stream, against the
                 MI355X datasheet peak
                 (HBM 8 TB/s, bf16 dense MFMA 2.5 PF)
  decode_hbm_gbs, prefill_tflops
                 the same for each half present
  phases_ms      every phase of the step from an untimed calibration pass with
                 events between all phases
  step_roofline  max(t_mem, t_mfma) / step time and (t_mem + t_mfma) / step time,
                 t_mem and t_mfma being the step's algorithmic bytes at 8 TB/s and
                 FLOPs at 2.5 PF
  model_ms       the library's step-time model (mpa_predict_step) for the batch
  graph          (--graph) step time when the step is replayed from a HIP graph
  measured_peaks what the library's probes sustain on this device (HBM stream
                 read, dense bf16 MFMA) and the roofline's fraction of that
  cpu_baseline   the CPU oracle, timed on a bounded sample of the same step

    python bench.py [--steps K] [--warmup W] [--config longctx] [--seed 0]
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "mixed-step attention tokens/s; decode HBM GB/s and prefill MFMA % of peak"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
MFMA_F32_PEAK_TFLOPS = 157.3
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_27085_amd", "csrc", "mpa_kernels.hip")

WORKLOADS = {
    "decode8b": "64 decode rows, ctx U{512..8192}; 32 q / 8 kv heads, head_dim 128, block 16, bf16",
    "lent": "128 decode rows (ctx 1k-16k) + 2 prefill chunks of 2048 on prefixes 0-8k; 32/8/128, bf16",
    "agentic": "256 decode rows (lognormal ctx, median 6k, cap 32k) + 4 chunks 512-4096 on 50-90% cached "
               "4k-24k prompts; 64/8/128, bf16",
    "budget0": "256 decode rows (ctx 4k-8k), no prefill; 32/8/128, bf16",
    "budget256": "256 decode rows (ctx 4k-8k) + a 256-token chunk on a 4k prefix; 32/8/128, bf16",
    "budget1024": "256 decode rows (ctx 4k-8k) + a 1024-token chunk on a 4k prefix; 32/8/128, bf16",
    "budget4096": "256 decode rows (ctx 4k-8k) + a 4096-token chunk on a 4k prefix; 32/8/128, bf16",
    "longctx": "32 decode rows (ctx 32k-128k) + one 8192-token chunk on a 64k prefix; 32/8/128, bf16",
}


def algorithmic_work(seq_lens, qsl, hq, hkv, d, elem_bytes, block=16, kv_bytes=None):
    """Bytes and FLOPs the step must move / compute at minimum, with e the
    bytes of a query / output element and c those of a cache element (c = e
    unless the cache is fp8):

    decode row (context L):   K+V read 2*L*Hkv*d*c, q read + out write
                              2*Hq*d*e, block ids 4*ceil(L/16)
    prefill chunk (C on P):   K+V read 2*(P+C)*Hkv*d*c, q + out 2*C*Hq*d*e
    append:                   new K/V read 2*T*Hkv*d*e, written 2*T*Hkv*d*c
    FLOPs: 4*d*Hq per attended (query, key) pair; decode attends L pairs,
    a chunk C*P + C*(C+1)/2."""
    c = elem_bytes if kv_bytes is None else kv_bytes
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    q_lens = np.diff(np.asarray(qsl, dtype=np.int64))
    dec = q_lens == 1
    pre = q_lens > 1
    L = seq_lens
    P = L - q_lens
    C = q_lens
    dec_bytes = int(np.sum((2 * L * hkv * d * c + 2 * hq * d * elem_bytes + 4 * ((L + block - 1) // block))[dec]))
    pre_bytes = int(np.sum((2 * L * hkv * d * c + 2 * C * hq * d * elem_bytes)[pre]))
    app_bytes = int(2 * q_lens.sum() * hkv * d * (elem_bytes + c))
    dec_flops = int(4 * d * hq * np.sum(L[dec]))
    pre_flops = int(4 * d * hq * np.sum((C * P + C * (C + 1) // 2)[pre]))
    return {
        "decode_bytes": dec_bytes,
        "prefill_bytes": pre_bytes,
        "append_bytes": app_bytes,
        "decode_flops": dec_flops,
        "prefill_flops": pre_flops,
        "decode_rows": int(dec.sum()),
        "prefill_chunks": int(pre.sum()),
        "query_tokens": int(q_lens.sum()),
    }


def kernel_source_sha() -> str:
    """Hash of the kernel source with comments and blank lines removed, so
    that a comment-only edit keeps the recorded counters valid."""
    import re

    with open(KERNEL_SOURCE, encoding="utf-8") as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = [re.sub(r"//.*$", "", ln).rstrip() for ln in text.splitlines()]
    code = "\n".join(ln for ln in lines if ln.strip())
    return hashlib.sha256(code.encode()).hexdigest()[:16]


def measured_traffic(workload: str, phase: str):
    """HBM bytes per launch from the committed rocprofv3 counter runs, or None
    if there are none for this workload/phase or the kernels changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f).get(workload, {}).get(phase)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("kernel_source_sha") != kernel_source_sha():
        return None
    return rec.get("bytes_per_launch")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def blas_threads() -> int:
    try:
        from threadpoolctl import threadpool_info

        n = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
        return max(n) if n else 1
    except Exception:
        return 1


def cpu_baseline(d, budget_s: float, seed: int):
    """Time the CPU oracle on a bounded, seeded sample of the step's rows.

    Sequences are visited in a seeded order, pass after pass, until the oracle
    time reaches ``budget_s``; a prefill chunk contributes up to 64 uniformly
    drawn rows per visit.  Host copies of each sequence are made once, before
    any timer starts; only the oracle's gather and attention are timed."""
    from oracle import ref
    from workloads.device import host_subbatch

    rng = np.random.default_rng(10_000 + seed)
    order = [int(s) for s in rng.permutation(d.num_seqs) if d.qsl_host[s + 1] > d.qsl_host[s]]
    hkv, hd, bs = d.heads.num_kv_heads, d.heads.head_dim, d.heads.block_size
    cache = {}
    rows_done = 0
    visits = 0
    elapsed = 0.0
    passes = 0
    while elapsed < budget_s and order and passes < 1000:
        for s in order:
            if s not in cache:
                cache[s] = host_subbatch(d, [s])["batch"]
            sub = cache[s]
            c = int(sub.query_start_loc[1])
            rows = np.arange(c) if c <= 64 else np.sort(rng.choice(c, size=64, replace=False))
            t0 = time.perf_counter()
            prefix = int(sub.seq_lens[0]) - c
            kp, vp = ref.gather_kv(sub.k_cache, sub.v_cache, sub.block_tables[0], prefix, hkv, hd, bs, sub.dtype)
            if sub.dtype == "fp8":
                k = np.concatenate([kp, ref.decode_raw(ref.fp8_codes(sub.k_new, sub.k_scale), "fp8")]) * sub.k_scale
                v = np.concatenate([vp, ref.decode_raw(ref.fp8_codes(sub.v_new, sub.v_scale), "fp8")]) * sub.v_scale
            else:
                k = np.concatenate([kp, ref.decode_raw(sub.k_new, sub.dtype)])
                v = np.concatenate([vp, ref.decode_raw(sub.v_new, sub.dtype)])
            ref.sequence_attention(ref.decode_raw(sub.q, sub.qdtype), k, v, prefix, sub.scale, hkv, rows=rows)
            elapsed += time.perf_counter() - t0
            rows_done += len(rows)
            visits += 1
            if elapsed >= budget_s:
                break
        passes += 1
    return {
        "value": rows_done / elapsed if elapsed > 0 else None,
        "unit": "query tokens/s",
        "cores": blas_threads(),
        "kind": "oracle",
        "sample": f"{rows_done} query rows over {visits} sequence visits ({len(cache)} distinct of {d.num_seqs}; "
                  f"seeded order, <=64 random rows per prefill-chunk visit), {elapsed:.1f} s of float64 numpy "
                  f"on {cpu_model()}, {os.cpu_count()} logical CPUs visible",
    }


def measured_peaks(torch, mpa, read_bytes: int = 2 << 30, mfma_iters: int = 20000, reps: int = 5) -> dict:
    """The library's probes (mpa_probe_stream_read, mpa_probe_mfma_bf16),
    median of `reps` launches after two untimed ones: HBM read GB/s over a
    buffer 8x the 256 MB last-level cache, and dense bf16 MFMA TFLOP/s."""
    buf = torch.empty(read_bytes, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(4, dtype=torch.float32, device="cuda")

    def timed(launch):
        for _ in range(2):
            launch()
        ms = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            launch()
            b.record()
            b.synchronize()
            ms.append(a.elapsed_time(b))
        return float(np.median(ms))

    read_ms = timed(lambda: mpa.probe_stream_read(buf, sink))
    flops = []
    mfma_ms = timed(lambda: flops.append(mpa.probe_mfma_bf16(mfma_iters, sink)))
    del buf
    return {"stream_read_gbs": round(read_bytes / (read_ms * 1e-3) / 1e9, 1),
            "mfma_bf16_tflops": round(flops[-1] / (mfma_ms * 1e-3) / 1e12, 1),
            "how": f"median of {reps}: one {read_bytes >> 20} MiB read with 16-byte non-temporal loads; "
                   f"{mfma_iters} rounds of 4 independent 32x32x16 bf16 MFMAs in 4096 waves"}


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="longctx", choices=sorted(WORKLOADS))
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probes", action="store_true",
                    help="skip the measured-peak probes (HBM stream read, bf16 MFMA) after the timed steps")
    ap.add_argument("--streams", type=int, default=1, choices=(1, 2),
                    help="2: the decode and prefill halves of the step run concurrently on two streams "
                         "(the library's mpa_decode_attention / mpa_prefill_attention); 1 (default): one after the other")
    ap.add_argument("--kv", default="bf16", choices=("bf16", "fp8"),
                    help="KV-cache element type: bf16 (default) or fp8 (OCP E4M3 codes, one scale per cache; "
                         "queries and outputs stay bf16)")
    ap.add_argument("--exec", default="serial", choices=("serial", "auto"),
                    help="auto: run the attention halves as mpa_plan_coexec picks -- one stream, or concurrently "
                         "on CU-partitioned streams (decode on 1-3 quarters of every XCD)")
    ap.add_argument("--tp", type=int, default=1, choices=(1, 2, 4, 8),
                    help="run one GPU's share of a tp-way tensor-parallel layout: the same sequences with "
                         "1/tp of the query and KV heads (the paper's decode workers run TP4)")
    ap.add_argument("--append", default="fused", choices=("fused", "separate"),
                    help="fused (default): the append inside the attention calls (mpa_append_prefill_attention, "
                         "mpa_append_decode_attention: the decode kernel writes the decode rows' new tokens); "
                         "separate: mpa_kv_append, then the attention")
    ap.add_argument("--flush-mb", type=int, default=512, metavar="MB",
                    help="read MB megabytes of device memory before every timed step (cache flush) and time each "
                         "step with its own events; value comes from the median step (default 512; 0: back-to-back "
                         "steps, wall clock)")
    ap.add_argument("--phase-reps", type=int, default=10, metavar="N",
                    help="at least N back-to-back launches (and at least 20 ms) of each attention half alone, after "
                         "at least 25 ms of untimed ones, between one event pair on its stream: the phase rates and the "
                         "roofline (default 10)")
    ap.add_argument("--graph", action="store_true",
                    help="also capture one step into a HIP graph (torch.cuda.graph) and time its replays")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes 5 times (the reference kernel "
                         "for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE readings) and exit")
    args = ap.parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the attention step has no cross-GPU exchange and this build runs "
              "on a single MI355X; run with --gpus 1.", file=sys.stderr)
        return 2

    import torch

    if args.copy_calibration:
        x = torch.ones(args.copy_calibration // 4, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(5):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": x.numel() * 4, "calls": 5}), flush=True)
        return 0

    import paper_2609_27085_amd as mpa
    from workloads.configs import config_specs
    from workloads.device import device_step

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    mpa.lib()
    specs, heads, nb, rng = config_specs(args.config, args.seed, tp=args.tp)
    d = device_step(specs, heads, args.kv, rng, args.seed, num_blocks=nb)
    work = algorithmic_work(d.seq_lens_host, d.qsl_host, heads.num_q_heads, heads.num_kv_heads, heads.head_dim, 2,
                            kv_bytes=1 if args.kv == "fp8" else 2)
    fused = args.append == "fused"
    sc = dict(k_scale=d.k_scale, v_scale=d.v_scale)
    ws = mpa.alloc_workspace(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.qsl_host, d.scale)
    out = torch.empty_like(d.q)
    lse = torch.empty(d.q.shape[:2], dtype=torch.float32, device=d.q.device)
    side = torch.cuda.Stream() if args.streams == 2 else None
    has_dec = work["decode_rows"] > 0
    has_pre = work["prefill_chunks"] > 0
    two = args.streams == 2 and has_dec and has_pre
    coexec_mode = 0
    if args.exec == "auto":
        if args.kv != "bf16" or args.streams != 1:
            raise SystemExit("--exec auto models bf16 caches on the one-stream step")
        coexec_mode = mpa.plan_coexec(mpa.shape_of(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.scale),
                                      d.seq_lens_host, d.qsl_host)[0]
    part = mpa.partition_streams(coexec_mode) if coexec_mode else None

    def step(ev=None):
        """append; then prefill half and decode half (concurrently with two
        streams).  ev maps a mark -- "start", "append", "prefill", "decode",
        "end" -- to the event recorded there; marks absent from ev are not
        recorded."""
        ev = ev or {}
        stream = torch.cuda.current_stream()  # the capture stream inside a graph capture

        def mark(name, s):
            if name in ev:
                ev[name].record(s)

        mark("start", stream)
        if not fused:
            mpa.kv_append(d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                          d.seq_lens_host, d.qsl_host, stream=stream, **sc)
        mark("append", stream)
        pre_stream = dec_stream = stream
        if two:
            side.wait_stream(stream)
            pre_stream = side
        if part:
            dec_stream, pre_stream = part
            dec_stream.wait_stream(stream)
            pre_stream.wait_stream(stream)
        if has_pre:
            if fused:
                mpa.append_attention(d.q, d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens,
                                     d.query_start_loc, d.seq_lens_host, d.qsl_host, out, lse=lse, workspace=ws,
                                     scale=d.scale, stream=pre_stream, which="mpa_append_prefill_attention", **sc)
            else:
                mpa.prefill_attention(d.q, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                                      d.seq_lens_host, d.qsl_host, out, lse=lse, workspace=ws, scale=d.scale,
                                      stream=pre_stream, **sc)
        mark("prefill", pre_stream)
        if has_dec:
            if fused:
                mpa.append_attention(d.q, d.k_new, d.v_new, d.k_cache, d.v_cache, d.block_tables, d.seq_lens,
                                     d.query_start_loc, d.seq_lens_host, d.qsl_host, out, lse=lse, workspace=ws,
                                     scale=d.scale, stream=dec_stream, which="mpa_append_decode_attention", **sc)
            else:
                mpa.decode_attention(d.q, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc,
                                     d.seq_lens_host, d.qsl_host, out, lse=lse, workspace=ws, scale=d.scale,
                                     stream=dec_stream, **sc)
        mark("decode", dec_stream)
        if two:
            stream.wait_stream(side)
        if part:
            stream.wait_stream(dec_stream)
            stream.wait_stream(pre_stream)
        mark("end", stream)

    def new_events(names):
        return {n: torch.cuda.Event(enable_timing=True) for n in names}

    # With one stream the halves run prefill-then-decode; with two they overlap.
    concurrent = two or bool(part)
    spans = {"append": ("start", "append"), "prefill": ("append", "prefill"),
             "decode": ("prefill", "decode") if not concurrent else ("append", "decode"), "step": ("start", "end")}

    def avg_ms(evs, span):
        a, b = spans[span]
        return float(np.mean([e[a].elapsed_time(e[b]) for e in evs]))

    for _ in range(args.warmup):
        step()
    # untimed calibration pass: every phase of the step, events between them
    calib = [new_events(["start", "append", "prefill", "decode", "end"]) for _ in range(max(3, min(10, args.steps)))]
    for e in calib:
        step(e)
    torch.cuda.synchronize()
    phase_ms = {k: avg_ms(calib, k) for k in spans}

    if args.flush_mb:
        # a streaming read of flush_mb MB before every timed step, which
        # evicts the step's data from L2 and the MALL without leaving dirty
        # lines (a write flush would leave its own write-back to drain into
        # the step), each step timed on its own with events from start to
        # end: value from the median step
        flush = torch.zeros(args.flush_mb << 20, dtype=torch.uint8, device="cuda")
        sink = torch.zeros(4, dtype=torch.uint8, device="cuda")
        mpa.probe_stream_read(flush, sink)
        events = [new_events(["start", "end"]) for _ in range(args.steps)]
        torch.cuda.synchronize()
        for k in range(args.steps):
            mpa.probe_stream_read(flush, sink)
            step(events[k])
        torch.cuda.synchronize()
        ms_per_step = float(np.median([e["start"].elapsed_time(e["end"]) for e in events]))
        value = work["query_tokens"] / (ms_per_step * 1e-3)
        del flush
    else:
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            step()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ms_per_step = wall * 1e3 / args.steps
        value = work["query_tokens"] * args.steps / wall

    # Each half's attention call alone (no append): back-to-back launches
    # between one event pair on the stream they run on (a partition stream in
    # co-execution mode), at least phase_reps of them and at least 20 ms,
    # after untimed launches that fill at least 25 ms of device time, so that
    # a short kernel is timed in the same steady state as a long one (the
    # first few milliseconds of launches after other work run slower).
    how_alone = {}

    def half_alone_ms(which):
        fn = mpa.decode_attention if which == "decode" else mpa.prefill_attention
        st = torch.cuda.current_stream()
        if part:
            st = part[0] if which == "decode" else part[1]

        def launch():
            fn(d.q, d.k_cache, d.v_cache, d.block_tables, d.seq_lens, d.query_start_loc, d.seq_lens_host,
               d.qsl_host, out, lse=lse, workspace=ws, scale=d.scale, stream=st, **sc)

        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(st)
        for _ in range(2):
            launch()
        b.record(st)
        torch.cuda.synchronize()
        per = max(a.elapsed_time(b) / 2, 1e-3)
        warm = 2 + min(1000, max(0, int(np.ceil((25.0 - 2 * per) / per))))
        for _ in range(warm - 2):
            launch()
        reps = max(1, args.phase_reps, min(2000, int(np.ceil(20.0 / per))))
        torch.cuda.synchronize()
        a.record(st)
        for _ in range(reps):
            launch()
        b.record(st)
        torch.cuda.synchronize()
        how_alone[which] = (reps, warm)
        return a.elapsed_time(b) / reps

    alone = {}
    if has_dec:
        alone["decode"] = half_alone_ms("decode")
    if has_pre:
        alone["prefill"] = half_alone_ms("prefill")
    dom = max(alone, key=alone.get)
    dom_ms = alone[dom]
    dec_gbs = work["decode_bytes"] / (alone["decode"] * 1e-3) / 1e9 if has_dec else None
    pre_tflops = work["prefill_flops"] / (alone["prefill"] * 1e-3) / 1e12 if has_pre else None
    info = mpa.plan_info(mpa.shape_of(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.scale, **sc),
                         d.seq_lens_host, d.qsl_host)
    if dom == "decode":
        achieved, peak, unit, bound = dec_gbs, HBM_PEAK_GBS, "GB/s", "hbm"
        split_rows = any(-(-int(L) // info.split_tokens) > 1
                         for L, c in zip(d.seq_lens_host, np.diff(d.qsl_host)) if c == 1)
        kernel = "decode_kernel+merge_kernel" if split_rows else "decode_kernel"
    else:
        achieved, peak, unit, bound = pre_tflops, MFMA_BF16_PEAK_TFLOPS, "TFLOP/s", "mfma"
        kernel = "prefill_mfma_kernel"
        if info.prefill_max_splits > 1:
            kernel += "+prefill_merge_kernel"
        if any(int(L) - int(c) < 64 for L, c in zip(d.seq_lens_host, np.diff(d.qsl_host)) if c > 1):
            kernel += "+prefill_kernel (rows of at most 64 keys)"
    roofline = {
        "bound": bound,
        "achieved": round(achieved, 2),
        "peak": peak,
        "unit": unit,
        "frac": round(achieved / peak, 4),
        "traffic": measured_traffic(args.config, dom) if args.kv == "bf16" and args.tp == 1 else None,
        "kernel": kernel,
        "phase_ms": round(dom_ms, 4),
        "algorithmic_per_launch": work["decode_bytes"] if dom == "decode" else work["prefill_flops"],
        "how": f"{how_alone[dom][0]} back-to-back launches of mpa_{dom}_attention alone (no append) between "
               f"one event pair on its stream, after {how_alone[dom][1]} untimed launches (at least 25 ms)",
    }
    total_bytes = work["decode_bytes"] + work["prefill_bytes"] + work["append_bytes"]
    total_flops = work["decode_flops"] + work["prefill_flops"]
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "query tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if args.kv == "bf16" else "fp8",
        "data": "synthetic (seeded N(0,1) values, shuffled block tables)",
        "config": {"workload": f"{args.config}: {WORKLOADS[args.config]}"
                               + (f"; one GPU's share of TP{args.tp}: {heads.num_q_heads}/{heads.num_kv_heads} heads"
                                  if args.tp > 1 else ""),
                   "seed": args.seed, "streams": args.streams if two else 1,
                   "append": ("fused into the attention halves (decode rows by the decode kernel)" if fused
                              else "mpa_kv_append before the attention"),
                   "timing": (f"median of {args.steps} steps, each between its own two events after a "
                              f"{args.flush_mb} MB device read" if args.flush_mb
                              else "wall clock over back-to-back steps"),
                   "kv_cache": "bf16" if args.kv == "bf16" else "fp8 e4m3 (per-cache scale; bf16 MFMA on the codes)",
                   "decode_rows": work["decode_rows"], "prefill_chunks": work["prefill_chunks"],
                   "query_tokens": work["query_tokens"],
                   "parallelism": f"one GPU's share of tp{args.tp}" if args.tp > 1 else "single GPU",
                   "exec": f"decode on {coexec_mode}/4 of every XCD beside prefill" if coexec_mode else "one stream"},
        "roofline": roofline,
        "phases_ms": {k: round(v, 4) for k, v in phase_ms.items()},
        "halves_alone_ms": {k: round(v, 4) for k, v in alone.items()},
        "decode_hbm_gbs": round(dec_gbs, 1) if dec_gbs else None,
        "decode_hbm_frac": round(dec_gbs / HBM_PEAK_GBS, 4) if dec_gbs else None,
        "prefill_tflops": round(pre_tflops, 2) if pre_tflops else None,
        "prefill_mfma_frac": round(pre_tflops / MFMA_BF16_PEAK_TFLOPS, 4) if pre_tflops else None,
        "step_hbm_gbs": round(total_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "step_attention_tflops": round(total_flops / (ms_per_step * 1e-3) / 1e12, 3),
    }
    # step roofline: the step's algorithmic bytes at 8 TB/s and FLOPs at the
    # bf16 MFMA peak, against the measured step time
    t_mem = total_bytes / (HBM_PEAK_GBS * 1e9)
    t_mfma = work["prefill_flops"] / (MFMA_BF16_PEAK_TFLOPS * 1e12)
    t_step = ms_per_step * 1e-3
    line["step_roofline"] = {"t_mem_ms": round(t_mem * 1e3, 4), "t_mfma_ms": round(t_mfma * 1e3, 4),
                             "max_frac": round(max(t_mem, t_mfma) / t_step, 4),
                             "sum_frac": round((t_mem + t_mfma) / t_step, 4)}
    if not args.no_probes:
        peaks = measured_peaks(torch, mpa)
        meas = peaks["stream_read_gbs"] if dom == "decode" else peaks["mfma_bf16_tflops"]
        peaks["roofline_frac_of_measured"] = round(achieved / meas, 4)
        line["measured_peaks"] = peaks
    # the library's step-time model (mpa_predict_step; bf16 caches) for this batch
    if args.kv == "bf16":
        pred = mpa.predict_step(mpa.shape_of(d.q, d.k_cache, d.block_tables, d.seq_lens_host, d.scale),
                                d.seq_lens_host, d.qsl_host)
        line["model_ms"] = {"append": round(pred.append_us * 1e-3, 4), "decode": round(pred.decode_us * 1e-3, 4),
                            "prefill": round(pred.prefill_us * 1e-3, 4), "step": round(pred.step_us * 1e-3, 4)}
    if args.graph:
        # the same step (no events) recorded once and replayed: every launch
        # carries its plan as kernel arguments, so the graph is a fixed
        # sequence of kernel nodes
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        for _ in range(max(1, args.warmup)):
            graph.replay()
        torch.cuda.synchronize()
        g0 = time.perf_counter()
        for _ in range(args.steps):
            graph.replay()
        torch.cuda.synchronize()
        gwall = time.perf_counter() - g0
        line["graph"] = {"ms_per_step": round(gwall * 1e3 / args.steps, 4),
                         "value": round(work["query_tokens"] * args.steps / gwall, 1)}
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(d, args.cpu_seconds, args.seed)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
