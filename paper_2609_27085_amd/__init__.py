"""Python binding of ``libmpa.so`` (include/mpa.h): argument marshalling only.

Every step of the attention path runs in the library's HIP kernels; this
module turns torch device tensors into pointers, host numpy arrays into int32
buffers and the current torch stream into a ``hipStream_t``.  If the library
is not built the calls raise ``MpaUnavailable``; there is no fallback.

    import paper_2609_27085_amd as mpa
    mpa.kv_append(k_new, v_new, k_cache, v_cache, block_tables, seq_lens, qsl,
                  seq_lens_host, qsl_host)
    ws = mpa.alloc_workspace(q, k_cache, block_tables, seq_lens_host, qsl_host)
    mpa.mixed_paged_attention(q, k_cache, v_cache, block_tables, seq_lens, qsl,
                              seq_lens_host, qsl_host, out, lse=lse, workspace=ws)
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmpa.so")

MPA_OK = 0
MPA_ERR_INVALID = -1
MPA_ERR_UNSUPPORTED = -2
MPA_ERR_WORKSPACE = -3
MPA_ERR_HIP = -4
MPA_ERR_SCRATCH = -5
MPA_SCRATCH_BYTES = 256 << 20  # the fixed device array behind mpa_append_attention_noalloc
MPA_BF16 = 0
MPA_F32 = 1
MPA_FP8 = 2  # fp8 (OCP E4M3) caches with bf16 queries, new rows and outputs
BLOCK_SIZE = 16

EXPORTS = (
    "mpa_kv_append",
    "mpa_mixed_paged_attention",
    "mpa_append_attention",
    "mpa_append_decode_attention",
    "mpa_append_prefill_attention",
    "mpa_append_attention_noalloc",
    "mpa_workspace_size",
    "mpa_status_string",
    "mpa_get_plan_info",
    "mpa_decode_attention",
    "mpa_prefill_attention",
    "mpa_default_rates",
    "mpa_kv_append_rope",
    "mpa_predict_step",
    "mpa_plan_coexec",
    "mpa_partition_streams",
    "mpa_probe_stream_read",
    "mpa_probe_mfma_bf16",
)


class MpaUnavailable(RuntimeError):
    pass


class MpaError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


class MpaShape(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("num_blocks", ctypes.c_int32),
        ("max_blocks_per_seq", ctypes.c_int32),
        ("total_q_tokens", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("dtype", ctypes.c_int32),
        ("k_scale", ctypes.c_float),
        ("v_scale", ctypes.c_float),
    ]


class MpaPlanInfo(ctypes.Structure):
    _fields_ = [
        ("num_decode_seqs", ctypes.c_int32),
        ("num_prefill_seqs", ctypes.c_int32),
        ("split_tokens", ctypes.c_int32),
        ("num_decode_items", ctypes.c_int32),
        ("num_prefill_tiles", ctypes.c_int32),
        ("decode_launches", ctypes.c_int32),
        ("prefill_max_splits", ctypes.c_int32),
    ]


class MpaRates(ctypes.Structure):
    _fields_ = [
        ("append_fixed_us", ctypes.c_double),
        ("append_gbs", ctypes.c_double),
        ("decode_fixed_us", ctypes.c_double),
        ("decode_gbs", ctypes.c_double),
        ("decode_wave_gbs", ctypes.c_double),
        ("merge_us", ctypes.c_double),
        ("prefill_wg_us", ctypes.c_double),
        ("prefill_tile_us", ctypes.c_double),
        ("prefill_merge_us", ctypes.c_double),
        ("prefill_fixup_us", ctypes.c_double),
        ("prefill_slots", ctypes.c_int32),
        ("append_block_us", ctypes.c_double),
        ("append_block_gbs", ctypes.c_double),
        ("coexec_decode_q1", ctypes.c_double),
        ("coexec_decode_q2", ctypes.c_double),
        ("coexec_decode_q3", ctypes.c_double),
        ("coexec_prefill_q1", ctypes.c_double),
        ("coexec_prefill_q2", ctypes.c_double),
        ("coexec_prefill_q3", ctypes.c_double),
        ("coexec_slowdown", ctypes.c_double),
        ("prefill_merge_row_us", ctypes.c_double),
        ("coexec_fixed_us", ctypes.c_double),
    ]


class MpaStepTime(ctypes.Structure):
    _fields_ = [
        ("append_us", ctypes.c_double),
        ("decode_us", ctypes.c_double),
        ("prefill_us", ctypes.c_double),
        ("step_us", ctypes.c_double),
    ]


_lib = None
_P = ctypes.c_void_p
_I32P = ctypes.POINTER(ctypes.c_int32)
_SHP = ctypes.POINTER(MpaShape)


def lib() -> ctypes.CDLL:
    """The loaded library (raises MpaUnavailable if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise MpaUnavailable(f"{LIB_PATH} is missing; build it with `python -m paper_2609_27085_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.mpa_kv_append.restype = ctypes.c_int
        L.mpa_kv_append.argtypes = [_SHP, _P, _P, _P, _P, _P, _P, _P, _I32P, _I32P, _I32P, _P]
        L.mpa_kv_append_rope.restype = ctypes.c_int
        L.mpa_kv_append_rope.argtypes = [_SHP, _P, _P, _P, _P, _P, _P, _P, _P, _I32P, _I32P, _I32P, _P,
                                         ctypes.c_int32, ctypes.c_int32, _P]
        L.mpa_mixed_paged_attention.restype = ctypes.c_int
        L.mpa_mixed_paged_attention.argtypes = [
            _SHP, _P, _P, _P, _P, _P, _P, _I32P, _I32P, _I32P, _P, _P, _P, ctypes.c_size_t, _P]
        L.mpa_append_attention.restype = ctypes.c_int
        L.mpa_append_attention.argtypes = [
            _SHP, _P, _P, _P, _P, _P, _P, _P, _P, _I32P, _I32P, _I32P, _P, _P, _P, ctypes.c_size_t, _P]
        L.mpa_append_attention_noalloc.restype = ctypes.c_int
        L.mpa_append_attention_noalloc.argtypes = [
            _SHP, _P, _P, _P, _P, _P, _P, _P, _P, _I32P, _I32P, _I32P, _P, _P, _P]
        for name in ("mpa_append_decode_attention", "mpa_append_prefill_attention"):
            getattr(L, name).restype = ctypes.c_int
            getattr(L, name).argtypes = L.mpa_append_attention.argtypes
        L.mpa_decode_attention.restype = ctypes.c_int
        L.mpa_decode_attention.argtypes = L.mpa_mixed_paged_attention.argtypes
        L.mpa_prefill_attention.restype = ctypes.c_int
        L.mpa_prefill_attention.argtypes = L.mpa_mixed_paged_attention.argtypes
        L.mpa_workspace_size.restype = ctypes.c_size_t
        L.mpa_workspace_size.argtypes = [_SHP, _I32P, _I32P]
        L.mpa_status_string.restype = ctypes.c_char_p
        L.mpa_status_string.argtypes = [ctypes.c_int]
        L.mpa_get_plan_info.restype = ctypes.c_int
        L.mpa_get_plan_info.argtypes = [_SHP, _I32P, _I32P, ctypes.POINTER(MpaPlanInfo)]
        L.mpa_default_rates.restype = None
        L.mpa_default_rates.argtypes = [ctypes.POINTER(MpaRates)]
        L.mpa_predict_step.restype = ctypes.c_int
        L.mpa_predict_step.argtypes = [_SHP, _I32P, _I32P, ctypes.POINTER(MpaRates), ctypes.POINTER(MpaStepTime)]
        L.mpa_plan_coexec.restype = ctypes.c_int
        L.mpa_plan_coexec.argtypes = [_SHP, _I32P, _I32P, ctypes.POINTER(MpaRates), ctypes.POINTER(ctypes.c_int32),
                                      ctypes.POINTER(ctypes.c_double)]
        L.mpa_partition_streams.restype = ctypes.c_int
        L.mpa_partition_streams.argtypes = [ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p),
                                            ctypes.POINTER(ctypes.c_void_p)]
        L.mpa_probe_stream_read.restype = ctypes.c_int
        L.mpa_probe_stream_read.argtypes = [_P, ctypes.c_size_t, _P, _P]
        L.mpa_probe_mfma_bf16.restype = ctypes.c_int
        L.mpa_probe_mfma_bf16.argtypes = [ctypes.c_int32, _P, ctypes.POINTER(ctypes.c_double), _P]
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().mpa_status_string(int(status)).decode()


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.int32)


def _i32p(a: Optional[np.ndarray]):
    if a is None:
        return None
    return a.ctypes.data_as(_I32P)


def _dtype_code(t) -> int:
    import torch

    if t.dtype == torch.uint8 or t.dtype == getattr(torch, "float8_e4m3fn", None):
        return MPA_FP8
    if t.dtype == torch.bfloat16:
        return MPA_BF16
    if t.dtype == torch.float32:
        return MPA_F32
    raise ValueError(f"unsupported dtype {t.dtype}")


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def make_shape(num_seqs, num_q_heads, num_kv_heads, head_dim, num_blocks, max_blocks_per_seq, total_q_tokens,
               scale, dtype: int, block_size: int = BLOCK_SIZE, k_scale: float = 1.0,
               v_scale: float = 1.0) -> MpaShape:
    return MpaShape(int(num_seqs), int(num_q_heads), int(num_kv_heads), int(head_dim), int(block_size),
                    int(num_blocks), int(max_blocks_per_seq), int(total_q_tokens), float(scale), int(dtype),
                    float(k_scale), float(v_scale))


def shape_of(q, k_cache, block_tables, seq_lens_host, scale=None, k_scale=1.0, v_scale=1.0) -> MpaShape:
    """mpa_shape from the tensors: q [T, Hq, d], k_cache [NB, Hkv, d/X, 16, X]
    (or any view with NB and Hkv leading), block_tables [S, MB].  The dtype
    comes from the cache (uint8 = fp8 codes), the queries being bf16 then."""
    t, hq, d = q.shape
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    return make_shape(len(seq_lens_host), hq, k_cache.shape[1], d, k_cache.shape[0], block_tables.shape[1], t,
                      scale, _dtype_code(k_cache), k_scale=k_scale, v_scale=v_scale)


def plan_info(shape: MpaShape, seq_lens_host, qsl_host) -> MpaPlanInfo:
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    info = MpaPlanInfo()
    rc = lib().mpa_get_plan_info(ctypes.byref(shape), _i32p(sl), _i32p(qs), ctypes.byref(info))
    if rc != MPA_OK:
        raise MpaError(rc, "mpa_get_plan_info")
    return info


def default_rates() -> MpaRates:
    """The library's measured MI355X rates for the step-time model."""
    r = MpaRates()
    lib().mpa_default_rates(ctypes.byref(r))
    return r


def predict_step(shape: MpaShape, seq_lens_host, qsl_host, rates: Optional[MpaRates] = None) -> MpaStepTime:
    """Predicted device time (us) of kv_append + mixed attention for a batch
    (mpa_predict_step); rates None means the library's defaults."""
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    out = MpaStepTime()
    rc = lib().mpa_predict_step(ctypes.byref(shape), _i32p(sl), _i32p(qs),
                                ctypes.byref(rates) if rates is not None else None, ctypes.byref(out))
    if rc != MPA_OK:
        raise MpaError(rc, "mpa_predict_step")
    return out


def plan_coexec(shape: MpaShape, seq_lens_host, qsl_host, rates: Optional[MpaRates] = None):
    """mpa_plan_coexec: (mode, [predicted attention us of modes 0..3])."""
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    mode = ctypes.c_int32(-1)
    pred = (ctypes.c_double * 4)()
    rc = lib().mpa_plan_coexec(ctypes.byref(shape), _i32p(sl), _i32p(qs),
                               ctypes.byref(rates) if rates is not None else None, ctypes.byref(mode), pred)
    if rc != MPA_OK:
        raise MpaError(rc, "mpa_plan_coexec")
    return int(mode.value), [float(x) for x in pred]


_partition_streams = {}


def partition_streams(mode: int):
    """mpa_partition_streams on the current device, as torch streams
    (decode half's, prefill half's); cached, never destroyed."""
    import torch

    key = (torch.cuda.current_device(), int(mode))
    if key not in _partition_streams:
        d, p = ctypes.c_void_p(), ctypes.c_void_p()
        rc = lib().mpa_partition_streams(int(mode), ctypes.byref(d), ctypes.byref(p))
        if rc != MPA_OK:
            raise MpaError(rc, "mpa_partition_streams")
        _partition_streams[key] = (torch.cuda.ExternalStream(d.value), torch.cuda.ExternalStream(p.value))
    return _partition_streams[key]


def probe_stream_read(buf, sink, stream=None) -> None:
    """mpa_probe_stream_read over the bytes of the contiguous device tensor
    buf; sink: a device tensor of at least 4 bytes."""
    rc = lib().mpa_probe_stream_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), _stream(stream))
    if rc != MPA_OK:
        raise MpaError(rc, "mpa_probe_stream_read")


def probe_mfma_bf16(iters: int, sink, stream=None) -> float:
    """mpa_probe_mfma_bf16; returns the launch's FLOPs."""
    flops = ctypes.c_double()
    rc = lib().mpa_probe_mfma_bf16(int(iters), _ptr(sink), ctypes.byref(flops), _stream(stream))
    if rc != MPA_OK:
        raise MpaError(rc, "mpa_probe_mfma_bf16")
    return flops.value


def workspace_size(shape: MpaShape, seq_lens_host, qsl_host) -> int:
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    return int(lib().mpa_workspace_size(ctypes.byref(shape), _i32p(sl), _i32p(qs)))


def alloc_workspace(q, k_cache, block_tables, seq_lens_host, qsl_host, scale=None):
    """A device byte tensor large enough for this batch (None if none needed)."""
    import torch

    n = workspace_size(shape_of(q, k_cache, block_tables, seq_lens_host, scale), seq_lens_host, qsl_host)
    if n == 0:
        return None
    return torch.empty(n, dtype=torch.uint8, device=q.device)


def kv_append(k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host, qsl_host,
              block_tables_host=None, stream=None, k_scale=1.0, v_scale=1.0) -> None:
    """mpa_kv_append on torch device tensors (host metadata as arrays); with
    uint8 (fp8) caches the bf16 rows are stored as codes under the scales."""
    t, hkv, d = k_new.shape
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    bth = None if block_tables_host is None else _host_i32(block_tables_host)
    shape = make_shape(len(sl), hkv, hkv, d, k_cache.shape[0], block_tables.shape[1], t, 1.0, _dtype_code(k_cache),
                       k_scale=k_scale, v_scale=v_scale)
    rc = lib().mpa_kv_append(
        ctypes.byref(shape), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(block_tables),
        _ptr(seq_lens), _ptr(query_start_loc), _i32p(sl), _i32p(qs), _i32p(bth), _stream(stream))
    if rc != MPA_OK:
        raise MpaError(rc, "mpa_kv_append")


def kv_append_rope(q, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host,
                   qsl_host, cos_sin, rope_dim=None, block_tables_host=None, stream=None, k_scale=1.0,
                   v_scale=1.0) -> None:
    """mpa_kv_append_rope: q [T, Hq, d] rotated in place, k_new rotated into
    the cache, v_new appended; cos_sin is a float32 device tensor
    [max_pos, R/2, 2] (rope_dim R defaults to 2 * cos_sin.shape[1]).  With
    uint8 (fp8) caches the rows are stored as codes under the scales."""
    t, hkv, d = k_new.shape
    hq = q.shape[1]
    if rope_dim is None:
        rope_dim = 2 * int(cos_sin.shape[1])
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    bth = None if block_tables_host is None else _host_i32(block_tables_host)
    shape = make_shape(len(sl), hq, hkv, d, k_cache.shape[0], block_tables.shape[1], t, 1.0, _dtype_code(k_cache),
                       k_scale=k_scale, v_scale=v_scale)
    rc = lib().mpa_kv_append_rope(
        ctypes.byref(shape), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(block_tables),
        _ptr(seq_lens), _ptr(query_start_loc), _i32p(sl), _i32p(qs), _i32p(bth), _ptr(cos_sin), int(rope_dim),
        int(cos_sin.shape[0]), _stream(stream))
    if rc != MPA_OK:
        raise MpaError(rc, "mpa_kv_append_rope")


def _attention(which, q, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host, qsl_host, out,
               lse, workspace, scale, block_tables_host, stream, k_scale=1.0, v_scale=1.0) -> None:
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    bth = None if block_tables_host is None else _host_i32(block_tables_host)
    shape = shape_of(q, k_cache, block_tables, sl, scale, k_scale, v_scale)
    args = [ctypes.byref(shape), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(block_tables), _ptr(seq_lens),
            _ptr(query_start_loc), _i32p(sl), _i32p(qs), _i32p(bth), _ptr(out), _ptr(lse)]
    args += [None, 0] if workspace is None else [_ptr(workspace), workspace.numel() * workspace.element_size()]
    args.append(_stream(stream))
    rc = getattr(lib(), which)(*args)
    if rc != MPA_OK:
        raise MpaError(rc, which)


def mixed_paged_attention(q, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host, qsl_host,
                          out, lse=None, workspace=None, scale=None, block_tables_host=None, stream=None,
                          k_scale=1.0, v_scale=1.0) -> None:
    """mpa_mixed_paged_attention on torch device tensors (k_scale, v_scale:
    the scales of uint8 = fp8 caches)."""
    _attention("mpa_mixed_paged_attention", q, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
               seq_lens_host, qsl_host, out, lse, workspace, scale, block_tables_host, stream, k_scale, v_scale)


def append_attention(q, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host,
                     qsl_host, out, lse=None, workspace=None, scale=None, block_tables_host=None, stream=None,
                     k_scale=1.0, v_scale=1.0, which="mpa_append_attention") -> None:
    """mpa_append_attention: kv_append then mixed_paged_attention in one call
    (the decode rows' new tokens written by the decode kernel); `which` names
    one of its halves instead (mpa_append_decode_attention,
    mpa_append_prefill_attention)."""
    if which not in ("mpa_append_attention", "mpa_append_decode_attention", "mpa_append_prefill_attention"):
        raise ValueError(which)
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    bth = None if block_tables_host is None else _host_i32(block_tables_host)
    shape = shape_of(q, k_cache, block_tables, sl, scale, k_scale, v_scale)
    args = [ctypes.byref(shape), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(block_tables),
            _ptr(seq_lens), _ptr(query_start_loc), _i32p(sl), _i32p(qs), _i32p(bth), _ptr(out), _ptr(lse)]
    args += [None, 0] if workspace is None else [_ptr(workspace), workspace.numel() * workspace.element_size()]
    args.append(_stream(stream))
    rc = getattr(lib(), which)(*args)
    if rc != MPA_OK:
        raise MpaError(rc, which)


def append_attention_noalloc(q, k_new, v_new, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
                             seq_lens_host, qsl_host, out, lse=None, scale=None, block_tables_host=None, stream=None,
                             k_scale=1.0, v_scale=1.0) -> None:
    """mpa_append_attention_noalloc: the one-call step with its partial
    results in the library's fixed device array (no workspace argument)."""
    sl, qs = _host_i32(seq_lens_host), _host_i32(qsl_host)
    bth = None if block_tables_host is None else _host_i32(block_tables_host)
    shape = shape_of(q, k_cache, block_tables, sl, scale, k_scale, v_scale)
    rc = lib().mpa_append_attention_noalloc(
        ctypes.byref(shape), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache), _ptr(block_tables),
        _ptr(seq_lens), _ptr(query_start_loc), _i32p(sl), _i32p(qs), _i32p(bth), _ptr(out), _ptr(lse),
        _stream(stream))
    if rc != MPA_OK:
        raise MpaError(rc, "mpa_append_attention_noalloc")


def decode_attention(q, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host, qsl_host,
                     out, lse=None, workspace=None, scale=None, block_tables_host=None, stream=None,
                     k_scale=1.0, v_scale=1.0) -> None:
    """mpa_decode_attention: only the rows of sequences with q_len == 1."""
    _attention("mpa_decode_attention", q, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
               seq_lens_host, qsl_host, out, lse, workspace, scale, block_tables_host, stream, k_scale, v_scale)


def prefill_attention(q, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host, qsl_host,
                      out, lse=None, workspace=None, scale=None, block_tables_host=None, stream=None,
                      k_scale=1.0, v_scale=1.0) -> None:
    """mpa_prefill_attention: only the rows of sequences with q_len > 1."""
    _attention("mpa_prefill_attention", q, k_cache, v_cache, block_tables, seq_lens, query_start_loc,
               seq_lens_host, qsl_host, out, lse, workspace, scale, block_tables_host, stream, k_scale, v_scale)


def coexec_attention(q, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host, qsl_host, out,
                     lse=None, workspace=None, scale=None, block_tables_host=None, stream=None, k_scale=1.0,
                     v_scale=1.0, rates=None, mode=None) -> int:
    """The step's attention in the mode mpa_plan_coexec picks (or `mode`):
    0 runs mpa_mixed_paged_attention on `stream`; 1..3 runs the decode and
    prefill halves concurrently on the partition streams, ordered after
    `stream` and joined back to it.  Returns the mode used; the outputs are
    bit-identical in every mode."""
    import torch

    main = torch.cuda.current_stream() if stream is None else stream
    kw = dict(lse=lse, workspace=workspace, scale=scale, block_tables_host=block_tables_host, k_scale=k_scale,
              v_scale=v_scale)
    if mode is None:
        shape = shape_of(q, k_cache, block_tables, _host_i32(seq_lens_host), scale, k_scale, v_scale)
        mode, _ = plan_coexec(shape, seq_lens_host, qsl_host, rates)
    args = (q, k_cache, v_cache, block_tables, seq_lens, query_start_loc, seq_lens_host, qsl_host, out)
    if mode == 0:
        mixed_paged_attention(*args, stream=main, **kw)
        return 0
    ds, ps = partition_streams(mode)
    ds.wait_stream(main)
    ps.wait_stream(main)
    decode_attention(*args, stream=ds, **kw)
    prefill_attention(*args, stream=ps, **kw)
    main.wait_stream(ds)
    main.wait_stream(ps)
    return int(mode)
