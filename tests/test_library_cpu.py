"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/mpa.h declares, and rejects malformed batches before
touching the device (nothing here launches a kernel)."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2609_27085_amd as mpa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mpa.h")
FAKE = 0x1000  # a non-null pointer value; never dereferenced because validation fails first


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mpa_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = mpa.lib()
    names = declared_functions()
    assert set(names) == set(mpa.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


def declared_arity():
    """Parameter count of every function include/mpa.h declares."""
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    out = {}
    for name, params in re.findall(r"\b(mpa_[a-z0-9_]+)\s*\(([^;{]*?)\)\s*;", src, flags=re.S):
        params = params.strip()
        out[name] = 0 if params in ("", "void") else params.count(",") + 1
    return out


def test_binding_signatures_match_header():
    # a ctypes prototype with the wrong number of parameters would pass the
    # trailing ones (a size, the stream) mangled
    L = mpa.lib()
    arity = declared_arity()
    assert set(arity) == set(mpa.EXPORTS)
    for name, n in arity.items():
        assert len(getattr(L, name).argtypes) == n, name


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5):
        assert mpa.status_string(code)
    assert mpa.status_string(123) == "unknown status"


def shape(**kw):
    base = dict(num_seqs=2, num_q_heads=8, num_kv_heads=2, head_dim=128, num_blocks=64, max_blocks_per_seq=8,
                total_q_tokens=5, scale=0.1, dtype=mpa.MPA_BF16)
    base.update(kw)
    return mpa.make_shape(**base)


def attention_rc(sh, seq_lens, qsl, bt=None, ws=0, ws_ptr=None):
    L = mpa.lib()
    sl = np.asarray(seq_lens, np.int32)
    qs = np.asarray(qsl, np.int32)
    bth = None if bt is None else np.asarray(bt, np.int32)
    return L.mpa_mixed_paged_attention(
        ctypes.byref(sh), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, mpa._i32p(sl), mpa._i32p(qs), mpa._i32p(bth), FAKE,
        None, ws_ptr, ws, None)


def append_rc(sh, seq_lens, qsl, bt=None):
    L = mpa.lib()
    sl = np.asarray(seq_lens, np.int32)
    qs = np.asarray(qsl, np.int32)
    bth = None if bt is None else np.asarray(bt, np.int32)
    return L.mpa_kv_append(ctypes.byref(sh), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, mpa._i32p(sl), mpa._i32p(qs),
                           mpa._i32p(bth), None)


@pytest.mark.parametrize("kw,code", [
    (dict(head_dim=96), mpa.MPA_ERR_UNSUPPORTED),
    (dict(head_dim=256), mpa.MPA_ERR_UNSUPPORTED),
    (dict(block_size=32), mpa.MPA_ERR_UNSUPPORTED),
    (dict(num_q_heads=6, num_kv_heads=4), mpa.MPA_ERR_UNSUPPORTED),
    (dict(num_q_heads=64, num_kv_heads=2), mpa.MPA_ERR_UNSUPPORTED),
    (dict(dtype=7), mpa.MPA_ERR_UNSUPPORTED),
    (dict(num_kv_heads=0), mpa.MPA_ERR_INVALID),
    (dict(scale=float("nan")), mpa.MPA_ERR_INVALID),
    (dict(scale=0.0), mpa.MPA_ERR_INVALID),
    (dict(scale=-0.1), mpa.MPA_ERR_INVALID),
])
def test_unsupported_shapes_rejected(kw, code):
    sh = shape(**kw)
    assert attention_rc(sh, [40, 3], [0, 1, 5]) == code
    assert append_rc(sh, [40, 3], [0, 1, 5]) == code


@pytest.mark.parametrize("seq_lens,qsl", [
    ([40, 3], [1, 1, 5]),      # query_start_loc[0] != 0
    ([40, 3], [0, 1, 6]),      # query_start_loc[S] != T
    ([40, 2], [0, 2, 5]),      # q_len 3 > seq_len 2
    ([40, 3], [0, 6, 5]),      # negative q_len
    ([-1, 3], [0, 0, 5]),      # negative seq_len
    ([200, 3], [0, 1, 5]),     # 13 blocks > max_blocks_per_seq = 8
])
def test_bad_metadata_rejected(seq_lens, qsl):
    sh = shape()
    assert attention_rc(sh, seq_lens, qsl) == mpa.MPA_ERR_INVALID
    assert append_rc(sh, seq_lens, qsl) == mpa.MPA_ERR_INVALID
    assert mpa.lib().mpa_workspace_size(ctypes.byref(sh), mpa._i32p(np.asarray(seq_lens, np.int32)),
                                        mpa._i32p(np.asarray(qsl, np.int32))) == 0


def test_block_ids_checked_when_host_table_given():
    sh = shape(num_blocks=10)
    bt = np.zeros((2, 8), np.int32)
    bt[0, :3] = [1, 2, 3]
    bt[1, 0] = 4
    bad = bt.copy()
    bad[0, 2] = 10  # out of range, used by sequence 0 (40 tokens -> 3 blocks)
    assert attention_rc(sh, [40, 3], [0, 1, 5], bad) == mpa.MPA_ERR_INVALID
    assert append_rc(sh, [40, 3], [0, 1, 5], bad) == mpa.MPA_ERR_INVALID
    neg = bt.copy()
    neg[1, 0] = -1
    assert attention_rc(sh, [40, 3], [0, 1, 5], neg) == mpa.MPA_ERR_INVALID


def test_null_pointers_rejected():
    L = mpa.lib()
    sh = shape()
    sl = np.asarray([40, 3], np.int32)
    qs = np.asarray([0, 1, 5], np.int32)
    assert L.mpa_mixed_paged_attention(ctypes.byref(sh), None, FAKE, FAKE, FAKE, FAKE, FAKE, mpa._i32p(sl),
                                       mpa._i32p(qs), None, FAKE, None, None, 0, None) == mpa.MPA_ERR_INVALID
    assert L.mpa_mixed_paged_attention(ctypes.byref(sh), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, mpa._i32p(qs),
                                       None, FAKE, None, None, 0, None) == mpa.MPA_ERR_INVALID
    assert L.mpa_mixed_paged_attention(None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, mpa._i32p(sl), mpa._i32p(qs),
                                       None, FAKE, None, None, 0, None) == mpa.MPA_ERR_INVALID


def test_workspace_required_for_split_rows():
    sh = shape(max_blocks_per_seq=1024)
    seq_lens, qsl = [9000, 40], [0, 1, 5]
    n = mpa.workspace_size(sh, seq_lens, qsl)
    info = mpa.plan_info(sh, seq_lens, qsl)
    assert info.num_decode_seqs == 1 and info.num_prefill_seqs == 1
    assert 9000 > info.split_tokens and info.split_tokens % 16 == 0
    items = info.num_decode_items
    assert items == -(-9000 // info.split_tokens)
    assert n == items * 8 * (128 + 2) * 4
    assert attention_rc(sh, seq_lens, qsl, ws=n - 1) == mpa.MPA_ERR_WORKSPACE
    # the partials' (max, sum) pairs are read as 8-byte vectors: a workspace
    # that is not 16-byte aligned is refused before any launch
    for off in (4, 8):
        assert attention_rc(sh, seq_lens, qsl, ws=n + 64, ws_ptr=FAKE + off) == mpa.MPA_ERR_WORKSPACE


def test_no_workspace_for_short_rows():
    sh = shape()
    assert mpa.workspace_size(sh, [40, 3], [0, 1, 5]) == 0


def test_plan_info_counts():
    sh = shape(num_seqs=5, total_q_tokens=1 + 1 + 70 + 0 + 2, max_blocks_per_seq=64)
    seq_lens = [100, 1, 300, 50, 2]
    qsl = [0, 1, 2, 72, 72, 74]
    info = mpa.plan_info(sh, seq_lens, qsl)
    assert info.num_decode_seqs == 2 and info.num_prefill_seqs == 2
    # bf16 tiles hold 256 (token, head) rows: G = 4 -> 64 tokens per tile
    assert info.num_prefill_tiles == (-(-70 // 64) + 1) * 2
    # f32 tiles hold 64 rows: 16 tokens per tile
    sh32 = shape(num_seqs=5, total_q_tokens=74, max_blocks_per_seq=64, dtype=mpa.MPA_F32)
    assert mpa.plan_info(sh32, seq_lens, qsl).num_prefill_tiles == (-(-70 // 16) + 1) * 2
    assert info.decode_launches == 1


def test_prefill_kv_splits_planned_for_short_chunks():
    # one 256-token chunk on a 4096-token prefix, 32 q / 8 KV heads: 4 query
    # tiles (64 tokens each at G = 4) x 8 KV heads = 32 workgroups, under the
    # 256 target, so the 64-tile prefix is split 8 ways
    sh = shape(num_seqs=1, num_q_heads=32, num_kv_heads=8, total_q_tokens=256, max_blocks_per_seq=272)
    seq_lens, qsl = [4352], [0, 256]
    info = mpa.plan_info(sh, seq_lens, qsl)
    assert info.prefill_max_splits == 8
    assert info.num_prefill_tiles == 4 * 8 * 8
    n = mpa.workspace_size(sh, seq_lens, qsl)
    assert n == 8 * 256 * 32 * (128 + 2) * 4
    assert attention_rc(sh, seq_lens, qsl, ws=n - 1) == mpa.MPA_ERR_WORKSPACE
    # enough query tiles already: no split
    big = shape(num_seqs=1, num_q_heads=32, num_kv_heads=8, total_q_tokens=4096, max_blocks_per_seq=512)
    assert mpa.plan_info(big, [8192], [0, 4096]).prefill_max_splits == 1
    assert mpa.workspace_size(big, [8192], [0, 4096]) == 0
    # a prefix shorter than 8 tiles is not split, nor is the f32 path
    assert mpa.plan_info(sh, [256 + 300], qsl).prefill_max_splits == 1
    sh32 = shape(num_seqs=1, num_q_heads=32, num_kv_heads=8, total_q_tokens=256, max_blocks_per_seq=272,
                 dtype=mpa.MPA_F32)
    assert mpa.plan_info(sh32, seq_lens, qsl).prefill_max_splits == 1
    assert mpa.workspace_size(sh32, seq_lens, qsl) == 0


def test_rope_append_rejects_bad_arguments_before_any_launch():
    """Host validation of mpa_kv_append_rope runs before anything touches a
    device, so it can be exercised here with null device pointers."""
    import ctypes

    L = mpa.lib()
    sl = np.array([100, 40], np.int32)
    qsl = np.array([0, 1, 11], np.int32)
    sh = mpa.make_shape(num_seqs=2, num_q_heads=8, num_kv_heads=2, head_dim=128, num_blocks=16,
                        max_blocks_per_seq=8, total_q_tokens=11, scale=0.1, dtype=mpa.MPA_BF16)
    fake = ctypes.c_void_p(16)  # never dereferenced: every case fails validation first

    def call(rope_dim, max_pos, q=fake, table=fake):
        return L.mpa_kv_append_rope(ctypes.byref(sh), q, fake, fake, fake, fake, fake, fake, fake,
                                    sl.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                                    qsl.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), None, table,
                                    rope_dim, max_pos, None)

    assert call(0, 128) == mpa.MPA_ERR_INVALID
    assert call(24, 128) == mpa.MPA_ERR_INVALID       # not a multiple of 16
    assert call(256, 128) == mpa.MPA_ERR_INVALID      # wider than head_dim
    assert call(128, 99) == mpa.MPA_ERR_INVALID       # position 99 past a 99-row table
    assert call(128, 128, q=None) == mpa.MPA_ERR_INVALID
    assert call(128, 128, table=None) == mpa.MPA_ERR_INVALID


def test_debug_append_slot_checks(monkeypatch):
    """MPA_DEBUG=1: the slots an append writes must be pairwise distinct and
    must not hold a key that the step reads (shared prefix blocks are
    read-only); the check needs the host block tables.  Every case here is
    rejected before any launch."""
    monkeypatch.setenv("MPA_DEBUG", "1")
    sh = shape(num_seqs=2, total_q_tokens=3)
    # sequence 0: 20 keys, appends 1 at position 19 (block 1, slot 3);
    # sequence 1: 40 keys, appends 2 at positions 38, 39 (block 2, slots 6, 7)
    sl, qsl = [20, 40], [0, 1, 3]
    bt = np.arange(16, dtype=np.int32).reshape(2, 8)
    # no host tables: the check cannot run
    assert append_rc(sh, sl, qsl) == mpa.MPA_ERR_INVALID
    # two tokens, one slot: sequence 1 (36 keys) appends positions 34 and 35,
    # slots 2 and 3 of its block 2, which the table maps onto sequence 0's
    # block 1, whose slot 3 sequence 0 appends to
    dup = bt.copy()
    dup[1, 2] = dup[0, 1]
    assert append_rc(sh, [20, 36], [0, 1, 3], dup) == mpa.MPA_ERR_INVALID
    # an append over a key another sequence reads: sequence 1's first block
    # is sequence 0's last, and sequence 1 reads all 16 of its slots
    shared = bt.copy()
    shared[1, 0] = shared[0, 1]
    assert append_rc(sh, sl, qsl, shared) == mpa.MPA_ERR_INVALID
    # an append over the appending sequence's own prefix (a table that
    # repeats a block)
    own = bt.copy()
    own[1, 2] = own[1, 0]
    assert append_rc(sh, sl, qsl, own) == mpa.MPA_ERR_INVALID


def test_probe_arguments_rejected_before_launch():
    L = mpa.lib()
    sink = ctypes.c_void_p(FAKE)
    for buf, n in ((None, 16), (FAKE, 0), (FAKE, 24), (FAKE + 8, 32)):
        assert L.mpa_probe_stream_read(buf, n, sink, None) == mpa.MPA_ERR_INVALID
    assert L.mpa_probe_stream_read(FAKE, 16, None, None) == mpa.MPA_ERR_INVALID
    for iters in (0, -5):
        assert L.mpa_probe_mfma_bf16(iters, sink, None, None) == mpa.MPA_ERR_INVALID
    assert L.mpa_probe_mfma_bf16(10, None, None, None) == mpa.MPA_ERR_INVALID


def test_plan_memo_matches_fresh_planning(monkeypatch):
    """The per-thread memo of the split choices: planning batches A, B, A in
    turn gives what a fresh thread (empty memo) gives for each, a batch that
    differs in one length is planned anew, and the tuning overrides are part
    of the key."""
    import threading

    def batch(last):
        sl = [9000, 5000, 700, 4352 + 256, 2048 + last]
        qsl = [0, 1, 2, 3, 3 + 256, 3 + 256 + last]
        sh = mpa.make_shape(num_seqs=5, num_q_heads=8, num_kv_heads=2, head_dim=128, num_blocks=2000,
                            max_blocks_per_seq=1024, total_q_tokens=qsl[-1], scale=128 ** -0.5, dtype=mpa.MPA_BF16)
        return sh, np.asarray(sl, np.int32), np.asarray(qsl, np.int32)

    def plan(args):
        i = mpa.plan_info(*args)
        return (i.split_tokens, i.num_decode_items, i.prefill_max_splits, mpa.workspace_size(*args))

    def fresh(args):
        out = []
        t = threading.Thread(target=lambda: out.append(plan(args)))
        t.start()
        t.join()
        return out[0]

    a, b = batch(512), batch(640)
    pa, pb = plan(a), plan(b)
    assert plan(a) == pa == fresh(a) and pb == fresh(b)
    monkeypatch.setenv("MPA_SPLIT_TOKENS", "256")
    monkeypatch.setenv("MPA_PREFILL_SPLITS", "3")
    forced = plan(a)
    assert forced[0] == 256 and forced[2] == 3 and forced == fresh(a)
    monkeypatch.delenv("MPA_SPLIT_TOKENS")
    monkeypatch.delenv("MPA_PREFILL_SPLITS")
    assert plan(a) == pa


def test_append_attention_rejects_before_launch():
    """mpa_append_attention runs every check of both calls before its first
    launch: missing new rows, a short workspace and a malformed batch are
    errors here, on a host without a GPU, where any launch would fail."""
    L = mpa.lib()
    sh = shape(max_blocks_per_seq=1024)
    sl = np.asarray([9000, 40], np.int32)
    qs = np.asarray([0, 1, 5], np.int32)
    n = mpa.workspace_size(sh, sl, qs)

    def rc(k_new, ws_ptr, ws, qsl=qs):
        return L.mpa_append_attention(ctypes.byref(sh), FAKE, k_new, k_new, FAKE, FAKE, FAKE, FAKE, FAKE,
                                      mpa._i32p(sl), mpa._i32p(np.asarray(qsl, np.int32)), None, FAKE, None, ws_ptr,
                                      ws, None)

    assert rc(None, FAKE, n) == mpa.MPA_ERR_INVALID
    assert rc(FAKE, FAKE, n - 1) == mpa.MPA_ERR_WORKSPACE
    assert rc(FAKE, FAKE + 8, n + 64) == mpa.MPA_ERR_WORKSPACE
    assert rc(FAKE, FAKE, n, qsl=[0, 2, 1]) == mpa.MPA_ERR_INVALID


def test_empty_batch_without_metadata():
    """An empty step (num_seqs 0) may come with null seq_lens and
    query_start_loc: every planning entry point answers it, and the step's
    calls return ok without launching anything (there is no GPU here)."""
    L = mpa.lib()
    sh = mpa.make_shape(num_seqs=0, num_q_heads=8, num_kv_heads=2, head_dim=128, num_blocks=0, max_blocks_per_seq=0,
                        total_q_tokens=0, scale=0.1, dtype=mpa.MPA_BF16)
    assert L.mpa_workspace_size(ctypes.byref(sh), None, None) == 0
    info = mpa.MpaPlanInfo()
    assert L.mpa_get_plan_info(ctypes.byref(sh), None, None, ctypes.byref(info)) == mpa.MPA_OK
    assert info.num_decode_seqs == 0 and info.num_prefill_seqs == 0 and info.num_prefill_tiles == 0
    t = mpa.MpaStepTime()
    assert L.mpa_predict_step(ctypes.byref(sh), None, None, None, ctypes.byref(t)) == mpa.MPA_OK
    assert t.step_us == 0.0
    mode = ctypes.c_int32(-1)
    assert L.mpa_plan_coexec(ctypes.byref(sh), None, None, None, ctypes.byref(mode), None) == mpa.MPA_OK
    assert mode.value == 0
    assert L.mpa_kv_append(ctypes.byref(sh), None, None, None, None, None, None, None, None, None, None,
                           None) == mpa.MPA_OK
    assert L.mpa_mixed_paged_attention(ctypes.byref(sh), None, None, None, None, None, None, None, None, None,
                                       None, None, None, 0, None) == mpa.MPA_OK
    assert L.mpa_append_attention(ctypes.byref(sh), None, None, None, None, None, None, None, None, None, None,
                                  None, None, None, None, 0, None) == mpa.MPA_OK


def test_noalloc_refuses_batches_beyond_its_array():
    """mpa_append_attention_noalloc: a batch whose partial results exceed
    the fixed array is refused with MPA_ERR_SCRATCH before anything runs
    (here no device exists), and the array's size is the header's."""
    L = mpa.lib()
    src = open(HEADER).read()
    assert "#define MPA_SCRATCH_BYTES ((size_t)256 << 20)" in src and mpa.MPA_SCRATCH_BYTES == 256 << 20
    sl = np.full(256, 32768, np.int32)
    qs = np.arange(257, dtype=np.int32)
    sh = mpa.make_shape(num_seqs=256, num_q_heads=64, num_kv_heads=8, head_dim=128, num_blocks=600000,
                        max_blocks_per_seq=2048, total_q_tokens=256, scale=0.1, dtype=mpa.MPA_BF16)
    assert mpa.workspace_size(sh, sl, qs) > mpa.MPA_SCRATCH_BYTES
    rc = L.mpa_append_attention_noalloc(ctypes.byref(sh), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                        mpa._i32p(sl), mpa._i32p(qs), None, FAKE, None, None)
    assert rc == mpa.MPA_ERR_SCRATCH
    assert "scratch" in mpa.status_string(rc)
