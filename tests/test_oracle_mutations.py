"""Planted mistakes in the oracle (CPU only) must each break at least one pin.

Each mutant replaces one oracle function with a plausible wrong variant -- a
shifted causal diagonal, the interleaved head mapping, a dropped scale, a
transposed cache layout, a dropped term of the log-sum-exp -- and the test
asserts that the pins of ``test_oracle_pins`` reject it.
"""

import numpy as np
import pytest

import test_oracle_pins as pins
from oracle import ref


def _seq_attn_factory(visible_fn=None, head_map=None, scale_override=None):
    def seq_attn(q_rows, k, v, prefix, scale, num_kv_heads, row_tile=512):
        c, hq, d = q_rows.shape
        big_l = k.shape[0]
        g = hq // num_kv_heads
        o = np.empty((c, hq, d))
        lse = np.empty((c, hq))
        keys = np.arange(big_l)
        rows = np.arange(c)
        vis = visible_fn(keys, rows, prefix) if visible_fn else keys[None] <= (prefix + rows)[:, None]
        vis = vis | (keys[None] == 0)  # keep every row non-empty
        for h in range(hq):
            kv = head_map(h, g, num_kv_heads) if head_map else h // g
            o[:, h], lse[:, h] = ref.softmax_attention(
                q_rows[:, h], k[:, kv], v[:, kv], scale if scale_override is None else scale_override, vis)
        return o, lse
    return seq_attn


def _bad_lse(q, k, v, scale, visible):
    o, lse = _good_softmax(q, k, v, scale, visible)
    s = np.where(visible, scale * (q @ k.T), -np.inf)
    return o, lse - s.max(axis=1)  # drops the maximum from the log-sum-exp


_good_softmax = ref.softmax_attention


def _transposed_gather(k_cache, v_cache, block_row, n_tokens, num_kv_heads, head_dim, block_size, dtype):
    if n_tokens == 0:
        z = np.zeros((0, num_kv_heads, head_dim))
        return z, z.copy()
    nb = -(-n_tokens // block_size)
    blocks = np.asarray(block_row[:nb], dtype=np.int64)
    # wrong: reads K as [b][h][t][d] (the "natural" layout) instead of the header's
    kb = ref.decode_raw(k_cache.reshape(-1, num_kv_heads, block_size, head_dim)[blocks], dtype)
    vb = ref.decode_raw(v_cache.reshape(-1, num_kv_heads, head_dim, block_size)[blocks], dtype)
    k = kb.transpose(0, 2, 1, 3).reshape(-1, num_kv_heads, head_dim)
    v = vb.transpose(0, 3, 1, 2).reshape(-1, num_kv_heads, head_dim)
    return k[:n_tokens], v[:n_tokens]


def _rope_interleaved(x_raw, positions, cos_sin, rope_dim, dtype):
    # wrong: rotates adjacent pairs (2j, 2j+1) instead of (j, j + R/2)
    x = ref.decode_raw(x_raw, dtype).astype(np.float32)
    cs = np.asarray(cos_sin, np.float32)[np.asarray(positions)]
    c, s = cs[:, None, :, 0], cs[:, None, :, 1]
    y = x.copy()
    a, b = x[:, :, 0:rope_dim:2], x[:, :, 1:rope_dim:2]
    y[:, :, 0:rope_dim:2] = a * c - b * s
    y[:, :, 1:rope_dim:2] = b * c + a * s
    return ref.round_bf16(y) if dtype == "bf16" else y


def _rope_sign(x_raw, positions, cos_sin, rope_dim, dtype):
    # wrong: rotates the other way
    cs = np.asarray(cos_sin, np.float32).copy()
    cs[..., 1] = -cs[..., 1]
    return _good_rope(x_raw, positions, cs, rope_dim, dtype)


_good_rope = ref.rope_reference


def _e4m3_fnuz_values():
    # wrong: the "fnuz" variant's exponent bias 8 (and no negative zero)
    v = _good_e4m3() / 2.0
    v[0x80] = np.nan
    return v


def _quantize_truncating(y32):
    # wrong: rounds magnitudes toward zero instead of to nearest even
    vals = _good_e4m3()[:0x7F]
    a = np.abs(np.asarray(y32, np.float64))
    pick = np.clip(np.searchsorted(vals, a, side="right") - 1, 0, 0x7E)
    return (pick | np.where(np.signbit(y32), 0x80, 0)).astype(np.uint8)


_good_e4m3 = ref.e4m3_values


def _round_bf16_truncating(x32):
    # wrong: drops the low 16 bits of the float32 instead of rounding them
    return (np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _round_bf16_ties_away(x32):
    # wrong: rounds ties away from zero instead of to the even pattern
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + np.uint64(0x8000)) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(x32)
    r[nan] = 0x7FC0
    return r


def _fp8_codes_times_scale(x_raw_bf16, scale):
    # wrong: multiplies by the scale instead of by its reciprocal
    return ref.quantize_e4m3(ref.decode_raw(x_raw_bf16, "bf16").astype(np.float32) * np.float32(scale))


MUTANTS = {
    "rope_interleaved_pairs": ("rope_reference", _rope_interleaved),
    "rope_reversed": ("rope_reference", _rope_sign),
    "e4m3_fnuz_bias": ("e4m3_values", _e4m3_fnuz_values),
    "e4m3_truncating": ("quantize_e4m3", _quantize_truncating),
    "round_bf16_truncating": ("round_bf16", _round_bf16_truncating),
    "round_bf16_ties_away": ("round_bf16", _round_bf16_ties_away),
    "fp8_codes_times_scale": ("fp8_codes", _fp8_codes_times_scale),
    "top_left_causal": ("sequence_attention", _seq_attn_factory(
        visible_fn=lambda keys, rows, prefix: keys[None] <= rows[:, None])),
    "exclusive_diagonal": ("sequence_attention", _seq_attn_factory(
        visible_fn=lambda keys, rows, prefix: keys[None] < (prefix + rows)[:, None])),
    "interleaved_heads": ("sequence_attention", _seq_attn_factory(
        head_map=lambda h, g, hkv: h % hkv)),
    "dropped_scale": ("sequence_attention", _seq_attn_factory(scale_override=1.0)),
    "lse_without_max": ("softmax_attention", _bad_lse),
    "natural_k_layout": ("gather_kv", _transposed_gather),
}

PIN_TESTS = [
    lambda: pins.test_golden_hand_worked(),
    lambda: pins.test_brute_force("f32", 0),
    lambda: pins.test_brute_force("bf16", 1),
    lambda: pins.test_block_size_invariance_and_sdpa("f32"),
    lambda: pins.test_zero_query_gives_running_mean(),
    lambda: pins.test_rope_hand_worked(),
    lambda: pins.test_rope_zero_and_quarter_turn("f32"),
    lambda: pins.test_e4m3_table_fixed_points(),
    lambda: pins.test_e4m3_quantize_round_trip_ties_and_saturation(),
    lambda: pins.test_round_bf16_ties_carries_and_nan(),
    lambda: pins.test_rope_bf16_rounding_hand_worked(),
    lambda: pins.test_fp8_codes_scale_direction_and_round_trip(),
]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(ref, attr, fn)
    caught = 0
    for t in PIN_TESTS:
        try:
            t()
        except AssertionError:
            caught += 1
    assert caught > 0, f"no pin rejects the mutant {name}"
