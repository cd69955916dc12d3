"""Plant plausible mistakes in the oracle (CPU only) and check that some pin fails for each.

A pin that no mistake can break pins nothing. Each mutant below replaces one
oracle helper with a subtly wrong version; the pin checks of
``test_oracle_dense`` / ``test_oracle_moe`` must then raise.
"""
import numpy as np
import pytest

import oracle
import oracle.qgemm_oracle as qo
import synth
import test_oracle_dense as td
import test_oracle_moe as tm

_orig_decode_q = qo.decode_q
_orig_dequant = qo.dequant
_orig_decode_bf16 = qo.decode_bf16
_orig_round = qo.round_to_bf16


def _q4_swapped(wq, fmt, K):
    if fmt != qo.FMT_Q4:
        return _orig_decode_q(wq, fmt, K)
    b = np.asarray(wq).astype(np.int64)
    q = np.empty(b.shape[:-1] + (K,), np.int64)
    q[..., 0::2] = (b >> 4) & 0xF
    q[..., 1::2] = b & 0xF
    return q - 8


def _q4_neg_offset(wq, fmt, K):
    q = _orig_decode_q(wq, fmt, K)
    return -q if fmt == qo.FMT_Q4 else q


def _q4_no_offset(wq, fmt, K):
    q = _orig_decode_q(wq, fmt, K)
    return q + 8 if fmt == qo.FMT_Q4 else q


def _q8_unsigned(wq, fmt, K):
    if fmt != qo.FMT_Q8:
        return _orig_decode_q(wq, fmt, K)
    return np.ascontiguousarray(wq).view(np.uint8).astype(np.int64)


def _scale_tiled(wq, scales, fmt, K):
    q = _orig_decode_q(wq, fmt, K).astype(np.float64)
    s = np.asarray(scales, np.float16).astype(np.float64)
    return q * np.tile(s, (1, 32))                  # wrong block <-> k mapping


def _drop_last_block(wq, scales, fmt, K):
    w = _orig_dequant(wq, scales, fmt, K)
    w[..., K - 32:] = 0.0
    return w


def _bf16_bad_shift(bits):
    b = np.ascontiguousarray(np.asarray(bits, np.uint16)).astype(np.uint32) << np.uint32(15)
    return b.view(np.float32).astype(np.float64)


def _round_truncate(v):
    v = np.asarray(v, np.float64)
    bits = (v.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return _orig_decode_bf16(bits), bits


def _silu_wrong_sign(z):
    z = np.asarray(z, np.float64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(z))


def _moe_gather_by_assignment(x_bits, idx, offsets, wq_list, s_list, topk, fmt):
    # gathers x[a] instead of x[a // topk]
    idx = np.asarray(idx, np.int64)
    x = qo.decode_bf16(x_bits)
    K = x.shape[1]
    N = np.asarray(s_list[0]).shape[0]
    y = np.zeros((idx.size, N))
    b = np.zeros((idx.size, N))
    for e in range(len(wq_list)):
        rows = np.nonzero(idx == e)[0]
        if rows.size:
            xe = x[np.minimum(rows, x.shape[0] - 1)]
            w = qo.dequant(wq_list[e], s_list[e], fmt, K)
            y[rows] = xe @ w.T
            b[rows] = np.abs(xe) @ np.abs(w).T
    return y, b


def _combine_wrong_slot(y2, route_w, topk, bound2=None):
    w = np.roll(np.asarray(route_w), 1)
    return _orig_combine(y2, w, topk, bound2)


_orig_combine = qo.combine
_orig_moe_entries = qo.moe_entries
_orig_down_combine = qo.down_combine_tokens


def _down_combine_token_row(h_bits, idx, route_w, wd_q, wd_s, topk, fmt, tokens):
    # reads every slot's activations from row t (the token) instead of row t*topk+j (the slot)
    h = np.asarray(h_bits)
    fake = h.copy()
    for t in np.asarray(tokens, np.int64):
        for j in range(topk):
            fake[t * topk + j] = h[min(t, h.shape[0] - 1)]
    return _orig_down_combine(fake, idx, route_w, wd_q, wd_s, topk, fmt, tokens)
_orig_bar_ratio = qo.bar_ratio


def _entries_gather_by_assignment(x_bits, idx, wq_list, s_list, topk, fmt, assigns, cols, bf16_weights=False):
    # reads x[a] (clamped to the token count) instead of x[a // topk]
    a = np.asarray(assigns, np.int64)
    xb = np.asarray(x_bits)
    rows = np.minimum(a, xb.shape[0] - 1)
    # route through the real function with topk=1 on a row table that picks x[rows]
    return _orig_moe_entries(xb[rows], np.asarray(idx)[a], wq_list, s_list, 1, fmt, np.arange(a.size), cols,
                             bf16_weights)


def _entries_expert_of_token(x_bits, idx, wq_list, s_list, topk, fmt, assigns, cols, bf16_weights=False):
    # takes the expert of slot a // topk instead of slot a
    idx = np.asarray(idx, np.int64)
    wrong = idx[np.asarray(assigns, np.int64) // topk]
    fake = idx.copy()
    fake[np.asarray(assigns, np.int64)] = wrong
    return _orig_moe_entries(x_bits, fake, wq_list, s_list, topk, fmt, assigns, cols, bf16_weights)


def _bar_ratio_swapped(y, y_ref, bound, rel=qo.TOL_REL, abs_=qo.TOL_ABS):
    return _orig_bar_ratio(y, y_ref, bound, abs_, rel)


def _bar_ratio_no_abs(y, y_ref, bound, rel=qo.TOL_REL, abs_=qo.TOL_ABS):
    with np.errstate(divide="ignore", invalid="ignore"):
        return _orig_bar_ratio(y, y_ref, bound, rel, 0.0)


def _bar_ratio_ignores_nan(y, y_ref, bound, rel=qo.TOL_REL, abs_=qo.TOL_ABS):
    y = np.asarray(y, np.float64)
    if y.size == 0:
        return 0.0
    err = np.abs(y - np.asarray(y_ref, np.float64))
    return float(np.nanmax(np.where(np.isfinite(err), err, np.nan) / (rel * np.asarray(bound, np.float64) + abs_)))

MUTANTS = {
    "q4_nibbles_swapped": ("decode_q", _q4_swapped),
    "q4_offset_sign": ("decode_q", _q4_neg_offset),
    "q4_offset_dropped": ("decode_q", _q4_no_offset),
    "q8_read_unsigned": ("decode_q", _q8_unsigned),
    "scale_block_index": ("dequant", _scale_tiled),
    "last_k_block_dropped": ("dequant", _drop_last_block),
    "bf16_decode_shift": ("decode_bf16", _bf16_bad_shift),
    "bf16_round_truncates": ("round_to_bf16", _round_truncate),
    "silu_sign": ("silu", _silu_wrong_sign),
    "moe_gather_row": ("moe", _moe_gather_by_assignment),
    "combine_slot": ("combine", _combine_wrong_slot),
    "moe_entries_gather_row": ("moe_entries", _entries_gather_by_assignment),
    "moe_entries_expert_of_token": ("moe_entries", _entries_expert_of_token),
    "down_combine_token_row": ("down_combine_tokens", _down_combine_token_row),
    "bar_ratio_rel_abs_swapped": ("bar_ratio", _bar_ratio_swapped),
    "bar_ratio_no_abs_term": ("bar_ratio", _bar_ratio_no_abs),
    "bar_ratio_ignores_nan": ("bar_ratio", _bar_ratio_ignores_nan),
}


def _pins():
    F8, F4 = synth.FMT_Q8, synth.FMT_Q4
    p = []
    for fmt in (F8, F4):
        p += [(td.test_bruteforce_exact_rational, dict(fmt=fmt, M=3, N=5, K=64)),
              (td.test_bruteforce_exact_rational, dict(fmt=fmt, M=5, N=3, K=96)),
              (td.test_unit_scale_q_one_gives_row_sums, dict(fmt=fmt)),
              (td.test_one_hot_pins_column_mapping, dict(fmt=fmt, n0=1, k0=95)),
              (td.test_one_hot_scale_block_pins_block_index, dict(fmt=fmt, blk=1)),
              (tm.test_moe_exact_rational_tiny, dict(fmt=fmt)),
              (tm.test_moe_entries_exact_rational, dict(fmt=fmt)),
              (tm.test_moe_entries_match_moe, dict(fmt=fmt, bf16_weights=False)),
              (tm.test_down_combine_tokens_matches_chain, dict(fmt=fmt)),
              (tm.test_moe_ffn_weighted_per_expert_dense_loop, dict(fmt=fmt))]
    p += [(td.test_nibble_order_low_nibble_first, {}), (td.test_q4_decode_every_nibble, {}),
          (td.test_q8_extremes_and_fp16_max_scale, dict(qv=-128)), (td.test_bf16_decode_known_patterns, {}),
          (tm.test_silu_closed_forms, {}), (tm.test_bf16_rounding_closed_forms, {}),
          (tm.test_combine_closed_forms, {}), (tm.test_bar_ratio_closed_forms, {}),
          (tm.test_bar_ratio_agrees_with_within_bar, {})]
    return p


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_some_pin_catches_mutant(name, monkeypatch):
    attr, fn = MUTANTS[name]
    monkeypatch.setattr(qo, attr, fn)
    monkeypatch.setattr(oracle, attr, fn)
    caught = []
    for f, kw in _pins():
        try:
            f(**kw)
        except Exception as exc:  # an assertion, or a shape error the mistake provokes
            caught.append((f.__name__, type(exc).__name__))
    assert caught, f"no pin caught mutant {name}"


def test_pins_pass_unmutated():
    for f, kw in _pins():
        f(**kw)
