"""Plain fp64 CPU oracle for prefill attention.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, the smoke check and the bench may import this module.
It shares no code with the GPU library (``paper_2607_19438_amd``) and imports nothing from it.

What it computes. The paper's prefill attention kernel (Section 3.1, "Prefill attention" item)
runs the score product Q K^T and the output product P V on the matrix units and keeps an exact
online softmax (a running row maximum) between them, so its output is the same as ordinary
softmax attention. The oracle is that ordinary definition, in float64, per query row:

    s_j = scale * (q . k_j)            for every key j the row may see
    m   = max_j s_j                    (numerical stabilisation; cancels exactly)
    p_j = exp(s_j - m),  l = sum_j p_j
    o   = sum_j p_j v_j / l

Readings of points the paper leaves open (it gives no layout, mask, head grouping or dtype):

* prefill of one prompt from an empty cache: query i sees keys 0..i (causal); ``causal=False``
  lets every query see every key;
* grouped-query attention: H query heads share Hkv key/value heads, query head h reads key/value
  head ``h // (H // Hkv)`` (the layout of the Qwen3 and Llama 3.2 models the paper evaluates);
* q, k, v and the output are bf16, token-major: ``q[B][S][H][D]``, ``k, v[B][S][Hkv][D]``;
* ``scale`` is a caller parameter (1/sqrt(D) for these models).

Alongside the output the oracle returns, per output element, ``sum_j p_j |v_jd|`` (p the exact
softmax weights), the magnitude that the rounding of the weights to bf16 before the P V product
scales. The tolerance derived from it is in ``attn_tolerance``.
"""
from __future__ import annotations

import numpy as np

from .qgemm_oracle import decode_bf16

__all__ = ["attention", "attention_rows", "attn_tolerance", "attn_ratio", "kv_head_of",
           "ATTN_P_REL", "ATTN_OUT_REL"]

# Tolerance constants (see attn_tolerance): the weights p/l enter the output product as bf16
# (relative rounding 2**-9) and the output is stored as bf16 (relative 2**-9); each term is
# allowed twice its rounding unit, which also covers the fp32 score and exponent errors (relative
# ~1e-5 at D = 128 for unit-variance inputs).
ATTN_P_REL = 2.0 ** -7
ATTN_OUT_REL = 2.0 ** -8


def kv_head_of(h: int, H: int, Hkv: int) -> int:
    """Key/value head read by query head h under grouped-query attention."""
    if H % Hkv != 0:
        raise ValueError("H must be a multiple of Hkv")
    return h // (H // Hkv)


def _decode(q_bits, k_bits, v_bits):
    q = decode_bf16(q_bits)
    k = decode_bf16(k_bits)
    v = decode_bf16(v_bits)
    if q.ndim != 4 or k.ndim != 4 or v.shape != k.shape:
        raise ValueError("q must be [B][S][H][D], k and v [B][S][Hkv][D]")
    B, S, H, D = q.shape
    if k.shape[0] != B or k.shape[1] != S or k.shape[3] != D:
        raise ValueError("q, k and v disagree on B, S or D")
    return q, k, v


def _scores(qh, kh, scale):
    """s[i][j] = scale * (q_i . k_j): queries qh [n][D], keys kh [S][D]."""
    return (qh @ kh.T) * scale


def _visible(rows, S, causal):
    """Boolean [len(rows)][S]: may query row i see key j (j <= i when causal)."""
    rows = np.asarray(rows)
    if not causal:
        return np.ones((rows.size, S), dtype=bool)
    return np.arange(S)[None, :] <= rows[:, None]


def _softmax_weights(s, visible):
    """p_j = exp(s_j - m) over the visible keys (m their maximum), and l = sum_j p_j."""
    s = np.where(visible, s, -np.inf)
    m = np.max(s, axis=1, keepdims=True)
    p = np.exp(s - m)
    return p, np.sum(p, axis=1, keepdims=True)


def _combine(p, l, vh):
    """o = sum_j p_j v_j / l, and sum_j p_j |v_j| / l."""
    return (p @ vh) / l, (p @ np.abs(vh)) / l


def _head(qh, kh, vh, rows, causal, scale):
    s = _scores(qh, kh, scale)
    p, l = _softmax_weights(s, _visible(rows, kh.shape[0], causal))
    return _combine(p, l, vh)


def attention(q_bits, k_bits, v_bits, causal: bool, scale: float):
    """Returns (o, absv), both float64 [B][S][H][D]."""
    q, k, v = _decode(q_bits, k_bits, v_bits)
    B, S, H, D = q.shape
    Hkv = k.shape[2]
    o = np.zeros((B, S, H, D))
    absv = np.zeros((B, S, H, D))
    for b in range(B):
        for h in range(H):
            g = kv_head_of(h, H, Hkv)
            o[b, :, h, :], absv[b, :, h, :] = _head(q[b, :, h, :], k[b, :, g, :], v[b, :, g, :],
                                                    np.arange(S), causal, scale)
    return o, absv


def attention_rows(q_bits, k_bits, v_bits, causal: bool, scale: float, rows):
    """The rows (b, i, h) of ``attention`` one by one: returns (o, absv), each [n][D]."""
    q, k, v = _decode(q_bits, k_bits, v_bits)
    H = q.shape[2]
    Hkv = k.shape[2]
    out_o, out_a = [], []
    for b, i, h in rows:
        g = kv_head_of(int(h), H, Hkv)
        o, a = _head(q[b, i, h][None, :], k[b, :, g, :], v[b, :, g, :], [int(i)], causal, scale)
        out_o.append(o[0])
        out_a.append(a[0])
    return np.array(out_o), np.array(out_a)


def attn_tolerance(o_ref, absv):
    """Per-element bound on |o - o_ref| for a kernel that rounds the softmax weights to bf16 before
    the P V product (fp32 accumulation) and stores o as bf16:
        ATTN_P_REL * sum_j p_j |v_jd| / l  +  ATTN_OUT_REL * |o_ref|  (+ 1e-30)."""
    return ATTN_P_REL * np.asarray(absv) + ATTN_OUT_REL * np.abs(np.asarray(o_ref)) + 1e-30


def attn_ratio(o, o_ref, absv) -> float:
    """max |o - o_ref| / tolerance (inf if o has a non-finite entry)."""
    o = np.asarray(o, dtype=np.float64)
    if not np.all(np.isfinite(o)):
        return float("inf")
    return float(np.max(np.abs(o - o_ref) / attn_tolerance(o_ref, absv))) if o.size else 0.0
