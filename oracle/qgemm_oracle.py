"""Plain fp64 CPU oracle for the block-quantised prefill GEMM.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, the smoke check and the bench's
CPU-baseline leg may import this module. It shares no code with the GPU
library (``paper_2607_19438_amd``) and imports nothing from it.

What it computes. The paper's tensor-core kernels (Section 3.1) are fast
implementations of two plain operations:

* dense GEMM over 4-bit / 8-bit block-quantised projection weights
  (Section 3.1, "Dense GEMM" item): ``y = x . dequant(W)^T``;
* the MoE expert GEMM, which evaluates each active expert's projection over
  the tokens routed to it (Section 3.1, "MoE expert GEMM" item);

plus, around the MoE GEMMs, the SiLU-gated gate/up activation (Section 3.1,
"Fused MoE gate/up projection" item) and the router-weighted sum of the
selected experts' outputs. Since every one of these has a plain definition,
the oracle is that definition written out in float64, step by step.

Readings of points the paper leaves open (the paper gives no byte layout,
block size, scale type, rounding or tolerance):

* weights are ``W[N][K]`` with K contiguous; one fp16 scale per 32 consecutive
  K elements of a row (``scales[N][K/32]``);
* Q8 stores a signed int8 ``q`` and means ``q * s``;
* Q4 stores two nibbles per byte, element ``2j`` in the low nibble of byte
  ``j`` and element ``2j+1`` in the high nibble; a nibble ``u`` means
  ``(u - 8) * s``;
* activations are bf16; the MoE intermediate ``h = silu(gate) * up`` is rounded
  to bf16 (round to nearest, ties to even) because it is the next GEMM's
  activation; gate is columns ``[0, inter)`` and up is ``[inter, 2*inter)`` of
  the gate/up projection's output;
* the acceptance bar is, per output element,
  ``|y - y_ref| <= 1e-3 * sum_k |x_k * w_k| + 1e-6``.

``bf16_weights=True`` (dequant, dense, dense_entries, moe, moe_entries)
evaluates the same definition after rounding every dequantised weight
``q * s`` to bf16 (nearest, ties to even). It is not the paper's definition but
the precision the GPU library states for its weight tiles; since ``q * s`` is
exact in both float64 and float32, the rounded weights are bit-identical to the
library's, and the remaining GPU difference is fp32 summation order only. It
gives a much tighter check than the acceptance bar, whose 1e-3 is below the
bf16 rounding unit (2**-8) and so holds only statistically, for large K.

Every intermediate is exact in float64 up to the contraction's own rounding
(an int of at most 8 bits times an 11-bit fp16 significand fits in 53 bits);
the contraction's error is below ``K * 2**-53 * sum_k |x_k w_k|``.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = [
    "FMT_Q8", "FMT_Q4", "QBLOCK", "TOL_REL", "TOL_ABS",
    "decode_bf16", "decode_q", "dequant",
    "dense", "dense_entries",
    "moe", "moe_entries",
    "silu", "round_to_bf16", "swiglu", "combine", "moe_ffn", "moe_ffn_tokens", "down_combine_tokens",
    "within_bar", "bar_ratio", "fp32_sum_rel", "SILU_LIPSCHITZ", "swiglu_err_bound", "moe_abs_apply",
    "ffn_out_tolerance",
]

FMT_Q8 = 0
FMT_Q4 = 1
QBLOCK = 32
TOL_REL = 1e-3
TOL_ABS = 1e-6


# ---------------------------------------------------------------------------
# decoders (storage -> exact float64 / integer values)
# ---------------------------------------------------------------------------

def decode_bf16(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64. bf16 is the upper half of an IEEE binary32."""
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    wide = b.astype(np.uint32) << np.uint32(16)
    return wide.view(np.float32).astype(np.float64)


def decode_q(wq, fmt: int, K: int) -> np.ndarray:
    """Signed integer weight values ``[N][K]`` encoded by the Q8 / Q4 storage."""
    wq = np.asarray(wq)
    if fmt == FMT_Q8:
        if wq.shape[-1] != K:
            raise ValueError("Q8 storage must be [N][K]")
        return np.ascontiguousarray(wq).view(np.int8).astype(np.int64)
    if fmt == FMT_Q4:
        if wq.shape[-1] * 2 != K:
            raise ValueError("Q4 storage must be [N][K/2]")
        b = np.ascontiguousarray(wq).view(np.uint8).astype(np.int64)
        q = np.empty(b.shape[:-1] + (K,), dtype=np.int64)
        q[..., 0::2] = b & 0xF            # element 2j: low nibble of byte j
        q[..., 1::2] = (b >> 4) & 0xF     # element 2j+1: high nibble of byte j
        return q - 8
    raise ValueError(f"unknown format {fmt}")


def dequant(wq, scales, fmt: int, K: int, bf16_weights: bool = False) -> np.ndarray:
    """``w[n][k] = s[n][k // 32] * q[n][k]`` in float64 (exact); optionally rounded to bf16."""
    if K % QBLOCK:
        raise ValueError("K must be a multiple of 32")
    q = decode_q(wq, fmt, K).astype(np.float64)
    s = np.asarray(scales, dtype=np.float16).astype(np.float64)
    if s.shape[-1] != K // QBLOCK:
        raise ValueError("scales must be [N][K/32]")
    w = q * np.repeat(s, QBLOCK, axis=-1)
    return round_to_bf16(w)[0] if bf16_weights else w


# ---------------------------------------------------------------------------
# dense GEMM (Section 3.1, dense item)
# ---------------------------------------------------------------------------

def dense(x_bits, wq, scales, fmt: int, bf16_weights: bool = False):
    """``y[m][n] = sum_k x[m][k] * w[n][k]`` and its bar ``sum_k |x[m][k] * w[n][k]|``."""
    x = decode_bf16(x_bits)
    K = x.shape[1]
    w = dequant(wq, scales, fmt, K, bf16_weights)
    y = x @ w.T
    bound = np.abs(x) @ np.abs(w).T
    return y, bound


def dense_entries(x_bits, wq, scales, fmt: int, rows, cols, bf16_weights: bool = False):
    """The same definition evaluated one output element at a time, for sampled ``(rows[i], cols[i])``."""
    rows = np.asarray(rows, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    x = decode_bf16(np.asarray(x_bits)[rows])
    K = x.shape[1]
    ucols, inv = np.unique(cols, return_inverse=True)
    wq_sel = np.asarray(wq)[ucols]
    s_sel = np.asarray(scales)[ucols]
    w = dequant(wq_sel, s_sel, fmt, K, bf16_weights)[inv]
    y = np.einsum("pk,pk->p", x, w)
    bound = np.einsum("pk,pk->p", np.abs(x), np.abs(w))
    return y, bound


# ---------------------------------------------------------------------------
# MoE expert GEMM (Section 3.1, MoE expert GEMM item)
# ---------------------------------------------------------------------------

def _check_routing(idx, offsets, E):
    idx = np.asarray(idx, dtype=np.int64)
    if idx.size and (idx.min() < 0 or idx.max() >= E):
        raise ValueError("expert index out of range")
    if offsets is not None:
        counts = np.bincount(idx, minlength=E)[:E]
        ref = np.concatenate([[0], np.cumsum(counts)])
        if not np.array_equal(np.asarray(offsets, dtype=np.int64), ref):
            raise ValueError("expert_offsets is not the prefix sum of the routing counts")
    return idx


def moe(x_bits, idx, offsets, wq_list, s_list, topk: int, fmt: int, bf16_weights: bool = False):
    """Per active expert, project its routed token rows; rows come back in token-slot order.

    Assignment ``a = t*topk + j`` is token ``t``'s ``j``-th selected expert
    ``idx[a]``; its output row is ``y[a] = dequant(W_idx[a]) . x[t]``.
    """
    E = len(wq_list)
    idx = _check_routing(idx, offsets, E)
    x = decode_bf16(x_bits)
    K = x.shape[1]
    N = np.asarray(s_list[0]).shape[0]
    A = idx.size
    y = np.zeros((A, N))
    bound = np.zeros((A, N))
    for e in range(E):
        rows = np.nonzero(idx == e)[0]
        if rows.size == 0:
            continue                      # inactive expert: no work, no rows
        xe = x[rows // topk]
        w = dequant(wq_list[e], s_list[e], fmt, K, bf16_weights)
        y[rows] = xe @ w.T
        bound[rows] = np.abs(xe) @ np.abs(w).T
    return y, bound


def moe_entries(x_bits, idx, wq_list, s_list, topk: int, fmt: int, assigns, cols, bf16_weights: bool = False):
    """``y[a][n]`` for sampled ``(assigns[i], cols[i])``, one element at a time."""
    idx = np.asarray(idx, dtype=np.int64)
    assigns = np.asarray(assigns, dtype=np.int64)
    cols = np.asarray(cols, dtype=np.int64)
    x = decode_bf16(np.asarray(x_bits)[assigns // topk])
    K = x.shape[1]
    y = np.empty(assigns.size)
    bound = np.empty(assigns.size)
    experts = idx[assigns]
    for e in np.unique(experts):
        sel = np.nonzero(experts == e)[0]
        w = dequant(np.asarray(wq_list[e])[cols[sel]], np.asarray(s_list[e])[cols[sel]], fmt, K, bf16_weights)
        y[sel] = np.einsum("pk,pk->p", x[sel], w)
        bound[sel] = np.einsum("pk,pk->p", np.abs(x[sel]), np.abs(w))
    return y, bound


# ---------------------------------------------------------------------------
# around the MoE GEMMs: SiLU gate (Section 3.1, fused gate/up item) and combine
# ---------------------------------------------------------------------------

def silu(z):
    """``silu(z) = z / (1 + exp(-z))`` in float64."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def round_to_bf16(v):
    """Round float64 values to the nearest bf16 (ties to even); returns ``(values, bits)``."""
    v = np.asarray(v, dtype=np.float64)
    out = np.empty_like(v)
    a = np.abs(v)
    finite = np.isfinite(v)
    # bf16: 8 significant bits, exponent range of binary32 (min normal 2**-126).
    m, e = np.frexp(np.where(finite, a, 0.0))          # a = m * 2**e, m in [0.5, 1)
    e = np.maximum(e, -125)                              # below 2**-126: fixed step 2**-133
    r = np.rint(np.ldexp(np.where(finite, a, 0.0), 8 - e))   # rint rounds half to even
    mag = np.ldexp(r, e - 8)
    mag = np.where(mag > 3.3895313892515355e38, np.inf, mag)
    out[:] = np.where(finite, np.copysign(mag, v), v)
    bits = (out.astype(np.float32).view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    return out, bits


def swiglu(y1, inter: int):
    """``h = bf16(silu(gate) * up)`` with gate = columns ``[0, inter)``, up = ``[inter, 2*inter)``."""
    y1 = np.asarray(y1, dtype=np.float64)
    if y1.shape[1] != 2 * inter:
        raise ValueError("gate/up output must have 2*inter columns")
    h = silu(y1[:, :inter]) * y1[:, inter:]
    return round_to_bf16(h)


def combine(y2, route_w, topk: int, bound2=None):
    """``out[t] = sum_j w[t*topk+j] * y2[t*topk+j]`` and its bar ``sum_j |w| * bound2``."""
    y2 = np.asarray(y2, dtype=np.float64)
    w = np.asarray(route_w, dtype=np.float32).astype(np.float64)
    T = y2.shape[0] // topk
    out = np.zeros((T, y2.shape[1]))
    bnd = np.zeros((T, y2.shape[1]))
    for j in range(topk):
        rows = np.arange(T) * topk + j
        out += w[rows, None] * y2[rows]
        if bound2 is not None:
            bnd += np.abs(w[rows, None]) * np.asarray(bound2)[rows]
    return out, bnd


def moe_ffn(x_bits, idx, offsets, route_w, wgu_q, wgu_s, wd_q, wd_s, topk: int, inter: int, fmt: int):
    """Whole MoE FFN: gate/up expert GEMM, SiLU gate, down expert GEMM, router-weighted sum."""
    y1, b1 = moe(x_bits, idx, offsets, wgu_q, wgu_s, topk, fmt)
    h, h_bits = swiglu(y1, inter)
    y2, b2 = moe(h_bits, idx, offsets, wd_q, wd_s, 1, fmt)
    out, bout = combine(y2, route_w, topk, b2)
    return dict(y1=y1, bound1=b1, h=h, h_bits=h_bits, y2=y2, bound2=b2, out=out, bound_out=bout)


def moe_ffn_tokens(x_bits, idx, route_w, wgu_q, wgu_s, wd_q, wd_s, topk: int, inter: int, fmt: int,
                   tokens, cols=None, with_tolerance: bool = False):
    """The MoE FFN output ``out[t]`` for a few sampled tokens, evaluated token by token.

    Returns ``(out, bound_out)``, plus the propagated tolerance of ffn_out_tolerance when
    ``with_tolerance``."""
    idx = np.asarray(idx, dtype=np.int64)
    w = np.asarray(route_w, dtype=np.float32).astype(np.float64)
    xall = np.asarray(x_bits)
    res_out, res_bound, res_tol = [], [], []
    for t in np.asarray(tokens, dtype=np.int64):
        x = decode_bf16(xall[t:t + 1])
        K = x.shape[1]
        o = None
        bo = None
        to = None
        for j in range(topk):
            a = t * topk + j
            e = idx[a]
            wgu = dequant(wgu_q[e], wgu_s[e], fmt, K)
            g = (x @ wgu.T)[0]
            b1 = (np.abs(x) @ np.abs(wgu).T)[0]
            h, h_bits = round_to_bf16(silu(g[:inter]) * g[inter:])
            hx = decode_bf16(h_bits[None, :])
            wd = dequant(wd_q[e], wd_s[e], fmt, inter)
            if cols is not None:
                wd = wd[np.asarray(cols)]
            y2 = (hx @ wd.T)[0]
            b2 = (np.abs(hx) @ np.abs(wd).T)[0]
            eh = swiglu_err_bound(g[None, :], b1[None, :], inter)
            t2 = (eh @ np.abs(wd).T)[0] + TOL_REL * b2 + TOL_ABS
            o = w[a] * y2 if o is None else o + w[a] * y2
            bo = abs(w[a]) * b2 if bo is None else bo + abs(w[a]) * b2
            to = abs(w[a]) * t2 if to is None else to + abs(w[a]) * t2
        res_out.append(o)
        res_bound.append(bo)
        res_tol.append(to)
    if with_tolerance:
        return np.array(res_out), np.array(res_bound), np.array(res_tol)
    return np.array(res_out), np.array(res_bound)


def down_combine_tokens(h_bits, idx, route_w, wd_q, wd_s, topk: int, fmt: int, tokens):
    """``out[t] = sum_j w[t*topk+j] * (dequant(W_down[idx[t*topk+j]]) . h[t*topk+j])`` for sampled
    tokens, from given bf16 activations ``h`` (one row per token slot): the down expert projection
    (Section 3.1, MoE expert GEMM item) followed by the router-weighted sum, on the same inputs a
    GPU chain fed. Returns ``(out, bound_out)`` with ``bound_out[t] = sum_j |w| sum_i |h_i w_i|``."""
    idx = np.asarray(idx, dtype=np.int64)
    w = np.asarray(route_w, dtype=np.float32).astype(np.float64)
    hall = np.asarray(h_bits)
    outs, bounds = [], []
    for t in np.asarray(tokens, dtype=np.int64):
        o = None
        b = None
        for j in range(topk):
            a = t * topk + j
            hx = decode_bf16(hall[a:a + 1])
            wd = dequant(wd_q[idx[a]], wd_s[idx[a]], fmt, hx.shape[1])
            y2 = (hx @ wd.T)[0]
            b2 = (np.abs(hx) @ np.abs(wd).T)[0]
            o = w[a] * y2 if o is None else o + w[a] * y2
            b = abs(w[a]) * b2 if b is None else b + abs(w[a]) * b2
        outs.append(o)
        bounds.append(b)
    return np.array(outs), np.array(bounds)


# ---------------------------------------------------------------------------
# acceptance bar
# ---------------------------------------------------------------------------

def within_bar(y, y_ref, bound, rel: float = TOL_REL, abs_: float = TOL_ABS) -> np.ndarray:
    """Elementwise ``|y - y_ref| <= rel * bound + abs``; a NaN in ``y`` fails."""
    y = np.asarray(y, dtype=np.float64)
    err = np.abs(y - np.asarray(y_ref, dtype=np.float64))
    ok = err <= rel * np.asarray(bound, dtype=np.float64) + abs_
    return ok & np.isfinite(y)


# upper bound of |d silu(z) / dz| = |sigma(z) * (1 + z * (1 - sigma(z)))|, whose maximum 1.09984 is near z = 2.3994
SILU_LIPSCHITZ = 1.0999


def swiglu_err_bound(y1_ref, bound1, inter: int, rel: float = TOL_REL, abs_: float = TOL_ABS):
    """Largest ``|h' - h_ref|`` when ``y1'`` is within the bar of ``y1_ref`` and each side rounds h to bf16.

    First-order propagation: ``|dh| <= L |dg| (|u| + |du|) + |silu(g)| |du|`` with L the
    Lipschitz constant of silu, then one bf16 unit (2**-7 relative) for the two roundings.
    """
    y1_ref = np.asarray(y1_ref, dtype=np.float64)
    g, u = y1_ref[:, :inter], y1_ref[:, inter:]
    dg = rel * np.asarray(bound1)[:, :inter] + abs_
    du = rel * np.asarray(bound1)[:, inter:] + abs_
    dh = SILU_LIPSCHITZ * dg * (np.abs(u) + du) + np.abs(silu(g)) * du
    return dh + 2.0 ** -7 * (np.abs(silu(g) * u) + dh)


def moe_abs_apply(v, idx, wq_list, s_list, fmt: int):
    """``out[a] = |W_idx[a]| . v[a]`` for nonnegative float64 rows ``v`` (one row per assignment)."""
    idx = np.asarray(idx, dtype=np.int64)
    v = np.asarray(v, dtype=np.float64)
    K = v.shape[1]
    N = np.asarray(s_list[0]).shape[0]
    out = np.zeros((idx.size, N))
    for e in np.unique(idx):
        rows = np.nonzero(idx == e)[0]
        out[rows] = v[rows] @ np.abs(dequant(wq_list[e], s_list[e], fmt, K)).T
    return out


def ffn_out_tolerance(res, idx, route_w, wd_q, wd_s, topk: int, inter: int, fmt: int,
                      rel: float = TOL_REL, abs_: float = TOL_ABS):
    """Elementwise tolerance of the MoE FFN output when each GEMM meets the bar on its own inputs.

    The down projection's error is its own bar plus the h error of swiglu_err_bound carried
    through ``|W_down|``; the combine adds the per-slot tolerances weighted by ``|route_w|``.
    """
    eh = swiglu_err_bound(res["y1"], res["bound1"], inter, rel, abs_)
    t2 = moe_abs_apply(eh, idx, wd_q, wd_s, fmt) + rel * res["bound2"] + abs_
    w = np.abs(np.asarray(route_w, dtype=np.float32).astype(np.float64))
    T = t2.shape[0] // topk
    return (t2.reshape(T, topk, -1) * w.reshape(T, topk)[:, :, None]).sum(axis=1)


def fp32_sum_rel(K: int) -> float:
    """Relative bound ``K * 2**-23`` (twice the first-order fp32 bound) for a K-term fp32 sum of exact products."""
    return K * 2.0 ** -23


def bar_ratio(y, y_ref, bound, rel: float = TOL_REL, abs_: float = TOL_ABS) -> float:
    """Largest ``|y - y_ref| / (rel * bound + abs)``; below 1 means every element passes."""
    y = np.asarray(y, dtype=np.float64)
    if y.size == 0:
        return 0.0
    if not np.all(np.isfinite(y)):
        return math.inf
    err = np.abs(y - np.asarray(y_ref, dtype=np.float64))
    return float(np.max(err / (rel * np.asarray(bound, dtype=np.float64) + abs_)))
