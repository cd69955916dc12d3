"""Seeded synthetic inputs for the block-quantised prefill GEMM workloads.

This module is shared by the tests, the bench and the oracle's callers. It only
draws random numbers and encodes them into the storage formats the GEMM reads
(bf16 bit patterns, int8 / packed-nibble weights, fp16 block scales, routing
tables). It performs none of the GEMM's arithmetic: no dequantisation, no
contraction, no activation, no combine.

Storage formats (the paper names 4-bit and 8-bit block-quantised weights for
its dense and MoE GEMMs, Section 3.1, without a byte layout; the layout here is
the one the library's C header documents):

* activations ``x``: bf16, row-major ``[M][K]``, carried as ``uint16`` bits.
* Q8 weights: ``int8`` ``[N][K]``, K contiguous.
* Q4 weights: ``uint8`` ``[N][K/2]``; byte ``j`` of a row holds element
  ``2j`` in bits 0-3 and element ``2j+1`` in bits 4-7 (low nibble first).
  The stored nibble ``u`` in ``[0, 15]`` means the signed value ``u - 8``.
* scales: ``float16`` ``[N][K/32]``; scale ``b`` covers ``k`` in ``[32b, 32b+32)``.
* MoE routing: ``token_expert_idx[T*topk]`` (expert of assignment
  ``a = t*topk + j``), ``expert_offsets[E+1]`` (exclusive prefix sum of the
  per-expert assignment counts) and ``route_w[T*topk]`` (float32 router weights).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

QBLOCK = 32
FMT_Q8 = 0
FMT_Q4 = 1
FMT_NAMES = {FMT_Q8: "q8", FMT_Q4: "q4"}

# Per-format draw ranges of the workloads: weight integers and scale interval.
SCALE_RANGE = {FMT_Q8: (0.001, 0.01), FMT_Q4: (0.005, 0.02)}


def rng_for(seed: int, *stream: int) -> np.random.Generator:
    """One independent numpy stream per (seed, config, tensor) tuple."""
    return np.random.default_rng(np.random.SeedSequence([int(seed), *[int(s) for s in stream]]))


# ---------------------------------------------------------------------------
# encoders (value -> storage bits); used only to build inputs
# ---------------------------------------------------------------------------

def bf16_bits(a) -> np.ndarray:
    """Round values to bf16 (via float32, round-to-nearest-even) and return uint16 bits."""
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    u = f.view(np.uint32)
    # finite inputs have u <= 0xFF7FFFFF, so adding at most 0x8000 cannot wrap
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def pack_nibbles(u: np.ndarray) -> np.ndarray:
    """Pack unsigned nibbles ``[N][K]`` (values 0..15) into ``[N][K/2]`` bytes, low nibble first."""
    u = np.asarray(u)
    if u.shape[-1] % 2:
        raise ValueError("K must be even to pack nibbles")
    if u.size and (u.min() < 0 or u.max() > 15):
        raise ValueError("nibbles must lie in [0, 15]")
    u = u.astype(np.uint8, copy=False)
    return (u[..., 0::2] | (u[..., 1::2] << 4)).astype(np.uint8)


# ---------------------------------------------------------------------------
# tensors
# ---------------------------------------------------------------------------

@dataclass
class QWeight:
    """One block-quantised weight matrix ``W[N][K]`` in storage form.

    ``q`` keeps the signed integer values the storage encodes (``int8`` for Q8,
    ``nibble - 8`` for Q4) so that tests can build exact references without
    going through any decoder.
    """
    fmt: int
    N: int
    K: int
    wq: np.ndarray          # int8 [N][K] (Q8) or uint8 [N][K/2] (Q4)
    scales: np.ndarray      # float16 [N][K/32]
    q: np.ndarray | None    # int16 [N][K], signed values encoded by wq (None when not kept)


def make_qweight(rng: np.random.Generator, N: int, K: int, fmt: int,
                 scale_range=None, keep_q: bool = True) -> QWeight:
    if K % QBLOCK:
        raise ValueError("K must be a multiple of 32")
    lo, hi = scale_range or SCALE_RANGE[fmt]
    if fmt == FMT_Q8:
        wq = rng.integers(-127, 128, size=(N, K), dtype=np.int8)
        q = wq.astype(np.int16) if keep_q else None
    elif fmt == FMT_Q4:
        u = rng.integers(0, 16, size=(N, K), dtype=np.uint8)
        wq = pack_nibbles(u)
        q = (u.astype(np.int16) - 8) if keep_q else None
    else:
        raise ValueError(f"unknown fmt {fmt}")
    scales = rng.uniform(lo, hi, size=(N, K // QBLOCK)).astype(np.float16)
    return QWeight(fmt, N, K, np.ascontiguousarray(wq), np.ascontiguousarray(scales), q)


def qweight_from_q(q: np.ndarray, scales: np.ndarray, fmt: int) -> QWeight:
    """Encode given signed integers and fp16 scales into storage form."""
    q = np.asarray(q, dtype=np.int16)
    N, K = q.shape
    if fmt == FMT_Q8:
        if q.min(initial=0) < -128 or q.max(initial=0) > 127:
            raise ValueError("Q8 values must lie in [-128, 127]")
        wq = q.astype(np.int8)
    elif fmt == FMT_Q4:
        wq = pack_nibbles(q + 8)
    else:
        raise ValueError(f"unknown fmt {fmt}")
    s = np.ascontiguousarray(np.asarray(scales, dtype=np.float16).reshape(N, K // QBLOCK))
    return QWeight(fmt, N, K, np.ascontiguousarray(wq), s, q)


def make_x(rng: np.random.Generator, M: int, K: int) -> np.ndarray:
    """Activations ~ N(0, 1) rounded to bf16; returns uint16 bits ``[M][K]``."""
    return bf16_bits(rng.standard_normal((M, K), dtype=np.float32))


def make_x_product(rng: np.random.Generator, M: int, K: int) -> np.ndarray:
    """Heavy-tailed activations: the product of two independent N(0, 1) draws, rounded to bf16.

    Stand-in input of the MoE down projection, whose activations are products of
    two roughly normal projections."""
    a = rng.standard_normal((M, K), dtype=np.float32)
    b = rng.standard_normal((M, K), dtype=np.float32)
    return bf16_bits(a * b)


# ---------------------------------------------------------------------------
# routing (input of the MoE GEMM: which expert each token slot uses)
# ---------------------------------------------------------------------------

@dataclass
class Routing:
    T: int
    E: int
    topk: int
    token_expert_idx: np.ndarray   # int32 [T*topk]
    expert_offsets: np.ndarray     # int32 [E+1]
    route_w: np.ndarray            # float32 [T*topk]

    @property
    def counts(self) -> np.ndarray:
        return np.diff(self.expert_offsets)


def offsets_from_idx(idx: np.ndarray, E: int) -> np.ndarray:
    counts = np.bincount(np.asarray(idx, dtype=np.int64), minlength=E)[:E]
    return np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)


def route_topk(logits: np.ndarray, topk: int) -> Routing:
    """Softmax over experts, keep the top-k (ties to the lower expert index), renormalise."""
    logits = np.asarray(logits, dtype=np.float64)
    T, E = logits.shape
    z = logits - logits.max(axis=1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=1, keepdims=True)
    sel = np.argsort(-p, axis=1, kind="stable")[:, :topk]
    ps = np.take_along_axis(p, sel, axis=1)
    g = ps / ps.sum(axis=1, keepdims=True)
    idx = sel.reshape(-1).astype(np.int32)
    return Routing(T, E, topk, idx, offsets_from_idx(idx, E), g.reshape(-1).astype(np.float32))


def routing_from_idx(idx: np.ndarray, E: int, topk: int, route_w=None) -> Routing:
    idx = np.asarray(idx, dtype=np.int32).reshape(-1)
    T = idx.size // topk
    if route_w is None:
        route_w = np.full(idx.size, 1.0 / topk, dtype=np.float32)
    return Routing(T, E, topk, idx, offsets_from_idx(idx, E), np.asarray(route_w, dtype=np.float32))


def zipf_bias(E: int, s: float = 1.2) -> np.ndarray:
    """``s * log`` of an (unnormalised) Zipf pmf over expert rank ``e+1``."""
    return -s * np.log(np.arange(1, E + 1, dtype=np.float64))


def make_routing(rng: np.random.Generator, T: int, E: int, topk: int, skew: float = 0.0) -> Routing:
    logits = rng.standard_normal((T, E))
    if skew:
        logits = logits + zipf_bias(E, skew)[None, :]
    return route_topk(logits, topk)


# ---------------------------------------------------------------------------
# the five workloads
# ---------------------------------------------------------------------------

@dataclass
class DenseCase:
    name: str
    fmt: int
    M: int
    N: int
    K: int
    x: np.ndarray            # uint16 bf16 bits [M][K]
    w: QWeight

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K


@dataclass
class MoECase:
    """MoE FFN: gate_up grouped GEMM (N=2*inter, K=hidden), SwiGLU, down grouped GEMM, combine."""
    name: str
    fmt: int
    T: int
    E: int
    topk: int
    hidden: int
    inter: int
    x: np.ndarray                       # uint16 bf16 bits [T][hidden]
    routing: Routing
    w_gate_up: list = field(default_factory=list)   # E x QWeight [2*inter][hidden]
    w_down: list = field(default_factory=list)      # E x QWeight [hidden][inter]

    @property
    def flops_gate_up(self) -> int:
        return 2 * self.T * self.topk * (2 * self.inter) * self.hidden

    @property
    def flops_down(self) -> int:
        return 2 * self.T * self.topk * self.hidden * self.inter


def dense_case(name: str, fmt: int, M: int, N: int, K: int, seed: int = 0, stream=(0,)) -> DenseCase:
    x = make_x(rng_for(seed, *stream, 0), M, K)
    w = make_qweight(rng_for(seed, *stream, 1), N, K, fmt)
    return DenseCase(name, fmt, M, N, K, x, w)


def moe_case(name: str, fmt: int, T: int, E: int, topk: int, hidden: int, inter: int,
             skew: float = 0.0, seed: int = 0, stream=(3,)) -> MoECase:
    x = make_x(rng_for(seed, *stream, 0), T, hidden)
    r = moe_routing(T, E, topk, skew, seed, stream)
    rg = rng_for(seed, *stream, 2)
    rd = rng_for(seed, *stream, 3)
    wgu = [make_qweight(rg, 2 * inter, hidden, fmt, keep_q=False) for _ in range(E)]
    wd = [make_qweight(rd, hidden, inter, fmt, keep_q=False) for _ in range(E)]
    return MoECase(name, fmt, T, E, topk, hidden, inter, x, r, wgu, wd)


def moe_routing(T: int, E: int, topk: int, skew: float, seed: int, stream) -> Routing:
    return make_routing(rng_for(seed, *stream, 1), T, E, topk, skew)


MOE_SHAPES = dict(E=128, topk=8, hidden=2048, inter=768)


def config_routing(i: int, seed: int = 0, T_override: int | None = None) -> Routing:
    """Only the routing of MoE workload ``i`` (cheap: no weights are drawn)."""
    if i == 3:
        T = T_override or 2048
        return moe_routing(T, 128, 8, 0.0, seed, (3,))
    if i == 4:
        T = T_override or 8192
        return moe_routing(T, 128, 8, 1.2, seed, (4, T))
    raise ValueError(f"config {i} has no routing")


def config(i: int, seed: int = 0, T_override: int | None = None):
    """The five workloads; returns a list of cases (dense or MoE)."""
    if i == 0:
        return [dense_case("dense_q8_m128_k1024_n1024", FMT_Q8, 128, 1024, 1024, seed, (0,))]
    if i == 1:
        return [dense_case("dense_q4_m512_k3072_n8192", FMT_Q4, 512, 8192, 3072, seed, (1,))]
    if i == 2:
        return [dense_case("dense_q8_gate_up_m2048_k2048_n8192", FMT_Q8, 2048, 8192, 2048, seed, (2, 0)),
                dense_case("dense_q8_down_m2048_k8192_n2048", FMT_Q8, 2048, 2048, 8192, seed, (2, 1))]
    if i == 3:
        T = T_override or 2048
        return [moe_case(f"moe_q4_t{T}_e128_top8", FMT_Q4, T, 128, 8, 2048, 768, 0.0, seed, (3,))]
    if i == 4:
        T = T_override or 8192
        return [moe_case(f"moe_q4_skewed_t{T}_e128_top8", FMT_Q4, T, 128, 8, 2048, 768, 1.2, seed, (4, T))]
    raise ValueError(f"no config {i}")


# ---------------------------------------------------------------------------
# prefill attention inputs
# ---------------------------------------------------------------------------

@dataclass
class AttnCase:
    name: str
    B: int
    S: int
    H: int
    Hkv: int
    D: int
    causal: bool
    scale: float
    q: np.ndarray    # bf16 bits [B][S][H][D]
    k: np.ndarray    # bf16 bits [B][S][Hkv][D]
    v: np.ndarray    # bf16 bits [B][S][Hkv][D]

    @property
    def flops(self) -> float:
        """2 products (Q K^T, P V) x 2 flops per multiply-add x D, over the visible (query, key) pairs."""
        pairs = self.S * (self.S + 1) // 2 if self.causal else self.S * self.S
        return 4.0 * self.B * self.H * self.D * pairs


def attn_case(name: str, B: int, S: int, H: int, Hkv: int, D: int, causal: bool = True, seed: int = 0,
              stream=(5,), q_std: float = 1.0) -> AttnCase:
    """q, k, v ~ N(0, 1) (q scaled by q_std, which sharpens the softmax), bf16; scale 1/sqrt(D)."""
    q = bf16_bits(rng_for(seed, *stream, 0).standard_normal((B, S, H, D)) * q_std)
    k = bf16_bits(rng_for(seed, *stream, 1).standard_normal((B, S, Hkv, D)))
    v = bf16_bits(rng_for(seed, *stream, 2).standard_normal((B, S, Hkv, D)))
    return AttnCase(name, B, S, H, Hkv, D, causal, 1.0 / float(np.sqrt(D)), q, k, v)


# The attention layer of the MoE workload's model family (hidden 2048, 128 experts, top-8):
# 32 query heads and 4 key/value heads of dimension 128, a 2048-token prompt, causal.
ATTN_PREFILL = dict(B=1, S=2048, H=32, Hkv=4, D=128, causal=True)


def attn_prefill_case(seed: int = 0) -> AttnCase:
    return attn_case("attn_prefill_2048", seed=seed, stream=(6,), **ATTN_PREFILL)
