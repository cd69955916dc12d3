"""Seeded random-shape parity sweep over every GPU path against the fp64 oracle.

The shapes are drawn once from fixed seeds (so the set is reproducible and a failure names its
case): ragged M, N, K around and between the tile sizes, small-M rows, expert counts, top-k,
routing skew, and attention lengths and head groupings. Bars as in the per-path tests.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_levels, dev_experts, dev_i32, dev_w, dev_x, torch_or_skip

pytestmark = pytest.mark.gpu

FMTS = [synth.FMT_Q8, synth.FMT_Q4]


def q():
    import paper_2607_19438_amd as m
    return m


def dense_shapes(n):
    rng = synth.rng_for(9001)
    out = []
    for i in range(n):
        M = int(rng.choice([1, 2, 7, 16, 17, 33, 100, 255, 256, 300, 513]))
        N = int(rng.integers(1, 700))
        K = 32 * int(rng.integers(1, 80))
        out.append((i, M, N, K, int(rng.integers(0, 2))))
    return out


@pytest.mark.parametrize("i,M,N,K,fmt", dense_shapes(24))
def test_random_dense(i, M, N, K, fmt):
    torch = torch_or_skip()
    case = synth.dense_case(f"rand_dense_{i}", fmt, M, N, K, seed=31, stream=(i, M, N, K))
    wq, sc = dev_w(torch, case.w)
    y = q().dense(dev_x(torch, case.x), wq, sc, fmt)
    torch.cuda.synchronize()
    exact = oracle.dense(case.x, case.w.wq, case.w.scales, fmt)
    rounded = oracle.dense(case.x, case.w.wq, case.w.scales, fmt, bf16_weights=True)
    check_levels(case.name + f" {M}x{N}x{K} {synth.FMT_NAMES[fmt]}", y.cpu().numpy(), exact, rounded, K, K >= 512)


def moe_shapes(n):
    rng = synth.rng_for(9002)
    out = []
    for i in range(n):
        E = int(rng.choice([1, 2, 5, 16, 64, 129]))
        topk = int(rng.integers(1, min(E, 8) + 1))
        T = int(rng.choice([1, 3, 40, 200, 700]))
        N = int(rng.choice([32, 96, 160, 256, 300]))
        K = 32 * int(rng.integers(1, 40))
        skew = float(rng.choice([0.0, 1.2]))
        out.append((i, T, E, topk, N, K, skew, int(rng.integers(0, 2))))
    return out


@pytest.mark.parametrize("i,T,E,topk,N,K,skew,fmt", moe_shapes(16))
def test_random_moe(i, T, E, topk, N, K, skew, fmt):
    torch = torch_or_skip()
    rng = synth.rng_for(32, i)
    x = synth.make_x(rng, T, K)
    r = synth.make_routing(rng, T, E, topk, skew)
    ws = [synth.make_qweight(rng, N, K, fmt) for _ in range(E)]
    wq, sc = dev_experts(torch, ws)
    y = q().moe(dev_x(torch, x), dev_i32(torch, r.token_expert_idx), dev_i32(torch, r.expert_offsets), wq, sc,
                topk, fmt)
    torch.cuda.synchronize()
    args = (x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws], [w.scales for w in ws], topk, fmt)
    check_levels(f"rand_moe_{i} T={T} E={E} topk={topk} N={N} K={K} skew={skew} {synth.FMT_NAMES[fmt]}",
                 y.cpu().numpy(), oracle.moe(*args), oracle.moe(*args, bf16_weights=True), K, K >= 512)


def fused_shapes(n):
    rng = synth.rng_for(9003)
    return [(i, int(rng.choice([5, 60, 300])), int(rng.choice([3, 8, 20])), int(rng.integers(1, 4)),
             int(rng.choice([1, 7, 16, 40, 100])), 32 * int(rng.integers(1, 24)), int(rng.integers(0, 2)))
            for i in range(n)]


@pytest.mark.parametrize("i,T,E,topk,inter,K,fmt", fused_shapes(10))
def test_random_fused_swiglu(i, T, E, topk, inter, K, fmt):
    torch = torch_or_skip()
    topk = min(topk, E)
    rng = synth.rng_for(33, i)
    x = synth.make_x(rng, T, K)
    r = synth.make_routing(rng, T, E, topk, 0.7)
    ws = [synth.make_qweight(rng, 2 * inter, K, fmt) for _ in range(E)]
    m = q()
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    wq, sc = dev_experts(torch, ws)
    h = m.moe_gate_up_swiglu(dev_x(torch, x), perm, off, wq, sc, topk, fmt)
    torch.cuda.synchronize()
    hv = oracle.decode_bf16(h.cpu().view(torch.int16).numpy().view(np.uint16))
    y1b, b1b = oracle.moe(x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws], [w.scales for w in ws],
                          topk, fmt, bf16_weights=True)
    h_ref, _ = oracle.swiglu(y1b, inter)
    tol = oracle.swiglu_err_bound(y1b, b1b, inter, rel=oracle.fp32_sum_rel(K), abs_=1e-30)
    ratio = float(np.max(np.abs(hv - h_ref) / (tol + 1e-30)))
    print(f"[parity] rand_fused_{i} T={T} E={E} topk={topk} inter={inter} K={K}: ratio {ratio:.3e}", flush=True)
    assert np.isfinite(hv).all() and ratio <= 1.0


def attn_shapes(n):
    rng = synth.rng_for(9004)
    out = []
    for i in range(n):
        Hkv = int(rng.choice([1, 2, 4]))
        H = Hkv * int(rng.choice([1, 2, 3, 8]))
        out.append((i, int(rng.integers(1, 3)), int(rng.integers(1, 600)), H, Hkv, int(rng.choice([64, 128])),
                    bool(rng.integers(0, 2))))
    return out


@pytest.mark.parametrize("i,B,S,H,Hkv,D,causal", attn_shapes(12))
def test_random_attention(i, B, S, H, Hkv, D, causal):
    torch = torch_or_skip()
    case = synth.attn_case(f"rand_attn_{i}", B, S, H, Hkv, D, causal, seed=34, stream=(i,))
    t = lambda bits: torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()
    o = q().attention_prefill(t(case.q), t(case.k), t(case.v), causal, case.scale)
    torch.cuda.synchronize()
    ov = oracle.decode_bf16(o.cpu().view(torch.int16).numpy().view(np.uint16))
    o_ref, absv = oracle.attention(case.q, case.k, case.v, causal, case.scale)
    r = oracle.attn_ratio(ov, o_ref, absv)
    print(f"[parity] {case.name} B={B} S={S} H={H}/{Hkv} D={D} causal={causal}: ratio {r:.3e}", flush=True)
    assert r <= 1.0
