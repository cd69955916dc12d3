"""GPU parity of the fused MoE gate/up projection + SiLU gate (qgemm_moe_gate_up_swiglu).

The fused epilogue must reproduce the unfused chain (grouped GEMM to fp32 y1, then the SwiGLU
kernel) bit for bit; the unfused chain itself is held to the oracle elsewhere, and here the fused
h is also compared with the oracle directly, including sizes the unfused SwiGLU cannot take.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import dev_experts, dev_i32, dev_x, torch_or_skip

pytestmark = pytest.mark.gpu

FMTS = [synth.FMT_Q8, synth.FMT_Q4]


def q():
    import paper_2607_19438_amd as m
    return m


def small_case(seed, T, E, topk, inter, K, fmt, skew=0.0):
    rng = synth.rng_for(seed, T, E, topk, inter, K, fmt)
    x = synth.make_x(rng, T, K)
    r = synth.make_routing(rng, T, E, topk, skew)
    ws = [synth.make_qweight(rng, 2 * inter, K, fmt) for _ in range(E)]
    return x, r, ws


def bits(torch, h):
    return h.cpu().view(torch.int16).numpy().view(np.uint16)


def fused_and_unfused(torch, x, r, ws, fmt):
    m = q()
    xd = dev_x(torch, x)
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    wq, sc = dev_experts(torch, ws)
    table = m.ExpertTable(wq, sc, fmt)
    h = m.moe_gate_up_swiglu(xd, perm, off, table, None, r.topk, fmt)
    y1 = m.moe_grouped(xd, perm, off, table, None, r.topk, fmt)
    h_ref = m.swiglu(y1)
    torch.cuda.synchronize()
    return bits(torch, h), bits(torch, h_ref)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("T,E,topk,inter,K,skew", [
    (1, 1, 1, 8, 32, 0.0), (37, 5, 2, 72, 96, 0.0), (300, 16, 4, 200, 128, 1.2),
    (513, 8, 8, 128, 64, 0.0), (1000, 130, 3, 64, 64, 1.0),     # E > 128: two launches
    (200, 6, 2, 768, 1024, 0.5), (700, 4, 1, 136, 544, 0.0),
])
def test_fused_equals_unfused_bitwise(fmt, T, E, topk, inter, K, skew):
    torch = torch_or_skip()
    x, r, ws = small_case(3, T, E, topk, inter, K, fmt, skew)
    h, h_ref = fused_and_unfused(torch, x, r, ws, fmt)
    assert np.array_equal(h, h_ref), f"{int((h != h_ref).sum())} of {h.size} h entries differ"


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("T,E,topk,inter,K", [(50, 3, 2, 1, 64), (90, 4, 2, 13, 96), (64, 2, 1, 131, 160)])
def test_fused_odd_inter_vs_oracle(fmt, T, E, topk, inter, K):
    """inter not a multiple of 8 (the unfused SwiGLU kernel rejects it): straight against the oracle."""
    torch = torch_or_skip()
    x, r, ws = small_case(4, T, E, topk, inter, K, fmt, 0.7)
    m = q()
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    wq, sc = dev_experts(torch, ws)
    h = m.moe_gate_up_swiglu(dev_x(torch, x), perm, off, wq, sc, r.topk, fmt)
    torch.cuda.synchronize()
    hv = oracle.decode_bf16(bits(torch, h))
    y1b, b1b = oracle.moe(x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws], [w.scales for w in ws],
                          topk, fmt, bf16_weights=True)
    h_ref, _ = oracle.swiglu(y1b, inter)
    tol = oracle.swiglu_err_bound(y1b, b1b, inter, rel=oracle.fp32_sum_rel(K), abs_=1e-30)
    ratio = float(np.max(np.abs(hv - h_ref) / (tol + 1e-30)))
    print(f"[parity] fused h inter={inter} K={K}: ratio to fp32-sum + bf16 bound = {ratio:.3e}", flush=True)
    assert np.isfinite(hv).all() and ratio <= 1.0


def test_fused_medium_vs_oracle():
    """Every h entry of a medium MoE layer against the oracle's h, within the propagated bar."""
    torch = torch_or_skip()
    case = synth.moe_case("moe_medium", synth.FMT_Q4, 160, 16, 4, 1024, 768, skew=0.8, seed=2, stream=(77,))
    r = case.routing
    m = q()
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    wq, sc = dev_experts(torch, case.w_gate_up)
    h = m.moe_gate_up_swiglu(dev_x(torch, case.x), perm, off, wq, sc, r.topk, case.fmt)
    torch.cuda.synchronize()
    hv = oracle.decode_bf16(bits(torch, h))
    y1, b1 = oracle.moe(case.x, r.token_expert_idx, r.expert_offsets, [w.wq for w in case.w_gate_up],
                        [w.scales for w in case.w_gate_up], r.topk, case.fmt)
    h_ref, _ = oracle.swiglu(y1, case.inter)
    tol = oracle.swiglu_err_bound(y1, b1, case.inter)
    ratio = float(np.max(np.abs(hv - h_ref) / tol))
    print(f"[parity] fused h moe_medium: ratio to propagated bar = {ratio:.3e}", flush=True)
    assert np.isfinite(hv).all() and ratio <= 1.0


@pytest.mark.parametrize("cfg,T", [(3, None), (4, None), (4, 128)])
def test_fused_full_size_equals_unfused(cfg, T):
    """Full-size gate/up projections (hidden 2048, inter 768): fused h == SwiGLU of the grouped GEMM."""
    torch = torch_or_skip()
    (case,) = synth.config(cfg, T_override=T)
    h, h_ref = fused_and_unfused(torch, case.x, case.routing, case.w_gate_up, case.fmt)
    assert np.array_equal(h, h_ref), f"{int((h != h_ref).sum())} of {h.size} h entries differ"


def test_fused_skips_rows_absent_from_perm():
    """Assignments missing from perm (entries outside [0, T*topk)) leave their h rows untouched."""
    torch = torch_or_skip()
    T, E, topk, inter, K, fmt = 64, 4, 2, 96, 128, synth.FMT_Q8
    x, r, ws = small_case(5, T, E, topk, inter, K, fmt)
    m = q()
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    dropped = perm[[0, 5, 17]].cpu().numpy()
    perm[[0, 5, 17]] = -1
    wq, sc = dev_experts(torch, ws)
    xd = dev_x(torch, x)
    h = torch.full((T * topk, inter), 7.0, dtype=torch.bfloat16, device="cuda")
    m.moe_gate_up_swiglu(xd, perm, off, wq, sc, topk, fmt, out=h)
    y1 = m.moe_grouped(xd, m.moe_bucket(dev_i32(torch, r.token_expert_idx), off), off, wq, sc, topk, fmt)
    h_ref = bits(torch, m.swiglu(y1))
    hb = bits(torch, h)
    keep = np.setdiff1d(np.arange(T * topk), dropped)
    assert np.all(oracle.decode_bf16(hb[dropped]) == 7.0)
    assert np.array_equal(hb[keep], h_ref[keep])
