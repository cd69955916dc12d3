"""GPU: the MoE down projection with the router-weighted combine fused into it
(qgemm_moe_down_combine) gives bitwise the rows and outputs of the two-call chain
qgemm_moe_grouped + qgemm_moe_combine (which the oracle checks elsewhere), on small
shapes covering every tile configuration and partial column tiles, on the full-size
workloads, and on repeated calls."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import dev_experts, dev_f32, dev_i32, dev_x, torch_or_skip

pytestmark = pytest.mark.gpu


def q():
    import paper_2607_19438_amd as m
    return m


def run_both(torch, h, r, wd, fmt, N, repeats=1):
    m = q()
    idx = dev_i32(torch, r.token_expert_idx)
    off = dev_i32(torch, r.expert_offsets)
    rw = dev_f32(torch, r.route_w)
    wq, sc = dev_experts(torch, wd)
    hd = dev_x(torch, h)
    perm = m.moe_bucket(idx, off)
    y2_ref = m.moe_grouped(hd, perm, off, wq, sc, 1, fmt)
    out_ref = m.moe_combine(y2_ref, rw, r.topk)
    runs = []
    for _ in range(repeats):
        y2 = torch.full_like(y2_ref, float("nan"))
        out = torch.full_like(out_ref, float("nan"))
        m.moe_down_combine(hd, perm, off, wq, sc, rw, r.topk, fmt, y2=y2, out=out)
        # unrelated work in between (another grouped launch over the same slots)
        m.moe_grouped(hd, perm, off, wq, sc, 1, fmt)
        runs.append((y2, out))
    torch.cuda.synchronize()
    return y2_ref.cpu().numpy(), out_ref.cpu().numpy(), [(a.cpu().numpy(), b.cpu().numpy()) for a, b in runs]


def bits(a):
    return np.ascontiguousarray(a).view(np.uint32)


@pytest.mark.parametrize("fmt", [synth.FMT_Q8, synth.FMT_Q4])
@pytest.mark.parametrize("T,E,topk,N,K,skew", [
    (1, 1, 1, 128, 32, 0.0),          # one token, one expert
    (37, 5, 2, 160, 96, 0.0),         # one partial column tile (BN 256 or 128)
    (300, 16, 4, 260, 128, 1.2),      # N % 8 != 0: a 4-column last tile
    (513, 8, 8, 96, 64, 0.0),         # 8-wave tiles, N below one tile
    (1000, 130, 3, 128, 64, 1.0),     # E > 128: two launches share the counters
    (64, 12, 10, 512, 64, 0.3),       # topk > 8: slots in two groups
    (100, 64, 4, 384, 768, 0.5),      # mean 6 rows per expert: four-wave 128x128 tiles
    (200, 6, 2, 2048, 768, 0.5),      # the down projection's N and K
    (700, 4, 2, 256, 128, 3.0),       # 256x256 tiles (mean 350) beside a 27/28-row expert: 32-row tile
    (900, 4, 1, 512, 160, 3.0),       # 256x256 tiles, experts of 1-5 rows, two column tiles, ragged K
])
def test_fused_equals_grouped_plus_combine(fmt, T, E, topk, N, K, skew):
    torch = torch_or_skip()
    rng = synth.rng_for(51, T, E, topk, N, K, fmt)
    h = synth.make_x_product(rng, T * topk, K)
    r = synth.make_routing(rng, T, E, topk, skew)
    wd = [synth.make_qweight(rng, N, K, fmt, keep_q=False) for _ in range(E)]
    y2_ref, out_ref, runs = run_both(torch, h, r, wd, fmt, N, repeats=2)
    assert np.isfinite(out_ref).all()
    for y2, out in runs:
        assert np.array_equal(bits(y2), bits(y2_ref))
        assert np.array_equal(bits(out), bits(out_ref))
    if K >= 512:
        toks = np.arange(min(T, 24))
        s_ref, s_b = oracle.down_combine_tokens(h, r.token_expert_idx, r.route_w, [w.wq for w in wd],
                                                [w.scales for w in wd], topk, fmt, toks)
        ratio = oracle.bar_ratio(runs[0][1][toks], s_ref, s_b)
        print(f"[parity] fused down+combine T={T} E={E} topk={topk} N={N} K={K}: bar ratio {ratio:.3e}", flush=True)
        assert ratio <= 1.0


@pytest.mark.parametrize("cfg,T", [(3, None), (4, None), (4, 128)])
def test_fused_full_size_bitwise(cfg, T):
    """The MoE workloads' down projection (K=768, N=2048, Q4) at full size: every row and output
    bitwise equal to the two-call chain, on three calls."""
    torch = torch_or_skip()
    r = synth.config_routing(cfg, T_override=T)
    rng = synth.rng_for(52, cfg, r.T)
    h = synth.make_x_product(rng, r.T * r.topk, 768)
    wd = [synth.make_qweight(rng, 2048, 768, synth.FMT_Q4, keep_q=False) for _ in range(r.E)]
    y2_ref, out_ref, runs = run_both(torch, h, r, wd, synth.FMT_Q4, 2048, repeats=3)
    for i, (y2, out) in enumerate(runs):
        assert np.array_equal(bits(y2), bits(y2_ref)), i
        assert np.array_equal(bits(out), bits(out_ref)), i
    toks = np.unique(np.concatenate([synth.rng_for(53, cfg).integers(0, r.T, 6), [0, r.T - 1]]))
    s_ref, s_b = oracle.down_combine_tokens(h, r.token_expert_idx, r.route_w, [w.wq for w in wd],
                                            [w.scales for w in wd], r.topk, synth.FMT_Q4, toks)
    ratio = oracle.bar_ratio(runs[0][1][toks], s_ref, s_b)
    print(f"[parity] fused down+combine cfg{cfg} T={r.T}: {r.T} tokens bitwise equal to grouped + combine "
          f"on 3 calls; sampled bar ratio {ratio:.3e}", flush=True)
    assert ratio <= 1.0


def test_fused_rejects_bad_sizes():
    torch = torch_or_skip()
    m = q()
    T, E, topk, N, K = 8, 2, 2, 130, 64
    r = synth.make_routing(synth.rng_for(54), T, E, topk)
    rng = synth.rng_for(55)
    wd = [synth.make_qweight(rng, N, K, synth.FMT_Q8, keep_q=False) for _ in range(E)]
    wq, sc = dev_experts(torch, wd)
    h = dev_x(torch, synth.make_x(rng, T * topk, K))
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    with pytest.raises(m.QGemmError) as ei:
        m.moe_down_combine(h, perm, off, wq, sc, dev_f32(torch, r.route_w), topk, synth.FMT_Q8)
    assert ei.value.code == -1 and "multiple of 4" in str(ei.value)
