"""GPU parity of the MoE path (bucketing, grouped GEMM, SwiGLU, combine) against the fp64 oracle."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import (check_levels, dev_experts, dev_f32, dev_i32, dev_w, dev_x, report, sample_pairs,
                      torch_or_skip)

pytestmark = pytest.mark.gpu

FMTS = [synth.FMT_Q8, synth.FMT_Q4]


def q():
    import paper_2607_19438_amd as m
    return m


def small_case(seed, T, E, topk, N, K, fmt, skew=0.0, idx=None):
    rng = synth.rng_for(seed, T, E, topk, N, K, fmt)
    x = synth.make_x(rng, T, K)
    r = synth.make_routing(rng, T, E, topk, skew) if idx is None else synth.routing_from_idx(idx, E, topk)
    ws = [synth.make_qweight(rng, N, K, fmt) for _ in range(E)]
    return x, r, ws


def run_moe(torch, x, r, ws, fmt):
    xd = dev_x(torch, x)
    wq, sc = dev_experts(torch, ws)
    y = q().moe(xd, dev_i32(torch, r.token_expert_idx), dev_i32(torch, r.expert_offsets), wq, sc, r.topk, fmt)
    torch.cuda.synchronize()
    return y.cpu().numpy()


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("T,E,topk,N,K,skew", [
    (1, 1, 1, 128, 32, 0.0), (37, 5, 2, 160, 96, 0.0), (300, 16, 4, 256, 128, 1.2),
    (513, 8, 8, 96, 64, 0.0), (1000, 130, 3, 128, 64, 1.0),     # E > 128: two launches
    (200, 6, 2, 384, 768, 0.5),
    (600, 2, 2, 256, 160, 0.0),     # 256x256 ping-pong tiles, ragged last K step
    (400, 4, 1, 256, 224, 0.0),     # 192x256 ping-pong tiles, ragged last K step
])
def test_grouped_small_full(fmt, T, E, topk, N, K, skew):
    torch = torch_or_skip()
    x, r, ws = small_case(1, T, E, topk, N, K, fmt, skew)
    y = run_moe(torch, x, r, ws, fmt)
    args = (x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws], [w.scales for w in ws], topk, fmt)
    check_levels(f"moe T={T} E={E} topk={topk} N={N} K={K} {synth.FMT_NAMES[fmt]}", y,
                 oracle.moe(*args), oracle.moe(*args, bf16_weights=True), K, K >= 512)


def test_bucket_is_stable_argsort():
    torch = torch_or_skip()
    for T, E, topk, skew in [(1, 1, 1, 0.0), (2048, 128, 8, 0.0), (8192, 128, 8, 1.2), (777, 3, 2, 0.0),
                             (5000, 4096, 1, 0.0)]:
        r = synth.make_routing(synth.rng_for(2, T, E), T, E, topk, skew)
        perm = q().moe_bucket(dev_i32(torch, r.token_expert_idx), dev_i32(torch, r.expert_offsets))
        torch.cuda.synchronize()
        ref = np.argsort(r.token_expert_idx, kind="stable").astype(np.int32)
        assert np.array_equal(perm.cpu().numpy(), ref), (T, E, topk)


@pytest.mark.parametrize("fmt", FMTS)
def test_single_expert_equals_dense_bitwise(fmt):
    torch = torch_or_skip()
    T, N, K = 300, 256, 192
    x, r, ws = small_case(3, T, 1, 1, N, K, fmt, idx=np.zeros(T, np.int32))
    y = run_moe(torch, x, r, ws, fmt)
    wq, sc = dev_w(torch, ws[0])
    yd = q().dense(dev_x(torch, x), wq, sc, fmt)
    torch.cuda.synchronize()
    assert np.array_equal(y, yd.cpu().numpy())
    # all tokens on expert 0 of four experts
    x4, r4, ws4 = small_case(3, T, 4, 1, N, K, fmt, idx=np.zeros(T, np.int32))
    ws4[0] = ws[0]
    y4 = run_moe(torch, x, r4, ws4, fmt)
    assert np.array_equal(y4, y)


@pytest.mark.parametrize("fmt", FMTS)
def test_token_permutation_invariance_bitwise(fmt):
    torch = torch_or_skip()
    T, E, topk, N, K = 500, 12, 4, 128, 256
    x, r, ws = small_case(4, T, E, topk, N, K, fmt)
    y = run_moe(torch, x, r, ws, fmt)
    perm = synth.rng_for(6).permutation(T)
    idx_p = r.token_expert_idx.reshape(T, topk)[perm].reshape(-1)
    rp = synth.routing_from_idx(idx_p, E, topk)
    yp = run_moe(torch, x[perm], rp, ws, fmt)
    rows = (perm[:, None] * topk + np.arange(topk)[None, :]).reshape(-1)
    assert np.array_equal(yp, y[rows])


def test_empty_experts_never_read():
    """Experts without tokens carry NaN scales; the output stays finite."""
    torch = torch_or_skip()
    T, E, N, K = 64, 8, 128, 64
    idx = np.array([0, 3, 3, 7] * 16, np.int32)
    x, r, ws = small_case(5, T, E, 1, N, K, synth.FMT_Q4, idx=idx)
    for e in (1, 2, 4, 5, 6):
        ws[e].scales[:] = np.float16(np.nan)
    y = run_moe(torch, x, r, ws, synth.FMT_Q4)
    assert np.isfinite(y).all()


def test_inconsistent_routing_is_reported(monkeypatch):
    """Offsets that disagree with the expert ids: the rows concerned become NaN; validation reports it."""
    torch = torch_or_skip()
    T, E, N, K = 40, 4, 128, 64
    idx = np.array([0, 1, 2, 3] * 10, np.int32)
    x, r, ws = small_case(7, T, E, 1, N, K, synth.FMT_Q8, idx=idx)
    bad = r.expert_offsets.copy()
    bad[2] += 1                                   # experts 1 and 2 now disagree with their counts
    xd = dev_x(torch, x)
    wq, sc = dev_experts(torch, ws)
    y = q().moe(xd, dev_i32(torch, idx), dev_i32(torch, bad), wq, sc, 1, synth.FMT_Q8)
    torch.cuda.synchronize()
    yh = y.cpu().numpy()
    assert np.isnan(yh[idx == 1]).all() and np.isnan(yh[idx == 2]).all()
    yr, b = oracle.moe(x, idx, r.expert_offsets, [w.wq for w in ws], [w.scales for w in ws], 1, synth.FMT_Q8,
                       bf16_weights=True)
    good = (idx == 0) | (idx == 3)
    assert np.all(np.abs(yh[good] - yr[good]) <= oracle.fp32_sum_rel(K) * b[good])
    monkeypatch.setenv("QGEMM_VALIDATE", "1")
    with pytest.raises(q().QGemmError):
        q().moe(xd, dev_i32(torch, idx), dev_i32(torch, bad), wq, sc, 1, synth.FMT_Q8)
    q().moe(xd, dev_i32(torch, idx), dev_i32(torch, r.expert_offsets), wq, sc, 1, synth.FMT_Q8)


@pytest.mark.parametrize("T,topk", [(1024, 8), (3200, 8), (4200, 6)])
def test_combine_bitexact_both_mappings(T, topk):
    """The combine picks its column mapping by the size of y2 (at most 192 MiB: wave-contiguous
    chunks; above: consecutive outputs per thread). T=1024 top-8 (64 MiB), T=3200 top-8 (200 MiB)
    and T=4200 top-6 (197 MiB, the kernel with a runtime slot count), N=2048: sampled tokens equal
    the host's fp32 FMA in increasing slot order, bit for bit."""
    torch = torch_or_skip()
    N = 2048
    rng = synth.rng_for(41, T)
    y2 = rng.standard_normal((T * topk, N), dtype=np.float32)
    w = rng.uniform(0.01, 1.0, T * topk).astype(np.float32)
    out = q().moe_combine(dev_f32(torch, y2), dev_f32(torch, w), topk)
    torch.cuda.synchronize()
    toks = np.unique(np.concatenate([rng.integers(0, T, 48), [0, T - 1]]))
    got = out[torch.from_numpy(toks).cuda()].cpu().numpy()
    exp = np.zeros((len(toks), N), np.float32)
    for j in range(topk):
        rows = toks * topk + j
        exp = (w[rows, None].astype(np.float64) * y2[rows].astype(np.float64) + exp.astype(np.float64)).astype(np.float32)
    print(f"[parity] combine T={T} ({T * topk * N * 4 / 2**20:.0f} MiB y2): {len(toks)} tokens compared bitwise", flush=True)
    assert np.array_equal(got, exp)


def test_swiglu_and_combine_small():
    torch = torch_or_skip()
    rng = synth.rng_for(8)
    rows, inter, topk, N = 96, 64, 4, 48
    y1 = (rng.standard_normal((rows, 2 * inter)) * 4).astype(np.float32)
    y1[0, :8] = [0.0, -100.0, 100.0, 1e-30, -1e-30, 88.0, -88.0, 3.0]
    h = q().swiglu(dev_f32(torch, y1)).cpu()
    hb = h.view(torch.int16).numpy().view(np.uint16)
    href, _ = oracle.swiglu(y1.astype(np.float64), inter)
    hv = oracle.decode_bf16(hb)
    # bf16 output: within one bf16 ulp-ish of the fp64 value (2^-7 relative) plus tiny absolute slack
    assert np.all(np.abs(hv - href) <= 2.0 ** -7 * np.abs(href) + 1e-30)
    # the three combine kernels: 8 outputs per thread with top-8 fixed, 8 with any top-k, 4 (N % 8 != 0)
    for topk_c, N_c in ((topk, N), (8, 48), (8, 52), (3, 44)):
        rows_c = 24 * topk_c
        y2 = rng.standard_normal((rows_c, N_c)).astype(np.float32)
        w = rng.uniform(0.01, 1.0, rows_c).astype(np.float32)
        out = q().moe_combine(dev_f32(torch, y2), dev_f32(torch, w), topk_c).cpu().numpy()
        oref, bnd = oracle.combine(y2.astype(np.float64), w, topk_c, np.abs(y2).astype(np.float64))
        assert oracle.within_bar(out, oref, bnd).all(), (topk_c, N_c)
        # fp32 FMA in increasing slot order: reproduce it exactly on the host
        exp = np.zeros((rows_c // topk_c, N_c), np.float32)
        for j in range(topk_c):
            exp = (w[j::topk_c, None].astype(np.float64) * y2[j::topk_c].astype(np.float64)
                   + exp.astype(np.float64)).astype(np.float32)
        assert np.array_equal(out, exp), (topk_c, N_c)


def moe_ffn_gpu(torch, case, split=False):
    """bucket -> gate/up grouped GEMM -> SwiGLU -> down grouped GEMM -> combine, on the GPU."""
    m = q()
    r = case.routing
    xd = dev_x(torch, case.x)
    idx = dev_i32(torch, r.token_expert_idx)
    off = dev_i32(torch, r.expert_offsets)
    rw = dev_f32(torch, r.route_w)
    wgu, sgu = dev_experts(torch, case.w_gate_up)
    wd, sd = dev_experts(torch, case.w_down)
    if split:
        perm = m.moe_bucket(idx, off)
        y1 = m.moe_grouped(xd, perm, off, wgu, sgu, r.topk, case.fmt)
    else:
        y1 = m.moe(xd, idx, off, wgu, sgu, r.topk, case.fmt)
    h = m.swiglu(y1)
    if split:
        y2 = m.moe_grouped(h, perm, off, wd, sd, 1, case.fmt)
    else:
        y2 = m.moe(h, idx, off, wd, sd, 1, case.fmt)
    out = m.moe_combine(y2, rw, r.topk)
    torch.cuda.synchronize()
    return y1.cpu().numpy(), out.cpu().numpy(), h.cpu().view(torch.int16).numpy().view(np.uint16)


def check_moe_case(torch, case, n_tokens, n_samples, split=False):
    r = case.routing
    y1, out, h = moe_ffn_gpu(torch, case, split)
    assert np.isfinite(y1).all() and np.isfinite(out).all()
    wq = [w.wq for w in case.w_gate_up]
    ws = [w.scales for w in case.w_gate_up]
    rng = synth.rng_for(123, case.T)
    A = case.T * case.topk
    big = int(np.argmax(r.counts))
    big_rows = np.nonzero(r.token_expert_idx == big)[0]
    rows, cols = sample_pairs(rng, A, 2 * case.inter, n_samples,
                              extra_rows=list(big_rows[[0, -1]]) + [A - 1], extra_cols=[0, 767, 768, 1535])
    eargs = (case.x, r.token_expert_idx, wq, ws, r.topk, case.fmt, rows, cols)
    check_levels(case.name + " gate_up (sampled)", y1[rows, cols], oracle.moe_entries(*eargs),
                 oracle.moe_entries(*eargs, bf16_weights=True), case.hidden, True)
    toks = np.unique(np.concatenate([rng.integers(0, case.T, n_tokens), [0, case.T - 1, big_rows[0] // r.topk]]))
    o_ref, o_b, o_tol = oracle.moe_ffn_tokens(case.x, r.token_expert_idx, r.route_w, wq, ws,
                                              [w.wq for w in case.w_down], [w.scales for w in case.w_down],
                                              r.topk, case.inter, case.fmt, toks, with_tolerance=True)
    s_ref, s_b = oracle.down_combine_tokens(h, r.token_expert_idx, r.route_w, [w.wq for w in case.w_down],
                                            [w.scales for w in case.w_down], r.topk, case.fmt, toks)
    check_chain(case.name + " ffn out (sampled tokens)", out[toks], o_ref, o_b, o_tol, s_ref, s_b)


def check_chain(name, out, o_ref, o_b, o_tol, s_ref, s_b):
    """The MoE FFN output ``out`` (router-weighted sum of the down projections):

    * the plain acceptance bar ``|out - ref| <= 1e-3 * sum_j |w_j| sum_i |h_i W_down| + 1e-6``
      against the oracle's down projection + combine fed the same bf16 activations ``h`` as the
      GPU (s_ref, s_b): the bar on the same inputs, as for every GEMM;
    * against the oracle's own chain from x (o_ref), the tolerance that carries each GEMM's bar
      through SiLU and the bf16 rounding of h (o_tol). The plain bar against that chain is
      reported, not required: both sides round h to bf16, and where the GPU's gate/up output
      (within its own bar) sits across a rounding boundary from the exact one, the two h differ
      by a whole bf16 unit; carried through W_down that can exceed 1e-3 of the bound."""
    assert np.isfinite(out).all()
    r_same = oracle.bar_ratio(out, s_ref, s_b)
    r_tol = float(np.max(np.abs(out - o_ref) / o_tol))
    r_end = oracle.bar_ratio(out, o_ref, o_b)
    print(f"[parity] {name}: plain 1e-3 bar ratio on the same h = {r_same:.3e}; "
          f"ratio to propagated tolerance from x = {r_tol:.3e} (plain bar against the oracle's own h, "
          f"not required: {r_end:.3e})", flush=True)
    assert r_same <= 1.0, f"{name}: FFN output exceeds the acceptance bar on the same h ({r_same})"
    assert r_tol <= 1.0, f"{name}: FFN output exceeds the propagated tolerance ({r_tol})"


@pytest.mark.parametrize("cfg,T", [(3, None), (4, None), (4, 128)])
def test_down_projection_full_size_seeded(cfg, T):
    """The MoE down projection (K=768, N=2048) at full size on seeded bf16 activations, sampled outputs."""
    torch = torch_or_skip()
    m = q()
    r = synth.config_routing(cfg, T_override=T)
    A = r.T * r.topk
    rng = synth.rng_for(31, cfg, r.T)
    h = synth.make_x_product(rng, A, 768)
    wd = [synth.make_qweight(rng, 2048, 768, synth.FMT_Q4, keep_q=False) for _ in range(r.E)]
    wq, sc = dev_experts(torch, wd)
    y2 = m.moe(dev_x(torch, h), dev_i32(torch, r.token_expert_idx), dev_i32(torch, r.expert_offsets), wq, sc, 1,
               synth.FMT_Q4)
    torch.cuda.synchronize()
    y2 = y2.cpu().numpy()
    assert np.isfinite(y2).all()
    rows, cols = sample_pairs(rng, A, 2048, 5000, extra_rows=[0, A - 1], extra_cols=[0, 1023, 2047])
    eargs = (h, r.token_expert_idx, [w.wq for w in wd], [w.scales for w in wd], 1, synth.FMT_Q4, rows, cols)
    check_levels(f"moe down cfg{cfg} T={r.T} (sampled)", y2[rows, cols], oracle.moe_entries(*eargs),
                 oracle.moe_entries(*eargs, bf16_weights=True), 768, True)


def test_config3_moe_q4_t2048():
    torch = torch_or_skip()
    (case,) = synth.config(3)
    check_moe_case(torch, case, n_tokens=12, n_samples=4000)


def test_config4_moe_q4_skewed_t8192():
    torch = torch_or_skip()
    (case,) = synth.config(4)
    check_moe_case(torch, case, n_tokens=8, n_samples=4000, split=True)


def test_config4_moe_q4_skewed_t128():
    torch = torch_or_skip()
    (case,) = synth.config(4, T_override=128)
    check_moe_case(torch, case, n_tokens=32, n_samples=4000)


def test_moe_ffn_full_oracle_medium():
    """Whole FFN chain on a medium shape, every output element against the oracle."""
    torch = torch_or_skip()
    case = synth.moe_case("moe_medium", synth.FMT_Q4, 160, 16, 4, 1024, 768, skew=0.8, seed=2, stream=(77,))
    y1, out, h = moe_ffn_gpu(torch, case)
    r = case.routing
    Q = lambda L: [w.wq for w in L]  # noqa: E731
    S = lambda L: [w.scales for w in L]  # noqa: E731
    res = oracle.moe_ffn(case.x, r.token_expert_idx, r.expert_offsets, r.route_w, Q(case.w_gate_up),
                         S(case.w_gate_up), Q(case.w_down), S(case.w_down), r.topk, case.inter, case.fmt)
    y1b = oracle.moe(case.x, r.token_expert_idx, r.expert_offsets, Q(case.w_gate_up), S(case.w_gate_up), r.topk,
                     case.fmt, bf16_weights=True)
    check_levels("moe_medium y1", y1, (res["y1"], res["bound1"]), y1b, case.hidden, True)
    tol = oracle.ffn_out_tolerance(res, r.token_expert_idx, r.route_w, Q(case.w_down), S(case.w_down), r.topk,
                                   case.inter, case.fmt)
    y2h, b2h = oracle.moe(h, r.token_expert_idx, r.expert_offsets, Q(case.w_down), S(case.w_down), 1, case.fmt)
    s_ref, s_b = oracle.combine(y2h, r.route_w, r.topk, b2h)
    check_chain("moe_medium out", out, res["out"], res["bound_out"], tol, s_ref, s_b)
    # the down projection alone, on the oracle's own activations h (same inputs on both sides)
    wd, sd = dev_experts(torch, case.w_down)
    y2 = q().moe(dev_x(torch, res["h_bits"]), dev_i32(torch, r.token_expert_idx), dev_i32(torch, r.expert_offsets),
                 wd, sd, 1, case.fmt)
    torch.cuda.synchronize()
    y2b = oracle.moe(res["h_bits"], r.token_expert_idx, r.expert_offsets, Q(case.w_down), S(case.w_down), 1,
                     case.fmt, bf16_weights=True)
    check_levels("moe_medium down on oracle h", y2.cpu().numpy(), (res["y2"], res["bound2"]), y2b, case.inter, True)
