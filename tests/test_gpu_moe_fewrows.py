"""GPU parity of grouped MoE GEMMs whose experts have few routed rows (short prompts, light experts
of skewed routing): partial row tiles, 16- and 32-row edges, empty experts, and small experts
beside large ones in one launch.

Group sizes are set exactly (tokens assigned to experts by hand), with ragged K, N and SwiGLU
widths. Bar: the oracle's elementwise acceptance bar and the fp32-summation bound against
bf16-rounded weights (``check_levels``); fused SwiGLU output against the oracle's h within the
propagated bound.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_levels, dev_experts, dev_i32, dev_x, torch_or_skip

pytestmark = pytest.mark.gpu

FMTS = [synth.FMT_Q8, synth.FMT_Q4]


def q():
    import paper_2607_19438_amd as m
    return m


def routed_case(seed, counts, topk, N, K, fmt):
    """Routing with exactly counts[e] assignments on expert e (token-slot order shuffled)."""
    rng = synth.rng_for(seed, len(counts), topk, N, K, fmt, *counts)
    A = int(sum(counts))
    assert A % topk == 0
    idx = np.repeat(np.arange(len(counts), dtype=np.int32), counts)
    rng.shuffle(idx)
    T = A // topk
    r = synth.routing_from_idx(idx, len(counts), topk, rng.uniform(0.1, 1.0, A).astype(np.float32))
    x = synth.make_x(rng, T, K)
    ws = [synth.make_qweight(rng, N, K, fmt) for _ in counts]
    return x, r, ws


def grouped(torch, x, r, ws, fmt):
    m = q()
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    wq, sc = dev_experts(torch, ws)
    y = m.moe_grouped(dev_x(torch, x), perm, off, m.ExpertTable(wq, sc, fmt), None, r.topk, fmt)
    torch.cuda.synchronize()
    return y


def check(name, x, r, ws, fmt, y, K):
    args = (x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws], [w.scales for w in ws], r.topk, fmt)
    check_levels(name, y, oracle.moe(*args), oracle.moe(*args, bf16_weights=True), K, K >= 512)


# per-expert row counts: 16- and 32-row edges (15, 16, 17, 32, 33), 64 and 65, empty experts, and
# a large expert in the same launch
COUNTS = [
    [1],
    [15, 0, 16, 17],
    [32, 33, 48, 63, 64],
    [64, 65, 1, 0, 130],
    [2, 3, 5, 7, 11, 13, 300, 0, 64],
]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("ci", range(len(COUNTS)))
@pytest.mark.parametrize("N,K", [(96, 64), (100, 96), (256, 2048), (33, 32), (2048, 768)])
def test_small_groups_vs_oracle(fmt, ci, N, K):
    torch = torch_or_skip()
    counts = COUNTS[ci]
    x, r, ws = routed_case(21, counts, 1, N, K, fmt)
    y = grouped(torch, x, r, ws, fmt).cpu().numpy()
    check(f"moe_fewrows counts={counts} N={N} K={K} {synth.FMT_NAMES[fmt]}", x, r, ws, fmt, y, K)


@pytest.mark.parametrize("fmt", FMTS)
def test_small_groups_topk_gather(fmt):
    """topk > 1: the gathered activation row is assignment / topk."""
    torch = torch_or_skip()
    x, r, ws = routed_case(22, [6, 40, 2, 64, 80, 0, 8], 2, 160, 1024, fmt)
    y = grouped(torch, x, r, ws, fmt).cpu().numpy()
    check(f"moe_fewrows topk=2 {synth.FMT_NAMES[fmt]}", x, r, ws, fmt, y, 1024)


@pytest.mark.parametrize("fmt", FMTS)
def test_small_groups_long_k(fmt):
    """Long K (64 and more K steps) with a ragged last step."""
    torch = torch_or_skip()
    for K in (2048, 4096, 4096 + 64):
        x, r, ws = routed_case(23, [3, 20, 64, 65], 1, 64, K, fmt)
        y = grouped(torch, x, r, ws, fmt).cpu().numpy()
        check(f"moe_fewrows long K={K} {synth.FMT_NAMES[fmt]}", x, r, ws, fmt, y, K)


def test_small_groups_deterministic_and_permutation_invariant():
    """Repeat calls are bitwise equal, and a token's row does not depend on its position in the
    expert's group."""
    torch = torch_or_skip()
    fmt = synth.FMT_Q4
    x, r, ws = routed_case(24, [50, 17, 64, 3], 1, 192, 512, fmt)
    y1 = grouped(torch, x, r, ws, fmt).cpu().numpy()
    for _ in range(3):
        assert np.array_equal(grouped(torch, x, r, ws, fmt).cpu().numpy().view(np.uint32), y1.view(np.uint32))
    T = x.shape[0]
    pi = synth.rng_for(25).permutation(T)
    r2 = synth.routing_from_idx(r.token_expert_idx[pi], r.E, 1, r.route_w[pi])
    y2 = grouped(torch, x[pi], r2, ws, fmt).cpu().numpy()
    assert np.array_equal(y2.view(np.uint32), y1[pi].view(np.uint32))


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("inter", [16, 13, 40, 768])
def test_small_groups_fused_swiglu_vs_oracle(fmt, inter):
    """Fused gate/up + SiLU on small groups: h against the oracle, and bitwise equal to the unfused
    chain when the SwiGLU kernel can take the width."""
    torch = torch_or_skip()
    counts = [1, 16, 17, 64, 65, 0, 33]
    K = 512
    x, r, ws = routed_case(26, counts, 1, 2 * inter, K, fmt)
    m = q()
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    wq, sc = dev_experts(torch, ws)
    table = m.ExpertTable(wq, sc, fmt)
    h = m.moe_gate_up_swiglu(dev_x(torch, x), perm, off, table, None, 1, fmt)
    torch.cuda.synchronize()
    hb = h.cpu().view(torch.int16).numpy().view(np.uint16)
    hv = oracle.decode_bf16(hb)
    y1b, b1b = oracle.moe(x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws], [w.scales for w in ws], 1,
                          fmt, bf16_weights=True)
    h_ref, _ = oracle.swiglu(y1b, inter)
    tol = oracle.swiglu_err_bound(y1b, b1b, inter, rel=oracle.fp32_sum_rel(K), abs_=1e-30)
    ratio = float(np.max(np.abs(hv - h_ref) / (tol + 1e-30)))
    print(f"[parity] small-group fused h inter={inter}: ratio to fp32-sum + bf16 bound = {ratio:.3e}", flush=True)
    assert np.isfinite(hv).all() and ratio <= 1.0
    if inter % 8 == 0:
        y1 = m.moe_grouped(dev_x(torch, x), perm, off, table, None, 1, fmt)
        h_unf = m.swiglu(y1)
        torch.cuda.synchronize()
        assert np.array_equal(h_unf.cpu().view(torch.int16).numpy().view(np.uint16), hb)


def test_small_groups_write_only_their_rows():
    """Memory around the output keeps its contents (partial tiles store only their group's rows)."""
    torch = torch_or_skip()
    fmt = synth.FMT_Q8
    x, r, ws = routed_case(27, [5, 0, 9], 1, 64, 256, fmt)
    m = q()
    off = dev_i32(torch, r.expert_offsets)
    perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
    wq, sc = dev_experts(torch, ws)
    A = r.token_expert_idx.size
    pad = 16
    big = torch.full((A + 2 * pad, 64), 7.5, dtype=torch.float32, device="cuda")
    y = big[pad:pad + A]
    m.moe_grouped(dev_x(torch, x), perm, off, m.ExpertTable(wq, sc, fmt), None, 1, fmt, out=y)
    torch.cuda.synchronize()
    b = big.cpu().numpy()
    assert np.all(b[:pad] == 7.5) and np.all(b[pad + A:] == 7.5)
    check("moe_fewrows guard", x, r, ws, fmt, y.cpu().numpy(), 256)


@pytest.mark.parametrize("fmt", FMTS)
def test_tile_choice_boundary_bitwise(fmt):
    """At most 32 rows per expert on average a launch takes 128x128 four-wave tiles, above that
    192x256 eight-wave tiles. Both add the same MFMA products in the same K order, so a row routed
    identically in a launch just below and one just above the boundary is bitwise equal; each
    launch also meets the oracle's bar. Plain grouped GEMM and the fused gate/up + SiLU epilogue."""
    torch = torch_or_skip()
    m = q()
    K, inter = 512, 128
    counts = [32, 40, 20, 36]                       # 128 rows over 4 experts: mean 32
    rng = synth.rng_for(28, fmt, *counts)
    idx_a = np.repeat(np.arange(len(counts), dtype=np.int32), counts)
    rng.shuffle(idx_a)
    idx_b = np.concatenate([idx_a, np.zeros(4, np.int32)])   # 132 rows: mean 33
    x_b = synth.make_x(rng, idx_b.size, K)
    x_a = np.ascontiguousarray(x_b[:idx_a.size])
    ws = [synth.make_qweight(rng, 2 * inter, K, fmt) for _ in counts]
    wq, sc = dev_experts(torch, ws)
    table = m.ExpertTable(wq, sc, fmt)
    ys, hs = [], []
    for x, idx in ((x_a, idx_a), (x_b, idx_b)):
        r = synth.routing_from_idx(idx, len(counts), 1, np.ones(idx.size, np.float32))
        off = dev_i32(torch, r.expert_offsets)
        perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
        y = m.moe_grouped(dev_x(torch, x), perm, off, table, None, 1, fmt)
        h = m.moe_gate_up_swiglu(dev_x(torch, x), perm, off, table, None, 1, fmt)
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        check(f"moe tile boundary rows={idx.size} {synth.FMT_NAMES[fmt]}", x, r, ws, fmt, y, K)
        ys.append(y)
        hs.append(h.cpu().view(torch.int16).numpy().view(np.uint16))
    n = idx_a.size
    assert np.array_equal(ys[0].view(np.uint32), ys[1][:n].view(np.uint32))
    assert np.array_equal(hs[0], hs[1][:n])


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("inter,K", [(128, 512), (384, 512), (128, 160)])
def test_small_groups_in_eight_wave_launches_bitwise(fmt, inter, K):
    """Small experts (1, 17, 20, 32 rows) and the short last groups of large ones beside a 33-row
    expert, in launches of 256x256 tiles (1544 rows over 8 experts: mean 193; 900 = 3 x 256 + 132,
    541 = 2 x 256 + 29) and of 192x256 tiles (the same routing over 9 experts: mean 171; 900 =
    4 x 192 + 132, 541 = 2 x 192 + 157). Plain and fused SwiGLU results meet the oracle's bar and
    are bitwise equal to the same routing over 49 experts (mean 31), which takes the four-wave
    tiles. inter = 384 gives three 256-column tiles (plain and gate/up), an odd count; K = 160 ends
    in half a K step."""
    torch = torch_or_skip()
    m = q()
    counts = [900, 1, 32, 33, 0, 17, 541, 20]
    rng = synth.rng_for(29, fmt, inter, K, *counts)
    idx = np.repeat(np.arange(len(counts), dtype=np.int32), counts)
    rng.shuffle(idx)
    x = synth.make_x(rng, idx.size, K)
    ws = [synth.make_qweight(rng, 2 * inter, K, fmt) for _ in counts]
    ys, hs = [], []
    for E in (8, 9, 49):
        wse = ws + [ws[0]] * (E - len(ws))              # experts past the routed ones stay empty
        wq, sc = dev_experts(torch, wse)
        table = m.ExpertTable(wq, sc, fmt)
        r = synth.routing_from_idx(idx, E, 1, np.ones(idx.size, np.float32))
        off = dev_i32(torch, r.expert_offsets)
        perm = m.moe_bucket(dev_i32(torch, r.token_expert_idx), off)
        y = m.moe_grouped(dev_x(torch, x), perm, off, table, None, 1, fmt)
        h = m.moe_gate_up_swiglu(dev_x(torch, x), perm, off, table, None, 1, fmt)
        torch.cuda.synchronize()
        y = y.cpu().numpy()
        check(f"moe small groups E={E} {synth.FMT_NAMES[fmt]}", x, r, wse, fmt, y, K)
        hb = h.cpu().view(torch.int16).numpy().view(np.uint16)
        y1b, b1b = oracle.moe(x, r.token_expert_idx, r.expert_offsets, [w.wq for w in wse],
                              [w.scales for w in wse], 1, fmt, bf16_weights=True)
        h_ref, _ = oracle.swiglu(y1b, inter)
        tol = oracle.swiglu_err_bound(y1b, b1b, inter, rel=oracle.fp32_sum_rel(K), abs_=1e-30)
        assert float(np.max(np.abs(oracle.decode_bf16(hb) - h_ref) / (tol + 1e-30))) <= 1.0
        ys.append(y.view(np.uint32))
        hs.append(hb)
    for i in (0, 1):
        assert np.array_equal(ys[i], ys[2]) and np.array_equal(hs[i], hs[2])
