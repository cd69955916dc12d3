"""Pins for the oracle's MoE expert GEMM, SiLU gate, bf16 rounding and combine (CPU only)."""
import math
import struct
from fractions import Fraction

import numpy as np
import pytest
from scipy.special import expit

import oracle
import synth

FMTS = [synth.FMT_Q8, synth.FMT_Q4]


def bf16_value_struct(bits: int) -> float:
    return struct.unpack(">f", struct.pack(">HH", int(bits), 0))[0]


def small_moe(seed, T=9, E=5, topk=2, N=7, K=64, fmt=synth.FMT_Q4, skew=0.0):
    rng = synth.rng_for(seed, T, E, topk, N, K, fmt)
    x = synth.make_x(rng, T, K)
    r = synth.make_routing(rng, T, E, topk, skew)
    ws = [synth.make_qweight(rng, N, K, fmt) for _ in range(E)]
    return x, r, ws


@pytest.mark.parametrize("fmt", FMTS)
def test_moe_exact_rational_tiny(fmt):
    x, r, ws = small_moe(1, T=3, E=4, topk=2, N=3, K=32, fmt=fmt)
    y, bound = oracle.moe(x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws],
                          [w.scales for w in ws], 2, fmt)
    for a in range(6):
        t, e = a // 2, int(r.token_expert_idx[a])
        for n in range(3):
            terms = [Fraction(bf16_value_struct(x[t, k])) * Fraction(float(ws[e].scales[n, k // 32]))
                     * int(ws[e].q[n, k]) for k in range(32)]
            ex = sum(terms)
            bx = sum(abs(v) for v in terms)
            assert abs(Fraction(y[a, n]) - ex) <= 32 * 2.0 ** -52 * bx
            assert abs(Fraction(bound[a, n]) - bx) <= 32 * 2.0 ** -52 * bx


@pytest.mark.parametrize("fmt", FMTS)
def test_moe_equals_token_major_dense_loop(fmt):
    """Expert-major gather/scatter equals evaluating each (token, slot) with the dense oracle."""
    x, r, ws = small_moe(2, T=17, E=6, topk=3, N=9, K=96, fmt=fmt)
    y, bound = oracle.moe(x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws],
                          [w.scales for w in ws], 3, fmt)
    for a in range(17 * 3):
        t, e = a // 3, int(r.token_expert_idx[a])
        yd, bd = oracle.dense(x[t:t + 1], ws[e].wq, ws[e].scales, fmt)
        np.testing.assert_allclose(y[a], yd[0], rtol=0, atol=96 * 2.0 ** -52 * bd.max())
        np.testing.assert_allclose(bound[a], bd[0], rtol=1e-14)


@pytest.mark.parametrize("fmt", FMTS)
def test_moe_ffn_weighted_per_expert_dense_loop(fmt):
    """Grouped FFN output equals the router-weighted sum of per-expert dense evaluations."""
    T, E, topk, hidden, inter = 11, 5, 2, 64, 32
    rng = synth.rng_for(3, fmt)
    x = synth.make_x(rng, T, hidden)
    r = synth.make_routing(rng, T, E, topk)
    wgu = [synth.make_qweight(rng, 2 * inter, hidden, fmt) for _ in range(E)]
    wd = [synth.make_qweight(rng, hidden, inter, fmt) for _ in range(E)]
    res = oracle.moe_ffn(x, r.token_expert_idx, r.expert_offsets, r.route_w,
                         [w.wq for w in wgu], [w.scales for w in wgu],
                         [w.wq for w in wd], [w.scales for w in wd], topk, inter, fmt)
    for t in range(T):
        acc = np.zeros(hidden)
        for j in range(topk):
            e = int(r.token_expert_idx[t * topk + j])
            g, _ = oracle.dense(x[t:t + 1], wgu[e].wq, wgu[e].scales, fmt)
            hv = [float(silu_scalar(g[0, i]) * g[0, inter + i]) for i in range(inter)]
            hb = np.array([round_bf16_scalar(v) for v in hv])
            y2, _ = oracle.dense(np.array([[bits_of(v) for v in hb]], dtype=np.uint16),
                                 wd[e].wq, wd[e].scales, fmt)
            acc += float(np.float32(r.route_w[t * topk + j])) * y2[0]
        np.testing.assert_allclose(res["out"][t], acc, rtol=0, atol=1e-12 * res["bound_out"][t].max() + 1e-300)
    tok = [0, 5, 10]
    o2, b2 = oracle.moe_ffn_tokens(x, r.token_expert_idx, r.route_w, [w.wq for w in wgu], [w.scales for w in wgu],
                                   [w.wq for w in wd], [w.scales for w in wd], topk, inter, fmt, tok)
    np.testing.assert_allclose(o2, res["out"][tok], rtol=0, atol=1e-12 * res["bound_out"].max())
    np.testing.assert_allclose(b2, res["bound_out"][tok], rtol=1e-12)


def silu_scalar(z: float) -> float:
    """Independent scalar SiLU via math.exp (stable branch per sign)."""
    if z >= 0:
        return z / (1.0 + math.exp(-z))
    ez = math.exp(z)
    return z * ez / (1.0 + ez)


def round_bf16_scalar(v: float) -> float:
    """Independent scalar RNE to 8 significant bits using exact rationals (normal range)."""
    if v == 0:
        return v
    m, e = math.frexp(abs(v))                 # |v| = m * 2**e
    scaled = Fraction(abs(v)) * Fraction(2) ** (8 - e)
    fl = math.floor(scaled)
    rem = scaled - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return math.copysign(float(Fraction(fl) * Fraction(2) ** (e - 8)), v)


def bits_of(v: float) -> int:
    return struct.unpack(">I", struct.pack(">f", v))[0] >> 16


@pytest.mark.parametrize("fmt", FMTS)
def test_token_permutation_invariance(fmt):
    x, r, ws = small_moe(4, T=13, E=5, topk=2, N=6, K=64, fmt=fmt)
    wq, ss = [w.wq for w in ws], [w.scales for w in ws]
    y, b = oracle.moe(x, r.token_expert_idx, r.expert_offsets, wq, ss, 2, fmt)
    perm = synth.rng_for(5).permutation(13)
    idx_p = r.token_expert_idx.reshape(13, 2)[perm].reshape(-1)
    yp, _ = oracle.moe(x[perm], idx_p, synth.offsets_from_idx(idx_p, 5), wq, ss, 2, fmt)
    rows = (perm[:, None] * 2 + np.arange(2)[None, :]).reshape(-1)
    np.testing.assert_allclose(yp, y[rows], rtol=0, atol=64 * 2.0 ** -52 * b.max())


@pytest.mark.parametrize("fmt", FMTS)
def test_single_expert_topk1_equals_dense(fmt):
    rng = synth.rng_for(6, fmt)
    T, N, K = 10, 8, 64
    x = synth.make_x(rng, T, K)
    w = synth.make_qweight(rng, N, K, fmt)
    r = synth.routing_from_idx(np.zeros(T, np.int32), 1, 1)
    y, b = oracle.moe(x, r.token_expert_idx, r.expert_offsets, [w.wq], [w.scales], 1, fmt)
    yd, bd = oracle.dense(x, w.wq, w.scales, fmt)
    np.testing.assert_allclose(y, yd, rtol=0, atol=64 * 2.0 ** -52 * bd.max())
    # every token on expert 0 of several experts, the others unused
    ws = [w] + [synth.make_qweight(rng, N, K, fmt) for _ in range(3)]
    r4 = synth.routing_from_idx(np.zeros(T, np.int32), 4, 1)
    y4, _ = oracle.moe(x, r4.token_expert_idx, r4.expert_offsets, [v.wq for v in ws], [v.scales for v in ws], 1, fmt)
    np.testing.assert_allclose(y4, yd, rtol=0, atol=64 * 2.0 ** -52 * bd.max())


def test_empty_experts_are_never_touched():
    """Experts with no routed tokens get NaN scales; the output stays finite."""
    x, r, ws = small_moe(7, T=8, E=6, topk=1, N=5, K=32)
    idx = np.array([0, 2, 2, 0, 5, 2, 0, 5], np.int32)
    r = synth.routing_from_idx(idx, 6, 1)
    ss = [w.scales.copy() for w in ws]
    for e in (1, 3, 4):
        ss[e][:] = np.float16(np.nan)
    y, _ = oracle.moe(x, r.token_expert_idx, r.expert_offsets, [w.wq for w in ws], ss, 1, synth.FMT_Q4)
    assert np.isfinite(y).all()


def test_inconsistent_offsets_rejected():
    x, r, ws = small_moe(8)
    bad = r.expert_offsets.copy()
    bad[1] += 1
    with pytest.raises(ValueError):
        oracle.moe(x, r.token_expert_idx, bad, [w.wq for w in ws], [w.scales for w in ws], 2, synth.FMT_Q4)


def test_silu_closed_forms():
    assert oracle.silu(0.0) == 0.0
    z = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(oracle.silu(z) - oracle.silu(-z), z, rtol=0, atol=1e-13)
    big = np.array([40.0, 100.0, 1e3])
    assert np.array_equal(oracle.silu(big), big)
    assert np.all(oracle.silu(-big) <= 0) and np.all(oracle.silu(-big) > -1e-15)
    np.testing.assert_allclose(oracle.silu(z), z * expit(z), rtol=1e-14, atol=1e-300)
    assert abs(oracle.silu(1.0) - 1 / (1 + math.exp(-1))) < 1e-16


def test_bf16_rounding_closed_forms():
    vals = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, 1 + 2.0 ** -8 + 2.0 ** -30, -(1 + 2.0 ** -8),
                     2.0 ** -134, 3 * 2.0 ** -134, 1e39, -1e39, 0.0, 2.0 ** -126 * (1 + 2.0 ** -8)])
    out, bits = oracle.round_to_bf16(vals)
    assert out[0] == 1.0                      # tie -> even
    assert out[1] == 1 + 2.0 ** -6            # tie -> even (up)
    assert out[2] == 1 + 2.0 ** -7            # above the tie
    assert out[3] == -1.0
    assert out[4] == 0.0                      # subnormal tie -> even (zero)
    assert out[5] == 2.0 ** -132              # subnormal tie -> even (up)
    assert out[6] == math.inf and out[7] == -math.inf
    assert out[8] == 0.0
    assert out[9] == 2.0 ** -126              # smallest normal, tie -> even
    assert bits[0] == 0x3F80 and bits[3] == 0xBF80 and bits[6] == 0x7F80


def test_bf16_rounding_matches_torch_and_scalar_rule():
    torch = pytest.importorskip("torch")
    v = synth.rng_for(9).standard_normal(20000) * np.exp(synth.rng_for(10).uniform(-20, 20, 20000))
    v32 = v.astype(np.float32).astype(np.float64)      # float32-representable: torch rounds once
    out, bits = oracle.round_to_bf16(v32)
    ref = torch.from_numpy(v32.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(out, ref)
    for val in v[:300]:
        assert oracle.round_to_bf16(np.array([val]))[0][0] == round_bf16_scalar(float(val))


def test_combine_closed_forms():
    T, topk, N = 4, 3, 5
    y2 = synth.rng_for(11).standard_normal((T * topk, N))
    w = np.zeros(T * topk, np.float32)
    w[np.arange(T) * topk + 1] = 1.0
    out, _ = oracle.combine(y2, w, topk)
    assert np.array_equal(out, y2[np.arange(T) * topk + 1])
    same = np.repeat(y2[::topk], topk, axis=0)
    w2 = np.array([0.25, 0.25, 0.5] * T, np.float32)
    out2, _ = oracle.combine(same, w2, topk)
    assert np.array_equal(out2, y2[::topk])
    b = np.abs(y2)
    _, bnd = oracle.combine(y2, -w2, topk, b)
    np.testing.assert_allclose(bnd, (b.reshape(T, topk, N) * np.array([0.25, 0.25, 0.5])[None, :, None]).sum(1))


def test_silu_lipschitz_constant_bounds_derivative():
    z = np.linspace(-40, 40, 800001)
    d = np.gradient(oracle.silu(z), z)
    assert np.max(np.abs(d)) <= oracle.SILU_LIPSCHITZ
    assert np.max(np.abs(d)) > oracle.SILU_LIPSCHITZ - 1e-3      # and it is tight


@pytest.mark.parametrize("fmt", FMTS)
def test_ffn_tolerance_covers_perturbed_chains(fmt):
    """Perturb each GEMM's output within the bar (worst-case signs and random), recompute the rest
    of the chain exactly as the oracle does, and check the FFN output stays within the tolerance."""
    T, E, topk, hidden, inter = 24, 4, 2, 64, 32
    rng = synth.rng_for(40, fmt)
    x = synth.make_x(rng, T, hidden)
    r = synth.make_routing(rng, T, E, topk)
    wgu = [synth.make_qweight(rng, 2 * inter, hidden, fmt) for _ in range(E)]
    wd = [synth.make_qweight(rng, hidden, inter, fmt) for _ in range(E)]
    args = (x, r.token_expert_idx, r.expert_offsets, r.route_w, [w.wq for w in wgu], [w.scales for w in wgu],
            [w.wq for w in wd], [w.scales for w in wd], topk, inter, fmt)
    res = oracle.moe_ffn(*args)
    tol = oracle.ffn_out_tolerance(res, r.token_expert_idx, r.route_w, [w.wq for w in wd], [w.scales for w in wd],
                                   topk, inter, fmt)
    worst = 0.0
    for trial in range(40):
        rr = synth.rng_for(41, trial)
        s1 = rr.choice([-1.0, 1.0], size=res["y1"].shape) if trial % 2 else rr.uniform(-1, 1, res["y1"].shape)
        y1p = res["y1"] + s1 * (oracle.TOL_REL * res["bound1"] + oracle.TOL_ABS)
        _, hb = oracle.swiglu(y1p, inter)
        y2p, _ = oracle.moe(hb, r.token_expert_idx, r.expert_offsets, [w.wq for w in wd], [w.scales for w in wd], 1, fmt)
        s2 = rr.choice([-1.0, 1.0], size=y2p.shape)
        y2p = y2p + s2 * (oracle.TOL_REL * res["bound2"] + oracle.TOL_ABS)
        outp, _ = oracle.combine(y2p, r.route_w, topk)
        worst = max(worst, float(np.max(np.abs(outp - res["out"]) / tol)))
    assert worst <= 1.0
    assert worst > 0.05          # the tolerance is not vacuous


# ---------------------------------------------------------------------------
# moe_entries: the per-element MoE evaluation the full-size GPU checks sample
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("fmt", FMTS)
def test_moe_entries_exact_rational(fmt):
    """Every (assignment, column) of a tiny top-3 case against exact rational arithmetic:
    row a reads token a // topk and the weights of expert idx[a] (not of another slot)."""
    T, E, topk, N, K = 4, 5, 3, 3, 64
    x, r, ws = small_moe(21, T=T, E=E, topk=topk, N=N, K=K, fmt=fmt)
    A = T * topk
    assigns = np.repeat(np.arange(A), N)
    cols = np.tile(np.arange(N), A)
    y, bound = oracle.moe_entries(x, r.token_expert_idx, [w.wq for w in ws], [w.scales for w in ws], topk, fmt,
                                  assigns, cols)
    for i, (a, n) in enumerate(zip(assigns, cols)):
        t, e = int(a) // topk, int(r.token_expert_idx[a])
        terms = [Fraction(bf16_value_struct(x[t, k])) * Fraction(float(ws[e].scales[n, k // 32])) * int(ws[e].q[n, k])
                 for k in range(K)]
        ex = sum(terms)
        bx = sum(abs(v) for v in terms)
        assert abs(Fraction(y[i]) - ex) <= K * 2.0 ** -52 * bx, (a, n)
        assert abs(Fraction(bound[i]) - bx) <= K * 2.0 ** -52 * bx, (a, n)


@pytest.mark.parametrize("bf16_weights", [False, True])
@pytest.mark.parametrize("fmt", FMTS)
def test_moe_entries_match_moe(fmt, bf16_weights):
    """Sampled entries (random pairs, every corner, every row of one expert at the last column)
    equal the expert-major oracle, with empty experts (NaN scales that must never be read)."""
    T, E, topk, N, K = 23, 9, 3, 40, 96
    x, r, ws = small_moe(22, T=T, E=E, topk=topk, N=N, K=K, fmt=fmt)
    idx = r.token_expert_idx.copy()
    idx[idx == 4] = 0                       # experts 4 and 7 receive nothing
    idx[idx == 7] = 8
    # keep each token's experts distinct (top-k never repeats an expert)
    idx = idx.reshape(T, topk)
    for t in range(T):
        seen = set()
        for j in range(topk):
            while idx[t, j] in seen or idx[t, j] in (4, 7):
                idx[t, j] = (idx[t, j] + 1) % E
            seen.add(int(idx[t, j]))
    idx = idx.reshape(-1)
    rr = synth.routing_from_idx(idx, E, topk)
    assert rr.counts[4] == 0 and rr.counts[7] == 0
    ss = [w.scales.copy() for w in ws]
    for e in (4, 7):
        ss[e][:] = np.float16(np.nan)
    wq = [w.wq for w in ws]
    y, b = oracle.moe(x, idx, rr.expert_offsets, wq, ss, topk, fmt, bf16_weights=bf16_weights)
    rng = synth.rng_for(23, fmt)
    A = T * topk
    rows = list(rng.integers(0, A, 300)) + [0, 0, A - 1, A - 1]
    cols = list(rng.integers(0, N, 300)) + [0, N - 1, 0, N - 1]
    for a in np.nonzero(idx == 0)[0]:
        rows.append(int(a))
        cols.append(N - 1)
    rows, cols = np.array(rows), np.array(cols)
    ye, be = oracle.moe_entries(x, idx, wq, ss, topk, fmt, rows, cols, bf16_weights=bf16_weights)
    assert np.isfinite(ye).all()
    np.testing.assert_allclose(ye, y[rows, cols], rtol=0, atol=K * 2.0 ** -52 * b.max())
    np.testing.assert_allclose(be, b[rows, cols], rtol=1e-13)


def test_moe_entries_bf16_weights_round_each_weight():
    """With bf16_weights each q*s is rounded to bf16 once: a weight 1 + 2^-8 (a tie) becomes 1."""
    K, N = 32, 2
    q = np.zeros((N, K), np.int16)
    q[1, 5] = 1
    s = np.full((N, 1), 1 + 2.0 ** -8, np.float64).astype(np.float16)   # 1.00390625, exact in fp16
    w = synth.qweight_from_q(q, s, synth.FMT_Q8)
    x = synth.bf16_bits(np.eye(1, K, 5))          # x = e_5
    idx = np.array([0], np.int32)
    ye, _ = oracle.moe_entries(x, idx, [w.wq], [w.scales], 1, synth.FMT_Q8, [0], [1])
    yb, _ = oracle.moe_entries(x, idx, [w.wq], [w.scales], 1, synth.FMT_Q8, [0], [1], bf16_weights=True)
    assert ye[0] == 1 + 2.0 ** -8 and yb[0] == 1.0


# ---------------------------------------------------------------------------
# bar_ratio: every GPU parity assertion goes through it
# ---------------------------------------------------------------------------

def test_bar_ratio_closed_forms():
    # the relative term alone: err 1 against 1e-3 * 1000 + 1e-6
    assert oracle.bar_ratio([1.0], [0.0], [1000.0]) == 1.0 / (1.0 + 1e-6)
    # the absolute term alone: zero bound, err 2e-6 -> ratio 2
    assert math.isclose(oracle.bar_ratio([2e-6], [0.0], [0.0]), 2.0, rel_tol=1e-12)
    # sign of the error does not matter; the largest ratio wins, not the largest error
    r = oracle.bar_ratio([5.0, -0.5, 3.0], [4.0, 0.0, 3.0], [1e6, 100.0, 0.0])
    assert math.isclose(r, 0.5 / (0.1 + 1e-6), rel_tol=1e-12)
    # explicit tolerances take their roles
    assert math.isclose(oracle.bar_ratio([3.0], [1.0], [10.0], rel=0.1, abs_=1.0), 1.0, rel_tol=1e-12)
    assert math.isclose(oracle.bar_ratio([3.0], [1.0], [1.0], rel=1.0, abs_=0.0), 2.0, rel_tol=1e-12)
    # non-finite results fail; an empty comparison passes
    assert oracle.bar_ratio([1.0, np.nan], [1.0, 0.0], [1.0, 1.0]) == math.inf
    assert oracle.bar_ratio([np.inf], [0.0], [1.0]) == math.inf
    assert oracle.bar_ratio(np.zeros(0), np.zeros(0), np.zeros(0)) == 0.0
    assert oracle.bar_ratio([7.0], [7.0], [0.0]) == 0.0


def test_bar_ratio_agrees_with_within_bar():
    rng = synth.rng_for(24)
    for trial in range(50):
        bound = rng.uniform(0.0, 10.0, 64) * (rng.random(64) < 0.8)
        y_ref = rng.standard_normal(64)
        y = y_ref + rng.choice([-1, 1], 64) * (1e-3 * bound + 1e-6) * rng.uniform(0.0, 1.0 + 0.3 * (trial % 2), 64)
        r = oracle.bar_ratio(y, y_ref, bound)
        assert (r <= 1.0) == bool(oracle.within_bar(y, y_ref, bound).all())


@pytest.mark.parametrize("fmt", FMTS)
def test_down_combine_tokens_matches_chain(fmt):
    """Fed the oracle's own h, the token-wise down projection + combine equals the FFN chain's
    output and bound; a one-hot router weight returns that slot's dense projection."""
    T, E, topk, hidden, inter = 9, 5, 3, 64, 32
    rng = synth.rng_for(25, fmt)
    x = synth.make_x(rng, T, hidden)
    r = synth.make_routing(rng, T, E, topk)
    wgu = [synth.make_qweight(rng, 2 * inter, hidden, fmt) for _ in range(E)]
    wd = [synth.make_qweight(rng, hidden, inter, fmt) for _ in range(E)]
    res = oracle.moe_ffn(x, r.token_expert_idx, r.expert_offsets, r.route_w, [w.wq for w in wgu],
                         [w.scales for w in wgu], [w.wq for w in wd], [w.scales for w in wd], topk, inter, fmt)
    toks = [0, 4, 8]
    o, b = oracle.down_combine_tokens(res["h_bits"], r.token_expert_idx, r.route_w, [w.wq for w in wd],
                                      [w.scales for w in wd], topk, fmt, toks)
    np.testing.assert_allclose(o, res["out"][toks], rtol=0, atol=1e-12 * res["bound_out"].max())
    np.testing.assert_allclose(b, res["bound_out"][toks], rtol=1e-12)
    one_hot = np.zeros(T * topk, np.float32)
    one_hot[np.arange(T) * topk + 2] = 1.0
    o1, _ = oracle.down_combine_tokens(res["h_bits"], r.token_expert_idx, one_hot, [w.wq for w in wd],
                                       [w.scales for w in wd], topk, fmt, toks)
    for i, t in enumerate(toks):
        a = t * topk + 2
        e = int(r.token_expert_idx[a])
        yd, bd = oracle.dense(res["h_bits"][a:a + 1], wd[e].wq, wd[e].scales, fmt)
        np.testing.assert_allclose(o1[i], yd[0], rtol=0, atol=inter * 2.0 ** -52 * bd.max())
