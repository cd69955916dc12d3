"""Pins for the oracle's dense block-quantised GEMM (CPU only).

Every check here compares the oracle with something other than itself:
exact rational arithmetic on tiny shapes, closed forms that a dropped term,
a wrong sign, a swapped nibble or a wrong block index would break, and
independent decoders (Python ``struct`` for bf16, the generator's pre-packing
integers for Q4/Q8).
"""
import math
import struct
from fractions import Fraction

import numpy as np
import pytest

import oracle
import synth

FMTS = [synth.FMT_Q8, synth.FMT_Q4]


def bf16_value_struct(bits: int) -> float:
    """Independent bf16 decode: place the 16 bits on top of a big-endian binary32."""
    return struct.unpack(">f", struct.pack(">HH", int(bits), 0))[0]


def exact_dense(x_bits, w: synth.QWeight):
    """y and bound in exact rationals from the generator's integers and scales."""
    M, K = x_bits.shape
    X = [[Fraction(bf16_value_struct(b)) for b in row] for row in x_bits]
    S = [[Fraction(float(s)) for s in row] for row in w.scales]
    Q = w.q.astype(int).tolist()
    y = [[None] * w.N for _ in range(M)]
    b = [[None] * w.N for _ in range(M)]
    for m in range(M):
        for n in range(w.N):
            acc = Fraction(0)
            acb = Fraction(0)
            for k in range(K):
                t = X[m][k] * S[n][k // 32] * Q[n][k]
                acc += t
                acb += abs(t)
            y[m][n] = acc
            b[m][n] = acb
    return y, b


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,N,K", [(1, 1, 32), (3, 5, 64), (5, 3, 96), (5, 5, 32), (1, 3, 96)])
def test_bruteforce_exact_rational(fmt, M, N, K):
    rng = synth.rng_for(1234, fmt, M, N, K)
    x = synth.make_x(rng, M, K)
    w = synth.make_qweight(rng, N, K, fmt)
    y, bound = oracle.dense(x, w.wq, w.scales, fmt)
    ye, be = exact_dense(x, w)
    eps = K * 2.0 ** -52
    for m in range(M):
        for n in range(N):
            assert abs(Fraction(y[m, n]) - ye[m][n]) <= eps * be[m][n]
            assert abs(Fraction(bound[m, n]) - be[m][n]) <= eps * be[m][n]


@pytest.mark.parametrize("fmt", FMTS)
def test_unit_scale_q_one_gives_row_sums(fmt):
    rng = synth.rng_for(7, fmt)
    M, N, K = 6, 4, 160
    x = synth.make_x(rng, M, K)
    w = synth.qweight_from_q(np.ones((N, K), np.int16), np.ones((N, K // 32)), fmt)
    y, bound = oracle.dense(x, w.wq, w.scales, fmt)
    for m in range(M):
        vals = [bf16_value_struct(b) for b in x[m]]
        ref = math.fsum(vals)
        babs = math.fsum(abs(v) for v in vals)
        for n in range(N):
            assert abs(y[m, n] - ref) <= K * 2.0 ** -53 * babs
            assert abs(bound[m, n] - babs) <= K * 2.0 ** -53 * babs


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("n0,k0", [(0, 0), (2, 31), (3, 32), (1, 95), (3, 70)])
def test_one_hot_pins_column_mapping(fmt, n0, k0):
    rng = synth.rng_for(11, fmt, n0, k0)
    M, N, K = 5, 4, 96
    x = synth.make_x(rng, M, K)
    q = np.zeros((N, K), np.int16)
    v = -7 if fmt == synth.FMT_Q4 else -101
    q[n0, k0] = v
    s = rng.uniform(0.5, 2.0, size=(N, K // 32)).astype(np.float16)
    w = synth.qweight_from_q(q, s, fmt)
    y, _ = oracle.dense(x, w.wq, w.scales, fmt)
    for m in range(M):
        expect = bf16_value_struct(x[m, k0]) * float(s[n0, k0 // 32]) * v   # exact in float64
        assert y[m, n0] == expect
    others = [n for n in range(N) if n != n0]
    assert np.all(y[:, others] == 0.0)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("blk", [0, 1, 2])
def test_one_hot_scale_block_pins_block_index(fmt, blk):
    rng = synth.rng_for(13, fmt, blk)
    M, N, K = 3, 2, 96
    x = synth.make_x(rng, M, K)
    w0 = synth.make_qweight(rng, N, K, fmt)
    s = np.zeros((N, K // 32), np.float16)
    s[1, blk] = np.float16(0.0078125)
    w = synth.qweight_from_q(w0.q, s, fmt)
    y, _ = oracle.dense(x, w.wq, w.scales, fmt)
    assert np.all(y[:, 0] == 0.0)
    for m in range(M):
        ks = range(32 * blk, 32 * blk + 32)
        exact = sum(Fraction(bf16_value_struct(x[m, k])) * int(w0.q[1, k]) for k in ks) * Fraction(0.0078125)
        assert abs(Fraction(y[m, 1]) - exact) <= 32 * 2.0 ** -53 * sum(
            abs(Fraction(bf16_value_struct(x[m, k])) * int(w0.q[1, k])) for k in ks) * Fraction(0.0078125)


def test_nibble_order_low_nibble_first():
    """Every byte 0x79: low nibble 9 -> +1 at even k, high nibble 7 -> -1 at odd k."""
    rng = synth.rng_for(17)
    M, N, K = 4, 3, 64
    x = synth.make_x(rng, M, K)
    wq = np.full((N, K // 2), 0x79, dtype=np.uint8)          # built by hand, not by the packer
    s = np.ones((N, K // 32), np.float16)
    y, _ = oracle.dense(x, wq, s, synth.FMT_Q4)
    for m in range(M):
        vals = [bf16_value_struct(b) for b in x[m]]
        ref = Fraction(math.fsum(vals[0::2])) - Fraction(math.fsum(vals[1::2]))
        babs = math.fsum(abs(v) for v in vals)
        for n in range(N):
            assert abs(Fraction(y[m, n]) - ref) <= 2 * K * 2.0 ** -53 * babs


def test_q4_decode_every_nibble():
    wq = np.array([[0x10, 0x32, 0x54, 0x76, 0x98, 0xBA, 0xDC, 0xFE]], dtype=np.uint8)
    q = oracle.decode_q(wq, synth.FMT_Q4, 16)
    assert q.tolist() == [[u - 8 for u in range(16)]]


@pytest.mark.parametrize("qv", [-128, 127, -127, 1])
def test_q8_extremes_and_fp16_max_scale(qv):
    rng = synth.rng_for(19, qv + 200)
    M, N, K = 3, 2, 32
    x = synth.make_x(rng, M, K)
    q = np.zeros((N, K), np.int16)
    q[1, 5] = qv
    s = np.full((N, 1), np.float16(65504.0))
    w = synth.qweight_from_q(q, s, synth.FMT_Q8)
    y, _ = oracle.dense(x, w.wq, w.scales, synth.FMT_Q8)
    for m in range(M):
        assert y[m, 1] == bf16_value_struct(x[m, 5]) * 65504.0 * qv
    assert np.all(y[:, 0] == 0)


def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x7F80, 0x0001, 0x3F81, 0x8000, 0x4049], dtype=np.uint16)
    v = oracle.decode_bf16(bits)
    assert v[0] == 1.0 and v[1] == -2.0 and v[2] == math.inf
    assert v[3] == 2.0 ** -133 and v[4] == 1 + 2.0 ** -7
    assert v[5] == 0.0 and math.copysign(1, v[5]) == -1
    assert v[6] == 3.140625
    rnd = synth.rng_for(23).integers(0, 0x7F80, size=200).astype(np.uint16)
    for b, val in zip(rnd, oracle.decode_bf16(rnd)):
        assert val == bf16_value_struct(b)


@pytest.mark.parametrize("fmt", FMTS)
def test_sampled_entries_match_full(fmt):
    rng = synth.rng_for(29, fmt)
    M, N, K = 37, 45, 128
    x = synth.make_x(rng, M, K)
    w = synth.make_qweight(rng, N, K, fmt)
    y, b = oracle.dense(x, w.wq, w.scales, fmt)
    rows = rng.integers(0, M, 100)
    cols = rng.integers(0, N, 100)
    ys, bs = oracle.dense_entries(x, w.wq, w.scales, fmt, rows, cols)
    np.testing.assert_allclose(ys, y[rows, cols], rtol=0, atol=1e-12 * b.max())
    np.testing.assert_allclose(bs, b[rows, cols], rtol=1e-13)


def test_bar_definition():
    y_ref = np.array([1.0, 2.0, -3.0])
    bound = np.array([10.0, 0.0, 100.0])
    assert oracle.within_bar(y_ref + np.array([0.0099, 9e-7, -0.0999]), y_ref, bound).all()
    assert not oracle.within_bar(y_ref + np.array([0.0102, 0, 0]), y_ref, bound)[0]
    assert not oracle.within_bar(y_ref + np.array([0, 2e-6, 0]), y_ref, bound)[1]
    assert not oracle.within_bar(np.array([np.nan, 2.0, -3.0]), y_ref, bound)[0]


def test_rejects_bad_shapes():
    with pytest.raises(ValueError):
        oracle.dequant(np.zeros((2, 40), np.int8), np.ones((2, 1), np.float16), synth.FMT_Q8, 40)
    with pytest.raises(ValueError):
        oracle.decode_q(np.zeros((2, 16), np.uint8), synth.FMT_Q4, 64)


@pytest.mark.parametrize("fmt", FMTS)
def test_bf16_weight_variant_rounds_each_exact_weight_once(fmt):
    """bf16_weights=True: each q*s rounded to nearest bf16 (ties even), checked with exact rationals."""
    from test_oracle_moe import round_bf16_scalar
    rng = synth.rng_for(31, fmt)
    M, N, K = 3, 4, 64
    x = synth.make_x(rng, M, K)
    w = synth.make_qweight(rng, N, K, fmt)
    wr = oracle.dequant(w.wq, w.scales, fmt, K, bf16_weights=True)
    for n in range(N):
        for k in range(K):
            exact = float(w.scales[n, k // 32]) * int(w.q[n, k])      # exact in float64
            assert wr[n, k] == round_bf16_scalar(exact)
    y, b = oracle.dense(x, w.wq, w.scales, fmt, bf16_weights=True)
    for m in range(M):
        for n in range(N):
            terms = [Fraction(bf16_value_struct(x[m, k])) * Fraction(round_bf16_scalar(
                float(w.scales[n, k // 32]) * int(w.q[n, k]))) for k in range(K)]
            ex = sum(terms)
            bx = sum(abs(t) for t in terms)
            assert abs(Fraction(y[m, n]) - ex) <= K * 2.0 ** -52 * bx
    # and the rounding really moves weights: the variant differs from the exact weights
    assert np.any(wr != oracle.dequant(w.wq, w.scales, fmt, K))
