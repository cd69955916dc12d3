"""Pins of the prefill-attention oracle (CPU only): a hand-derived fixture, closed forms, a
high-precision brute force on tiny inputs, and invariants that a dropped normalisation, a wrong
mask, a wrong head mapping or a wrong scale would break (see the planted mistakes at the end)."""
import json
import math
import os
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np
import pytest

import oracle
import oracle.attention_oracle as ao
import synth

HERE = os.path.dirname(os.path.abspath(__file__))


def bits(a):
    return synth.bf16_bits(np.asarray(a, dtype=np.float64))


def test_hand_derived_fixture():
    with open(os.path.join(HERE, "golden", "attention_hand.json")) as f:
        g = json.load(f)
    S, D = g["S"], g["D"]
    q = bits(g["q"]).reshape(1, S, 1, D)
    k = bits(g["k"]).reshape(1, S, 1, D)
    v = bits(g["v"]).reshape(1, S, 1, D)
    for c in g["cases"]:
        o, absv = oracle.attention(q, k, v, c["causal"], math.log(3.0))
        want = np.array([[float(Fraction(x)) for x in row] for row in c["o"]])
        np.testing.assert_allclose(o[0, :, 0, :], want, rtol=1e-14, atol=1e-14)
        np.testing.assert_allclose(absv[0, :, 0, :], want, rtol=1e-14, atol=1e-14)   # v >= 0


@pytest.mark.parametrize("causal", [True, False])
def test_constant_values_give_that_value(causal):
    """Softmax weights sum to one: if every key carries the same v, every output is that v."""
    B, S, H, Hkv, D = 2, 37, 4, 2, 16
    case = synth.attn_case("c", B, S, H, Hkv, D, causal, seed=1)
    c = np.linspace(-3, 3, D)
    v = np.broadcast_to(bits(c), (B, S, Hkv, D))
    o, absv = oracle.attention(case.q, case.k, v, causal, case.scale)
    cv = oracle.decode_bf16(bits(c))
    np.testing.assert_allclose(o, np.broadcast_to(cv, o.shape), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(absv, np.broadcast_to(np.abs(cv), o.shape), rtol=1e-13, atol=1e-13)


def test_equal_scores_give_prefix_means():
    """All keys zero -> every score is 0 -> causal row i is the mean of v_0..v_i."""
    B, S, H, D = 1, 50, 2, 8
    case = synth.attn_case("z", B, S, H, H, D, True, seed=2)
    k = np.zeros_like(case.k)
    o, _ = oracle.attention(case.q, k, case.v, True, case.scale)
    v = oracle.decode_bf16(case.v)
    want = np.cumsum(v, axis=1) / np.arange(1, S + 1)[None, :, None, None]
    np.testing.assert_allclose(o, want, rtol=1e-12, atol=1e-13)


def test_one_dominant_key_selects_its_value():
    """A key whose score exceeds the others by ~80 gets weight 1 - O(e^-80)."""
    S, D = 20, 8
    q = np.zeros((1, S, 1, D)); q[..., 0] = 10.0
    k = np.zeros((1, S, 1, D)); k[0, 7, 0, 0] = 8.0
    v = synth.rng_for(3).standard_normal((1, S, 1, D))
    o, _ = oracle.attention(bits(q), bits(k), bits(v), False, 1.0)
    vv = oracle.decode_bf16(bits(v))
    np.testing.assert_allclose(o[0, :, 0, :], np.broadcast_to(vv[0, 7, 0], (S, D)), rtol=1e-12, atol=1e-12)


def test_causal_rows_ignore_later_tokens():
    """Changing the keys and values of tokens t.. leaves the causal rows before t unchanged."""
    case = synth.attn_case("p", 1, 40, 4, 2, 16, True, seed=4)
    o1, _ = oracle.attention(case.q, case.k, case.v, True, case.scale)
    k2, v2 = case.k.copy(), case.v.copy()
    t = 23
    k2[:, t:] = bits(synth.rng_for(5).standard_normal(k2[:, t:].shape))
    v2[:, t:] = bits(synth.rng_for(6).standard_normal(v2[:, t:].shape))
    o2, _ = oracle.attention(case.q, k2, v2, True, case.scale)
    np.testing.assert_allclose(o1[:, :t], o2[:, :t], rtol=1e-15, atol=0)
    assert not np.allclose(o1[:, t:], o2[:, t:])


def test_grouped_query_head_mapping():
    """Key/value head g carries the constant value c_g: query head h must return c_{h // (H/Hkv)}."""
    B, S, H, Hkv, D = 1, 12, 8, 2, 4
    case = synth.attn_case("g", B, S, H, Hkv, D, True, seed=7)
    v = np.zeros((B, S, Hkv, D))
    v[:, :, 0, :] = 1.0
    v[:, :, 1, :] = 5.0
    o, _ = oracle.attention(case.q, case.k, bits(v), True, case.scale)
    for h in range(H):
        np.testing.assert_allclose(o[0, :, h, :], 1.0 if h < 4 else 5.0, rtol=1e-14)


def test_key_permutation_invariance_without_mask():
    case = synth.attn_case("perm", 1, 33, 2, 1, 8, False, seed=8)
    perm = synth.rng_for(9).permutation(33)
    o1, _ = oracle.attention(case.q, case.k, case.v, False, case.scale)
    o2, _ = oracle.attention(case.q, case.k[:, perm], case.v[:, perm], False, case.scale)
    np.testing.assert_allclose(o1, o2, rtol=1e-13, atol=1e-14)


def _decimal_attention(q, k, v, causal, scale, H, Hkv):
    """Plain loops in 40-digit decimal arithmetic: q, k, v float64 arrays [S][H][D] / [S][Hkv][D]."""
    getcontext().prec = 40
    S, _, D = q.shape
    out = np.zeros(q.shape)
    sc = Decimal(scale)
    for h in range(H):
        g = h * Hkv // H
        for i in range(S):
            n = i + 1 if causal else S
            s = [sc * sum(Decimal(q[i, h, d]) * Decimal(k[j, g, d]) for d in range(D)) for j in range(n)]
            m = max(s)
            p = [(x - m).exp() for x in s]
            l = sum(p)
            for d in range(D):
                out[i, h, d] = float(sum(p[j] * Decimal(v[j, g, d]) for j in range(n)) / l)
    return out


@pytest.mark.parametrize("causal", [True, False])
def test_matches_decimal_brute_force(causal):
    case = synth.attn_case("tiny", 1, 6, 4, 2, 5, causal, seed=10, q_std=3.0)
    o, _ = oracle.attention(case.q, case.k, case.v, causal, case.scale)
    q, k, v = (oracle.decode_bf16(a)[0] for a in (case.q, case.k, case.v))
    want = _decimal_attention(q, k, v, causal, case.scale, 4, 2)
    np.testing.assert_allclose(o[0], want, rtol=1e-13, atol=1e-14)


def test_rows_path_matches_full_path():
    case = synth.attn_case("rows", 2, 30, 4, 2, 8, True, seed=11)
    o, a = oracle.attention(case.q, case.k, case.v, True, case.scale)
    rows = [(0, 0, 0), (1, 29, 3), (0, 17, 2), (1, 5, 1)]
    ro, ra = oracle.attention_rows(case.q, case.k, case.v, True, case.scale, rows)
    for n, (b, i, h) in enumerate(rows):
        np.testing.assert_allclose(ro[n], o[b, i, h], rtol=1e-14, atol=1e-15)
        np.testing.assert_allclose(ra[n], a[b, i, h], rtol=1e-14, atol=1e-15)


def test_tolerance_formula():
    o_ref = np.array([1.0, -2.0, 0.0])
    absv = np.array([3.0, 2.0, 1.0])
    tol = oracle.attn_tolerance(o_ref, absv)
    np.testing.assert_allclose(tol, 2.0 ** -7 * absv + 2.0 ** -8 * np.abs(o_ref) + 1e-30)
    assert oracle.attn_ratio(o_ref + tol * 0.5, o_ref, absv) == pytest.approx(0.5)
    assert oracle.attn_ratio(np.array([np.nan, 0, 0]), o_ref, absv) == float("inf")


# ---------------------------------------------------------------------------
# planted mistakes: each must make at least one pin above fail
# ---------------------------------------------------------------------------

PINS = [test_hand_derived_fixture,
        lambda: test_constant_values_give_that_value(True),
        test_equal_scores_give_prefix_means,
        test_grouped_query_head_mapping,
        lambda: test_matches_decimal_brute_force(True),
        lambda: test_matches_decimal_brute_force(False),
        test_causal_rows_ignore_later_tokens]


def _no_normalise(p, l, vh):
    return p @ vh, p @ np.abs(vh)


def _strict_causal(rows, S, causal):
    vis = np.arange(S)[None, :] < np.asarray(rows)[:, None]
    vis[:, 0] = True                  # keep every row non-empty
    return vis if causal else np.ones((np.asarray(rows).size, S), dtype=bool)


def _head_modulo(h, H, Hkv):
    return h % Hkv


def _scale_dropped(qh, kh, scale):
    return qh @ kh.T


MUTANTS = {"_combine": _no_normalise, "_visible": _strict_causal, "kv_head_of": _head_modulo,
           "_scores": _scale_dropped}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistake_is_caught(name, monkeypatch):
    monkeypatch.setattr(ao, name, MUTANTS[name])
    failed = 0
    for pin in PINS:
        try:
            pin()
        except AssertionError:
            failed += 1
    assert failed > 0, f"no pin caught the planted mistake {name}"
