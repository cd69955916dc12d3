"""Checks of the seeded input generators and routing tables (CPU only)."""
import numpy as np
import pytest

import synth


def test_pack_nibbles_hand_example():
    u = np.array([[1, 2, 3, 4, 15, 0]], np.uint8)
    assert synth.pack_nibbles(u).tolist() == [[0x21, 0x43, 0x0F]]
    with pytest.raises(ValueError):
        synth.pack_nibbles(np.array([[16, 0]]))


def test_bf16_encoder_rne():
    v = np.array([1.0, 1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -2.0, 3.140625], np.float64)
    assert synth.bf16_bits(v).tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC000, 0x4049]


@pytest.mark.parametrize("skew", [0.0, 1.2])
def test_routing_invariants(skew):
    r = synth.make_routing(synth.rng_for(1, int(skew * 10)), 300, 16, 4, skew)
    idx = r.token_expert_idx.reshape(300, 4)
    assert all(len(set(row)) == 4 for row in idx.tolist())
    np.testing.assert_allclose(r.route_w.reshape(300, 4).astype(np.float64).sum(1), 1.0, atol=1e-6)
    assert np.all(r.route_w > 0)
    assert r.expert_offsets[0] == 0 and r.expert_offsets[-1] == 1200
    assert np.all(np.diff(r.expert_offsets) >= 0)
    assert np.array_equal(np.diff(r.expert_offsets), np.bincount(idx.reshape(-1), minlength=16))


def test_topk_picks_largest_and_breaks_ties_low():
    logits = np.array([[0.0, 3.0, 1.0, 3.0, -1.0]])
    r = synth.route_topk(logits, 3)
    assert r.token_expert_idx.tolist() == [1, 3, 2]
    p = np.exp(logits[0] - 3.0)
    sel = p[[1, 3, 2]]
    np.testing.assert_allclose(r.route_w, (sel / sel.sum()).astype(np.float32))


def test_skewed_workload_group_sizes():
    """Zipf-biased routing at T=8192 spans near-empty experts to groups above 1000 tokens."""
    c = synth.config_routing(4).counts
    assert c.sum() == 8192 * 8
    assert c.min() <= 2 and c.max() > 1000
    c3 = synth.config_routing(3).counts
    assert c3.min() > 50 and c3.max() < 250           # uniform logits: balanced groups
    c128 = synth.config_routing(4, T_override=128).counts
    assert (c128 == 0).sum() > 30                      # small-M tail: many inactive experts


def test_config_shapes_small():
    (c0,) = synth.config(0)
    assert (c0.M, c0.N, c0.K, c0.fmt) == (128, 1024, 1024, synth.FMT_Q8)
    assert c0.x.dtype == np.uint16 and c0.x.shape == (128, 1024)
    assert c0.w.wq.dtype == np.int8 and c0.w.wq.shape == (1024, 1024)
    assert c0.w.scales.dtype == np.float16 and c0.w.scales.shape == (1024, 32)
    assert c0.w.q.min() >= -127 and c0.w.q.max() <= 127
    s = c0.w.scales.astype(np.float64)
    assert s.min() >= 0.000999 and s.max() <= 0.01001


def test_seeded_reproducible():
    a = synth.dense_case("a", synth.FMT_Q4, 8, 16, 64, seed=3, stream=(9,))
    b = synth.dense_case("b", synth.FMT_Q4, 8, 16, 64, seed=3, stream=(9,))
    assert np.array_equal(a.x, b.x) and np.array_equal(a.w.wq, b.w.wq)
    assert np.array_equal(a.w.scales, b.w.scales)
    assert a.w.wq.shape == (16, 32) and a.w.q.min() >= -8 and a.w.q.max() <= 7
