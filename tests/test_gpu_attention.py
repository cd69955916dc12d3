"""GPU parity of prefill attention (``qgemm_attention_prefill``) against the fp64 oracle.

Bar (derived in the oracle's ``attn_tolerance``): per output element
``|o - o_ref| <= 2^-7 sum_j p_j |v_j| + 2^-8 |o_ref|`` -- the kernel rounds the softmax weights to
bf16 before the output product and stores o as bf16; everything else is fp32.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import torch_or_skip

pytestmark = pytest.mark.gpu


def q():
    import paper_2607_19438_amd as m
    return m


def dev(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def run(torch, case, out=None):
    o = q().attention_prefill(dev(torch, case.q), dev(torch, case.k), dev(torch, case.v), case.causal, case.scale,
                              out=out)
    torch.cuda.synchronize()
    return o


def host(torch, o):
    return oracle.decode_bf16(o.cpu().view(torch.int16).numpy().view(np.uint16))


def check_full(torch, case):
    o = host(torch, run(torch, case))
    o_ref, absv = oracle.attention(case.q, case.k, case.v, case.causal, case.scale)
    r = oracle.attn_ratio(o, o_ref, absv)
    print(f"[parity] {case.name}: max |err| / bar = {r:.3e}", flush=True)
    assert r <= 1.0, f"{case.name}: ratio {r}"
    return o


SHAPES = [  # B, S, H, Hkv, D
    (1, 1, 1, 1, 128), (1, 17, 2, 1, 128), (1, 64, 4, 4, 128), (1, 100, 4, 2, 128), (1, 128, 2, 1, 128),
    (1, 129, 2, 2, 128), (2, 300, 8, 2, 128), (1, 1000, 4, 1, 128), (1, 200, 4, 4, 64), (2, 513, 8, 4, 64),
]


@pytest.mark.parametrize("causal", [True, False])
@pytest.mark.parametrize("B,S,H,Hkv,D", SHAPES)
def test_attention_shapes(B, S, H, Hkv, D, causal):
    torch = torch_or_skip()
    case = synth.attn_case(f"attn_{B}x{S}x{H}/{Hkv}x{D}_{'c' if causal else 'f'}", B, S, H, Hkv, D, causal,
                           seed=1, stream=(B, S, H, Hkv, D))
    check_full(torch, case)


@pytest.mark.parametrize("q_std", [4.0, 16.0])
def test_attention_peaked_softmax(q_std):
    """Sharper score distributions (running maximum changes often, many weights underflow)."""
    torch = torch_or_skip()
    case = synth.attn_case(f"attn_peaked_{q_std}", 1, 700, 4, 2, 128, True, seed=2, q_std=q_std)
    check_full(torch, case)


def test_attention_full_size():
    """The attention layer of the MoE model family: S=2048, 32 query heads, 4 key/value heads, D=128,
    causal; every output element against the oracle."""
    torch = torch_or_skip()
    check_full(torch, synth.attn_prefill_case())


def test_attention_deterministic_and_constant_values():
    torch = torch_or_skip()
    case = synth.attn_case("det", 1, 777, 8, 2, 128, True, seed=3)
    o1 = run(torch, case).cpu()
    for _ in range(3):
        assert torch.equal(run(torch, case).cpu(), o1)
    # every value row equal -> every output row equals it (within the bar: weights rounded to bf16)
    vconst = np.broadcast_to(synth.bf16_bits(np.linspace(-2, 2, 128)), case.v.shape).copy()
    c2 = synth.AttnCase("const_v", 1, 777, 8, 2, 128, True, case.scale, case.q, case.k, vconst)
    check_full(torch, c2)


def test_attention_causal_rows_ignore_later_tokens():
    torch = torch_or_skip()
    case = synth.attn_case("causal_prefix", 1, 400, 4, 2, 128, True, seed=4)
    o1 = run(torch, case).cpu()
    k2, v2 = case.k.copy(), case.v.copy()
    t = 261
    k2[:, t:] = synth.bf16_bits(synth.rng_for(5).standard_normal(k2[:, t:].shape))
    v2[:, t:] = synth.bf16_bits(synth.rng_for(6).standard_normal(v2[:, t:].shape))
    c2 = synth.AttnCase("causal_prefix2", 1, 400, 4, 2, 128, True, case.scale, case.q, k2, v2)
    o2 = run(torch, c2).cpu()
    assert torch.equal(o1[:, :t], o2[:, :t])


def test_attention_writes_only_o_and_rejects_bad_args():
    torch = torch_or_skip()
    m = q()
    case = synth.attn_case("guard", 1, 70, 4, 2, 64, True, seed=7)
    n = case.q.size
    big = torch.full((n + 64,), 3.0, dtype=torch.bfloat16, device="cuda")
    o = big[32:32 + n].view(case.q.shape)
    run(torch, case, out=o)
    b = big.float().cpu().numpy()
    assert np.all(b[:32] == 3.0) and np.all(b[32 + n:] == 3.0)
    qd, kd, vd = dev(torch, case.q), dev(torch, case.k), dev(torch, case.v)
    with pytest.raises(m.QGemmError):
        m.attention_prefill(qd, kd, vd, True, 0.0)
    with pytest.raises(m.QGemmError):
        m.attention_prefill(qd[:, :, :3].contiguous(), kd, vd)   # 3 query heads over 2 key/value heads
