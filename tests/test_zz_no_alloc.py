"""GPU: the allocation-free MoE entry point (qgemm_moe_noalloc, static device scratch) against
qgemm_moe on the same inputs, called through the C ABI: bitwise equal on two calls in a row, the
second smaller than the first; sizes beyond the scratch are rejected before anything runs."""
import ctypes

import numpy as np
import pytest

import synth
from gpu_util import dev_experts, dev_i32, dev_x, torch_or_skip

pytestmark = pytest.mark.gpu


def q():
    import paper_2607_19438_amd as m
    return m


def call_noalloc(torch, m, x, idx, off, wq, sc, topk, fmt, N):
    """qgemm_moe_noalloc through ctypes, into a y buffer allocated beforehand."""
    T, K = x.shape
    E = off.shape[0] - 1
    y = torch.full((T * topk, N), float("nan"), dtype=torch.float32, device=x.device)
    wp = (ctypes.c_void_p * E)(*[wq[e].data_ptr() for e in range(E)])
    sp = (ctypes.c_void_p * E)(*[sc[e].data_ptr() for e in range(E)])
    rc = m.lib().qgemm_moe_noalloc(x.data_ptr(), idx.data_ptr(), off.data_ptr(), wp, sp, y.data_ptr(), T, E, topk, N,
                                   K, fmt, torch.cuda.current_stream().cuda_stream)
    assert rc == 0, m.last_error()
    return y


@pytest.mark.parametrize("fmt", [synth.FMT_Q8, synth.FMT_Q4])
def test_noalloc_equals_moe_two_calls_shrinking(fmt):
    torch = torch_or_skip()
    m = q()
    results = []
    # the second call is smaller (fewer tokens, slots and experts) and runs right after the first
    for (T, E, topk, N, K, skew, seed) in ((2048, 128, 8, 512, 256, 1.2, 61), (300, 16, 4, 384, 128, 0.5, 62)):
        rng = synth.rng_for(seed, fmt)
        x = synth.make_x(rng, T, K)
        r = synth.make_routing(rng, T, E, topk, skew)
        ws = [synth.make_qweight(rng, N, K, fmt, keep_q=False) for _ in range(E)]
        xd = dev_x(torch, x)
        idx = dev_i32(torch, r.token_expert_idx)
        off = dev_i32(torch, r.expert_offsets)
        wq, sc = dev_experts(torch, ws)
        y_na = call_noalloc(torch, m, xd, idx, off, wq, sc, topk, fmt, N)
        y_ref = m.moe(xd, idx, off, wq, sc, topk, fmt)
        torch.cuda.synchronize()
        results.append((y_na.cpu().numpy(), y_ref.cpu().numpy()))
    for y_na, y_ref in results:
        assert np.isfinite(y_ref).all()
        assert np.array_equal(y_na.view(np.uint32), y_ref.view(np.uint32))


def test_noalloc_rejects_sizes_beyond_scratch():
    torch = torch_or_skip()
    m = q()
    ptrs = (ctypes.c_void_p * 4)(16, 32, 48, 64)
    lib = m.lib()
    # T*topk = 270000 slots > 262144
    assert lib.qgemm_moe_noalloc(16, 16, 16, ptrs, ptrs, 16, 135000, 4, 2, 128, 64, 0, None) == -3
    assert "static scratch" in m.last_error()
    assert lib.qgemm_moe_noalloc(16, 16, 16, ptrs, ptrs, 16, 0, 4, 2, 128, 64, 0, None) == 0
