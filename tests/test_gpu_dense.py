"""GPU parity of the dense block-quantised GEMM (``qgemm_dense``) against the fp64 oracle.

Bar: ``|y - y_ref| <= 1e-3 * sum_k |x_k w_k| + 1e-6`` elementwise, on the same
seeded inputs; full outputs where the oracle finishes in seconds, sampled
outputs (computed one by one by the oracle) at the largest workloads.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_levels, dev_w, dev_x, report, sample_pairs, tight_ratio, torch_or_skip

pytestmark = pytest.mark.gpu

FMTS = [synth.FMT_Q8, synth.FMT_Q4]


def run_dense(torch, case):
    import paper_2607_19438_amd as q
    x = dev_x(torch, case.x)
    wq, sc = dev_w(torch, case.w)
    y = q.dense(x, wq, sc, case.fmt)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def full_check(name, y, case, require_bar=True):
    exact = oracle.dense(case.x, case.w.wq, case.w.scales, case.fmt)
    rounded = oracle.dense(case.x, case.w.wq, case.w.scales, case.fmt, bf16_weights=True)
    check_levels(name, y, exact, rounded, case.K, require_bar)


def test_config0_dense_q8_full():
    torch = torch_or_skip()
    (case,) = synth.config(0)
    full_check(case.name, run_dense(torch, case), case)


def test_config1_dense_q4_full():
    torch = torch_or_skip()
    (case,) = synth.config(1)
    full_check(case.name, run_dense(torch, case), case)


@pytest.mark.parametrize("which", [0, 1])
def test_config2_dense_q8_sampled(which):
    """Full-size gate_up (2048x8192x2048) and down (2048x2048x8192), sampled outputs."""
    torch = torch_or_skip()
    case = synth.config(2)[which]
    y = run_dense(torch, case)
    assert np.isfinite(y).all()
    rng = synth.rng_for(99, which)
    rows, cols = sample_pairs(rng, case.M, case.N, 6000, extra_rows=[0, 255, 256, case.M - 1],
                              extra_cols=list(range(0, case.N, 97)))
    exact = oracle.dense_entries(case.x, case.w.wq, case.w.scales, case.fmt, rows, cols)
    rounded = oracle.dense_entries(case.x, case.w.wq, case.w.scales, case.fmt, rows, cols, bf16_weights=True)
    check_levels(case.name + " (sampled)", y[rows, cols], exact, rounded, case.K, True)


RAGGED = [
    (1, 1, 32), (1, 128, 64), (7, 33, 96), (31, 200, 160), (129, 130, 64),
    (255, 257, 288), (300, 1000, 32), (64, 64, 2048 + 32),
    (3857, 3684, 96),      # 256x256 tiles with ragged M and N tails
    (4096, 4096, 64),      # 256x256 tiles, exact
    (300, 1000, 1536),     # split-K over 2 workgroups per 256x256 tile, ragged M and N
    (1000, 700, 4096 + 32),  # split-K over 5, K tail inside the last split
    (512, 512, 8192),      # split-K over 8 on 128x256 tiles (the down-projection shape class)
    (1500, 4000, 160),     # 128x256 tiles above 1024 rows (no split), ragged M and N
    (1100, 4352, 1056),    # the same with an odd K-step count and a K tail
]
# every K-step count modulo the unrolled loop period (2 or 6 steps) and each K tail position,
# on the 128x128 tile (M < 256) and the 256x256 tile
K_STEPS = [(255, 257, 64 * s + t) for s, t in ((3, 32), (4, 0), (4, 32), (5, 0), (6, 32), (7, 0), (9, 32), (11, 0), (13, 32))]
K_STEPS += [(3584, 3840, K) for K in (288, 448, 736)]       # 210 tiles of 256x256, no split


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M,N,K", RAGGED + K_STEPS)
def test_ragged_shapes(fmt, M, N, K):
    torch = torch_or_skip()
    case = synth.dense_case(f"ragged_{synth.FMT_NAMES[fmt]}_{M}x{N}x{K}", fmt, M, N, K, seed=5, stream=(M, N, K))
    full_check(case.name, run_dense(torch, case), case, require_bar=K >= 512)


def test_empty_m_is_noop_and_errors_leave_y_untouched():
    torch = torch_or_skip()
    import paper_2607_19438_amd as q
    case = synth.dense_case("e", synth.FMT_Q8, 16, 64, 64, seed=1)
    x = dev_x(torch, case.x)
    wq, sc = dev_w(torch, case.w)
    y = torch.full((16, 64), 7.0, device="cuda")
    lib = q.lib()
    s = torch.cuda.current_stream().cuda_stream
    assert lib.qgemm_dense(x.data_ptr(), wq.data_ptr(), sc.data_ptr(), y.data_ptr(), 0, 64, 64, 0, s) == 0
    assert lib.qgemm_dense(x.data_ptr() + 2, wq.data_ptr(), sc.data_ptr(), y.data_ptr(), 16, 64, 64, 0, s) == -2
    assert lib.qgemm_dense(x.data_ptr(), wq.data_ptr(), sc.data_ptr(), y.data_ptr(), 16, 64, 48, 0, s) == -1
    assert lib.qgemm_dense(x.data_ptr(), wq.data_ptr(), sc.data_ptr(), y.data_ptr(), 16, 64, 64, 3, s) == -1
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())


@pytest.mark.parametrize("fmt", FMTS)
def test_bitwise_deterministic_and_tile_independent(fmt):
    """Repeat runs are bitwise equal; rows do not depend on which tile shape computed them."""
    torch = torch_or_skip()
    import paper_2607_19438_amd as q
    case = synth.dense_case("det", fmt, 4096, 4096, 256, seed=3)
    x = dev_x(torch, case.x)
    wq, sc = dev_w(torch, case.w)
    y1 = q.dense(x, wq, sc, fmt)        # 256x256 tiles
    y2 = q.dense(x, wq, sc, fmt)
    y3 = q.dense(x[:200].contiguous(), wq, sc, fmt)   # 128x128 tiles
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    assert torch.equal(y1[:200], y3)


@pytest.mark.parametrize("fmt", FMTS)
def test_split_k_bitwise_repeatable(fmt):
    """Split-K partials are summed in split order: repeat runs are bitwise equal."""
    torch = torch_or_skip()
    import paper_2607_19438_amd as q
    case = synth.dense_case("splitk", fmt, 1024, 1024, 4096, seed=8)
    x = dev_x(torch, case.x)
    wq, sc = dev_w(torch, case.w)
    y1 = q.dense(x, wq, sc, fmt)
    y2 = q.dense(x, wq, sc, fmt)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    rows = synth.rng_for(3).integers(0, 1024, 300)
    cols = synth.rng_for(4).integers(0, 1024, 300)
    exact = oracle.dense_entries(case.x, case.w.wq, case.w.scales, fmt, rows, cols)
    rounded = oracle.dense_entries(case.x, case.w.wq, case.w.scales, fmt, rows, cols, bf16_weights=True)
    check_levels("split-K 1024x1024x4096 (sampled)", y1.cpu().numpy()[rows, cols], exact, rounded, 4096, True)


def test_unit_scale_q_one_gives_row_sums_on_gpu():
    torch = torch_or_skip()
    M, N, K = 64, 256, 1024
    x = synth.make_x(synth.rng_for(4), M, K)
    for fmt in FMTS:
        w = synth.qweight_from_q(np.ones((N, K), np.int16), np.ones((N, K // 32)), fmt)
        case = synth.DenseCase("unit", fmt, M, N, K, x, w)
        y = run_dense(torch, case)
        rs = oracle.decode_bf16(x).sum(axis=1)
        babs = np.abs(oracle.decode_bf16(x)).sum(axis=1)
        # unit weights are exact in bf16: only fp32 summation error remains
        assert np.all(np.abs(y - rs[:, None]) <= oracle.fp32_sum_rel(K) * babs[:, None])


@pytest.mark.parametrize("fmt", FMTS)
def test_every_k_step_count_repeated(fmt):
    """One 128x128 tile for K = 64 .. 832 (1 to 13 K steps, with and without a half step), each
    run four times: the prefetch pipeline's waits must hold on every repetition, in every
    position of the unrolled loop period."""
    torch = torch_or_skip()
    for steps in range(1, 14):
        for K in (64 * steps, 64 * steps - 32):
            case = synth.dense_case(f"repeat_{synth.FMT_NAMES[fmt]}_K{K}", fmt, 128, 128, K, seed=9, stream=(K,))
            ref = oracle.dense(case.x, case.w.wq, case.w.scales, fmt, bf16_weights=True)
            for _ in range(4):
                y = run_dense(torch, case)
                assert tight_ratio(y, ref[0], ref[1], K) <= 1.0, f"K={K}"

