"""GPU parity of the small-M dense path against the fp64 oracle: ``qgemm_dense`` with M <= 16, and
with 16 < M <= 128 when the 128x128 tiles would occupy few CUs (then in blocks of 16 columns).

Small M is the decode / speculative-verification shape (and a short prompt's): every weight is read
once and dequantised straight into MFMA operand registers, K is split over waves and workgroups,
and the partial sums are added in a fixed order. Bar: ``|y - y_ref| <= 1e-3 * sum_k |x_k w_k| + 1e-6`` elementwise,
plus the fp32-summation bound against the oracle with bf16-rounded weights.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import check_levels, dev_w, dev_x, torch_or_skip

pytestmark = pytest.mark.gpu

FMTS = [synth.FMT_Q8, synth.FMT_Q4]


def q():
    import paper_2607_19438_amd as m
    return m


def run(torch, case, out=None):
    x = dev_x(torch, case.x)
    wq, sc = dev_w(torch, case.w)
    y = q().dense(x, wq, sc, case.fmt, out=out)
    torch.cuda.synchronize()
    return y


def check(case, y, require_bar=None):
    exact = oracle.dense(case.x, case.w.wq, case.w.scales, case.fmt)
    rounded = oracle.dense(case.x, case.w.wq, case.w.scales, case.fmt, bf16_weights=True)
    check_levels(case.name, y, exact, rounded, case.K, case.K >= 512 if require_bar is None else require_bar)


# (N, K): one row block and one chunk; ragged N; every Q8 / Q4 K tail inside a chunk; K splits
# over many workgroups (long K, few rows); several splits with a short last split
SHAPES = [(1, 32), (17, 64), (33, 96), (100, 224), (257, 1056), (31, 2048 + 96), (64, 8192 + 32),
          (1000, 4096), (96, 160), (513, 640)]


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("M", [1, 2, 3, 5, 8, 12, 15, 16, 17, 24, 32, 33, 48, 64, 100, 128])
@pytest.mark.parametrize("N,K", SHAPES)
def test_small_m_shapes(fmt, M, N, K):
    torch = torch_or_skip()
    case = synth.dense_case(f"small_{synth.FMT_NAMES[fmt]}_{M}x{N}x{K}", fmt, M, N, K, seed=8, stream=(M, N, K))
    check(case, run(torch, case).cpu().numpy())


@pytest.mark.parametrize("M", [1, 4, 16])
@pytest.mark.parametrize("fmt,N,K", [(synth.FMT_Q4, 8192, 3072), (synth.FMT_Q8, 8192, 2048),
                                     (synth.FMT_Q8, 2048, 8192), (synth.FMT_Q4, 1536, 2048),
                                     (synth.FMT_Q4, 2048, 768)])
def test_small_m_full_size(fmt, N, K, M):
    """Projection shapes of the prefill workloads at decode / verification batch sizes, every output."""
    torch = torch_or_skip()
    case = synth.dense_case(f"small_full_{synth.FMT_NAMES[fmt]}_{M}x{N}x{K}", fmt, M, N, K, seed=9,
                            stream=(M, N, K))
    check(case, run(torch, case).cpu().numpy(), require_bar=True)


@pytest.mark.parametrize("M,fmt,N,K", [(128, synth.FMT_Q8, 1024, 1024), (96, synth.FMT_Q4, 2048, 3072),
                                       (40, synth.FMT_Q8, 4096, 2048), (128, synth.FMT_Q4, 512, 8192)])
def test_wide_small_m_full(M, fmt, N, K):
    """Short-prompt shapes on the blocks-of-16-columns path, every output against the oracle and
    bitwise repeatable."""
    torch = torch_or_skip()
    case = synth.dense_case(f"wide_{synth.FMT_NAMES[fmt]}_{M}x{N}x{K}", fmt, M, N, K, seed=14, stream=(M, N, K))
    y = run(torch, case).cpu().numpy()
    check(case, y, require_bar=True)
    y2 = run(torch, case).cpu().numpy()
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32))


def test_small_m_deterministic_across_split_counts():
    """Repeated calls are bitwise equal, also when calls with other split counts run in between
    (the per-row-block arrival counters must be back at zero after every call)."""
    torch = torch_or_skip()
    a = synth.dense_case("det_a", synth.FMT_Q8, 9, 200, 8192, seed=10, stream=(1,))     # many splits
    b = synth.dense_case("det_b", synth.FMT_Q4, 16, 8192, 3072, seed=10, stream=(2,))   # few splits
    c = synth.dense_case("det_c", synth.FMT_Q4, 3, 64, 256, seed=10, stream=(3,))       # one split
    first = [run(torch, k).cpu().numpy() for k in (a, b, c)]
    for _ in range(3):
        for k, y0 in zip((a, b, c, a), first + [first[0]]):
            y = run(torch, k).cpu().numpy()
            assert np.array_equal(y.view(np.uint32), y0.view(np.uint32)), k.name
    check(a, first[0])
    check(b, first[1])


def test_small_m_writes_only_y():
    """Entries of a larger buffer around y stay untouched (no stores past M rows or N columns)."""
    torch = torch_or_skip()
    M, N, K = 5, 70, 4096
    case = synth.dense_case("small_guard", synth.FMT_Q4, M, N, K, seed=11, stream=(4,))
    pad = 64                                     # keeps y 16-byte aligned
    big = torch.full((2 * pad + M * N,), 3.5, dtype=torch.float32, device="cuda")
    y = big[pad:pad + M * N].view(M, N)
    run(torch, case, out=y)
    b = big.cpu().numpy()
    assert np.all(b[:pad] == 3.5) and np.all(b[pad + M * N:] == 3.5)
    check(case, y.cpu().numpy())
