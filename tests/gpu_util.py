"""Shared helpers of the GPU parity tests: moving seeded inputs to the device and sampling."""
import numpy as np
import pytest

import synth


def torch_or_skip():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU in this environment")
    return torch


def dev_x(torch, bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def dev_w(torch, w: synth.QWeight):
    return torch.from_numpy(np.ascontiguousarray(w.wq)).cuda(), torch.from_numpy(np.ascontiguousarray(w.scales)).cuda()


def dev_experts(torch, ws):
    """Stack E expert weights into contiguous [E, N, K'] / [E, N, K/32] device tensors."""
    wq = torch.from_numpy(np.ascontiguousarray(np.stack([w.wq for w in ws]))).cuda()
    sc = torch.from_numpy(np.ascontiguousarray(np.stack([w.scales for w in ws]))).cuda()
    return wq, sc


def dev_i32(torch, a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.int32))).cuda()


def dev_f32(torch, a):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a, dtype=np.float32))).cuda()


def sample_pairs(rng, R, C, n, extra_rows=(), extra_cols=()):
    """n random (row, col) pairs plus the corners and the given rows x cols cross."""
    rows = list(rng.integers(0, R, n)) + [0, R - 1, 0, R - 1]
    cols = list(rng.integers(0, C, n)) + [0, 0, C - 1, C - 1]
    for r in extra_rows:
        for c in extra_cols:
            rows.append(r)
            cols.append(c)
    return np.array(rows, np.int64), np.array(cols, np.int64)


def report(name, ratio):
    print(f"[parity] {name}: max |err| / bar = {ratio:.3e}", flush=True)


def tight_ratio(y, y_b, bound_b, K):
    """Ratio to the fp32-summation bound against the oracle evaluated with bf16-rounded weights."""
    import oracle
    tol = oracle.fp32_sum_rel(K) * np.asarray(bound_b) + 1e-30
    y = np.asarray(y, np.float64)
    if not np.all(np.isfinite(y)):
        return np.inf
    return float(np.max(np.abs(y - y_b) / tol)) if y.size else 0.0


def check_levels(name, y, exact, rounded, K, require_bar):
    """Tight check against bf16-rounded weights; the 1e-3 acceptance bar against exact weights.

    exact / rounded: (y_ref, bound) pairs from the oracle without / with bf16-rounded weights.
    The bar is required at the workload sizes (K >= 512), where bf16 weight rounding
    (relative 2**-8 per weight, random sign) averages well below 1e-3 of the bound.
    """
    import oracle
    t = tight_ratio(y, rounded[0], rounded[1], K)
    r = oracle.bar_ratio(y, exact[0], exact[1])
    print(f"[parity] {name}: fp32-sum ratio vs bf16-weight oracle = {t:.3e}; "
          f"acceptance-bar ratio vs exact oracle = {r:.3e}", flush=True)
    assert t <= 1.0, f"{name}: exceeds the fp32 summation bound ({t})"
    if require_bar:
        assert r <= 1.0, f"{name}: exceeds the acceptance bar ({r})"
