"""Python binding of ``libqgemm.so``, the gfx950 block-quantised prefill GEMM library.

Argument marshalling only: every step runs in the library's HIP kernels.
PyTorch provides device memory and the current HIP stream. The C entry points
and their contracts are declared in ``include/qgemm.h``; the Python functions
carry the same names without the ``qgemm_`` prefix.

The library must be built (``python -m paper_2607_19438_amd.build``); there is
no fallback path, and a missing library raises ``QGemmError``.
"""
from __future__ import annotations

import ctypes
import os

import torch  # imported before the library so that both share one HIP runtime

__all__ = ["Q8", "Q4", "QGemmError", "lib", "lib_path", "dense", "moe", "moe_noalloc", "moe_bucket", "moe_grouped",
           "moe_gate_up_swiglu", "moe_down_combine", "swiglu", "moe_combine", "attention_prefill", "probe_mfma_clock", "last_error", "release", "version", "EXPORTS", "ExpertTable"]

Q8 = 0
Q4 = 1
_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libqgemm.so")

_vp = ctypes.c_void_p
_i = ctypes.c_int
# name -> (restype, argtypes); mirrors include/qgemm.h
EXPORTS = {
    "qgemm_dense": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp]),
    "qgemm_moe": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "qgemm_moe_noalloc": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "qgemm_moe_bucket": (_i, [_vp, _vp, _vp, _i, _i, _vp]),
    "qgemm_moe_grouped": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "qgemm_moe_gate_up_swiglu": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "qgemm_moe_down_combine": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _i, _vp]),
    "qgemm_swiglu": (_i, [_vp, _vp, _i, _i, _vp]),
    "qgemm_moe_combine": (_i, [_vp, _vp, _vp, _i, _i, _i, _vp]),
    "qgemm_attention_prefill": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, ctypes.c_float, _i, _vp]),
    "qgemm_probe_mfma_clock": (_i, [_i, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double), _vp]),
    "qgemm_last_error": (ctypes.c_char_p, []),
    "qgemm_release": (_i, []),
    "qgemm_version": (_i, []),
}


class QGemmError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"qgemm error {code}: {msg}")
        self.code = code


_lib = None


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """Load ``libqgemm.so`` (once) and declare every exported symbol's signature."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise QGemmError(-4, f"{_LIB_PATH} is not built; run `python -m paper_2607_19438_amd.build`")
        handle = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def _check(rc: int):
    if rc != 0:
        raise QGemmError(rc, lib().qgemm_last_error().decode())


def _stream(t: torch.Tensor):
    return torch.cuda.current_stream(t.device).cuda_stream


def _need(t: torch.Tensor, name: str, dtypes, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype not in dtypes:
        raise TypeError(f"{name} has dtype {t.dtype}, expected one of {dtypes}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dimensions")


_W_DTYPES = (torch.int8, torch.uint8)


def _wshape_k(wq: torch.Tensor, fmt: int) -> int:
    return wq.shape[-1] if fmt == Q8 else wq.shape[-1] * 2


def version() -> int:
    return lib().qgemm_version()


def last_error() -> str:
    return lib().qgemm_last_error().decode()


def release():
    _check(lib().qgemm_release())


def dense(x: torch.Tensor, wq: torch.Tensor, scales: torch.Tensor, fmt: int, out: torch.Tensor | None = None):
    """``y[M][N] = x[M][K] . dequant(wq, scales)^T`` in fp32 (``qgemm_dense``)."""
    _need(x, "x", (torch.bfloat16,), 2)
    _need(wq, "wq", _W_DTYPES, 2)
    _need(scales, "scales", (torch.float16,), 2)
    M, K = x.shape
    N = wq.shape[0]
    if _wshape_k(wq, fmt) != K or scales.shape != (N, K // 32):
        raise ValueError("x, wq and scales disagree on N or K")
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=x.device)
    _need(out, "out", (torch.float32,), 2)
    if out.shape != (M, N):
        raise ValueError("out must be [M][N]")
    _check(lib().qgemm_dense(x.data_ptr(), wq.data_ptr(), scales.data_ptr(), out.data_ptr(), M, N, K, fmt,
                             _stream(x)))
    return out


class ExpertTable:
    """Validated per-expert weights with their host pointer arrays, built once and reused.

    ``wq`` / ``scales``: lists of E tensors or stacked ``[E, N, K']`` / ``[E, N, K/32]`` tensors.
    """

    def __init__(self, wq, scales, fmt: int):
        if isinstance(wq, torch.Tensor):
            wq = list(wq.unbind(0))
        if isinstance(scales, torch.Tensor):
            scales = list(scales.unbind(0))
        if len(wq) != len(scales) or not wq:
            raise ValueError("need one weight and one scale tensor per expert")
        for t in wq:
            _need(t, "wq[e]", _W_DTYPES, 2)
        for t in scales:
            _need(t, "scales[e]", (torch.float16,), 2)
        self.E = len(wq)
        self.N = wq[0].shape[0]
        self.K = _wshape_k(wq[0], fmt)
        self.fmt = fmt
        if any(w.shape[0] != self.N or _wshape_k(w, fmt) != self.K for w in wq) or any(
                s.shape != (self.N, self.K // 32) for s in scales):
            raise ValueError("expert weights disagree on N or K")
        self.wq, self.scales = wq, scales          # keep the tensors alive
        self.wp = (ctypes.c_void_p * self.E)(*[t.data_ptr() for t in wq])
        self.sp = (ctypes.c_void_p * self.E)(*[t.data_ptr() for t in scales])


def _expert_tables(wq, scales, E, fmt=None):
    """Host arrays of per-expert device pointers from lists or stacked [E, ...] tensors."""
    if isinstance(wq, ExpertTable):
        if wq.E != E:
            raise ValueError("expert table has the wrong number of experts")
        return wq.wq, wq.scales, wq.wp, wq.sp
    if isinstance(wq, torch.Tensor):
        wq = list(wq.unbind(0))
    if isinstance(scales, torch.Tensor):
        scales = list(scales.unbind(0))
    if len(wq) != E or len(scales) != E:
        raise ValueError("need one weight and one scale tensor per expert")
    for t in wq:
        _need(t, "wq[e]", _W_DTYPES, 2)
    for t in scales:
        _need(t, "scales[e]", (torch.float16,), 2)
    wp = (ctypes.c_void_p * E)(*[t.data_ptr() for t in wq])
    sp = (ctypes.c_void_p * E)(*[t.data_ptr() for t in scales])
    return wq, scales, wp, sp


def moe(x, token_expert_idx, expert_offsets, wq, scales, topk: int, fmt: int, out=None):
    """MoE expert GEMM over token slots (``qgemm_moe``): ``y[T*topk][N]`` fp32 in slot order.

    ``wq`` may be an ExpertTable (then ``scales`` is ignored)."""
    _need(x, "x", (torch.bfloat16,), 2)
    _need(token_expert_idx, "token_expert_idx", (torch.int32,), 1)
    _need(expert_offsets, "expert_offsets", (torch.int32,), 1)
    T, K = x.shape
    E = expert_offsets.shape[0] - 1
    wq, scales, wp, sp = _expert_tables(wq, scales, E)
    N = wq[0].shape[0]
    if token_expert_idx.shape[0] != T * topk:
        raise ValueError("token_expert_idx must have T*topk entries")
    if any(_wshape_k(w, fmt) != K or w.shape[0] != N for w in wq):
        raise ValueError("expert weights disagree with x on K or with each other on N")
    if out is None:
        out = torch.empty((T * topk, N), dtype=torch.float32, device=x.device)
    _need(out, "out", (torch.float32,), 2)
    _check(lib().qgemm_moe(x.data_ptr(), token_expert_idx.data_ptr(), expert_offsets.data_ptr(), wp, sp,
                           out.data_ptr(), T, E, topk, N, K, fmt, _stream(x)))
    return out


def moe_noalloc(x, token_expert_idx, expert_offsets, wq, scales, topk: int, fmt: int, out=None):
    """``qgemm_moe_noalloc``: as ``moe`` with the bucketing buffers in the library's static device
    scratch (no device allocation in the call; ``out`` should be given by callers that cannot
    allocate). ``wq`` may be an ExpertTable."""
    _need(x, "x", (torch.bfloat16,), 2)
    _need(token_expert_idx, "token_expert_idx", (torch.int32,), 1)
    _need(expert_offsets, "expert_offsets", (torch.int32,), 1)
    T, K = x.shape
    E = expert_offsets.shape[0] - 1
    wq, scales, wp, sp = _expert_tables(wq, scales, E)
    N = wq[0].shape[0]
    if token_expert_idx.shape[0] != T * topk:
        raise ValueError("token_expert_idx must have T*topk entries")
    if out is None:
        out = torch.empty((T * topk, N), dtype=torch.float32, device=x.device)
    _need(out, "out", (torch.float32,), 2)
    _check(lib().qgemm_moe_noalloc(x.data_ptr(), token_expert_idx.data_ptr(), expert_offsets.data_ptr(), wp, sp,
                                   out.data_ptr(), T, E, topk, N, K, fmt, _stream(x)))
    return out


def moe_bucket(token_expert_idx, expert_offsets, out=None):
    """Assignments grouped by expert, stable (``qgemm_moe_bucket``)."""
    _need(token_expert_idx, "token_expert_idx", (torch.int32,), 1)
    _need(expert_offsets, "expert_offsets", (torch.int32,), 1)
    n = token_expert_idx.shape[0]
    E = expert_offsets.shape[0] - 1
    if out is None:
        out = torch.empty((n,), dtype=torch.int32, device=token_expert_idx.device)
    _need(out, "out", (torch.int32,), 1)
    _check(lib().qgemm_moe_bucket(token_expert_idx.data_ptr(), expert_offsets.data_ptr(), out.data_ptr(), n, E,
                                  _stream(token_expert_idx)))
    return out


def moe_grouped(x, perm, expert_offsets, wq, scales, topk: int, fmt: int, out=None):
    """Grouped GEMM from an existing bucketing (``qgemm_moe_grouped``); ``wq`` may be an ExpertTable."""
    _need(x, "x", (torch.bfloat16,), 2)
    _need(perm, "perm", (torch.int32,), 1)
    _need(expert_offsets, "expert_offsets", (torch.int32,), 1)
    T, K = x.shape
    E = expert_offsets.shape[0] - 1
    wq, scales, wp, sp = _expert_tables(wq, scales, E)
    N = wq[0].shape[0]
    if out is None:
        out = torch.empty((T * topk, N), dtype=torch.float32, device=x.device)
    _need(out, "out", (torch.float32,), 2)
    _check(lib().qgemm_moe_grouped(x.data_ptr(), perm.data_ptr(), expert_offsets.data_ptr(), wp, sp,
                                   out.data_ptr(), T, E, topk, N, K, fmt, _stream(x)))
    return out


def moe_gate_up_swiglu(x, perm, expert_offsets, wq, scales, topk: int, fmt: int, out=None):
    """Fused gate/up projection + SiLU gate (``qgemm_moe_gate_up_swiglu``): bf16 ``h[T*topk][inter]``.

    Expert weights are ``[2*inter][K]`` (gate rows, then up rows); ``wq`` may be an ExpertTable."""
    _need(x, "x", (torch.bfloat16,), 2)
    _need(perm, "perm", (torch.int32,), 1)
    _need(expert_offsets, "expert_offsets", (torch.int32,), 1)
    T, K = x.shape
    E = expert_offsets.shape[0] - 1
    wq, scales, wp, sp = _expert_tables(wq, scales, E)
    N = wq[0].shape[0]
    if N % 2 != 0:
        raise ValueError("gate/up weights need an even number of rows")
    inter = N // 2
    if out is None:
        out = torch.empty((T * topk, inter), dtype=torch.bfloat16, device=x.device)
    _need(out, "out", (torch.bfloat16,), 2)
    if out.shape != (T * topk, inter):
        raise ValueError("out must be [T*topk][inter]")
    _check(lib().qgemm_moe_gate_up_swiglu(x.data_ptr(), perm.data_ptr(), expert_offsets.data_ptr(), wp, sp,
                                          out.data_ptr(), T, E, topk, inter, K, fmt, _stream(x)))
    return out


def moe_down_combine(h, perm, expert_offsets, wq, scales, route_w, topk: int, fmt: int, y2=None, out=None):
    """Down projection over token slots with the router-weighted combine fused in
    (``qgemm_moe_down_combine``): returns ``(y2 [T*topk][N], out [T][N])``, both fp32.
    ``wq`` may be an ExpertTable."""
    _need(h, "h", (torch.bfloat16,), 2)
    _need(perm, "perm", (torch.int32,), 1)
    _need(expert_offsets, "expert_offsets", (torch.int32,), 1)
    _need(route_w, "route_w", (torch.float32,), 1)
    A, K = h.shape
    if A % topk != 0 or route_w.shape[0] != A:
        raise ValueError("h and route_w need T*topk rows")
    T = A // topk
    E = expert_offsets.shape[0] - 1
    wq, scales, wp, sp = _expert_tables(wq, scales, E)
    N = wq[0].shape[0]
    if any(_wshape_k(w, fmt) != K or w.shape[0] != N for w in wq):
        raise ValueError("expert weights disagree with h on K or with each other on N")
    if y2 is None:
        y2 = torch.empty((A, N), dtype=torch.float32, device=h.device)
    if out is None:
        out = torch.empty((T, N), dtype=torch.float32, device=h.device)
    _need(y2, "y2", (torch.float32,), 2)
    _need(out, "out", (torch.float32,), 2)
    if y2.shape != (A, N) or out.shape != (T, N):
        raise ValueError("y2 must be [T*topk][N] and out [T][N]")
    _check(lib().qgemm_moe_down_combine(h.data_ptr(), perm.data_ptr(), expert_offsets.data_ptr(), wp, sp,
                                        route_w.data_ptr(), y2.data_ptr(), out.data_ptr(), T, E, topk, N, K, fmt,
                                        _stream(h)))
    return y2, out


def swiglu(y1, out=None):
    """``h = bf16(silu(gate) * up)`` over ``y1 = [gate | up]`` (``qgemm_swiglu``)."""
    _need(y1, "y1", (torch.float32,), 2)
    rows, two_inter = y1.shape
    inter = two_inter // 2
    if out is None:
        out = torch.empty((rows, inter), dtype=torch.bfloat16, device=y1.device)
    _need(out, "out", (torch.bfloat16,), 2)
    _check(lib().qgemm_swiglu(y1.data_ptr(), out.data_ptr(), rows, inter, _stream(y1)))
    return out


def moe_combine(y2, route_w, topk: int, out=None):
    """``out[t] = sum_j route_w[t*topk+j] * y2[t*topk+j]`` (``qgemm_moe_combine``)."""
    _need(y2, "y2", (torch.float32,), 2)
    _need(route_w, "route_w", (torch.float32,), 1)
    A, N = y2.shape
    T = A // topk
    if out is None:
        out = torch.empty((T, N), dtype=torch.float32, device=y2.device)
    _need(out, "out", (torch.float32,), 2)
    _check(lib().qgemm_moe_combine(y2.data_ptr(), route_w.data_ptr(), out.data_ptr(), T, topk, N, _stream(y2)))
    return out


def attention_prefill(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, causal: bool = True,
                      scale: float | None = None, out: torch.Tensor | None = None):
    """``qgemm_attention_prefill``: q ``[B][S][H][D]``, k / v ``[B][S][Hkv][D]`` bf16 -> o ``[B][S][H][D]`` bf16."""
    _need(q, "q", (torch.bfloat16,), 4)
    _need(k, "k", (torch.bfloat16,), 4)
    _need(v, "v", (torch.bfloat16,), 4)
    B, S, H, D = q.shape
    if k.shape != v.shape or k.shape[0] != B or k.shape[1] != S or k.shape[3] != D:
        raise ValueError("q, k and v disagree on B, S or D")
    Hkv = k.shape[2]
    if scale is None:
        scale = 1.0 / float(D) ** 0.5
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", (torch.bfloat16,), 4)
    if out.shape != q.shape:
        raise ValueError("out must have the shape of q")
    _check(lib().qgemm_attention_prefill(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, S, H, Hkv, D,
                                         float(scale), int(bool(causal)), _stream(q)))
    return out


def probe_mfma_clock(iters: int = 100000):
    """Sustained shader clock (MHz) and bf16 MFMA throughput (TFLOP/s) under full matrix-core load
    (``qgemm_probe_mfma_clock``; synchronises the current stream). A measurement utility."""
    mhz = ctypes.c_double(0.0)
    tf = ctypes.c_double(0.0)
    _check(lib().qgemm_probe_mfma_clock(int(iters), ctypes.byref(mhz), ctypes.byref(tf),
                                        torch.cuda.current_stream().cuda_stream))
    return {"sclk_mhz": mhz.value, "mfma_tflops": tf.value}
