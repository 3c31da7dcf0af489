"""ctypes binding of libhstu (include/hstu.h), argument marshalling only.

Each C entry point has a Python function of the same name that takes
torch tensors (device memory) and passes their data pointers, strides and
the current HIP stream.  Every step of the computation runs in the HIP
kernels of libhstu.so; if the library is missing or fails to load, import
of this module raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhstu.so")

HSTU_F32, HSTU_BF16 = 0, 1
STATUS = {0: "HSTU_OK", 1: "HSTU_ERR_INVALID_ARGUMENT", 2: "HSTU_ERR_UNSUPPORTED",
          3: "HSTU_ERR_WORKSPACE", 4: "HSTU_ERR_HIP", 5: "HSTU_ERR_DATA"}

EXPORTED = ("hstu_workspace_bytes", "hstu_attn_fwd", "hstu_attn_bwd", "hstu_layer_fwd",
            "hstu_time_bucketize", "hstu_complete_cumsum", "hstu_pair_offsets", "hstu_validate",
            "hstu_last_error", "hstu_abi_version", "hstu_timing_enable", "hstu_timing_read",
            "hstu_timing_reset", "hstu_probe_mfma_bf16", "hstu_layer_bwd",
            "hstu_attn_fwd_cached", "hstu_attn_fwd_cached_workspace_bytes",
            "hstu_proj_workspace_bytes", "hstu_proj_in_fwd",
            "hstu_proj_out_fwd", "hstu_proj_out_bwd", "hstu_proj_in_bwd",
            "hstu_sl_subseq_len", "hstu_sl_keep_numerator", "hstu_sl_workspace_bytes",
            "hstu_stochastic_length", "hstu_gather_rows", "hstu_sl_sparsity",
            "hstu_attn_fwd_noalloc")


class Problem(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("total_tokens", ctypes.c_int64),
                ("max_seq_len", ctypes.c_int32), ("num_heads", ctypes.c_int32),
                ("d_qk", ctypes.c_int32), ("d_v", ctypes.c_int32),
                ("num_time_buckets", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class Jagged(ctypes.Structure):
    _fields_ = [("seq_offsets", ctypes.c_void_p), ("timestamps", ctypes.c_void_p),
                ("num_targets", ctypes.c_void_p), ("rab_pos", ctypes.c_void_p),
                ("rab_time", ctypes.c_void_p)]


class HstuError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz, f32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t,
                            ctypes.c_float)
    PP, PJ = ctypes.POINTER(Problem), ctypes.POINTER(Jagged)
    sig = {
        "hstu_workspace_bytes": (sz, [PP]),
        "hstu_attn_fwd": (i32, [PP, PJ, P, i64, P, i64, P, i64, P, P, sz, P]),
        "hstu_attn_bwd": (i32, [PP, PJ, P, i64, P, i64, P, i64, P, P, P, P, P, P, P, sz, P]),
        "hstu_layer_fwd": (i32, [PP, PJ, P, i64, P, i64, P, i64, P, i64, P, P, f32, P, P, P, P,
                                 P, sz, P]),
        "hstu_layer_bwd": (i32, [PP, PJ, P, i64, P, i64, P, i64, P, i64, P, P, P, P, P, P,
                                 P, P, P, P, P, P, P, P, P, sz, P]),
        "hstu_attn_fwd_cached": (i32, [PP, PJ, P, i64, P, i64, P, i64, P, P, i64, P, i64, P, i64,
                                       P, P, sz, P]),
        "hstu_time_bucketize": (i32, [i32, i64, i32, P, P, P, i64, P, P]),
        "hstu_complete_cumsum": (i32, [i32, P, P, P]),
        "hstu_pair_offsets": (i32, [i32, P, P, P]),
        "hstu_validate": (i32, [PP, PJ, P]),
        "hstu_last_error": (ctypes.c_char_p, []),
        "hstu_abi_version": (i32, []),
        "hstu_timing_enable": (i32, [i32]),
        "hstu_timing_read": (i32, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(ctypes.c_int64)]),
        "hstu_timing_reset": (i32, []),
        "hstu_probe_mfma_bf16": (i32, [i32, i32, P, ctypes.POINTER(ctypes.c_double), P]),
        "hstu_proj_workspace_bytes": (sz, [PP, i32]),
        "hstu_attn_fwd_cached_workspace_bytes": (sz, [PP]),
        "hstu_sl_subseq_len": (i32, [i32, ctypes.c_double]),
        "hstu_sl_keep_numerator": (ctypes.c_double, [i32, ctypes.c_double]),
        "hstu_attn_fwd_noalloc": (i32, [PP, PJ, P, i64, P, i64, P, i64, P, P]),
        "hstu_sl_workspace_bytes": (sz, [i32]),
        "hstu_stochastic_length": (i32, [i32, P, P, P, i32, ctypes.c_double, i32, P, P, P, P, P,
                                         sz, P]),
        "hstu_gather_rows": (i32, [P, i64, i64, P, P, i64, P, i64, P]),
        "hstu_sl_sparsity": (i32, [i32, P, i32, ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(ctypes.c_double)]),
        "hstu_proj_in_fwd": (i32, [PP, i32, P, i64, P, P, P, P, P]),
        "hstu_proj_out_fwd": (i32, [PP, i32, P, i64, P, P, P, P, P]),
        "hstu_proj_out_bwd": (i32, [PP, i32, P, i64, P, P, P, P, P, P, sz, P]),
        "hstu_proj_in_bwd": (i32, [PP, i32, P, i64, P, P, P, P, P, P, P, P, P, P, P, sz, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def _check(status: int):
    if status != 0:
        raise HstuError(status, lib.hstu_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return HSTU_BF16
    if t.dtype == torch.float32:
        return HSTU_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _row_stride(t: torch.Tensor) -> int:
    """Row stride in elements of a [T, h, d] (or [T, h*d]) view whose rows
    are [h][d]-contiguous."""
    if t.dim() == 3:
        if t.stride(2) != 1 or t.stride(1) != t.shape[2]:
            raise ValueError("rows must be [h][d] contiguous")
    elif t.dim() == 2:
        if t.stride(1) != 1:
            raise ValueError("rows must be contiguous")
    else:
        raise ValueError("expected a [T, h, d] or [T, h*d] tensor")
    return t.stride(0)


def make_problem(num_seqs, total_tokens, max_seq_len, num_heads, d_qk, d_v, num_time_buckets,
                 dtype) -> Problem:
    return Problem(int(num_seqs), int(total_tokens), int(max_seq_len), int(num_heads), int(d_qk),
                   int(d_v), int(num_time_buckets), int(dtype))


def make_jagged(seq_offsets, timestamps, rab_pos, rab_time, num_targets=None) -> Jagged:
    return Jagged(seq_offsets.data_ptr(), timestamps.data_ptr(),
                  None if num_targets is None else num_targets.data_ptr(),
                  rab_pos.data_ptr(), rab_time.data_ptr())


def problem_for(q, v, seq_offsets, max_seq_len, rab_time) -> Problem:
    T, H, dqk = q.shape[0], q.shape[1], q.shape[2]
    dv = v.shape[2]
    return make_problem(seq_offsets.numel() - 1, T, max_seq_len, H, dqk, dv, rab_time.numel(),
                        _dtype_code(q))


# ---------------------------------------------------------------- raw names

def hstu_abi_version() -> int:
    return int(lib.hstu_abi_version())


def hstu_last_error() -> str:
    return lib.hstu_last_error().decode()


def hstu_workspace_bytes(problem: Problem) -> int:
    return int(lib.hstu_workspace_bytes(ctypes.byref(problem)))


def workspace(problem: Problem, device=None) -> torch.Tensor:
    n = hstu_workspace_bytes(problem)
    if n == 0:
        raise HstuError(1, "invalid problem")
    return torch.empty(n, dtype=torch.uint8, device=device or "cuda")


def hstu_attn_fwd(q, k, v, seq_offsets, timestamps, rab_pos, rab_time, max_seq_len,
                  num_targets=None, out=None, ws=None, stream=None):
    """O [T, h, d_v] of Eq. 2 (see include/hstu.h)."""
    p = problem_for(q, v, seq_offsets, max_seq_len, rab_time)
    j = make_jagged(seq_offsets, timestamps, rab_pos, rab_time, num_targets)
    if out is None:
        out = torch.empty((q.shape[0], q.shape[1], v.shape[2]), dtype=q.dtype, device=q.device)
    if ws is None:
        ws = workspace(p, q.device)
    _check(lib.hstu_attn_fwd(ctypes.byref(p), ctypes.byref(j), _ptr(q), _row_stride(q), _ptr(k),
                             _row_stride(k), _ptr(v), _row_stride(v), _ptr(out), _ptr(ws),
                             ws.numel(), _stream(stream)))
    return out


def hstu_attn_fwd_noalloc(q, k, v, seq_offsets, timestamps, rab_pos, rab_time, max_seq_len, out,
                          num_targets=None, stream=None):
    """hstu_attn_fwd with its scratch in the library's static device array
    (no workspace; `out` [T, h, d_v] is required, nothing is allocated)."""
    p = problem_for(q, v, seq_offsets, max_seq_len, rab_time)
    j = make_jagged(seq_offsets, timestamps, rab_pos, rab_time, num_targets)
    _check(lib.hstu_attn_fwd_noalloc(ctypes.byref(p), ctypes.byref(j), _ptr(q), _row_stride(q),
                                     _ptr(k), _row_stride(k), _ptr(v), _row_stride(v), _ptr(out),
                                     _stream(stream)))
    return out


def hstu_attn_fwd_cached_workspace_bytes(problem: Problem) -> int:
    return int(lib.hstu_attn_fwd_cached_workspace_bytes(ctypes.byref(problem)))


def cached_workspace(problem: Problem, device=None) -> torch.Tensor:
    n = hstu_attn_fwd_cached_workspace_bytes(problem)
    if n == 0:
        raise HstuError(1, "invalid problem")
    return torch.empty(n, dtype=torch.uint8, device=device or "cuda")


def hstu_attn_fwd_cached(q, k, v, seq_offsets, timestamps, k_cache, v_cache, cache_offsets,
                         cache_timestamps, rab_pos, rab_time, max_seq_len, out=None, ws=None,
                         stream=None):
    """O [T, h, d_v] of the candidate rows q, k, v (offsets seq_offsets) against
    the cached history keys and values k_cache, v_cache (offsets
    cache_offsets); see include/hstu.h."""
    p = problem_for(q, v, seq_offsets, max_seq_len, rab_time)
    j = make_jagged(seq_offsets, timestamps, rab_pos, rab_time, None)
    if out is None:
        out = torch.empty((q.shape[0], q.shape[1], v.shape[2]), dtype=q.dtype, device=q.device)
    if ws is None:
        ws = cached_workspace(p, q.device)
    _check(lib.hstu_attn_fwd_cached(ctypes.byref(p), ctypes.byref(j), _ptr(q), _row_stride(q),
                                    _ptr(k), _row_stride(k), _ptr(v), _row_stride(v),
                                    _ptr(cache_offsets), _ptr(cache_timestamps),
                                    int(k_cache.shape[0]), _ptr(k_cache), _row_stride(k_cache),
                                    _ptr(v_cache), _row_stride(v_cache), _ptr(out), _ptr(ws),
                                    ws.numel(), _stream(stream)))
    return out


def hstu_attn_bwd(q, k, v, d_out, seq_offsets, timestamps, rab_pos, rab_time, max_seq_len,
                  num_targets=None, grads=None, ws=None, stream=None):
    """(dq, dk, dv, d_rab_pos, d_rab_time) for the loss <O, d_out>."""
    p = problem_for(q, v, seq_offsets, max_seq_len, rab_time)
    j = make_jagged(seq_offsets, timestamps, rab_pos, rab_time, num_targets)
    if grads is None:
        T, H = q.shape[0], q.shape[1]
        grads = (torch.empty((T, H, q.shape[2]), dtype=q.dtype, device=q.device),
                 torch.empty((T, H, k.shape[2]), dtype=q.dtype, device=q.device),
                 torch.empty((T, H, v.shape[2]), dtype=q.dtype, device=q.device),
                 torch.empty_like(rab_pos), torch.empty_like(rab_time))
    dq, dk, dv, drp, drt = grads
    if ws is None:
        ws = workspace(p, q.device)
    _check(lib.hstu_attn_bwd(ctypes.byref(p), ctypes.byref(j), _ptr(q), _row_stride(q), _ptr(k),
                             _row_stride(k), _ptr(v), _row_stride(v), _ptr(d_out), _ptr(dq),
                             _ptr(dk), _ptr(dv), _ptr(drp), _ptr(drt), _ptr(ws), ws.numel(),
                             _stream(stream)))
    return grads


def hstu_layer_fwd(q, k, v, u, seq_offsets, timestamps, rab_pos, rab_time, max_seq_len,
                   num_targets=None, ln_weight=None, ln_bias=None, ln_eps=1e-5, attn_out=None,
                   y=None, ln_mean=None, ln_rstd=None, ws=None, stream=None):
    """(attn_out [T, D] fp32, y [T, D], ln_mean [T], ln_rstd [T]) of Eq. 2-3."""
    p = problem_for(q, v, seq_offsets, max_seq_len, rab_time)
    j = make_jagged(seq_offsets, timestamps, rab_pos, rab_time, num_targets)
    T, D = q.shape[0], q.shape[1] * v.shape[2]
    if attn_out is None:
        attn_out = torch.empty((T, D), dtype=torch.float32, device=q.device)
    if y is None:
        y = torch.empty((T, D), dtype=q.dtype, device=q.device)
    if ln_mean is None:
        ln_mean = torch.empty(T, dtype=torch.float32, device=q.device)
    if ln_rstd is None:
        ln_rstd = torch.empty(T, dtype=torch.float32, device=q.device)
    if ws is None:
        ws = workspace(p, q.device)
    _check(lib.hstu_layer_fwd(ctypes.byref(p), ctypes.byref(j), _ptr(q), _row_stride(q), _ptr(k),
                              _row_stride(k), _ptr(v), _row_stride(v), _ptr(u), _row_stride(u),
                              _ptr(ln_weight), _ptr(ln_bias), float(ln_eps), _ptr(attn_out),
                              _ptr(y), _ptr(ln_mean), _ptr(ln_rstd), _ptr(ws), ws.numel(),
                              _stream(stream)))
    return attn_out, y, ln_mean, ln_rstd


def hstu_layer_bwd(q, k, v, u, attn_out, ln_mean, ln_rstd, d_y, seq_offsets, timestamps,
                   rab_pos, rab_time, max_seq_len, num_targets=None, ln_weight=None,
                   ln_bias=None, want_ln_grads=None, grads=None, ws=None, stream=None):
    """(dq, dk, dv, du, d_ln_weight, d_ln_bias, d_rab_pos, d_rab_time) for the
    loss <Y, d_y> of Eq. 2-3; attn_out, ln_mean, ln_rstd from hstu_layer_fwd.
    d_ln_weight / d_ln_bias are computed when want_ln_grads (default: when
    ln_weight is given), else None."""
    p = problem_for(q, v, seq_offsets, max_seq_len, rab_time)
    j = make_jagged(seq_offsets, timestamps, rab_pos, rab_time, num_targets)
    T, D = q.shape[0], q.shape[1] * v.shape[2]
    if want_ln_grads is None:
        want_ln_grads = ln_weight is not None
    if grads is None:
        H = q.shape[1]
        grads = (torch.empty((T, H, q.shape[2]), dtype=q.dtype, device=q.device),
                 torch.empty((T, H, k.shape[2]), dtype=q.dtype, device=q.device),
                 torch.empty((T, H, v.shape[2]), dtype=q.dtype, device=q.device),
                 torch.empty((T, D), dtype=q.dtype, device=q.device),
                 torch.empty(D, dtype=torch.float32, device=q.device) if want_ln_grads else None,
                 torch.empty(D, dtype=torch.float32, device=q.device) if want_ln_grads else None,
                 torch.empty_like(rab_pos), torch.empty_like(rab_time))
    dq, dk, dv, du, dw, db, drp, drt = grads
    if ws is None:
        ws = workspace(p, q.device)
    _check(lib.hstu_layer_bwd(ctypes.byref(p), ctypes.byref(j), _ptr(q), _row_stride(q), _ptr(k),
                              _row_stride(k), _ptr(v), _row_stride(v), _ptr(u), _row_stride(u),
                              _ptr(attn_out), _ptr(ln_weight), _ptr(ln_bias), _ptr(ln_mean),
                              _ptr(ln_rstd), _ptr(d_y), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(du),
                              _ptr(dw), _ptr(db), _ptr(drp), _ptr(drt), _ptr(ws), ws.numel(),
                              _stream(stream)))
    return grads


def hstu_complete_cumsum(x: torch.Tensor, out=None, stream=None):
    if out is None:
        out = torch.empty(x.numel() + 1, dtype=torch.int64, device=x.device)
    _check(lib.hstu_complete_cumsum(x.numel(), _ptr(x), _ptr(out), _stream(stream)))
    return out


def hstu_pair_offsets(seq_offsets: torch.Tensor, out=None, stream=None):
    if out is None:
        out = torch.empty_like(seq_offsets)
    _check(lib.hstu_pair_offsets(seq_offsets.numel() - 1, _ptr(seq_offsets), _ptr(out),
                                 _stream(stream)))
    return out


def hstu_time_bucketize(seq_offsets, timestamps, num_time_buckets, pair_offsets=None,
                        total_pairs=None, out=None, stream=None):
    """uint8 buckets, one L_b x L_b row-major matrix per sequence."""
    if pair_offsets is None:
        pair_offsets = hstu_pair_offsets(seq_offsets, stream=stream)
    if total_pairs is None:
        total_pairs = int(pair_offsets[-1].item())  # host read, synchronises
    if out is None:
        out = torch.empty(max(total_pairs, 1), dtype=torch.uint8, device=timestamps.device)
    _check(lib.hstu_time_bucketize(seq_offsets.numel() - 1, timestamps.numel(),
                                   int(num_time_buckets), _ptr(seq_offsets), _ptr(timestamps),
                                   _ptr(pair_offsets), int(total_pairs), _ptr(out),
                                   _stream(stream)))
    return out[:total_pairs]


def hstu_validate(seq_offsets, timestamps, rab_pos, rab_time, max_seq_len, num_heads, d_qk, d_v,
                  dtype=HSTU_BF16, num_targets=None, stream=None):
    p = make_problem(seq_offsets.numel() - 1, timestamps.numel(), max_seq_len, num_heads, d_qk,
                     d_v, rab_time.numel(), dtype)
    j = make_jagged(seq_offsets, timestamps, rab_pos, rab_time, num_targets)
    _check(lib.hstu_validate(ctypes.byref(p), ctypes.byref(j), _stream(stream)))


def hstu_timing_enable(on: bool = True):
    _check(lib.hstu_timing_enable(1 if on else 0))


def hstu_timing_reset():
    _check(lib.hstu_timing_reset())


# ------------------------------------------------ linear maps (Eq. 1, Eq. 3)

def proj_problem(x, num_heads, d_qk, d_v) -> Problem:
    """Problem of a projection call: only T, h, d_qk, d_v and the dtype
    matter (one placeholder sequence, N = 1, one time bucket)."""
    return make_problem(1, x.shape[0], 1, num_heads, d_qk, d_v, 1, _dtype_code(x))


def _row_stride2(t: torch.Tensor) -> int:
    if t.dim() == 2 and t.shape[0] == 0:
        return t.shape[1]
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a [T, width] tensor with contiguous rows")
    return t.stride(0)


def hstu_proj_workspace_bytes(p: Problem, d_model: int) -> int:
    return int(lib.hstu_proj_workspace_bytes(ctypes.byref(p), int(d_model)))


def proj_workspace(p: Problem, d_model: int, device=None) -> torch.Tensor:
    n = int(lib.hstu_proj_workspace_bytes(ctypes.byref(p), int(d_model)))
    if n == 0:
        raise HstuError(1, "invalid projection problem")
    return torch.empty(n, dtype=torch.uint8, device=device or "cuda")


def hstu_proj_in_fwd(x, w1, b1, num_heads, d_qk, d_v, z=None, z_pre=None, want_pre=True,
                     stream=None):
    """Eq. 1: returns (z, z_pre), z [T, F] = SiLU(x w1^T + b1) laid out U|V|Q|K."""
    p = proj_problem(x, num_heads, d_qk, d_v)
    F = 2 * num_heads * (d_qk + d_v)
    if z is None:
        z = torch.empty((x.shape[0], F), dtype=x.dtype, device=x.device)
    if z_pre is None and want_pre:
        z_pre = torch.empty_like(z)
    _check(lib.hstu_proj_in_fwd(ctypes.byref(p), int(x.shape[1]), _ptr(x), _row_stride2(x),
                                _ptr(w1), _ptr(b1), _ptr(z), _ptr(z_pre), _stream(stream)))
    return z, z_pre


def split_uvqk(z, num_heads, d_qk, d_v):
    """[T, h, d] views U, V, Q, K of z [T, F] (row stride F)."""
    T = z.shape[0]
    hv, hq = num_heads * d_v, num_heads * d_qk
    F = z.shape[1]

    def view(c0, d):
        return z.as_strided((T, num_heads, d), (F, d, 1), z.storage_offset() + c0)
    return view(0, d_v), view(hv, d_v), view(2 * hv, d_qk), view(2 * hv + hq, d_qk)


def hstu_proj_out_fwd(g, w2, b2, residual, num_heads, d_qk, d_v, y=None, stream=None):
    """Eq. 3's f_2 plus the residual: y [T, D] = g w2^T + b2 + residual."""
    p = proj_problem(g, num_heads, d_qk, d_v)
    D = w2.shape[0]
    if y is None:
        y = torch.empty((g.shape[0], D), dtype=g.dtype, device=g.device)
    _check(lib.hstu_proj_out_fwd(ctypes.byref(p), int(D), _ptr(g), _row_stride2(g), _ptr(w2),
                                 _ptr(b2), _ptr(residual), _ptr(y), _stream(stream)))
    return y


def hstu_proj_out_bwd(g, w2, dy, num_heads, d_qk, d_v, want_db=True, out=None, ws=None,
                      stream=None):
    """Returns (dg, dw2, db2) for the loss <y, dy>."""
    p = proj_problem(g, num_heads, d_qk, d_v)
    D, hv = w2.shape
    if out is None:
        out = (torch.empty((g.shape[0], hv), dtype=g.dtype, device=g.device),
               torch.empty((D, hv), dtype=torch.float32, device=g.device),
               torch.empty(D, dtype=torch.float32, device=g.device) if want_db else None)
    dg, dw2, db2 = out
    if ws is None:
        ws = proj_workspace(p, D, g.device)
    _check(lib.hstu_proj_out_bwd(ctypes.byref(p), int(D), _ptr(g), _row_stride2(g), _ptr(w2),
                                 _ptr(dy), _ptr(dg), _ptr(dw2), _ptr(db2), _ptr(ws), ws.numel(),
                                 _stream(stream)))
    return dg, dw2, db2


def hstu_proj_in_bwd(x, w1, z_pre, du, dv, dq, dk, num_heads, d_qk, d_v, dx_add=None,
                     want_db=True, out=None, ws=None, stream=None):
    """Returns (dx, dw1, db1) for the loss <z, [du|dv|dq|dk]>."""
    p = proj_problem(x, num_heads, d_qk, d_v)
    F, D = w1.shape
    if out is None:
        out = (torch.empty_like(x, memory_format=torch.contiguous_format),
               torch.empty((F, D), dtype=torch.float32, device=x.device),
               torch.empty(F, dtype=torch.float32, device=x.device) if want_db else None)
    dx, dw1, db1 = out
    if ws is None:
        ws = proj_workspace(p, D, x.device)
    _check(lib.hstu_proj_in_bwd(ctypes.byref(p), int(D), _ptr(x), _row_stride2(x), _ptr(w1),
                                _ptr(z_pre), _ptr(du), _ptr(dv), _ptr(dq), _ptr(dk),
                                _ptr(dx_add), _ptr(dx), _ptr(dw1), _ptr(db1), _ptr(ws),
                                ws.numel(), _stream(stream)))
    return dx, dw1, db1


# ------------------------------------------------ Stochastic Length (Eq. 4)

HSTU_SL_GREEDY, HSTU_SL_RANDOM, HSTU_SL_WEIGHTED = 0, 1, 2


def hstu_sl_subseq_len(max_seq_len: int, alpha: float) -> int:
    return int(lib.hstu_sl_subseq_len(int(max_seq_len), float(alpha)))


def hstu_sl_keep_numerator(max_seq_len: int, alpha: float) -> float:
    return float(lib.hstu_sl_keep_numerator(int(max_seq_len), float(alpha)))


def hstu_sl_workspace_bytes(num_seqs: int) -> int:
    return int(lib.hstu_sl_workspace_bytes(int(num_seqs)))


def hstu_stochastic_length(seq_offsets, timestamps, subseq_len, keep_numerator, selection, u_keep,
                           e_rand=None, num_targets=None, out=None, ws=None, stream=None):
    """(new_offsets [B+1], gather [T]) on the device; the first
    new_offsets[B] entries of gather are valid (see include/hstu.h)."""
    B = seq_offsets.numel() - 1
    T = timestamps.numel()
    if out is None:
        out = (torch.empty(B + 1, dtype=torch.int64, device=seq_offsets.device),
               torch.empty(max(T, 1), dtype=torch.int64, device=seq_offsets.device))
    new_offsets, gather = out
    if ws is None:
        ws = torch.empty(int(lib.hstu_sl_workspace_bytes(B)), dtype=torch.uint8,
                         device=seq_offsets.device)
    _check(lib.hstu_stochastic_length(B, _ptr(seq_offsets), _ptr(timestamps), _ptr(num_targets),
                                      int(subseq_len), float(keep_numerator), int(selection),
                                      _ptr(u_keep), _ptr(e_rand),
                                      _ptr(new_offsets), _ptr(gather), _ptr(ws), ws.numel(),
                                      _stream(stream)))
    return new_offsets, gather


def hstu_gather_rows(src, gather, count, max_rows=None, dst=None, stream=None):
    """dst[r] = src[gather[r]] for r < count[0] (a one-element device tensor,
    e.g. new_offsets[-1:]); src rows are its first dimension."""
    rows = src.shape[0]
    row_elems = src[0].numel() if rows else int(np.prod(src.shape[1:]))
    if max_rows is None:
        max_rows = gather.numel()
    if dst is None:
        dst = torch.empty((max_rows,) + tuple(src.shape[1:]), dtype=src.dtype, device=src.device)
    es = src.element_size()
    _check(lib.hstu_gather_rows(_ptr(src), src.stride(0) * es, row_elems * es, _ptr(gather),
                                _ptr(count), int(max_rows), _ptr(dst), dst.stride(0) * es,
                                _stream(stream)))
    return dst


def hstu_sl_sparsity(seq_offsets_host, max_seq_len):
    """(sparsity, s2) of a batch from host int64 offsets."""
    offs = np.ascontiguousarray(seq_offsets_host, dtype=np.int64)
    sp, s2 = ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(lib.hstu_sl_sparsity(len(offs) - 1, offs.ctypes.data_as(ctypes.c_void_p),
                                int(max_seq_len), ctypes.byref(sp), ctypes.byref(s2)))
    return sp.value, s2.value


def hstu_probe_mfma_bf16(iters: int, waves_per_simd: int, sink: torch.Tensor, stream=None):
    """Launches the matrix-core rate probe; returns its flop count."""
    flop = ctypes.c_double(0.0)
    _check(lib.hstu_probe_mfma_bf16(int(iters), int(waves_per_simd), _ptr(sink),
                                    ctypes.byref(flop), _stream(stream)))
    return flop.value


def hstu_timing_read(name: str):
    ms = ctypes.c_double(0.0)
    n = ctypes.c_int64(0)
    _check(lib.hstu_timing_read(name.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
