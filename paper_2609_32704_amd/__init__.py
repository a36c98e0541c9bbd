"""CoWindow Attention (CoWA) on AMD MI355X.

Python binding of ``libcowa.so`` (C ABI in ``include/cowa.h``).  Every step of
the method runs in the library's HIP kernels; this module only marshals
arguments, and uses torch for device memory and streams.  There is no CPU or
eager fallback: if the library is missing, every call raises.

Entry points with the names of the C ABI live in ``paper_2609_32704_amd._abi``;
the helpers below wrap them for torch tensors:

* ``make_params`` / ``make_decode_params`` -- fill the ABI structs
* ``Schedule``  -- sizes, allocates and builds the block schedule (cowa_schedule)
* ``fwd``       -- cowa_fwd: O and LSE
* ``bwd``       -- cowa_bwd: dQ, dK, dV
* ``decode``    -- cowa_decode: one decoding step over a KV cache
"""

import math

from . import _abi
from ._abi import (CowaError, COWA_BF16, COWA_FP32, cowa_version, cowa_last_error, cowa_windows,  # noqa: F401
                   cowa_schedule_size)

__all__ = ["CowaError", "make_params", "make_decode_params", "Schedule", "fwd", "bwd", "decode", "windows",
           "cowa_version"]


def _torch():
    import torch
    return torch


def _dtype_code(dtype):
    torch = _torch()
    if dtype == torch.bfloat16:
        return COWA_BF16
    if dtype == torch.float32:
        return COWA_FP32
    raise ValueError(f"unsupported dtype {dtype}; use torch.bfloat16 or torch.float32")


def make_params(batch, n_q, n_k, h_q, h_k, head_dim, w_sink, w_near, tile_q, tile_k, softmax_scale=None,
                dtype=COWA_BF16, h_k_total=None, h_k_offset=0):
    p = _abi.cowa_params()
    p.batch, p.n_q, p.n_k, p.h_q, p.h_k, p.head_dim = batch, n_q, n_k, h_q, h_k, head_dim
    p.w_sink, p.w_near = w_sink, w_near
    p.h_k_total = h_k if h_k_total is None else h_k_total
    p.h_k_offset = h_k_offset
    p.tile_q, p.tile_k = tile_q, tile_k
    p.softmax_scale = 1.0 / math.sqrt(head_dim) if softmax_scale is None else softmax_scale
    p.dtype = dtype
    return p


def make_decode_params(batch, h_q, h_k, head_dim, n_max, w_sink, w_near, softmax_scale=None, h_k_total=None,
                       h_k_offset=0, split_keys=0, dtype=COWA_BF16):
    p = _abi.cowa_decode_params()
    p.batch, p.h_q, p.h_k, p.head_dim, p.n_max = batch, h_q, h_k, head_dim, n_max
    p.w_sink, p.w_near = w_sink, w_near
    p.h_k_total = h_k if h_k_total is None else h_k_total
    p.h_k_offset = h_k_offset
    p.split_keys = split_keys
    p.softmax_scale = 1.0 / math.sqrt(head_dim) if softmax_scale is None else softmax_scale
    p.dtype = dtype
    return p


def windows(params):
    """cowa_windows: the (sink, near, gap, width) tuple of every local KV head."""
    return cowa_windows(params)


def _stream(stream):
    torch = _torch()
    return torch.cuda.current_stream().cuda_stream if stream is None else stream


class Schedule:
    """A block schedule on the current device: sized on the host
    (cowa_schedule_size), its buffer allocated through torch, built on the
    device (cowa_schedule)."""

    def __init__(self, params, device="cuda", stream=None, build=True):
        torch = _torch()
        self.s = cowa_schedule_size(params)
        self.buf = torch.empty(max(int(self.s.bytes), 256), dtype=torch.uint8, device=device)
        self.s.buf = self.buf.data_ptr()
        if build:
            _abi.cowa_schedule(self.s, _stream(stream))

    @property
    def nnz(self):
        return int(self.s.nnz)

    def arrays(self):
        """Views of the four schedule arrays (int32 / uint32 as int32 bits)."""
        torch = _torch()
        s = self.s
        rows_f = s.p.h_k * s.n_qt + 1
        rows_b = s.p.h_k * s.n_kt + 1

        def view(off, n):
            return self.buf[off:off + 4 * n].view(torch.int32)
        return {"fwd_row_ptr": view(s.off_fwd_row_ptr, rows_f), "bwd_col_ptr": view(s.off_bwd_col_ptr, rows_b),
                "fwd_ent": view(s.off_fwd_ent, s.nnz), "bwd_ent": view(s.off_bwd_ent, s.nnz)}


def _check(t, name, dtype, ndim):
    torch = _torch()
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if t.dim() != ndim or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {ndim}-d tensor")


def fwd(q, k, v, w_sink, w_near, tile_q, tile_k, softmax_scale=None, h_k_total=None, h_k_offset=0, schedule=None,
        out=None, lse=None, stream=None):
    """cowa_fwd.  q [B,H_q,N_q,d], k/v [B,H_k,N_k,d] (bf16 or fp32, contiguous).
    Returns (o, lse).  ``schedule`` may be a prebuilt Schedule for these shapes."""
    torch = _torch()
    _check(q, "q", q.dtype, 4)
    _check(k, "k", q.dtype, 4)
    _check(v, "v", q.dtype, 4)
    bsz, h_q, n_q, d = q.shape
    h_k, n_k = k.shape[1], k.shape[2]
    if k.shape != v.shape or k.shape[0] != bsz or k.shape[3] != d:
        raise ValueError("k and v must be [B, H_k, N_k, d] matching q")
    p = make_params(bsz, n_q, n_k, h_q, h_k, d, w_sink, w_near, tile_q, tile_k, softmax_scale,
                    _dtype_code(q.dtype), h_k_total, h_k_offset)
    if schedule is None:
        schedule = Schedule(p, q.device, stream)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((bsz, h_q, n_q), dtype=torch.float32, device=q.device)
    _check(out, "out", q.dtype, 4)
    _check(lse, "lse", torch.float32, 3)
    _abi.cowa_fwd(p, schedule.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                  _stream(stream))
    return out, lse


def bwd(q, k, v, o, lse, do, w_sink, w_near, tile_q, tile_k, softmax_scale=None, h_k_total=None, h_k_offset=0,
        schedule=None, workspace=None, dq=None, dk=None, dv=None, stream=None):
    """cowa_bwd.  Returns (dq, dk, dv) for bf16 inputs."""
    torch = _torch()
    for t, n in ((q, "q"), (o, "o"), (do, "do")):
        _check(t, n, q.dtype, 4)
    _check(k, "k", q.dtype, 4)
    _check(v, "v", q.dtype, 4)
    _check(lse, "lse", torch.float32, 3)
    bsz, h_q, n_q, d = q.shape
    h_k, n_k = k.shape[1], k.shape[2]
    p = make_params(bsz, n_q, n_k, h_q, h_k, d, w_sink, w_near, tile_q, tile_k, softmax_scale,
                    _dtype_code(q.dtype), h_k_total, h_k_offset)
    if schedule is None:
        schedule = Schedule(p, q.device, stream)
    need = _abi.cowa_bwd_workspace_size(p)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    _check(dq, "dq", q.dtype, 4)
    _check(dk, "dk", q.dtype, 4)
    _check(dv, "dv", q.dtype, 4)
    _abi.cowa_bwd(p, schedule.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                  do.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), workspace.data_ptr(),
                  workspace.numel(), _stream(stream))
    return dq, dk, dv


def decode(q, k_cache, v_cache, seqlens_k, w_sink, w_near, softmax_scale=None, h_k_total=None, h_k_offset=0,
           split_keys=0, workspace=None, out=None, lse=None, stream=None):
    """cowa_decode.  q [B,H_q,d], caches [B,H_k,n_max,d] bf16, seqlens_k int32 [B]
    on the device.  Returns (o [B,H_q,d], lse [B,H_q])."""
    torch = _torch()
    _check(q, "q", q.dtype, 3)
    _check(k_cache, "k_cache", q.dtype, 4)
    _check(v_cache, "v_cache", q.dtype, 4)
    _check(seqlens_k, "seqlens_k", torch.int32, 1)
    bsz, h_q, d = q.shape
    h_k, n_max = k_cache.shape[1], k_cache.shape[2]
    p = make_decode_params(bsz, h_q, h_k, d, n_max, w_sink, w_near, softmax_scale, h_k_total, h_k_offset,
                           split_keys, _dtype_code(q.dtype))
    need = _abi.cowa_decode_workspace_size(p)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((bsz, h_q), dtype=torch.float32, device=q.device)
    _abi.cowa_decode(p, q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), seqlens_k.data_ptr(), out.data_ptr(),
                     lse.data_ptr(), workspace.data_ptr(), workspace.numel(), _stream(stream))
    return out, lse
