"""CoWindow Attention (CoWA) on AMD MI355X.

Python binding of ``libcowa.so`` (C ABI in ``include/cowa.h``).  Every step of
the method runs in the library's HIP kernels; this module only marshals
arguments, and uses torch for device memory and streams.  There is no CPU or
eager fallback: if the library is missing, every call raises.

Entry points with the names of the C ABI live in ``paper_2609_32704_amd._abi``;
the helpers below wrap them for torch tensors:

* ``make_params`` / ``make_decode_params`` -- fill the ABI structs
* ``Schedule``  -- sizes, allocates and builds the block schedule (cowa_schedule)
* ``fwd`` / ``fwd_varlen`` -- cowa_fwd: O and LSE (fixed lengths / ragged batch)
* ``bwd`` / ``bwd_varlen`` -- cowa_bwd: dQ, dK, dV
* ``decode``    -- cowa_decode: one decoding step over a KV cache
* ``attention`` / ``attention_varlen`` -- differentiable attention
                   (torch.autograd.Function over cowa_fwd and cowa_bwd)

Windows: by default every call uses the paper's default rule (shared sink and
near windows, complementary long-range windows from the global KV-head index).
``windows=[(sink, near, gap, width), ...]`` (one tuple per local KV head)
gives explicit per-head windows instead (Sec. 2.1 four-tuple interface).

Ragged batches (``*_varlen``): tensors are packed head-major, Q [H_q, N_q, d]
and K, V [H_k, N_k, d], sequence b owning rows cu_seqlens[b] .. cu_seqlens[b+1]
with its queries aligned to the end of its keys.
"""

import math

from . import _abi
from ._abi import (CowaError, COWA_BF16, COWA_FP32, cowa_version, cowa_last_error, cowa_windows,  # noqa: F401
                   cowa_schedule_size)

__all__ = ["CowaError", "make_params", "make_decode_params", "Schedule", "fwd", "bwd", "fwd_varlen", "bwd_varlen",
           "decode", "windows", "attention", "attention_varlen", "cowa_version"]


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


def _host_ints(x, name):
    """A list of Python ints from a list, tuple, numpy array or torch tensor
    (a device tensor is copied to the host)."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().tolist()
    except ImportError:
        pass
    vals = [int(v) for v in (x.tolist() if hasattr(x, "tolist") else x)]
    if not vals:
        raise ValueError(f"{name} must have at least one entry")
    return vals


def make_params(batch, n_q, n_k, h_q, h_k, head_dim, w_sink, w_near, tile_q, tile_k, softmax_scale=None,
                dtype=COWA_BF16, h_k_total=None, h_k_offset=0, windows=None, cu_seqlens_q=None, cu_seqlens_k=None):
    """cowa_params.  windows: None or h_k tuples (sink, near, gap, width).
    cu_seqlens_q/k: None (fixed lengths) or batch + 1 cumulative lengths of a
    ragged batch, whose n_q/n_k are then the packed totals."""
    p = _abi.cowa_params()
    p.batch, p.n_q, p.n_k, p.h_q, p.h_k, p.head_dim = batch, n_q, n_k, h_q, h_k, head_dim
    p.w_sink, p.w_near = w_sink, w_near
    p.h_k_total = h_k if h_k_total is None else h_k_total
    p.h_k_offset = h_k_offset
    p.tile_q, p.tile_k = tile_q, tile_k
    p.softmax_scale = 1.0 / math.sqrt(head_dim) if softmax_scale is None else softmax_scale
    p.dtype = dtype
    keep = []
    if windows is not None:
        if len(windows) != h_k:
            raise ValueError(f"windows has {len(windows)} tuples, expected one per local KV head ({h_k})")
        arr = _abi.window_array(windows)
        keep.append(arr)
        p.windows = arr
    if (cu_seqlens_q is None) != (cu_seqlens_k is None):
        raise ValueError("cu_seqlens_q and cu_seqlens_k must both be given or both be None")
    if cu_seqlens_q is not None:
        cq, ck = _host_ints(cu_seqlens_q, "cu_seqlens_q"), _host_ints(cu_seqlens_k, "cu_seqlens_k")
        if len(cq) != batch + 1 or len(ck) != batch + 1:
            raise ValueError(f"cu_seqlens must have batch + 1 = {batch + 1} entries")
        aq, ak = _abi.int32_array(cq), _abi.int32_array(ck)
        keep += [aq, ak]
        p.cu_seqlens_q, p.cu_seqlens_k = aq, ak
    p._keep = keep
    return p


def make_decode_params(batch, h_q, h_k, head_dim, n_max, w_sink, w_near, softmax_scale=None, h_k_total=None,
                       h_k_offset=0, split_keys=0, dtype=COWA_BF16, windows=None):
    p = _abi.cowa_decode_params()
    p.batch, p.h_q, p.h_k, p.head_dim, p.n_max = batch, h_q, h_k, head_dim, n_max
    p.w_sink, p.w_near = w_sink, w_near
    p.h_k_total = h_k if h_k_total is None else h_k_total
    p.h_k_offset = h_k_offset
    p.split_keys = split_keys
    p.softmax_scale = 1.0 / math.sqrt(head_dim) if softmax_scale is None else softmax_scale
    p.dtype = dtype
    p._keep = []
    if windows is not None:
        if len(windows) != h_k:
            raise ValueError(f"windows has {len(windows)} tuples, expected one per local KV head ({h_k})")
        arr = _abi.window_array(windows)
        p._keep.append(arr)
        p.windows = arr
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
        self.params = params  # its host arrays back the pointer fields of self.s.p
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


def _validate(specs):
    """specs: (tensor, name, dtype, shape) per tensor; None tensors are skipped.
    Raise ValueError unless every tensor is a contiguous torch tensor of its
    dtype and exact shape (all of them checked first), and then unless all of
    them are on the GPU of the first.  Every check runs before anything is
    passed to the library, whose kernels index every buffer by the shapes
    taken from q and k."""
    torch = _torch()
    specs = [sp for sp in specs if sp[0] is not None]
    for t, name, dtype, shape in specs:
        if not isinstance(t, torch.Tensor):
            raise ValueError(f"{name} must be a torch.Tensor")
        if t.dtype != dtype:
            raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
    dev = specs[0][0].device
    for t, name, _, _ in specs:
        if not t.is_cuda:
            raise ValueError(f"{name} must be a device tensor")
        if t.device != dev:
            raise ValueError(f"{name} is on {t.device}, expected {dev}")


def _dims(q, k, name_q="q", name_k="k"):
    """(B, H_q, N_q, d, H_k, N_k) from q [B,H_q,N_q,d] and k [B,H_k,N_k,d]."""
    torch = _torch()
    for t, n in ((q, name_q), (k, name_k)):
        if not isinstance(t, torch.Tensor) or t.dim() != 4:
            raise ValueError(f"{n} must be a 4-d tensor [B, H, N, d]")
    bsz, h_q, n_q, d = q.shape
    if k.shape[0] != bsz or k.shape[3] != d:
        raise ValueError(f"{name_k} has shape {tuple(k.shape)}; expected [B={bsz}, H_k, N_k, d={d}]")
    return bsz, h_q, n_q, d, k.shape[1], k.shape[2]


def _dims_varlen(q, k, cu_seqlens_q, cu_seqlens_k):
    """(B, H_q, N_q, d, H_k, N_k) of packed q [H_q,N_q,d], k [H_k,N_k,d] and
    the host cumulative lengths."""
    torch = _torch()
    for t, n in ((q, "q"), (k, "k")):
        if not isinstance(t, torch.Tensor) or t.dim() != 3:
            raise ValueError(f"{n} must be a 3-d packed tensor [H, N_total, d]")
    h_q, n_q, d = q.shape
    h_k, n_k = k.shape[0], k.shape[1]
    if k.shape[2] != d:
        raise ValueError(f"k has shape {tuple(k.shape)}; expected [H_k, N_k, d={d}]")
    cq, ck = _host_ints(cu_seqlens_q, "cu_seqlens_q"), _host_ints(cu_seqlens_k, "cu_seqlens_k")
    if len(cq) != len(ck):
        raise ValueError("cu_seqlens_q and cu_seqlens_k must have the same length")
    if cq[-1] != n_q or ck[-1] != n_k:
        raise ValueError(f"cu_seqlens end at ({cq[-1]}, {ck[-1]}) but q and k hold ({n_q}, {n_k}) rows")
    return len(cq) - 1, h_q, n_q, d, h_k, n_k, cq, ck


def _fwd(p, q, k, v, qs, ks, ls, schedule, out, lse, stream):
    torch = _torch()
    _validate([(q, "q", q.dtype, qs), (k, "k", q.dtype, ks), (v, "v", q.dtype, ks), (out, "out", q.dtype, qs),
               (lse, "lse", torch.float32, ls)])
    if schedule is None:
        schedule = Schedule(p, q.device, stream)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty(ls, dtype=torch.float32, device=q.device)
    _abi.cowa_fwd(p, schedule.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                  _stream(stream))
    return out, lse


def fwd(q, k, v, w_sink, w_near, tile_q, tile_k, softmax_scale=None, h_k_total=None, h_k_offset=0, schedule=None,
        out=None, lse=None, stream=None, windows=None):
    """cowa_fwd.  q [B,H_q,N_q,d], k/v [B,H_k,N_k,d] (bf16 or fp32, contiguous).
    Returns (o, lse).  ``schedule`` may be a prebuilt Schedule for these shapes."""
    bsz, h_q, n_q, d, h_k, n_k = _dims(q, k)
    p = make_params(bsz, n_q, n_k, h_q, h_k, d, w_sink, w_near, tile_q, tile_k, softmax_scale,
                    _dtype_code(q.dtype), h_k_total, h_k_offset, windows)
    return _fwd(p, q, k, v, (bsz, h_q, n_q, d), (bsz, h_k, n_k, d), (bsz, h_q, n_q), schedule, out, lse, stream)


def fwd_varlen(q, k, v, cu_seqlens_q, cu_seqlens_k, w_sink, w_near, tile_q, tile_k, softmax_scale=None,
               h_k_total=None, h_k_offset=0, schedule=None, out=None, lse=None, stream=None, windows=None):
    """cowa_fwd on a ragged batch.  q [H_q,N_q,d], k/v [H_k,N_k,d] packed;
    cu_seqlens_* hold batch + 1 cumulative lengths.  Returns (o, lse [H_q,N_q])."""
    bsz, h_q, n_q, d, h_k, n_k, cq, ck = _dims_varlen(q, k, cu_seqlens_q, cu_seqlens_k)
    p = make_params(bsz, n_q, n_k, h_q, h_k, d, w_sink, w_near, tile_q, tile_k, softmax_scale,
                    _dtype_code(q.dtype), h_k_total, h_k_offset, windows, cq, ck)
    return _fwd(p, q, k, v, (h_q, n_q, d), (h_k, n_k, d), (h_q, n_q), schedule, out, lse, stream)


def _bwd(p, q, k, v, o, lse, do, qs, ks, ls, schedule, workspace, dq, dk, dv, stream):
    torch = _torch()
    _validate([(q, "q", q.dtype, qs), (k, "k", q.dtype, ks), (v, "v", q.dtype, ks), (o, "o", q.dtype, qs),
               (do, "do", q.dtype, qs), (lse, "lse", torch.float32, ls), (dq, "dq", q.dtype, qs),
               (dk, "dk", q.dtype, ks), (dv, "dv", q.dtype, ks),
               (workspace, "workspace", torch.uint8, (None if workspace is None else workspace.numel(),))])
    need = _abi.cowa_bwd_workspace_size(p)
    if workspace is not None and workspace.numel() < need:
        raise ValueError(f"workspace has {workspace.numel()} bytes, the backward needs {need}")
    if schedule is None:
        schedule = Schedule(p, q.device, stream)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    _abi.cowa_bwd(p, schedule.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                  do.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), workspace.data_ptr(),
                  workspace.numel(), _stream(stream))
    return dq, dk, dv


def bwd(q, k, v, o, lse, do, w_sink, w_near, tile_q, tile_k, softmax_scale=None, h_k_total=None, h_k_offset=0,
        schedule=None, workspace=None, dq=None, dk=None, dv=None, stream=None, windows=None):
    """cowa_bwd.  Returns (dq, dk, dv) for bf16 inputs."""
    bsz, h_q, n_q, d, h_k, n_k = _dims(q, k)
    p = make_params(bsz, n_q, n_k, h_q, h_k, d, w_sink, w_near, tile_q, tile_k, softmax_scale,
                    _dtype_code(q.dtype), h_k_total, h_k_offset, windows)
    return _bwd(p, q, k, v, o, lse, do, (bsz, h_q, n_q, d), (bsz, h_k, n_k, d), (bsz, h_q, n_q), schedule,
                workspace, dq, dk, dv, stream)


def bwd_varlen(q, k, v, o, lse, do, cu_seqlens_q, cu_seqlens_k, w_sink, w_near, tile_q, tile_k,
               softmax_scale=None, h_k_total=None, h_k_offset=0, schedule=None, workspace=None, dq=None, dk=None,
               dv=None, stream=None, windows=None):
    """cowa_bwd on a ragged batch (packed tensors as in fwd_varlen)."""
    bsz, h_q, n_q, d, h_k, n_k, cq, ck = _dims_varlen(q, k, cu_seqlens_q, cu_seqlens_k)
    p = make_params(bsz, n_q, n_k, h_q, h_k, d, w_sink, w_near, tile_q, tile_k, softmax_scale,
                    _dtype_code(q.dtype), h_k_total, h_k_offset, windows, cq, ck)
    return _bwd(p, q, k, v, o, lse, do, (h_q, n_q, d), (h_k, n_k, d), (h_q, n_q), schedule, workspace, dq, dk, dv,
                stream)


def decode(q, k_cache, v_cache, seqlens_k, w_sink, w_near, softmax_scale=None, h_k_total=None, h_k_offset=0,
           split_keys=0, workspace=None, out=None, lse=None, stream=None, windows=None):
    """cowa_decode.  q [B,H_q,d], caches [B,H_k,n_max,d] bf16, seqlens_k int32 [B]
    on the device.  Returns (o [B,H_q,d], lse [B,H_q])."""
    torch = _torch()
    if not isinstance(q, torch.Tensor) or q.dim() != 3:
        raise ValueError("q must be a 3-d tensor [B, H_q, d]")
    if not isinstance(k_cache, torch.Tensor) or k_cache.dim() != 4:
        raise ValueError("k_cache must be a 4-d tensor [B, H_k, n_max, d]")
    bsz, h_q, d = q.shape
    h_k, n_max = k_cache.shape[1], k_cache.shape[2]
    cs = (bsz, h_k, n_max, d)
    _validate([(q, "q", q.dtype, (bsz, h_q, d)), (k_cache, "k_cache", q.dtype, cs), (v_cache, "v_cache", q.dtype, cs),
               (seqlens_k, "seqlens_k", torch.int32, (bsz,)), (out, "out", q.dtype, (bsz, h_q, d)),
               (lse, "lse", torch.float32, (bsz, h_q)),
               (workspace, "workspace", torch.uint8, (None if workspace is None else workspace.numel(),))])
    p = make_decode_params(bsz, h_q, h_k, d, n_max, w_sink, w_near, softmax_scale, h_k_total, h_k_offset,
                           split_keys, _dtype_code(q.dtype), windows)
    need = _abi.cowa_decode_workspace_size(p)
    if workspace is not None and workspace.numel() < need:
        raise ValueError(f"workspace has {workspace.numel()} bytes, decoding needs {need}")
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((bsz, h_q), dtype=torch.float32, device=q.device)
    _abi.cowa_decode(p, q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), seqlens_k.data_ptr(), out.data_ptr(),
                     lse.data_ptr(), workspace.data_ptr(), workspace.numel(), _stream(stream))
    return out, lse


class _Attention:
    """torch.autograd.Function around cowa_fwd / cowa_bwd (built lazily so that
    importing the package does not import torch).  The function takes the
    tensors and one ``cfg`` tuple: (w_sink, w_near, tile_q, tile_k,
    softmax_scale, h_k_total, h_k_offset, windows, cu_seqlens_q, cu_seqlens_k),
    the last two None for fixed lengths."""
    fn = None

    @classmethod
    def get(cls):
        if cls.fn is None:
            torch = _torch()

            class CowaAttentionFn(torch.autograd.Function):
                @staticmethod
                def forward(ctx, q, k, v, cfg):
                    q, k, v = q.contiguous(), k.contiguous(), v.contiguous()
                    w_sink, w_near, tq, tk, scale, h_tot, h_off, wins, cq, ck = cfg
                    if cq is None:
                        sched_p = make_params(q.shape[0], q.shape[2], k.shape[2], q.shape[1], k.shape[1], q.shape[3],
                                              w_sink, w_near, tq, tk, scale, _dtype_code(q.dtype), h_tot, h_off, wins)
                        sched = Schedule(sched_p, q.device)
                        o, lse = fwd(q, k, v, w_sink, w_near, tq, tk, scale, h_tot, h_off, schedule=sched,
                                     windows=wins)
                    else:
                        sched_p = make_params(len(cq) - 1, q.shape[1], k.shape[1], q.shape[0], k.shape[0],
                                              q.shape[2], w_sink, w_near, tq, tk, scale, _dtype_code(q.dtype), h_tot,
                                              h_off, wins, cq, ck)
                        sched = Schedule(sched_p, q.device)
                        o, lse = fwd_varlen(q, k, v, cq, ck, w_sink, w_near, tq, tk, scale, h_tot, h_off,
                                            schedule=sched, windows=wins)
                    ctx.save_for_backward(q, k, v, o, lse)
                    ctx.mark_non_differentiable(lse)
                    ctx.set_materialize_grads(False)
                    ctx.cfg = cfg
                    ctx.sched = sched
                    return o, lse

                @staticmethod
                def backward(ctx, d_o, d_lse):
                    q, k, v, o, lse = ctx.saved_tensors
                    if d_o is None:
                        return None, None, None, None
                    w_sink, w_near, tq, tk, scale, h_tot, h_off, wins, cq, ck = ctx.cfg
                    if cq is None:
                        dq, dk, dv = bwd(q, k, v, o, lse, d_o.contiguous(), w_sink, w_near, tq, tk, scale, h_tot,
                                         h_off, schedule=ctx.sched, windows=wins)
                    else:
                        dq, dk, dv = bwd_varlen(q, k, v, o, lse, d_o.contiguous(), cq, ck, w_sink, w_near, tq, tk,
                                                scale, h_tot, h_off, schedule=ctx.sched, windows=wins)
                    return dq, dk, dv, None

            cls.fn = CowaAttentionFn
        return cls.fn


def attention(q, k, v, w_sink, w_near, tile_q=128, tile_k=128, softmax_scale=None, h_k_total=None, h_k_offset=0,
              return_lse=False, windows=None):
    """Differentiable CoWA attention (torch autograd): the forward runs cowa_fwd
    and saves O and LSE; the backward runs cowa_bwd (deterministic: the same
    inputs give bitwise the same gradients).  q [B,H_q,N_q,d], k/v
    [B,H_k,N_k,d], bf16 for the backward.  Returns O (and LSE, treated as a
    non-differentiable output, if return_lse)."""
    cfg = (w_sink, w_near, tile_q, tile_k, softmax_scale, h_k_total, h_k_offset,
           None if windows is None else [tuple(w) for w in windows], None, None)
    o, lse = _Attention.get().apply(q, k, v, cfg)
    return (o, lse) if return_lse else o


def attention_varlen(q, k, v, cu_seqlens_q, cu_seqlens_k, w_sink, w_near, tile_q=128, tile_k=128,
                     softmax_scale=None, h_k_total=None, h_k_offset=0, return_lse=False, windows=None):
    """attention() on a ragged batch: q [H_q,N_q,d], k/v [H_k,N_k,d] packed,
    cu_seqlens_* with batch + 1 cumulative lengths."""
    cfg = (w_sink, w_near, tile_q, tile_k, softmax_scale, h_k_total, h_k_offset,
           None if windows is None else [tuple(w) for w in windows],
           _host_ints(cu_seqlens_q, "cu_seqlens_q"), _host_ints(cu_seqlens_k, "cu_seqlens_k"))
    o, lse = _Attention.get().apply(q, k, v, cfg)
    return (o, lse) if return_lse else o
