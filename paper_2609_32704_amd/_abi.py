"""ctypes declarations of the C ABI in include/cowa.h (argument marshalling only).

Every function here has the name of the C entry point it calls.  Device
pointers are passed as integers (``tensor.data_ptr()``), streams as the integer
handle of a HIP stream (``torch.cuda.current_stream().cuda_stream``).
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcowa.so")

COWA_OK = 0
COWA_ERR_INVALID_ARG = -1
COWA_ERR_UNSUPPORTED = -2
COWA_ERR_WORKSPACE = -3
COWA_ERR_SCHEDULE_MISMATCH = -4
COWA_ERR_NO_DEVICE = -5
COWA_ERR_HIP = -6
STATUS_NAMES = {0: "COWA_OK", -1: "COWA_ERR_INVALID_ARG", -2: "COWA_ERR_UNSUPPORTED", -3: "COWA_ERR_WORKSPACE",
                -4: "COWA_ERR_SCHEDULE_MISMATCH", -5: "COWA_ERR_NO_DEVICE", -6: "COWA_ERR_HIP"}

COWA_BF16 = 0
COWA_FP32 = 1


class cowa_window(ctypes.Structure):
    _fields_ = [("sink", ctypes.c_int32), ("near", ctypes.c_int32), ("gap", ctypes.c_int32),
                ("width", ctypes.c_int32)]


class cowa_params(ctypes.Structure):
    """The C struct.  The pointer fields reference host arrays that the
    Python object keeps alive in ``_keep`` (set by make_params)."""
    _fields_ = [("batch", ctypes.c_int32), ("n_q", ctypes.c_int32), ("n_k", ctypes.c_int32),
                ("h_q", ctypes.c_int32), ("h_k", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("w_sink", ctypes.c_int32), ("w_near", ctypes.c_int32), ("h_k_total", ctypes.c_int32),
                ("h_k_offset", ctypes.c_int32), ("tile_q", ctypes.c_int32), ("tile_k", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("windows", ctypes.POINTER(cowa_window)), ("cu_seqlens_q", ctypes.POINTER(ctypes.c_int32)),
                ("cu_seqlens_k", ctypes.POINTER(ctypes.c_int32))]


class cowa_schedule_t(ctypes.Structure):
    _fields_ = [("p", cowa_params), ("n_qt", ctypes.c_int32), ("n_kt", ctypes.c_int32),
                ("max_row", ctypes.c_int32), ("max_col", ctypes.c_int32), ("nnz", ctypes.c_int64),
                ("off_fwd_row_ptr", ctypes.c_size_t), ("off_bwd_col_ptr", ctypes.c_size_t),
                ("off_fwd_ent", ctypes.c_size_t), ("off_bwd_ent", ctypes.c_size_t),
                ("off_windows", ctypes.c_size_t), ("off_seqs", ctypes.c_size_t),
                ("off_qt_seq", ctypes.c_size_t), ("off_kt_seq", ctypes.c_size_t),
                ("max_qt", ctypes.c_int32), ("max_kt", ctypes.c_int32), ("digest", ctypes.c_uint64),
                ("bytes", ctypes.c_size_t), ("buf", ctypes.c_void_p)]


class cowa_decode_params(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("h_q", ctypes.c_int32), ("h_k", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("n_max", ctypes.c_int32), ("w_sink", ctypes.c_int32),
                ("w_near", ctypes.c_int32), ("h_k_total", ctypes.c_int32), ("h_k_offset", ctypes.c_int32),
                ("split_keys", ctypes.c_int32), ("softmax_scale", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("windows", ctypes.POINTER(cowa_window))]


def window_array(tuples):
    """A C array of cowa_window from (sink, near, gap, width) tuples."""
    arr = (cowa_window * len(tuples))()
    for x, t in enumerate(tuples):
        arr[x].sink, arr[x].near, arr[x].gap, arr[x].width = (int(v) for v in t)
    return arr


def int32_array(values):
    return (ctypes.c_int32 * len(values))(*[int(v) for v in values])


_P = ctypes.POINTER
_vp = ctypes.c_void_p
_SIGNATURES = {
    "cowa_version": (ctypes.c_char_p, []),
    "cowa_last_error": (ctypes.c_char_p, []),
    "cowa_windows": (ctypes.c_int, [_P(cowa_params), _P(cowa_window)]),
    "cowa_schedule_size": (ctypes.c_int, [_P(cowa_params), _P(cowa_schedule_t)]),
    "cowa_schedule": (ctypes.c_int, [_P(cowa_schedule_t), _vp]),
    "cowa_legal_pairs": (ctypes.c_int, [_P(cowa_params), _P(ctypes.c_int64)]),
    "cowa_decode_visible_keys": (ctypes.c_int, [_P(cowa_decode_params), _P(ctypes.c_int32), _P(ctypes.c_int64)]),
    "cowa_fwd": (ctypes.c_int, [_P(cowa_params), _P(cowa_schedule_t), _vp, _vp, _vp, _vp, _vp, _vp]),
    "cowa_bwd_workspace_size": (ctypes.c_int, [_P(cowa_params), _P(ctypes.c_size_t)]),
    "cowa_bwd": (ctypes.c_int, [_P(cowa_params), _P(cowa_schedule_t), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                _vp, _vp, ctypes.c_size_t, _vp]),
    "cowa_bwd_prepare": (ctypes.c_int, [_P(cowa_params), _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]),
    "cowa_bwd_main": (ctypes.c_int, [_P(cowa_params), _P(cowa_schedule_t), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                     ctypes.c_size_t, _vp]),
    "cowa_bwd_dq": (ctypes.c_int, [_P(cowa_params), _P(cowa_schedule_t), _vp, _vp, _vp, _vp, _vp, _vp,
                                   ctypes.c_size_t, _vp]),
    "cowa_decode_workspace_size": (ctypes.c_int, [_P(cowa_decode_params), _P(ctypes.c_size_t)]),
    "cowa_decode": (ctypes.c_int, [_P(cowa_decode_params), _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                   _vp]),
    "cowa_decode_noalloc": (ctypes.c_int, [_P(cowa_decode_params), _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
}

_lib = None


class CowaError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def lib():
    """The loaded library.  Fails loudly when it has not been built: there is no
    fallback path."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"CoWA HIP library not built: {LIB_PATH} is missing "
                              "(run __graft_entry__.build())")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def check(status):
    if status != COWA_OK:
        raise CowaError(status, lib().cowa_last_error().decode())
    return status


def cowa_version():
    return lib().cowa_version().decode()


def cowa_last_error():
    return lib().cowa_last_error().decode()


def cowa_windows(params):
    out = (cowa_window * params.h_k)()
    check(lib().cowa_windows(ctypes.byref(params), out))
    return [(w.sink, w.near, w.gap, w.width) for w in out]


def cowa_schedule_size(params):
    s = cowa_schedule_t()
    check(lib().cowa_schedule_size(ctypes.byref(params), ctypes.byref(s)))
    return s


def cowa_schedule(sched, stream):
    check(lib().cowa_schedule(ctypes.byref(sched), _vp(stream)))


def cowa_legal_pairs(params):
    n = ctypes.c_int64()
    check(lib().cowa_legal_pairs(ctypes.byref(params), ctypes.byref(n)))
    return n.value


def cowa_decode_visible_keys(dparams, seqlens_host):
    arr = (ctypes.c_int32 * len(seqlens_host))(*[int(x) for x in seqlens_host])
    n = ctypes.c_int64()
    check(lib().cowa_decode_visible_keys(ctypes.byref(dparams), arr, ctypes.byref(n)))
    return n.value


def cowa_fwd(params, sched, q, k, v, o, lse, stream):
    check(lib().cowa_fwd(ctypes.byref(params), ctypes.byref(sched), _vp(q), _vp(k), _vp(v), _vp(o), _vp(lse),
                         _vp(stream)))


def cowa_bwd_workspace_size(params):
    n = ctypes.c_size_t()
    check(lib().cowa_bwd_workspace_size(ctypes.byref(params), ctypes.byref(n)))
    return n.value


def cowa_bwd(params, sched, q, k, v, o, lse, d_o, dq, dk, dv, workspace, ws_bytes, stream):
    check(lib().cowa_bwd(ctypes.byref(params), ctypes.byref(sched), _vp(q), _vp(k), _vp(v), _vp(o), _vp(lse),
                         _vp(d_o), _vp(dq), _vp(dk), _vp(dv), _vp(workspace), ws_bytes, _vp(stream)))


def cowa_bwd_prepare(params, o, d_o, lse, workspace, ws_bytes, stream):
    check(lib().cowa_bwd_prepare(ctypes.byref(params), _vp(o), _vp(d_o), _vp(lse), _vp(workspace), ws_bytes,
                                 _vp(stream)))


def cowa_bwd_main(params, sched, q, k, v, d_o, dk, dv, workspace, ws_bytes, stream):
    check(lib().cowa_bwd_main(ctypes.byref(params), ctypes.byref(sched), _vp(q), _vp(k), _vp(v), _vp(d_o),
                              _vp(dk), _vp(dv), _vp(workspace), ws_bytes, _vp(stream)))


def cowa_bwd_dq(params, sched, q, k, v, d_o, dq, workspace, ws_bytes, stream):
    check(lib().cowa_bwd_dq(ctypes.byref(params), ctypes.byref(sched), _vp(q), _vp(k), _vp(v), _vp(d_o), _vp(dq),
                            _vp(workspace), ws_bytes, _vp(stream)))


def cowa_decode_workspace_size(dparams):
    n = ctypes.c_size_t()
    check(lib().cowa_decode_workspace_size(ctypes.byref(dparams), ctypes.byref(n)))
    return n.value


def cowa_decode(dparams, q, k_cache, v_cache, seqlens_k, o, lse, workspace, ws_bytes, stream):
    check(lib().cowa_decode(ctypes.byref(dparams), _vp(q), _vp(k_cache), _vp(v_cache), _vp(seqlens_k), _vp(o),
                            _vp(lse), _vp(workspace), ws_bytes, _vp(stream)))


def cowa_decode_noalloc(dparams, q, k_cache, v_cache, seqlens_k, o, lse, stream):
    check(lib().cowa_decode_noalloc(ctypes.byref(dparams), _vp(q), _vp(k_cache), _vp(v_cache), _vp(seqlens_k),
                                    _vp(o), _vp(lse), _vp(stream)))
