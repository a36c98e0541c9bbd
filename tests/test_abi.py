"""The C ABI on the host: the library loads, exports every symbol the header
declares, sizes schedules and windows like the oracle, and rejects invalid
arguments with the documented status before touching any device.
(No kernel is launched here.)"""

import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT
from oracle import windows as ow, schedule as osched

cowa = pytest.importorskip("paper_2609_32704_amd")
abi = cowa._abi

HEADER = os.path.join(ROOT, "include", "cowa.h")


def _lib():
    try:
        return abi.lib()
    except ImportError as e:
        pytest.fail(f"library not built: {e}")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+char\s*\*|cowa_status)\s*(cowa_\w+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for n in ("cowa_schedule", "cowa_fwd", "cowa_bwd", "cowa_decode", "cowa_schedule_size", "cowa_windows",
              "cowa_bwd_workspace_size", "cowa_decode_workspace_size", "cowa_last_error", "cowa_version"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = _lib()
    for n in declared_functions():
        assert hasattr(lib, n), n
    assert "gfx950" in abi.cowa_version()


def test_struct_layouts_match_header(tmp_path):
    """Every struct of the header has the same size and field offsets in C
    (compiled here with gcc against include/cowa.h) as in the ctypes binding."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = [abi.cowa_window, abi.cowa_params, abi.cowa_schedule_t, abi.cowa_decode_params]
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "cowa.h"', "int main(void) {"]
    for st in structs:
        lines.append(f'  printf("{st.__name__} %zu\\n", sizeof({st.__name__}));')
        for name, _ in st._fields_:
            lines.append(f'  printf("{st.__name__}.{name} %zu\\n", offsetof({st.__name__}, {name}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = dict(line.split() for line in subprocess.run([str(exe)], capture_output=True, text=True,
                                                       check=True).stdout.splitlines())
    for st in structs:
        assert int(out[st.__name__]) == ctypes.sizeof(st), st.__name__
        for name, _ in st._fields_:
            assert int(out[f"{st.__name__}.{name}"]) == getattr(st, name).offset, f"{st.__name__}.{name}"


@pytest.mark.parametrize("n_k,ws,wn,ht,ho,hk", [(131072, 128, 4096, 8, 0, 8), (512, 16, 64, 2, 0, 2),
                                                (100, 0, 0, 3, 1, 2), (5, 10, 10, 4, 0, 4),
                                                (2 ** 30 - 1, 7, 9, 64, 60, 4)])
def test_windows_match_oracle(n_k, ws, wn, ht, ho, hk):
    p = cowa.make_params(1, 1, n_k, hk, hk, 128, ws, wn, 64, 64, h_k_total=ht, h_k_offset=ho)
    got = cowa.windows(p)
    assert got == [ow.window_tuple(n_k, ws, wn, ho + h, ht) for h in range(hk)]


@pytest.mark.parametrize("case", [(512, 512, 32, 32, 16, 64, 2, 2, 0), (8192, 8192, 64, 64, 64, 1024, 8, 8, 0),
                                  (333, 1000, 64, 128, 3, 77, 3, 5, 2), (1, 1, 32, 32, 0, 1, 1, 1, 0)])
def test_schedule_size_matches_oracle(case):
    n_q, n_k, tq, tk, ws, wn, hk, ht, ho = case
    p = cowa.make_params(1, n_q, n_k, hk, hk, 128, ws, wn, tq, tk, h_k_total=ht, h_k_offset=ho)
    s = abi.cowa_schedule_size(p)
    ref = osched.build(n_q, n_k, tq, tk, ws, wn, hk, ht, ho)
    assert s.nnz == len(ref["fwd_ent"])
    assert s.n_qt == ref["n_qt"] and s.n_kt == ref["n_kt"]
    assert s.max_row == int(np.diff(ref["fwd_row_ptr"]).max())
    assert s.max_col == int(np.diff(ref["bwd_col_ptr"]).max())
    for off in (s.off_fwd_row_ptr, s.off_bwd_col_ptr, s.off_fwd_ent, s.off_bwd_ent):
        assert off % 256 == 0
    assert s.bytes >= s.off_bwd_ent + 4 * s.nnz


def _good():
    return cowa.make_params(1, 256, 256, 4, 2, 128, 8, 32, 64, 64)


def _status(fn, *args):
    return fn(*args)


@pytest.mark.parametrize("field,value,status", [
    ("n_q", 300, abi.COWA_ERR_INVALID_ARG), ("n_q", 0, abi.COWA_ERR_INVALID_ARG),
    ("h_q", 5, abi.COWA_ERR_INVALID_ARG), ("tile_q", 48, abi.COWA_ERR_INVALID_ARG),
    ("tile_k", 256, abi.COWA_ERR_INVALID_ARG), ("w_sink", -1, abi.COWA_ERR_INVALID_ARG),
    ("w_near", -5, abi.COWA_ERR_INVALID_ARG), ("h_k_offset", 1, abi.COWA_ERR_INVALID_ARG),
    ("h_k_total", 1, abi.COWA_ERR_INVALID_ARG), ("head_dim", 96, abi.COWA_ERR_UNSUPPORTED),
    ("dtype", 7, abi.COWA_ERR_INVALID_ARG), ("batch", -1, abi.COWA_ERR_INVALID_ARG),
    ("softmax_scale", float("inf"), abi.COWA_ERR_INVALID_ARG), ("softmax_scale", 0.0, abi.COWA_ERR_INVALID_ARG),
    ("softmax_scale", -0.125, abi.COWA_ERR_INVALID_ARG),
])
def test_invalid_params_rejected_on_host(field, value, status):
    lib = _lib()
    p = _good()
    setattr(p, field, value)
    s = abi.cowa_schedule_t()
    assert lib.cowa_schedule_size(ctypes.byref(p), ctypes.byref(s)) == status
    assert lib.cowa_last_error()
    out = (abi.cowa_window * 4)()
    assert lib.cowa_windows(ctypes.byref(p), out) == status


def _sized(p):
    s = abi.cowa_schedule_size(p)
    s.buf = 1 << 20  # a fake, aligned address: these calls must fail before any launch
    return s


def test_fwd_argument_errors_on_host():
    lib = _lib()
    p = _good()
    s = _sized(p)
    ok = 1 << 24
    vp = ctypes.c_void_p
    call = lambda *a: lib.cowa_fwd(ctypes.byref(p), ctypes.byref(s), *[vp(x) for x in a])
    assert call(0, ok, ok, ok, ok, 0) == abi.COWA_ERR_INVALID_ARG            # q NULL
    assert call(ok + 8, ok, ok, ok, ok, 0) == abi.COWA_ERR_INVALID_ARG       # q misaligned
    assert call(ok, ok, ok, ok, ok + 2, 0) == abi.COWA_ERR_INVALID_ARG       # lse misaligned
    other = _good()
    other.w_near = 33
    assert lib.cowa_fwd(ctypes.byref(other), ctypes.byref(s), *[vp(ok)] * 5, vp(0)) == \
        abi.COWA_ERR_SCHEDULE_MISMATCH
    s.buf = 4096 + 16
    assert call(ok, ok, ok, ok, ok, 0) == abi.COWA_ERR_INVALID_ARG           # schedule buffer misaligned
    s.buf = 0
    assert call(ok, ok, ok, ok, ok, 0) == abi.COWA_ERR_INVALID_ARG           # schedule buffer NULL
    # bf16 with a 32-row query block is not built
    p32 = _good()
    p32.tile_q = 32
    s32 = _sized(p32)
    assert lib.cowa_fwd(ctypes.byref(p32), ctypes.byref(s32), *[vp(ok)] * 5, vp(0)) == abi.COWA_ERR_UNSUPPORTED
    # ... nor with a 32-key block
    k32 = _good()
    k32.tile_k = 32
    sk32 = _sized(k32)
    assert lib.cowa_fwd(ctypes.byref(k32), ctypes.byref(sk32), *[vp(ok)] * 5, vp(0)) == abi.COWA_ERR_UNSUPPORTED


def test_batch_zero_is_a_no_op():
    lib = _lib()
    p = _good()
    p.batch = 0
    s = _sized(p)
    assert lib.cowa_fwd(ctypes.byref(p), ctypes.byref(s), *[ctypes.c_void_p(0)] * 6) == abi.COWA_OK


def test_schedule_fields_must_come_from_sizing():
    lib = _lib()
    p = _good()
    s = _sized(p)
    s.nnz += 1
    assert lib.cowa_schedule(ctypes.byref(s), None) == abi.COWA_ERR_SCHEDULE_MISMATCH


def test_bwd_workspace_and_errors_on_host():
    lib = _lib()
    p = _good()
    need = abi.cowa_bwd_workspace_size(p)
    rows = p.batch * p.h_q * p.n_q
    assert need >= rows * 8
    p32 = _good()
    p32.dtype = abi.COWA_FP32
    s = _sized(p32)
    vp = ctypes.c_void_p
    assert lib.cowa_bwd(ctypes.byref(p32), ctypes.byref(s), *[vp(1 << 24)] * 10, ctypes.c_size_t(need),
                        vp(0)) == abi.COWA_ERR_UNSUPPORTED


def _split_ws(n_rows, n_cols, parts, tile_k, d):
    arr = -(-n_rows * 4 // 256) * 256
    part = -(-n_cols * parts * 2 * tile_k * d * 4 // 256) * 256 if parts > 1 else 0
    return 2 * arr + part


@pytest.mark.parametrize("offset", [0, 7])
def test_bwd_workspace_holds_sink_column_parts(offset):
    """One rank of an 8-way KV-head split at 131072 tokens: the sink block's
    query list spans all 1024 query blocks, a column past the sink holds at
    most (128 + 4096 - 2) // 128 + 2 = 34 near and (128 + 15856 - 2) // 128 + 2
    = 126 long-range blocks, so the sink column is cut into ceil(2 x 1024 / 160)
    = 13 parts (about half an ordinary column each), whose float32 dK/dV
    partials (2 x 128 x 128 x 4 bytes each) follow the two per-row arrays in
    the workspace."""
    p = cowa.make_params(1, 131072, 131072, 4, 1, 128, 128, 4096, 128, 128, h_k_total=8, h_k_offset=offset)
    assert abi.cowa_bwd_workspace_size(p) == _split_ws(4 * 131072, 1, 13, 128, 128)


def test_bwd_workspace_without_sink_has_no_parts():
    # no sink keys (the dense causal twin): nothing is split
    p = cowa.make_params(1, 8192, 8192, 32, 8, 128, 0, 8192, 64, 64)
    assert abi.cowa_bwd_workspace_size(p) == _split_ws(32 * 8192, 0, 1, 64, 128)
    # the 8K workload (64-token blocks): sink column of 128 blocks, others at
    # most (64 + 1024 - 2) // 64 + 2 + (64 + 888 - 2) // 64 + 2 = 34 -> ceil(256 / 34)
    # = 8 parts, for each of the 8 KV heads
    p = cowa.make_params(1, 8192, 8192, 32, 8, 128, 64, 1024, 64, 64)
    assert abi.cowa_bwd_workspace_size(p) == _split_ws(32 * 8192, 8, 8, 64, 128)


def test_decode_argument_errors_on_host():
    lib = _lib()
    d = cowa.make_decode_params(4, 8, 2, 128, 1000, 16, 64)
    need = abi.cowa_decode_workspace_size(d)
    vp = ctypes.c_void_p
    ok = 1 << 24
    assert lib.cowa_decode(ctypes.byref(d), vp(0), vp(ok), vp(ok), vp(ok), vp(ok), vp(ok), vp(ok),
                           ctypes.c_size_t(need), vp(0)) == abi.COWA_ERR_INVALID_ARG
    if need > 0:
        assert lib.cowa_decode(ctypes.byref(d), *[vp(ok)] * 7, ctypes.c_size_t(need - 1), vp(0)) == \
            abi.COWA_ERR_WORKSPACE
    bad = cowa.make_decode_params(4, 8, 3, 128, 1000, 16, 64)
    n = ctypes.c_size_t()
    assert lib.cowa_decode_workspace_size(ctypes.byref(bad), ctypes.byref(n)) == abi.COWA_ERR_INVALID_ARG
    bad = cowa.make_decode_params(4, 8, 2, 128, 1000, 16, 64, split_keys=100)
    assert lib.cowa_decode_workspace_size(ctypes.byref(bad), ctypes.byref(n)) == abi.COWA_ERR_INVALID_ARG


@pytest.mark.parametrize("case", [(1, 512, 512, 4, 2, 16, 64, 2, 0), (1, 8192, 8192, 32, 8, 64, 1024, 8, 0),
                                  (2, 300, 1000, 6, 3, 5, 77, 8, 4), (1, 50, 50, 2, 2, 0, 0, 2, 0)])
def test_legal_pairs_match_oracle(case):
    from oracle import counts
    bsz, n_q, n_k, h_q, h_k, ws, wn, ht, ho = case
    p = cowa.make_params(bsz, n_q, n_k, h_q, h_k, 128, ws, wn, 64, 64, h_k_total=ht, h_k_offset=ho)
    assert abi.cowa_legal_pairs(p) == counts.legal_pairs(bsz, n_q, n_k, h_q, h_k, ws, wn, ht, ho)


def test_legal_pairs_128k_workload():
    p = cowa.make_params(1, 131072, 131072, 32, 8, 128, 128, 4096, 128, 128)
    assert abi.cowa_legal_pairs(p) == 49612416768


def test_decode_visible_keys_match_oracle():
    from oracle import counts
    d = cowa.make_decode_params(5, 8, 2, 128, 5000, 16, 300, h_k_total=4, h_k_offset=1)
    lens = [5000, 1, 316, 4000, 0]
    ref = counts.decode_visible_keys([x for x in lens if 1 <= x <= 5000], 16, 300, 2, 4, 1).sum()
    assert abi.cowa_decode_visible_keys(d, lens) == ref
    d = cowa.make_decode_params(64, 32, 8, 128, 131072, 128, 4096)
    assert abi.cowa_decode_visible_keys(d, [131072] * 64) == 64 * 8 * 20080


@pytest.mark.parametrize("n_q,n_k,ok", [(16000 * 128, 16000 * 128, False), (8192 * 128, 8192 * 128, True),
                                        (8192 * 128 + 1, 8192 * 128 + 1, False)])
def test_bwd_shape_limits_on_host(n_q, n_k, ok):
    """The backward passes keep one schedule row / column of block entries in
    LDS; shapes beyond those limits are rejected before any launch (checked on
    the host, so the error comes back without a device)."""
    lib = _lib()
    p = cowa.make_params(1, n_q, n_k, 4, 1, 128, 128, 4096, 128, 128)
    need = ctypes.c_size_t()
    st = lib.cowa_bwd_workspace_size(ctypes.byref(p), ctypes.byref(need))
    assert st == abi.COWA_OK
    s = abi.cowa_schedule_t()
    vp = ctypes.c_void_p
    st = lib.cowa_bwd_main(ctypes.byref(p), ctypes.byref(s), *[vp(1 << 24)] * 7, need, vp(0))
    if ok:
        assert st != abi.COWA_ERR_UNSUPPORTED
    else:
        assert st == abi.COWA_ERR_UNSUPPORTED
        assert b"blocks" in lib.cowa_last_error()


def test_bwd_checks_every_stage_before_any_launch():
    """cowa_bwd runs three stages; a limit of its last stage (the dQ pass's
    grid of n_qt x h_q x batch workgroups) is rejected before the first stage
    is launched: the status is COWA_ERR_UNSUPPORTED even without a device
    (a launch attempt would need one and report COWA_ERR_NO_DEVICE)."""
    lib = _lib()
    bsz = (1 << 31) // (1000 * 64) + 1
    p = cowa.make_params(bsz, 128000, 128000, 64, 1, 128, 128, 4096, 128, 128)
    need = abi.cowa_bwd_workspace_size(p)
    s = _sized(p)
    vp = ctypes.c_void_p
    st = lib.cowa_bwd(ctypes.byref(p), ctypes.byref(s), *[vp(1 << 24)] * 10, ctypes.c_size_t(need), vp(0))
    assert st == abi.COWA_ERR_UNSUPPORTED
    assert b"query blocks" in lib.cowa_last_error()
    # each stage on its own applies the same check
    st = lib.cowa_bwd_main(ctypes.byref(p), ctypes.byref(s), *[vp(1 << 24)] * 7, ctypes.c_size_t(need), vp(0))
    assert st == abi.COWA_ERR_UNSUPPORTED


# ---- explicit window tuples and ragged batches (host side) ----

RAGGED = [([0, 70, 70, 200, 233], [0, 100, 131, 300, 500]), ([0, 1], [0, 1]), ([0, 0, 5], [0, 3, 9]),
          ([0, 300, 1000], [0, 300, 1000])]
TUPLES = [None, [(1, 16, 5, 40), (0, 33, 0, 100), (50, 0, 3, 3)]]


@pytest.mark.parametrize("cu", RAGGED)
@pytest.mark.parametrize("tuples", TUPLES)
def test_ragged_schedule_size_matches_oracle(cu, tuples):
    cu_q, cu_k = cu
    p = cowa.make_params(len(cu_q) - 1, cu_q[-1], cu_k[-1], 3, 3, 128, 4, 20, 64, 32, windows=tuples,
                         cu_seqlens_q=cu_q, cu_seqlens_k=cu_k)
    s = abi.cowa_schedule_size(p)
    ref = osched.build_varlen(cu_q, cu_k, 64, 32, 4, 20, 3, windows=tuples)
    assert s.nnz == len(ref["fwd_ent"])
    assert (s.n_qt, s.n_kt) == (ref["n_qt"], ref["n_kt"])
    rows, cols = np.diff(ref["fwd_row_ptr"]), np.diff(ref["bwd_col_ptr"])
    assert s.max_row == (int(rows.max()) if rows.size else 0)
    assert s.max_col == (int(cols.max()) if cols.size else 0)
    lens_q, lens_k = np.diff(cu_q), np.diff(cu_k)
    assert s.max_qt == int((-(-lens_q // 64)).max()) and s.max_kt == int((-(-lens_k // 32)).max())


@pytest.mark.parametrize("tuples", TUPLES[1:])
def test_tuple_schedule_size_matches_oracle(tuples):
    p = cowa.make_params(2, 333, 1000, 6, 3, 128, 4, 20, 64, 128, windows=tuples)
    s = abi.cowa_schedule_size(p)
    ref = osched.build(333, 1000, 64, 128, 4, 20, 3, windows=tuples)
    assert s.nnz == len(ref["fwd_ent"])
    assert cowa.windows(p) == [tuple(t) for t in tuples]


def test_legal_pairs_with_tuples_and_ragged():
    from oracle import windows as w
    cu_q, cu_k = [0, 70, 70, 200, 233], [0, 100, 131, 300, 500]
    for tuples in TUPLES:
        p = cowa.make_params(4, 233, 500, 6, 3, 128, 4, 20, 64, 32, windows=tuples, cu_seqlens_q=cu_q,
                             cu_seqlens_k=cu_k)
        ref = 0
        for b in range(4):
            n_q, n_k = cu_q[b + 1] - cu_q[b], cu_k[b + 1] - cu_k[b]
            for h in range(3):
                bounds = w.head_bounds(n_k, 4, 20, h, 3, None if tuples is None else tuples[h])
                ref += int(w.visible_mask_bounds(n_q, n_k, *bounds).sum())
        assert abi.cowa_legal_pairs(p) == 2 * ref


@pytest.mark.parametrize("cu_q,cu_k", [([1, 5], [0, 5]), ([0, 6], [0, 5]), ([0, 5, 3], [0, 5, 9]),
                                       ([0, 5], [0, 7])])
def test_invalid_cu_seqlens_rejected(cu_q, cu_k):
    lib = _lib()
    p = cowa.make_params(len(cu_q) - 1, cu_q[-1], 5, 2, 1, 128, 1, 4, 64, 64, cu_seqlens_q=cu_q, cu_seqlens_k=cu_k)
    s = abi.cowa_schedule_t()
    assert lib.cowa_schedule_size(ctypes.byref(p), ctypes.byref(s)) == abi.COWA_ERR_INVALID_ARG


def test_invalid_tuples_rejected():
    lib = _lib()
    p = cowa.make_params(1, 100, 100, 2, 2, 128, 1, 4, 64, 64, windows=[(1, 4, 0, 10), (1, -1, 0, 10)])
    s = abi.cowa_schedule_t()
    assert lib.cowa_schedule_size(ctypes.byref(p), ctypes.byref(s)) == abi.COWA_ERR_INVALID_ARG
    d = cowa.make_decode_params(2, 4, 2, 128, 1000, 4, 8, windows=[(1, 4, 0, 10), (1, 4, -2, 10)])
    n = ctypes.c_size_t()
    assert lib.cowa_decode_workspace_size(ctypes.byref(d), ctypes.byref(n)) == abi.COWA_ERR_INVALID_ARG


def test_schedule_digest_guards_windows_and_lengths():
    """A schedule sized for one set of tuples or lengths is refused (before any
    launch) for another of the same shapes."""
    lib = _lib()
    vp = ctypes.c_void_p
    ok = 1 << 24
    p1 = cowa.make_params(1, 256, 256, 4, 2, 128, 8, 32, 64, 64, windows=[(8, 32, 0, 50), (8, 32, 50, 50)])
    s1 = _sized(p1)
    p2 = cowa.make_params(1, 256, 256, 4, 2, 128, 8, 32, 64, 64, windows=[(8, 32, 0, 50), (8, 32, 51, 50)])
    assert lib.cowa_fwd(ctypes.byref(p2), ctypes.byref(s1), *[vp(ok)] * 5, vp(0)) == abi.COWA_ERR_SCHEDULE_MISMATCH
    r1 = cowa.make_params(2, 200, 300, 4, 2, 128, 8, 32, 64, 64, cu_seqlens_q=[0, 100, 200], cu_seqlens_k=[0, 150, 300])
    sr = _sized(r1)
    r2 = cowa.make_params(2, 200, 300, 4, 2, 128, 8, 32, 64, 64, cu_seqlens_q=[0, 90, 200], cu_seqlens_k=[0, 150, 300])
    assert lib.cowa_fwd(ctypes.byref(r2), ctypes.byref(sr), *[vp(ok)] * 5, vp(0)) == abi.COWA_ERR_SCHEDULE_MISMATCH
    assert lib.cowa_fwd(ctypes.byref(r1), ctypes.byref(sr), *[vp(ok)] * 5, vp(0)) == abi.COWA_ERR_NO_DEVICE


def test_decode_noalloc_rejects_steps_beyond_its_scratch():
    """The allocation-free decode keeps split partials in a 32 MiB device
    array; a step that needs more is refused before any device call."""
    lib = _lib()
    vp = ctypes.c_void_p
    ok = 1 << 24
    big = cowa.make_decode_params(256, 64, 8, 128, 131072, 128, 4096, split_keys=64)
    assert abi.cowa_decode_workspace_size(big) > 32 << 20
    assert lib.cowa_decode_noalloc(ctypes.byref(big), *[vp(ok)] * 6, vp(0)) == abi.COWA_ERR_UNSUPPORTED
    assert b"scratch" in lib.cowa_last_error()
    fits = cowa.make_decode_params(64, 32, 8, 128, 131072, 128, 4096)
    assert abi.cowa_decode_workspace_size(fits) <= 32 << 20
    assert lib.cowa_decode_noalloc(ctypes.byref(fits), *[vp(ok)] * 6, vp(0)) == abi.COWA_ERR_NO_DEVICE
