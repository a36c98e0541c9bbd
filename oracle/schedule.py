"""KV-block sets J_h(i) and QO-block sets I_h(j), built two independent ways.

Test infrastructure (see the package docstring): never used by the product.

Sec. 2.3 (forward execution): for QO block I_i, J_h(i) holds the KV blocks
with at least one legal pair under Eq. fwa_support; Alg. 1 visits them with j
descending.  Sec. 2.3 (backward execution): I_h(j) holds the QO blocks with at
least one legal pair with KV block J_j; Alg. 2 visits them with i ascending.
Only blocks that cross a causal, window or sequence boundary need the
element mask; every other listed block is FULL.

Canonical schedule (what the GPU builder must reproduce bit for bit), for the
local KV heads h = 0..H_k-1 of one device:

* ``fwd_row_ptr`` int32 [H_k * n_qt + 1]; row r = h * n_qt + i.
* ``fwd_ent``     uint32 [nnz]; (j << 1) | partial, j descending within a row.
* ``bwd_col_ptr`` int32 [H_k * n_kt + 1]; column c = h * n_kt + j.
* ``bwd_ent``     uint32 [nnz]; (i << 1) | partial, i ascending within a column.

partial = 0 (FULL) iff every one of the B_q * B_k element pairs of the tile
rectangle lies inside the sequences (i_q < N_q, i_k < N_k) and is legal.
"""

import numpy as np

from .windows import visible_mask_bounds, visible_intervals_bounds, head_bounds


def _pack(row_lists, n_rows):
    ptr = np.zeros(n_rows + 1, dtype=np.int64)
    for r, lst in enumerate(row_lists):
        ptr[r + 1] = ptr[r] + len(lst)
    ent = np.zeros(int(ptr[-1]), dtype=np.uint32)
    for r, lst in enumerate(row_lists):
        if lst:
            ent[ptr[r]:ptr[r + 1]] = np.asarray(lst, dtype=np.uint32)
    return ptr.astype(np.int32), ent


def _assemble(listed, full, n_qt, n_kt):
    """listed/full: bool [H_k, n_qt, n_kt] -> canonical CSR pair."""
    h_k = listed.shape[0]
    fwd_rows, bwd_cols = [], []
    for h in range(h_k):
        for i in range(n_qt):
            js = np.nonzero(listed[h, i])[0][::-1]          # descending (Alg. 1)
            fwd_rows.append([(int(j) << 1) | int(not full[h, i, j]) for j in js])
        for j in range(n_kt):
            is_ = np.nonzero(listed[h, :, j])[0]             # ascending (Alg. 2)
            bwd_cols.append([(int(i) << 1) | int(not full[h, i, j]) for i in is_])
    fwd_row_ptr, fwd_ent = _pack(fwd_rows, h_k * n_qt)
    bwd_col_ptr, bwd_ent = _pack(bwd_cols, h_k * n_kt)
    return {"fwd_row_ptr": fwd_row_ptr, "fwd_ent": fwd_ent,
            "bwd_col_ptr": bwd_col_ptr, "bwd_ent": bwd_ent,
            "n_qt": n_qt, "n_kt": n_kt, "listed": listed, "full": full}


def tile_flags_bruteforce(n_q, n_k, tile_q, tile_k, w_sink, w_near, h_k, h_total, h_offset, windows=None):
    """Method A: reduce the element mask over every tile rectangle.

    Out-of-sequence positions are padded as illegal, so a tile that sticks out
    of either sequence is never FULL.  Memory is O(N_q * N_k) per head: use it
    up to a few thousand tokens.
    """
    n_qt = -(-n_q // tile_q)
    n_kt = -(-n_k // tile_k)
    listed = np.zeros((h_k, n_qt, n_kt), dtype=bool)
    full = np.zeros((h_k, n_qt, n_kt), dtype=bool)
    for h in range(h_k):
        bounds = head_bounds(n_k, w_sink, w_near, h_offset + h, h_total, None if windows is None else windows[h])
        m = visible_mask_bounds(n_q, n_k, *bounds)
        pad = np.zeros((n_qt * tile_q, n_kt * tile_k), dtype=bool)
        pad[:n_q, :n_k] = m
        blocks = pad.reshape(n_qt, tile_q, n_kt, tile_k)
        listed[h] = blocks.any(axis=(1, 3))
        full[h] = blocks.all(axis=(1, 3))
    return listed, full


def tile_flags_intervals(n_q, n_k, tile_q, tile_k, w_sink, w_near, h_k, h_total, h_offset, windows=None):
    """Method B: per query, the merged key runs of A_h(i_q) mark the tiles they
    touch and the tiles they cover completely.

    A tile (i, j) is listed iff some query of QO block i has a run touching KV
    block j; it is FULL iff it lies inside both sequences and every one of its
    B_q queries has a single run covering all B_k keys of block j (runs of one
    query are merged, so full coverage can only come from one run).
    Memory is O(N_q + n_qt * n_kt) per head.
    """
    n_qt = -(-n_q // tile_q)
    n_kt = -(-n_k // tile_k)
    listed = np.zeros((h_k, n_qt, n_kt), dtype=bool)
    full = np.zeros((h_k, n_qt, n_kt), dtype=bool)
    for h in range(h_k):
        touch = np.zeros((n_qt, n_kt + 1), dtype=np.int64)
        cover = np.zeros((n_qt, n_kt + 1), dtype=np.int64)
        rows_t, cols_t, vals_t = [], [], []
        rows_c, cols_c, vals_c = [], [], []
        bounds = head_bounds(n_k, w_sink, w_near, h_offset + h, h_total, None if windows is None else windows[h])
        for i_q in range(n_q):
            qt = i_q // tile_q
            for a, b in visible_intervals_bounds(i_q, n_q, n_k, *bounds):
                ja, jb = a // tile_k, (b - 1) // tile_k          # touched blocks [ja, jb]
                rows_t += [qt, qt]
                cols_t += [ja, jb + 1]
                vals_t += [1, -1]
                fa, fb = -(-a // tile_k), b // tile_k            # fully covered [fa, fb)
                if fa < fb:
                    rows_c += [qt, qt]
                    cols_c += [fa, fb]
                    vals_c += [1, -1]
        np.add.at(touch, (np.asarray(rows_t, dtype=np.int64), np.asarray(cols_t, dtype=np.int64)),
                  np.asarray(vals_t, dtype=np.int64))
        if rows_c:
            np.add.at(cover, (np.asarray(rows_c, dtype=np.int64), np.asarray(cols_c, dtype=np.int64)),
                      np.asarray(vals_c, dtype=np.int64))
        listed[h] = np.cumsum(touch, axis=1)[:, :n_kt] > 0
        covered_by = np.cumsum(cover, axis=1)[:, :n_kt]
        q_inside = np.array([(i + 1) * tile_q <= n_q for i in range(n_qt)], dtype=bool)
        k_inside = np.array([(j + 1) * tile_k <= n_k for j in range(n_kt)], dtype=bool)
        full[h] = (covered_by == tile_q) & q_inside[:, None] & k_inside[None, :]
    return listed, full


def build(n_q, n_k, tile_q, tile_k, w_sink, w_near, h_k, h_total=None, h_offset=0, method="intervals",
          windows=None):
    """Canonical CSR schedule of the local KV heads (see the module docstring).
    ``windows``: None (default rule) or one (sink, near, gap, width) per head."""
    if h_total is None:
        h_total = h_k
    fn = tile_flags_intervals if method == "intervals" else tile_flags_bruteforce
    listed, full = fn(n_q, n_k, tile_q, tile_k, w_sink, w_near, h_k, h_total, h_offset, windows)
    return _assemble(listed, full, listed.shape[1], listed.shape[2])


def build_varlen(cu_q, cu_k, tile_q, tile_k, w_sink, w_near, h_k, h_total=None, h_offset=0, method="intervals",
                 windows=None):
    """Canonical CSR schedule of a ragged batch: each sequence's blocks are
    found from its own lengths (its queries aligned to the end of its keys,
    Eq. fwa_distance), and the blocks of sequence b follow those of b - 1:
    row h * n_qt + (first block of b) + i, column h * n_kt + (first block of b)
    + j, with n_qt / n_kt the block counts over the batch; entries hold blocks
    within the sequence."""
    if h_total is None:
        h_total = h_k
    fn = tile_flags_intervals if method == "intervals" else tile_flags_bruteforce
    per = []
    for b in range(len(cu_q) - 1):
        n_q, n_k = int(cu_q[b + 1] - cu_q[b]), int(cu_k[b + 1] - cu_k[b])
        if n_k == 0:
            per.append(None)
            continue
        per.append(fn(n_q, n_k, tile_q, tile_k, w_sink, w_near, h_k, h_total, h_offset, windows))
    fwd_rows, bwd_cols = [], []
    for h in range(h_k):
        for flags in per:
            if flags is None:
                continue
            listed, full = flags
            for i in range(listed.shape[1]):
                js = np.nonzero(listed[h, i])[0][::-1]
                fwd_rows.append([(int(j) << 1) | int(not full[h, i, j]) for j in js])
        for flags in per:
            if flags is None:
                continue
            listed, full = flags
            for j in range(listed.shape[2]):
                is_ = np.nonzero(listed[h, :, j])[0]
                bwd_cols.append([(int(i) << 1) | int(not full[h, i, j]) for i in is_])
    fwd_row_ptr, fwd_ent = _pack(fwd_rows, len(fwd_rows))
    bwd_col_ptr, bwd_ent = _pack(bwd_cols, len(bwd_cols))
    return {"fwd_row_ptr": fwd_row_ptr, "fwd_ent": fwd_ent, "bwd_col_ptr": bwd_col_ptr, "bwd_ent": bwd_ent,
            "n_qt": len(fwd_rows) // h_k, "n_kt": len(bwd_cols) // h_k}
