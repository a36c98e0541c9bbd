"""CoWA attention in float64: forward, exact gradient, decoding.

Test infrastructure (see the package docstring): never used by the product.

The method computes exactly masked softmax attention over each query's
visible-key set A_h(i_q) (Eq. fwa_support): Alg. 1 is an online-softmax
evaluation of it and Sec. 2.3 states that the probabilities rebuilt from the
saved log-sum-exp give the exact gradient (Alg. 2).  So the oracle is that
plain definition, per (batch, QO head), in float64:

    S  = scale * Q K^T,  S[~M] = -inf           (M = visible mask of KV head h_k)
    m  = rowmax S,  P = exp(S - m),  l = rowsum P
    O  = P V / l,  LSE = m + ln l               (Alg. 1: final rescale and LSE)

and the gradient of <dO, O> (Alg. 2):

    P  = exp(S - LSE) on M, 0 elsewhere
    dP = dO V^T,  D = rowsum(O * dO),  dS = P * (dP - D)
    dQ = scale * dS K,  dK = sum over the QO-head group of scale * dS^T Q,
    dV = sum over the QO-head group of P^T dO.

QO head h uses KV head floor(h * H_k / H_q) (Sec. 2.1).  The scale multiplies
Q K^T; the paper assumes Q pre-scaled by 1/sqrt(d_h) (Sec. 2.3), which is
scale = 1/sqrt(d_h) applied here instead.

A row whose visible set is empty (possible only with w_near = 0) has O = 0,
LSE = -inf and contributes nothing to any gradient.

Arrays: Q, O, dO [B, H_q, N_q, d]; K, V [B, H_k, N_k, d]; LSE [B, H_q, N_q].
``h_total`` / ``h_offset`` are the global KV-head count and the global index
of local KV head 0 (Eq. fwa_global_head); the defaults describe one device.

For large shapes the work is split into blocks of query rows, and each block
only gathers the keys that some row of the block can see (the union of the
rows' visible runs); the mask is still evaluated element by element on that
gather, so the result is the same exact definition.
"""

import numpy as np

from .windows import kv_head_of, visible_mask_bounds, visible_intervals_bounds, head_bounds


def _bounds(n_k, w_sink, w_near, h_offset, hk, h_total, windows):
    """(sink, near, lo, hi) of local KV head hk: its explicit four-tuple when
    ``windows`` (one (sink, near, gap, width) per local KV head) is given, else
    the default rule over the global head index (Sec. 2.1)."""
    return head_bounds(n_k, w_sink, w_near, h_offset + hk, h_total, None if windows is None else windows[hk])


def _union_keys(rows, n_q, n_k, bounds):
    runs = []
    for i_q in rows:
        runs += visible_intervals_bounds(int(i_q), n_q, n_k, *bounds)
    if not runs:
        return np.zeros(0, dtype=np.int64)
    runs.sort()
    merged = [list(runs[0])]
    for a, b in runs[1:]:
        if a <= merged[-1][1]:
            merged[-1][1] = max(merged[-1][1], b)
        else:
            merged.append([a, b])
    return np.concatenate([np.arange(a, b, dtype=np.int64) for a, b in merged])


def _rows_forward(qh, kh, vh, rows, n_q, n_k, bounds, scale):
    """Exact O and LSE of the given query rows of one (batch, QO head) whose
    KV head has the window bounds (sink, near, lo, hi).

    qh [N_q, d]; kh, vh [N_k, d]; rows: sorted int array (a block of nearby rows).
    Returns (o [len(rows), d], lse [len(rows)], keys, p) where ``keys`` are the
    gathered key positions and p the normalised probabilities on them.
    """
    keys = _union_keys(rows, n_q, n_k, bounds)
    d = qh.shape[1]
    if keys.size == 0:
        return (np.zeros((len(rows), d)), np.full(len(rows), -np.inf), keys,
                np.zeros((len(rows), 0)))
    mask = visible_mask_bounds(n_q, n_k, *bounds, rows=rows, cols=keys)
    s = scale * (qh[rows] @ kh[keys].T)
    s = np.where(mask, s, -np.inf)
    m = s.max(axis=1)
    m_safe = np.where(np.isfinite(m), m, 0.0)
    p = np.where(mask, np.exp(s - m_safe[:, None]), 0.0)
    l = p.sum(axis=1)
    l_safe = np.where(l > 0, l, 1.0)
    o = (p @ vh[keys]) / l_safe[:, None]
    lse = np.where(l > 0, m_safe + np.log(l_safe), -np.inf)
    return o, lse, keys, p / l_safe[:, None]


def _blocks(rows, size):
    rows = np.asarray(rows, dtype=np.int64)
    for s in range(0, len(rows), size):
        yield rows[s:s + size]


def forward(q, k, v, w_sink, w_near, scale, h_total=None, h_offset=0, block=256, windows=None):
    """Full forward: returns (O, LSE) in float64.  ``windows``: None (default
    rule) or one (sink, near, gap, width) tuple per local KV head."""
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    bsz, h_q, n_q, d = q.shape
    h_k, n_k = k.shape[1], k.shape[2]
    h_total = h_k if h_total is None else h_total
    o = np.zeros((bsz, h_q, n_q, v.shape[3]))
    lse = np.zeros((bsz, h_q, n_q))
    for b in range(bsz):
        for h in range(h_q):
            hk = kv_head_of(h, h_q, h_k)
            bounds = _bounds(n_k, w_sink, w_near, h_offset, hk, h_total, windows)
            for rows in _blocks(np.arange(n_q), block):
                ob, lb, _, _ = _rows_forward(q[b, h], k[b, hk], v[b, hk], rows, n_q, n_k, bounds, scale)
                o[b, h, rows] = ob
                lse[b, h, rows] = lb
    return o, lse


def forward_rows(q, k, v, rows, w_sink, w_near, scale, h_total=None, h_offset=0, block=128, windows=None):
    """O and LSE of selected rows.  ``rows``: iterable of (b, h, i_q).
    Returns (o [n, d], lse [n]) in the order given."""
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    h_q, n_q = q.shape[1], q.shape[2]
    h_k, n_k = k.shape[1], k.shape[2]
    h_total = h_k if h_total is None else h_total
    rows = [tuple(int(t) for t in r) for r in rows]
    out_o = np.zeros((len(rows), v.shape[3]))
    out_l = np.zeros(len(rows))
    groups = {}
    for n, (b, h, i) in enumerate(rows):
        groups.setdefault((b, h), []).append((i, n))
    for (b, h), lst in groups.items():
        lst.sort()
        hk = kv_head_of(h, h_q, h_k)
        bounds = _bounds(n_k, w_sink, w_near, h_offset, hk, h_total, windows)
        for s in range(0, len(lst), block):
            chunk = lst[s:s + block]
            idx = np.array([i for i, _ in chunk], dtype=np.int64)
            ob, lb, _, _ = _rows_forward(q[b, h], k[b, hk], v[b, hk], idx, n_q, n_k, bounds, scale)
            for t, (_, n) in enumerate(chunk):
                out_o[n] = ob[t]
                out_l[n] = lb[t]
    return out_o, out_l


def backward(q, k, v, do, w_sink, w_near, scale, h_total=None, h_offset=0, block=256, rows=None, heads=None,
             windows=None):
    """Exact gradient of <dO, O(Q, K, V)>.  Returns (dQ, dK, dV, O, LSE).

    ``rows`` / ``heads`` restrict the work to those query rows and QO heads
    (default: all); dK and dV then hold only their contributions."""
    q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
    bsz, h_q, n_q, d = q.shape
    h_k, n_k = k.shape[1], k.shape[2]
    h_total = h_k if h_total is None else h_total
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    o = np.zeros_like(do)
    lse = np.zeros((bsz, h_q, n_q))
    row_set = np.arange(n_q) if rows is None else np.asarray(rows, dtype=np.int64)
    for b in range(bsz):
        for h in (range(h_q) if heads is None else heads):
            hk = kv_head_of(h, h_q, h_k)
            bounds = _bounds(n_k, w_sink, w_near, h_offset, hk, h_total, windows)
            for rows in _blocks(row_set, block):
                ob, lb, keys, p = _rows_forward(q[b, h], k[b, hk], v[b, hk], rows, n_q, n_k, bounds, scale)
                o[b, h, rows] = ob
                lse[b, h, rows] = lb
                if keys.size == 0:
                    continue
                dp = do[b, h, rows] @ v[b, hk, keys].T
                dsum = (ob * do[b, h, rows]).sum(axis=1)
                ds = p * (dp - dsum[:, None])
                dq[b, h, rows] = scale * (ds @ k[b, hk, keys])
                dk[b, hk, keys] += scale * (ds.T @ q[b, h, rows])
                dv[b, hk, keys] += p.T @ do[b, h, rows]
    return dq, dk, dv, o, lse


def backward_kv_rows(q, k, v, do, kv_rows, w_sink, w_near, scale, h_total=None, h_offset=0,
                     block=128, windows=None):
    """Exact dK and dV of selected key rows.  ``kv_rows``: iterable of
    (b, h_k, i_k).  Every query that sees one of the selected keys is
    evaluated over its whole visible set (its O and LSE are needed).
    Returns (dk [n, d], dv [n, d]) in the order given."""
    q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
    h_q, n_q = q.shape[1], q.shape[2]
    h_k, n_k = k.shape[1], k.shape[2]
    h_total = h_k if h_total is None else h_total
    kv_rows = [tuple(int(t) for t in r) for r in kv_rows]
    out_dk = np.zeros((len(kv_rows), k.shape[3]))
    out_dv = np.zeros((len(kv_rows), v.shape[3]))
    groups = {}
    for n, (b, hk, i) in enumerate(kv_rows):
        groups.setdefault((b, hk), []).append((i, n))
    for (b, hk), lst in groups.items():
        sel = np.array(sorted({i for i, _ in lst}), dtype=np.int64)
        pos = {int(i): t for t, i in enumerate(sel)}
        acc_k = np.zeros((len(sel), k.shape[3]))
        acc_v = np.zeros((len(sel), v.shape[3]))
        bounds = _bounds(n_k, w_sink, w_near, h_offset, hk, h_total, windows)
        # queries that see at least one selected key, per QO head of the group
        for h in range(h_q):
            if kv_head_of(h, h_q, h_k) != hk:
                continue
            sees = np.zeros(n_q, dtype=bool)
            for rows in _blocks(np.arange(n_q), 4096):
                sees[rows] = visible_mask_bounds(n_q, n_k, *bounds, rows=rows, cols=sel).any(axis=1)
            for rows in _blocks(np.nonzero(sees)[0], block):
                ob, lb, keys, p = _rows_forward(q[b, h], k[b, hk], v[b, hk], rows, n_q, n_k, bounds, scale)
                dp = do[b, h, rows] @ v[b, hk, keys].T
                dsum = (ob * do[b, h, rows]).sum(axis=1)
                ds = p * (dp - dsum[:, None])
                take = np.isin(keys, sel)
                kk = keys[take]
                idx = np.array([pos[int(x)] for x in kk], dtype=np.int64)
                acc_k[idx] += scale * (ds[:, take].T @ q[b, h, rows])
                acc_v[idx] += p[:, take].T @ do[b, h, rows]
        for i, n in lst:
            out_dk[n] = acc_k[pos[i]]
            out_dv[n] = acc_v[pos[i]]
    return out_dk, out_dv


def backward_q_rows(q, k, v, do, rows, w_sink, w_near, scale, h_total=None, h_offset=0, block=128, windows=None):
    """Exact dQ (and O, LSE) of selected query rows ``(b, h, i_q)``, evaluated in
    blocks of nearby rows of one (batch, QO head).
    Returns (dq [n, d], o [n, d], lse [n]) in the order given."""
    q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
    h_q, n_q = q.shape[1], q.shape[2]
    h_k, n_k = k.shape[1], k.shape[2]
    h_total = h_k if h_total is None else h_total
    rows = [tuple(int(t) for t in r) for r in rows]
    out_dq = np.zeros((len(rows), q.shape[3]))
    out_o = np.zeros((len(rows), v.shape[3]))
    out_l = np.zeros(len(rows))
    groups = {}
    for n, (b, h, i) in enumerate(rows):
        groups.setdefault((b, h), []).append((i, n))
    for (b, h), lst in groups.items():
        lst.sort()
        hk = kv_head_of(h, h_q, h_k)
        bounds = _bounds(n_k, w_sink, w_near, h_offset, hk, h_total, windows)
        for s in range(0, len(lst), block):
            chunk = lst[s:s + block]
            idx = np.array([i for i, _ in chunk], dtype=np.int64)
            ob, lb, keys, p = _rows_forward(q[b, h], k[b, hk], v[b, hk], idx, n_q, n_k, bounds, scale)
            dqb = np.zeros((len(idx), q.shape[3]))
            if keys.size:
                dp = do[b, h, idx] @ v[b, hk, keys].T
                dsum = (ob * do[b, h, idx]).sum(axis=1)
                ds = p * (dp - dsum[:, None])
                dqb = scale * (ds @ k[b, hk, keys])
            for t, (_, n) in enumerate(chunk):
                out_dq[n], out_o[n], out_l[n] = dqb[t], ob[t], lb[t]
    return out_dq, out_o, out_l


def decode(q, k_cache, v_cache, seqlens, w_sink, w_near, scale, h_total=None, h_offset=0, windows=None):
    """One decoding step (Sec. 2.3, decoding execution): the forward with N_q = 1
    per sequence, N_k = seqlens[b] (cached tokens plus the current one, whose
    K/V the caller has already appended), breakpoints from that N_k.

    q [B, H_q, d]; caches [B, H_k, n_max, d].  Returns (O [B, H_q, d], LSE [B, H_q])."""
    q, kc, vc = (np.asarray(x, dtype=np.float64) for x in (q, k_cache, v_cache))
    bsz, h_q, d = q.shape
    h_k = kc.shape[1]
    h_total = h_k if h_total is None else h_total
    o = np.zeros((bsz, h_q, vc.shape[3]))
    lse = np.zeros((bsz, h_q))
    for b in range(bsz):
        n_k = int(seqlens[b])
        for h in range(h_q):
            hk = kv_head_of(h, h_q, h_k)
            bounds = _bounds(n_k, w_sink, w_near, h_offset, hk, h_total, windows)
            ob, lb, _, _ = _rows_forward(q[b, h][None, :], kc[b, hk, :n_k], vc[b, hk, :n_k],
                                         np.array([0]), 1, n_k, bounds, scale)
            o[b, h], lse[b, h] = ob[0], lb[0]
    return o, lse


def _seq_slices(cu_q, cu_k):
    cu_q = [int(x) for x in cu_q]
    cu_k = [int(x) for x in cu_k]
    return [(slice(cu_q[b], cu_q[b + 1]), slice(cu_k[b], cu_k[b + 1])) for b in range(len(cu_q) - 1)]


def forward_varlen(q, k, v, cu_q, cu_k, w_sink, w_near, scale, h_total=None, h_offset=0, windows=None):
    """Forward of a ragged batch: sequence b has queries cu_q[b] .. cu_q[b+1] of
    the packed q [H_q, N_q, d] and keys cu_k[b] .. cu_k[b+1] of k, v [H_k, N_k, d];
    each sequence is its own attention problem, its queries aligned to the end
    of its own keys (Eq. fwa_distance), run through ``forward`` one at a time.
    Returns (O [H_q, N_q, d], LSE [H_q, N_q])."""
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    o = np.zeros((q.shape[0], q.shape[1], v.shape[2]))
    lse = np.zeros((q.shape[0], q.shape[1]))
    for sq, sk in _seq_slices(cu_q, cu_k):
        if sq.stop == sq.start:
            continue
        ob, lb = forward(q[None, :, sq], k[None, :, sk], v[None, :, sk], w_sink, w_near, scale, h_total, h_offset,
                         windows=windows)
        o[:, sq], lse[:, sq] = ob[0], lb[0]
    return o, lse


def backward_varlen(q, k, v, do, cu_q, cu_k, w_sink, w_near, scale, h_total=None, h_offset=0, windows=None):
    """Gradient of a ragged batch, one sequence at a time through ``backward``
    (keys of a sequence without queries get zero gradients).
    Returns (dQ, dK, dV, O, LSE) in the packed layouts."""
    q, k, v, do = (np.asarray(x, dtype=np.float64) for x in (q, k, v, do))
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    o = np.zeros_like(do)
    lse = np.zeros((q.shape[0], q.shape[1]))
    for sq, sk in _seq_slices(cu_q, cu_k):
        if sq.stop == sq.start:
            continue
        r = backward(q[None, :, sq], k[None, :, sk], v[None, :, sk], do[None, :, sq], w_sink, w_near, scale,
                     h_total, h_offset, windows=windows)
        dq[:, sq], dk[:, sk], dv[:, sk], o[:, sq], lse[:, sq] = (x[0] for x in r)
    return dq, dk, dv, o, lse
