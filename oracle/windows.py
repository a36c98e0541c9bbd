"""The CoWA window rule, written out from Sec. 2.1 of the paper.

Test infrastructure (see the package docstring): never used by the product.

Notation follows the paper: N_q, N_k are the query and key lengths, i_q, i_k
zero-based positions, H_q, H_k the QO and KV head counts, w_sink and w_near the
shared prefix-sink and near-diagonal widths.  ``h_total`` is the global number
of KV heads and ``h_global`` a global KV-head index (Eq. fwa_global_head); on
one device h_global = h_local and h_total = H_k.
"""

import numpy as np


def causal_distance(i_q, i_k, n_q, n_k):
    """Bottom-right aligned causal distance (Eq. fwa_distance):
    delta = i_q + (N_k - N_q) - i_k; the key is causal for the query iff delta >= 0."""
    return i_q + (n_k - n_q) - i_k


def kv_head_of(h, h_q, h_k):
    """GQA map of Sec. 2.1: QO head h uses KV head floor(h * H_k / H_q)."""
    return (h * h_k) // h_q


def global_kv_head(rank, h_k_local, h_local):
    """Eq. fwa_global_head: h_global = r * H_k^local + h_local."""
    return rank * h_k_local + h_local


def long_range_span(n_k, w_sink, w_near):
    """Eq. fwa_long_range_span: L = max(N_k - w_sink - w_near, 0)."""
    return max(n_k - w_sink - w_near, 0)


def breakpoints(n_k, w_sink, w_near, h_total):
    """Eq. fwa_long_range_span: b_h = floor(h * L / H_k) for h = 0..H_k, in exact
    integer arithmetic (Python ints never overflow)."""
    span = long_range_span(n_k, w_sink, w_near)
    return [(h * span) // h_total for h in range(h_total + 1)]


def window_tuple(n_k, w_sink, w_near, h_global, h_total):
    """Per-head four-tuple of Sec. 2.1 (sink width, near width, gap after the near
    window, long-range width) = (w_sink, w_near, b_h, b_{h+1} - b_h)."""
    b = breakpoints(n_k, w_sink, w_near, h_total)
    return (w_sink, w_near, b[h_global], b[h_global + 1] - b[h_global])


def long_window_bounds(n_k, w_sink, w_near, h_global, h_total):
    """Distances [lo, hi) of the long-range window of KV head h_global:
    w_near + b_h <= delta < w_near + b_{h+1} (Sec. 2.1, third window)."""
    b = breakpoints(n_k, w_sink, w_near, h_total)
    return w_near + b[h_global], w_near + b[h_global + 1]


def visible_mask(n_q, n_k, w_sink, w_near, h_global, h_total, rows=None, cols=None):
    """Element mask M[i_q, i_k] of the visible-key set A_h(i_q) (Eq. fwa_support).

    The three windows of Sec. 2.1 are built separately and joined with a
    logical OR, i.e. a set union: a key that lies in two windows is still one
    visible key.  ``rows`` / ``cols`` select query / key positions (default:
    all N_q / all N_k).  Returns a bool array [len(rows), len(cols)].
    """
    iq = np.arange(n_q, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    ik = np.arange(n_k, dtype=np.int64) if cols is None else np.asarray(cols, dtype=np.int64)
    delta = causal_distance(iq[:, None], ik[None, :], n_q, n_k)
    lo, hi = long_window_bounds(n_k, w_sink, w_near, h_global, h_total)
    near = (delta >= 0) & (delta < w_near)
    sink = (ik[None, :] < w_sink) & (delta >= 0)
    far = (delta >= lo) & (delta < hi)
    return near | sink | far


def visible_set(i_q, n_q, n_k, w_sink, w_near, h_global, h_total):
    """The same set A_h(i_q), built element by element with Python sets (for
    tiny brute-force checks; independent of the vectorised mask above)."""
    span = max(n_k - w_sink - w_near, 0)
    b_lo = (h_global * span) // h_total
    b_hi = ((h_global + 1) * span) // h_total
    near, sink, far = set(), set(), set()
    for i_k in range(n_k):
        d = i_q + (n_k - n_q) - i_k
        if 0 <= d < w_near:
            near.add(i_k)
        if i_k < w_sink and d >= 0:
            sink.add(i_k)
        if w_near + b_lo <= d < w_near + b_hi:
            far.add(i_k)
    return near | sink | far


def visible_intervals(i_q, n_q, n_k, w_sink, w_near, h_global, h_total):
    """A_h(i_q) as a sorted list of disjoint, non-touching half-open key
    intervals [a, b).

    Each window of Sec. 2.1 is a contiguous run of keys: with c = i_q + N_k - N_q
    the key at distance 0, delta in [x, y) is the key run (c - y, c - x].  The
    runs are clipped to [0, N_k) and merged (union, touching runs joined).
    """
    c = i_q + (n_k - n_q)
    lo, hi = long_window_bounds(n_k, w_sink, w_near, h_global, h_total)
    runs = [
        (c - w_near + 1, c + 1),          # near: 0 <= delta < w_near
        (0, min(w_sink, c + 1)),          # sink: i_k < w_sink and delta >= 0
        (c - hi + 1, c - lo + 1),         # long: lo <= delta < hi
    ]
    clipped = []
    for a, b in runs:
        a, b = max(a, 0), min(b, n_k, c + 1)
        if a < b:
            clipped.append((a, b))
    clipped.sort()
    merged = []
    for a, b in clipped:
        if merged and a <= merged[-1][1]:
            merged[-1] = (merged[-1][0], max(merged[-1][1], b))
        else:
            merged.append((a, b))
    return merged


def support_size(i_q, n_q, n_k, w_sink, w_near, h_global, h_total):
    """|A_h(i_q)|: the number of distinct visible keys of one query."""
    return sum(b - a for a, b in visible_intervals(i_q, n_q, n_k, w_sink, w_near, h_global, h_total))


def support_sizes(n_q, n_k, w_sink, w_near, h_global, h_total):
    """|A_h(i_q)| for every query i_q = 0..N_q-1 as an int64 array.

    Computed per query from the three windows' key runs with inclusion-exclusion
    over their pairwise overlaps (the near and long runs never overlap because
    lo >= w_near; sink may overlap either).
    """
    iq = np.arange(n_q, dtype=np.int64)
    c = iq + (n_k - n_q)
    lo, hi = long_window_bounds(n_k, w_sink, w_near, h_global, h_total)

    def run(a, b):
        a = np.maximum(a, 0)
        b = np.minimum(b, c + 1)
        return a, np.maximum(b, a)

    na, nb = run(c - w_near + 1, c + 1)
    sa, sb = run(np.zeros_like(c), np.minimum(w_sink, c + 1))
    fa, fb = run(c - hi + 1, c - lo + 1)

    def overlap(a1, b1, a2, b2):
        return np.maximum(np.minimum(b1, b2) - np.maximum(a1, a2), 0)

    total = (nb - na) + (sb - sa) + (fb - fa)
    total -= overlap(na, nb, sa, sb) + overlap(fa, fb, sa, sb) + overlap(na, nb, fa, fb)
    # A triple overlap would need near and long to overlap, which lo >= w_near forbids.
    return total
