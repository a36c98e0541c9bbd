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


def tuple_bounds(window):
    """Distance bounds of a four-tuple (sink, near, gap, width) (Sec. 2.1:
    sink width, near width, gap after the near window, long-range width):
    (sink, near, lo, hi) with the long window near + gap <= delta < near + gap + width."""
    sink, near, gap, width = (int(x) for x in window)
    return sink, near, near + gap, near + gap + width


def head_bounds(n_k, w_sink, w_near, h_global, h_total, window=None):
    """(sink, near, lo, hi) of one KV head: from its explicit four-tuple if one
    is given, else from the default rule (Eq. fwa_long_range_span)."""
    if window is not None:
        return tuple_bounds(window)
    lo, hi = long_window_bounds(n_k, w_sink, w_near, h_global, h_total)
    return w_sink, w_near, lo, hi


def visible_mask_bounds(n_q, n_k, sink, near, lo, hi, rows=None, cols=None):
    """Element mask M[i_q, i_k] of A(i_q) = near u sink u long (Eq. fwa_support)
    for the window bounds (sink, near, lo, hi).

    The three windows of Sec. 2.1 are built separately and joined with a
    logical OR, i.e. a set union: a key that lies in two windows is still one
    visible key.  ``rows`` / ``cols`` select query / key positions (default:
    all N_q / all N_k).  Returns a bool array [len(rows), len(cols)].
    """
    iq = np.arange(n_q, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    ik = np.arange(n_k, dtype=np.int64) if cols is None else np.asarray(cols, dtype=np.int64)
    delta = causal_distance(iq[:, None], ik[None, :], n_q, n_k)
    near_w = (delta >= 0) & (delta < near)
    sink_w = (ik[None, :] < sink) & (delta >= 0)
    far = (delta >= lo) & (delta < hi)
    return near_w | sink_w | far


def visible_mask(n_q, n_k, w_sink, w_near, h_global, h_total, rows=None, cols=None):
    """The mask of the default pattern's KV head h_global (Eq. fwa_support)."""
    lo, hi = long_window_bounds(n_k, w_sink, w_near, h_global, h_total)
    return visible_mask_bounds(n_q, n_k, w_sink, w_near, lo, hi, rows, cols)


def m_window_layout(n_k, w_sink, w_near, h_k, m):
    """The m-window layouts of the collective-coverage ablation (App. A.1,
    Table 1): the long-range history is cut into H_k equal-width regions W_1 ..
    W_{H_k}, W_1 next to the near window (the default pattern's long window of
    KV head 0) and W_{H_k} next to the sink; the m regions closest to the near
    window, W_1 .. W_m, are repeated across the H_k KV heads (head h takes
    W_{(h mod m) + 1}), with the shared sink and near windows unchanged.
    Returns one (sink, near, gap, width) tuple per KV head; m = H_k is the
    default pattern."""
    if h_k % m != 0:
        raise ValueError("m must divide the number of KV heads")
    return [window_tuple(n_k, w_sink, w_near, h % m, h_k) for h in range(h_k)]


def visible_set(i_q, n_q, n_k, w_sink, w_near, h_global, h_total, window=None):
    """The same set A_h(i_q), built element by element with Python sets (for
    tiny brute-force checks; independent of the vectorised mask above).  With
    ``window`` = (sink, near, gap, width) the head's explicit four-tuple is used
    as Sec. 2.1 defines it instead of the default rule."""
    if window is None:
        span = max(n_k - w_sink - w_near, 0)
        b_lo = (h_global * span) // h_total
        b_hi = ((h_global + 1) * span) // h_total
        sink_w, near_w, gap, width = w_sink, w_near, b_lo, b_hi - b_lo
    else:
        sink_w, near_w, gap, width = window
    near, sink, far = set(), set(), set()
    for i_k in range(n_k):
        d = i_q + (n_k - n_q) - i_k
        if 0 <= d < near_w:
            near.add(i_k)
        if i_k < sink_w and d >= 0:
            sink.add(i_k)
        if near_w + gap <= d < near_w + gap + width:
            far.add(i_k)
    return near | sink | far


def visible_intervals_bounds(i_q, n_q, n_k, sink, near, lo, hi):
    """A(i_q) for the window bounds (sink, near, lo, hi) as a sorted list of
    disjoint, non-touching half-open key intervals [a, b).

    Each window of Sec. 2.1 is a contiguous run of keys: with c = i_q + N_k - N_q
    the key at distance 0, delta in [x, y) is the key run (c - y, c - x].  The
    runs are clipped to [0, N_k) and merged (union, touching runs joined).
    """
    c = i_q + (n_k - n_q)
    runs = [
        (c - near + 1, c + 1),            # near: 0 <= delta < near
        (0, min(sink, c + 1)),            # sink: i_k < sink and delta >= 0
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


def visible_intervals(i_q, n_q, n_k, w_sink, w_near, h_global, h_total):
    """A_h(i_q) of the default pattern's KV head h_global as disjoint key intervals."""
    lo, hi = long_window_bounds(n_k, w_sink, w_near, h_global, h_total)
    return visible_intervals_bounds(i_q, n_q, n_k, w_sink, w_near, lo, hi)


def support_size(i_q, n_q, n_k, w_sink, w_near, h_global, h_total):
    """|A_h(i_q)|: the number of distinct visible keys of one query."""
    return sum(b - a for a, b in visible_intervals(i_q, n_q, n_k, w_sink, w_near, h_global, h_total))


def support_sizes(n_q, n_k, w_sink, w_near, h_global, h_total):
    """|A_h(i_q)| for every query i_q = 0..N_q-1 of the default pattern as an int64 array."""
    lo, hi = long_window_bounds(n_k, w_sink, w_near, h_global, h_total)
    return support_sizes_bounds(n_q, n_k, w_sink, w_near, lo, hi)


def support_sizes_bounds(n_q, n_k, sink, near, lo, hi):
    """|A(i_q)| for every query i_q = 0..N_q-1 and window bounds (sink, near,
    lo, hi) with lo >= near, as an int64 array.

    Computed per query from the three windows' key runs with inclusion-exclusion
    over their pairwise overlaps (the near and long runs never overlap because
    lo >= near; sink may overlap either).
    """
    if lo < near:
        raise ValueError("the long-range window starts after the near window (gap >= 0)")
    iq = np.arange(n_q, dtype=np.int64)
    c = iq + (n_k - n_q)

    def run(a, b):
        a = np.maximum(a, 0)
        b = np.minimum(b, c + 1)
        return a, np.maximum(b, a)

    na, nb = run(c - near + 1, c + 1)
    sa, sb = run(np.zeros_like(c), np.minimum(sink, c + 1))
    fa, fb = run(c - hi + 1, c - lo + 1)

    def overlap(a1, b1, a2, b2):
        return np.maximum(np.minimum(b1, b2) - np.maximum(a1, a2), 0)

    total = (nb - na) + (sb - sa) + (fb - fa)
    total -= overlap(na, nb, sa, sb) + overlap(fa, fb, sa, sb) + overlap(na, nb, fa, fb)
    # A triple overlap would need near and long to overlap, which lo >= near forbids.
    return total
