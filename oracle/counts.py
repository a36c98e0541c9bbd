"""Support sizes, legal-pair counts and FLOP accounting.

Test infrastructure (see the package docstring): never used by the product.

* Legal pairs: the number of (query, key) pairs with the key in A_h(i_q),
  summed over queries, QO heads and the batch.  The attention work of every
  kernel is priced on these pairs only (dense tiles skipped or masked do not
  count).
* FLOPs (App. A.2 and A.3, one multiply-accumulate = 2 FLOPs, d_qk = d_v = d):
  the forward does QK and PV, 2d + 2d = 4d per legal pair and QO head; the
  backward recomputes QK and then does dP, dV, dK and dQ, 5 * 2d = 10d.  This
  is the paper's per-token cost 8 s h d_qk + 6 s h d_v split as fwd 4d + bwd
  10d (the paper's total is 14d per pair).
* Decode bytes: the K and V rows of every visible key of every (sequence, KV
  head) are read once, plus q, O and LSE.
"""

import numpy as np

from .windows import support_sizes


def support_table(n_q, n_k, w_sink, w_near, h_k, h_total=None, h_offset=0):
    """|A_h(i_q)| for every local KV head and query: int64 [H_k, N_q]."""
    h_total = h_k if h_total is None else h_total
    return np.stack([support_sizes(n_q, n_k, w_sink, w_near, h_offset + h, h_total)
                     for h in range(h_k)])


def legal_pairs_per_kv_head(n_q, n_k, w_sink, w_near, h_k, h_total=None, h_offset=0):
    """Legal pairs of one query sequence for each local KV head (one QO head)."""
    return support_table(n_q, n_k, w_sink, w_near, h_k, h_total, h_offset).sum(axis=1)


def legal_pairs(batch, n_q, n_k, h_q, h_k, w_sink, w_near, h_total=None, h_offset=0):
    """Total legal pairs over the batch and all QO heads (each QO head of a
    group sees its KV head's set)."""
    per = legal_pairs_per_kv_head(n_q, n_k, w_sink, w_near, h_k, h_total, h_offset)
    return int(batch * (h_q // h_k) * per.sum())


def mean_support(n, w_sink, w_near, h_k):
    """s-bar of App. A.3: the exact support size averaged over all query
    positions and QO heads of a training sequence (N_q = N_k = n).  With equal
    QO-head groups this is the average over KV heads."""
    return float(support_table(n, n, w_sink, w_near, h_k).mean())


def final_query_budgets(n_k, w_sink, w_near, h_k):
    """|A_h(N_q - 1)| per KV head at the final query (Sec. 2.2)."""
    return [int(support_sizes(1, n_k, w_sink, w_near, h, h_k)[0]) for h in range(h_k)]


def fwd_flops(pairs, d):
    return 4 * d * pairs


def bwd_flops(pairs, d):
    return 10 * d * pairs


def dense_causal_pairs(batch, n_q, n_k, h_q):
    """Legal pairs of dense causal attention with the same alignment."""
    off = n_k - n_q
    per_row = np.minimum(np.arange(n_q, dtype=np.int64) + off + 1, n_k)
    return int(batch * h_q * per_row.sum())


def decode_visible_keys(seqlens, w_sink, w_near, h_k, h_total=None, h_offset=0):
    """Visible keys per (sequence, local KV head) at one decoding step: int64 [B, H_k]."""
    h_total = h_k if h_total is None else h_total
    out = np.zeros((len(seqlens), h_k), dtype=np.int64)
    for b, n_k in enumerate(seqlens):
        for h in range(h_k):
            out[b, h] = support_sizes(1, int(n_k), w_sink, w_near, h_offset + h, h_total)[0]
    return out


def decode_bytes(seqlens, h_q, h_k, d, w_sink, w_near, elem_bytes=2, h_total=None, h_offset=0):
    """Algorithmic HBM bytes of one decoding step: visible K and V rows, the
    query, the output and the fp32 LSE."""
    keys = int(decode_visible_keys(seqlens, w_sink, w_near, h_k, h_total, h_offset).sum())
    b = len(seqlens)
    return 2 * keys * d * elem_bytes + b * h_q * d * elem_bytes * 2 + b * h_q * 4
