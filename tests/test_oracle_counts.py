"""Pins of the oracle's work accounting (oracle/counts.py) and of the
attention oracle's multi-block path.

* Per-Selected-Token FLOPs (App. A.2 / A.5 tables): the forward FLOPs of one
  selected key for one query over all QO heads, counts.fwd_flops(h_q, d),
  equal the printed 2 h (d_qk + d_v) values (`tests/golden/accounting.json`).
* The per-token core-attention cost of App. A.3, 8 s h d_qk + 6 s h d_v with
  backward QK recomputation, is the forward plus backward count per legal
  pair (fwd 4d + bwd 10d at d_qk = d_v = d).
* Decoding bytes: one rank of the 8-way KV-head split at 128K reads the
  visible K and V rows plus q, O and LSE; in MiB this reproduces the printed
  peak decoding-operator memory of CoWA (8.441) and FullAttn (64.004) at
  three decimals, for every rank.
* attention.forward / backward split queries into row blocks that gather only
  the keys some row can see; on shapes longer than one block (several
  blocks, a ragged last one) they still equal torch's float64 SDPA with the
  explicit mask and its autograd.
"""

import json
import os

import numpy as np
import torch

from conftest import GOLDEN
from oracle import attention, counts, windows


def _golden():
    with open(os.path.join(GOLDEN, "accounting.json")) as f:
        return json.load(f)


def test_pst_flops_match_printed_tables():
    for row in _golden()["pst_flops"]:
        assert row["d_qk"] == row["d_v"]
        assert counts.fwd_flops(row["h_q"], row["d_qk"]) == row["printed"]


def test_forward_plus_backward_is_the_per_token_cost():
    # App. A.3: 8 s h d_qk + 6 s h d_v per token with s selected keys per QO head
    for d in (64, 128):
        for pairs in (1, 17, 12345):
            assert counts.fwd_flops(pairs, d) + counts.bwd_flops(pairs, d) == 8 * pairs * d + 6 * pairs * d
            assert counts.bwd_flops(pairs, d) > 2 * counts.fwd_flops(pairs, d)  # backward recomputes QK


def test_decode_bytes_match_printed_decoding_memory():
    g = _golden()
    sh, mem = g["decode_shape"], g["decode_memory_mib"]
    for rank in range(sh["h_total"]):
        b = counts.decode_bytes([sh["n_k"]], sh["h_q"], sh["h_k"], sh["d"], sh["w_sink"], sh["w_near"],
                                h_total=sh["h_total"], h_offset=rank)
        assert round(b / 2 ** 20, 3) == mem["cowa"], rank
        keys = int(counts.decode_visible_keys([sh["n_k"]], sh["w_sink"], sh["w_near"], sh["h_k"], sh["h_total"],
                                              rank).sum())
        assert keys == 17280  # the printed per-QO-head budget at 128K
    dense = counts.decode_bytes([sh["n_k"]], sh["h_q"], sh["h_k"], sh["d"], 0, sh["n_k"])
    assert round(dense / 2 ** 20, 3) == mem["fullattn"]


def _sdpa_masked(q, k, v, masks, scale, do=None):
    h_q, h_k = q.shape[1], k.shape[1]
    m = torch.from_numpy(np.stack(masks)).repeat_interleave(h_q // h_k, dim=0)[None]
    tq, tk, tv = (torch.from_numpy(x.copy()).requires_grad_(do is not None) for x in (q, k, v))
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=m, scale=scale, enable_gqa=True)
    if do is None:
        return out.detach().numpy(), None
    out.backward(torch.from_numpy(do))
    return out.detach().numpy(), (tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy())


def test_multi_block_forward_and_backward_vs_torch():
    rng = np.random.default_rng(31)
    n_q, n_k, h_q, h_k, d, w_sink, w_near, scale = 600, 650, 4, 2, 16, 7, 50, 0.3
    q = rng.standard_normal((1, h_q, n_q, d))
    k = rng.standard_normal((1, h_k, n_k, d))
    v = rng.standard_normal((1, h_k, n_k, d))
    do = rng.standard_normal((1, h_q, n_q, d))
    masks = [windows.visible_mask(n_q, n_k, w_sink, w_near, h, h_k) for h in range(h_k)]
    o_ref, (dq_r, dk_r, dv_r) = _sdpa_masked(q, k, v, masks, scale, do)
    o, _ = attention.forward(q, k, v, w_sink, w_near, scale)            # blocks of 256 rows: 256, 256, 88
    o_small, _ = attention.forward(q, k, v, w_sink, w_near, scale, block=97)
    np.testing.assert_allclose(o, o_ref, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(o_small, o_ref, rtol=1e-11, atol=1e-12)
    dq, dk, dv, o2, _ = attention.backward(q, k, v, do, w_sink, w_near, scale)
    np.testing.assert_allclose(o2, o_ref, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dq, dq_r, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(dk, dk_r, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(dv, dv_r, rtol=1e-9, atol=1e-10)
