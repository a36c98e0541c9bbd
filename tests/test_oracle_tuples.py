"""Pins of the oracle's explicit per-head windows and ragged batches.

Explicit windows (Sec. 2.1: each head's windows are a four-tuple of sink
width, near width, gap after the near window and long-range width, and the
same interface permits head-specific widths and gaps):
* the default rule's tuples reproduce the default rule exactly (two
  independent constructions: the per-element Python sets and the vectorised
  mask);
* random tuples: vectorised mask, key intervals and support sizes against
  the per-element Python sets;
* the m-window layouts of App. A.1 cover 12.5 / 25 / 50 / 100 % of the
  long-range history (Table 1) with matched per-head widths;
* attention with explicit tuples against torch's CPU float64 SDPA (forward)
  and autograd (gradient) with the brute-force mask; decoding equals the last
  forward row.

Ragged batches (Eq. fwa_distance aligns each sequence's queries to the end of
its own keys):
* equal lengths reproduce the batched oracle;
* the packed problem equals torch SDPA / autograd on the packed tensors with
  a block-diagonal mask built from per-sequence brute-force sets;
* the ragged schedule's two construction methods agree, and a one-sequence
  ragged batch is the ordinary schedule.
"""

import json
import os

import numpy as np
import pytest
import torch

from conftest import GOLDEN
from oracle import attention, windows as ow, schedule as osched


def _brute_mask(n_q, n_k, window):
    m = np.zeros((n_q, n_k), dtype=bool)
    for i in range(n_q):
        for j in ow.visible_set(i, n_q, n_k, 0, 0, 0, 1, window=window):
            m[i, j] = True
    return m


def _random_tuple(rng, n_k):
    return (int(rng.integers(0, n_k // 2 + 2)), int(rng.integers(0, n_k // 2 + 2)),
            int(rng.integers(0, n_k + 2)), int(rng.integers(0, n_k + 2)))


@pytest.mark.parametrize("n_q,n_k,ws,wn,ht", [(30, 30, 3, 5, 4), (17, 45, 0, 7, 3), (50, 50, 60, 10, 8),
                                              (9, 9, 0, 0, 2), (40, 64, 2, 1, 5)])
def test_default_tuples_reproduce_default_rule(n_q, n_k, ws, wn, ht):
    for hg in range(ht):
        tup = ow.window_tuple(n_k, ws, wn, hg, ht)
        for i in range(n_q):
            assert ow.visible_set(i, n_q, n_k, ws, wn, hg, ht, window=tup) == \
                ow.visible_set(i, n_q, n_k, ws, wn, hg, ht)
        lo, hi = ow.long_window_bounds(n_k, ws, wn, hg, ht)
        assert ow.head_bounds(n_k, ws, wn, hg, ht, window=tup) == (ws, wn, lo, hi)
        assert np.array_equal(ow.visible_mask_bounds(n_q, n_k, *ow.tuple_bounds(tup)),
                              ow.visible_mask(n_q, n_k, ws, wn, hg, ht))


def test_random_tuples_against_bruteforce():
    rng = np.random.default_rng(3)
    for _ in range(40):
        n_k = int(rng.integers(1, 60))
        n_q = int(rng.integers(1, n_k + 1))
        tup = _random_tuple(rng, n_k)
        brute = _brute_mask(n_q, n_k, tup)
        bounds = ow.tuple_bounds(tup)
        assert np.array_equal(ow.visible_mask_bounds(n_q, n_k, *bounds), brute), tup
        for i in range(n_q):
            keys = set()
            for a, b in ow.visible_intervals_bounds(i, n_q, n_k, *bounds):
                keys |= set(range(a, b))
            assert keys == set(np.nonzero(brute[i])[0].tolist())
        assert np.array_equal(ow.support_sizes_bounds(n_q, n_k, *bounds), brute.sum(axis=1))


def test_m_window_layouts_cover_table1_fractions():
    """Table 1: with matched per-head widths, the 1-, 2-, 4- and 8-window
    layouts cover 12.5, 25, 50 and 100 % of the long-range history.  Measured
    on the final query of a sequence whose long-range span L = N - w_sink -
    w_near is a multiple of 8: the keys that some head sees through a
    long-range window and no head through the shared sink or near windows,
    divided by L."""
    g = json.load(open(os.path.join(GOLDEN, "collective_coverage.json")))
    h_k, ws, wn = g["h_k"], g["w_sink"], g["w_near"]
    for n in (4096, 8192):
        span = ow.long_range_span(n, ws, wn)
        assert span % h_k == 0
        for m_str, pct in g["long_range_coverage_percent"].items():
            m = int(m_str)
            tuples = ow.m_window_layout(n, ws, wn, h_k, m)
            assert all(t[3] == span // h_k for t in tuples)          # matched per-head widths
            assert len({t[2] for t in tuples}) == m                   # m distinct long windows
            union = np.zeros(n, dtype=bool)
            for t in tuples:
                union |= ow.visible_mask_bounds(1, n, *ow.tuple_bounds(t), rows=[0])[0]
            shared = ow.visible_mask_bounds(1, n, ws, wn, wn, wn, rows=[0])[0]  # sink and near only
            covered = int((union & ~shared).sum())
            assert covered / span * 100 == pytest.approx(pct), (n, m)
    # the 8-window layout is the default pattern
    assert ow.m_window_layout(8192, ws, wn, h_k, h_k) == [ow.window_tuple(8192, ws, wn, h, h_k)
                                                           for h in range(h_k)]


def _head_masks(n_q, n_k, tuples):
    return [_brute_mask(n_q, n_k, t) for t in tuples]


def _sdpa_masked(q, k, v, masks, scale):
    h_q, h_k = q.shape[1], k.shape[1]
    m = torch.from_numpy(np.stack(masks)).repeat_interleave(h_q // h_k, dim=0)[None]
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), attn_mask=m, scale=scale, enable_gqa=True)


def test_forward_and_gradient_with_tuples():
    rng = np.random.default_rng(8)
    n_q, n_k, h_q, h_k, d = 23, 41, 4, 2, 8
    tuples = [(2, 5, 3, 9), (0, 9, 0, 30)]
    q, k, v, do = (rng.standard_normal(s) for s in ((1, h_q, n_q, d), (1, h_k, n_k, d), (1, h_k, n_k, d),
                                                    (1, h_q, n_q, d)))
    scale = 0.3
    masks = _head_masks(n_q, n_k, tuples)
    o, lse = attention.forward(q, k, v, 0, 0, scale, windows=tuples)
    ref = _sdpa_masked(q, k, v, masks, scale).numpy()
    assert np.allclose(o, ref, atol=1e-12, rtol=1e-12)
    tq, tk, tv = (torch.from_numpy(x).requires_grad_(True) for x in (q, k, v))
    m = torch.from_numpy(np.stack(masks)).repeat_interleave(h_q // h_k, dim=0)[None]
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=m, scale=scale, enable_gqa=True)
    (out * torch.from_numpy(do)).sum().backward()
    dq, dk, dv, _, _ = attention.backward(q, k, v, do, 0, 0, scale, windows=tuples)
    for a, b in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        assert np.allclose(a, b.numpy(), atol=1e-11, rtol=1e-11)
    # decoding with the same tuples is the last forward row of a sequence that ends there
    od, ld = attention.decode(q[:, :, -1], k, v, [n_k], 0, 0, scale, windows=tuples)
    assert np.allclose(od, o[:, :, -1], atol=1e-12) and np.allclose(ld, lse[:, :, -1], atol=1e-12)


def _packed(rng, cu_q, cu_k, h_q, h_k, d):
    return (rng.standard_normal((h_q, cu_q[-1], d)), rng.standard_normal((h_k, cu_k[-1], d)),
            rng.standard_normal((h_k, cu_k[-1], d)), rng.standard_normal((h_q, cu_q[-1], d)))


def test_varlen_equal_lengths_reproduce_batched_oracle():
    rng = np.random.default_rng(4)
    bsz, n_q, n_k, h_q, h_k, d = 3, 20, 33, 4, 2, 8
    q, k, v, do = (rng.standard_normal(s) for s in ((bsz, h_q, n_q, d), (bsz, h_k, n_k, d), (bsz, h_k, n_k, d),
                                                    (bsz, h_q, n_q, d)))
    ref = attention.backward(q, k, v, do, 2, 5, 0.4, h_total=4, h_offset=1)
    pack = lambda x: np.concatenate(list(x), axis=1)  # [B, H, N, d] -> [H, B N, d]
    cu_q, cu_k = [n_q * b for b in range(bsz + 1)], [n_k * b for b in range(bsz + 1)]
    got = attention.backward_varlen(pack(q), pack(k), pack(v), pack(do), cu_q, cu_k, 2, 5, 0.4, h_total=4,
                                    h_offset=1)
    for r, g in zip(ref[:4], got[:4]):
        assert np.allclose(pack(r), g, atol=1e-13)
    assert np.allclose(np.concatenate(list(ref[4]), axis=1), got[4], atol=1e-13)


@pytest.mark.parametrize("tuples", [None, [(1, 4, 2, 7), (3, 2, 0, 11)]])
def test_varlen_against_block_diagonal_sdpa(tuples):
    """The packed sequences as one attention problem whose mask is block
    diagonal: a query sees keys of its own sequence only, under that
    sequence's own window rule (its own N_k and bottom-right alignment)."""
    rng = np.random.default_rng(5)
    cu_q, cu_k = [0, 5, 5, 21, 40], [0, 12, 19, 21, 70]
    h_q, h_k, d, ws, wn, scale = 4, 2, 8, 2, 3, 0.35
    q, k, v, do = _packed(rng, cu_q, cu_k, h_q, h_k, d)
    masks = []
    for h in range(h_k):
        m = np.zeros((cu_q[-1], cu_k[-1]), dtype=bool)
        for b in range(len(cu_q) - 1):
            n_q, n_k = cu_q[b + 1] - cu_q[b], cu_k[b + 1] - cu_k[b]
            tup = tuples[h] if tuples else ow.window_tuple(n_k, ws, wn, h, h_k)
            m[cu_q[b]:cu_q[b + 1], cu_k[b]:cu_k[b + 1]] = _brute_mask(n_q, n_k, tup)
        masks.append(m)
    tq, tk, tv = (torch.from_numpy(x[None]).requires_grad_(True) for x in (q, k, v))
    mm = torch.from_numpy(np.stack(masks)).repeat_interleave(h_q // h_k, dim=0)[None]
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mm, scale=scale, enable_gqa=True)
    (out * torch.from_numpy(do[None])).sum().backward()
    o, _ = attention.forward_varlen(q, k, v, cu_q, cu_k, ws, wn, scale, windows=tuples)
    assert np.allclose(o, out.detach().numpy()[0], atol=1e-12)
    dq, dk, dv, _, _ = attention.backward_varlen(q, k, v, do, cu_q, cu_k, ws, wn, scale, windows=tuples)
    for a, b in ((dq, tq.grad), (dk, tk.grad), (dv, tv.grad)):
        assert np.allclose(a, b.numpy()[0], atol=1e-11)
    # keys of the sequence without queries (keys 12..18) get zero gradients
    assert not dk[:, 12:19].any() and not dv[:, 12:19].any()


def test_varlen_schedule_methods_agree():
    cu_q, cu_k = [0, 70, 70, 200, 233], [0, 100, 131, 300, 500]
    for tuples in (None, [(1, 16, 5, 40), (0, 33, 0, 100), (50, 0, 3, 3)]):
        a = osched.build_varlen(cu_q, cu_k, 32, 64, 4, 20, 3, method="intervals", windows=tuples)
        b = osched.build_varlen(cu_q, cu_k, 32, 64, 4, 20, 3, method="bruteforce", windows=tuples)
        for key in ("fwd_row_ptr", "fwd_ent", "bwd_col_ptr", "bwd_ent"):
            assert np.array_equal(a[key], b[key]), key
    one = osched.build_varlen([0, 150], [0, 300], 32, 64, 4, 20, 3)
    ref = osched.build(150, 300, 32, 64, 4, 20, 3)
    for key in ("fwd_row_ptr", "fwd_ent", "bwd_col_ptr", "bwd_ent"):
        assert np.array_equal(one[key], ref[key]), key
