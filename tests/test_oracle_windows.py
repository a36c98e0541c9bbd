"""Pins of the oracle's window rule against what the paper fixes.

* printed per-query budgets (App. A.2 table, App. A.1 window split)
* printed mean support s-bar at 4K and 32K (App. A.3)
* collective coverage (Eq. fwa_collective_coverage)
* disjoint, adjacent long-range windows (Eq. fwa_long_range_span)
* final-query count closed form and its cap (Eq. fwa_support_counts, Sec. 2.2)
* global KV-head indexing (Eq. fwa_global_head)
* brute force: three independent constructions of A_h(i_q) agree
"""

import json
import os

import numpy as np
import pytest

from oracle import windows, counts
from conftest import GOLDEN


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_printed_budgets_every_head():
    g = _golden("per_query_budgets.json")
    for n, budget in g["budgets"].items():
        got = counts.final_query_budgets(int(n), g["w_sink"], g["w_near"], g["h_k"])
        assert got == [budget] * g["h_k"], (n, got)


@pytest.mark.parametrize("split", [(1, 1023), (0, 1024), (64, 960), (512, 512)])
def test_printed_mean_support(split):
    g = _golden("mean_support.json")
    w_sink, w_near = split
    assert w_sink + w_near == g["shared_width"]
    for n, sbar in g["mean_support"].items():
        got = counts.mean_support(int(n), w_sink, w_near, g["h_k"])
        assert round(got, g["printed_decimals"]) == sbar, (n, got)


def test_mean_support_discriminates_double_counting():
    """Counting a key once per window it lies in (no set union) must miss the
    printed s-bar: the pin would catch that mistake."""
    g = _golden("mean_support.json")
    n = 4096
    w_sink, w_near = 1, 1023
    tot = 0
    for h in range(g["h_k"]):
        iq = np.arange(n)
        lo, hi = windows.long_window_bounds(n, w_sink, w_near, h, g["h_k"])
        near = np.minimum(iq + 1, w_near)
        sink = np.minimum(iq + 1, w_sink)
        far = np.clip(iq - lo + 1, 0, hi - lo)
        tot += (near + sink + far).sum()
    wrong = tot / (g["h_k"] * n)
    assert round(wrong, 2) != g["mean_support"]["4096"]


def _shapes(rng, count):
    out = []
    for _ in range(count):
        n_k = int(rng.integers(1, 90))
        n_q = int(rng.integers(1, n_k + 1))
        h_total = int(rng.integers(1, 9))
        w_sink = int(rng.integers(0, 12))
        w_near = int(rng.integers(0, 40))
        out.append((n_q, n_k, w_sink, w_near, h_total))
    return out


def test_collective_coverage_exhaustive_tiny():
    for n_k in range(1, 24):
        for n_q in range(1, n_k + 1):
            for h_total in (1, 2, 3, 5, 8):
                for w_sink in (0, 1, 3):
                    for w_near in (1, 2, 5):
                        causal = windows.causal_distance(np.arange(n_q)[:, None], np.arange(n_k)[None, :],
                                                         n_q, n_k) >= 0
                        union = np.zeros_like(causal)
                        for h in range(h_total):
                            union |= windows.visible_mask(n_q, n_k, w_sink, w_near, h, h_total)
                        assert np.array_equal(union, causal), (n_q, n_k, h_total, w_sink, w_near)


def test_collective_coverage_random():
    rng = np.random.default_rng(1)
    for n_q, n_k, w_sink, w_near, h_total in _shapes(rng, 200):
        causal = windows.causal_distance(np.arange(n_q)[:, None], np.arange(n_k)[None, :], n_q, n_k) >= 0
        union = np.zeros_like(causal)
        for h in range(h_total):
            union |= windows.visible_mask(n_q, n_k, w_sink, w_near, h, h_total)
        # holds for w_near = 0 too: the long windows then start at distance 0
        assert np.array_equal(union, causal)


def test_long_windows_tile_the_span():
    rng = np.random.default_rng(2)
    for _ in range(500):
        n_k = int(rng.integers(0, 10 ** 7))
        w_sink = int(rng.integers(0, 5000))
        w_near = int(rng.integers(0, 5000))
        h_total = int(rng.integers(1, 65))
        span = windows.long_range_span(n_k, w_sink, w_near)
        b = windows.breakpoints(n_k, w_sink, w_near, h_total)
        assert b[0] == 0 and b[-1] == span
        assert all(b[i] <= b[i + 1] for i in range(h_total))
        widths = [b[i + 1] - b[i] for i in range(h_total)]
        assert max(widths) - min(widths) <= 1
        # adjacent half-open intervals [w_near + b_h, w_near + b_{h+1}) tile [w_near, w_near + L)
        lo = [windows.long_window_bounds(n_k, w_sink, w_near, h, h_total) for h in range(h_total)]
        assert lo[0][0] == w_near and lo[-1][1] == w_near + span
        assert all(lo[i][1] == lo[i + 1][0] for i in range(h_total - 1))


def test_long_windows_pairwise_disjoint_elements():
    rng = np.random.default_rng(3)
    for n_q, n_k, w_sink, w_near, h_total in _shapes(rng, 100):
        delta = windows.causal_distance(np.arange(n_q)[:, None], np.arange(n_k)[None, :], n_q, n_k)
        owners = np.zeros(delta.shape, dtype=np.int64)
        for h in range(h_total):
            lo, hi = windows.long_window_bounds(n_k, w_sink, w_near, h, h_total)
            owners += ((delta >= lo) & (delta < hi))
        assert owners.max(initial=0) <= 1


def test_final_query_count_closed_form():
    rng = np.random.default_rng(4)
    for _ in range(300):
        h_total = int(rng.integers(1, 9))
        n_k = int(rng.integers(1, 400))
        n_q = int(rng.integers(1, n_k + 1))
        w_sink = int(rng.integers(0, 50))
        w_near = int(rng.integers(0, 120))
        sizes = [int(windows.visible_mask(n_q, n_k, w_sink, w_near, h, h_total, rows=[n_q - 1]).sum())
                 for h in range(h_total)]
        if w_sink + w_near <= n_k:
            assert sum(sizes) == h_total * (w_sink + w_near) + windows.long_range_span(n_k, w_sink, w_near)
        else:
            # near and sink already cover the causal prefix: every head sees all N_k keys, capped
            assert sizes == [n_k] * h_total


def test_dense_reduction_of_the_pattern():
    rng = np.random.default_rng(5)
    for n_q, n_k, w_sink, w_near, _ in _shapes(rng, 100):
        causal = windows.causal_distance(np.arange(n_q)[:, None], np.arange(n_k)[None, :], n_q, n_k) >= 0
        # a single KV head sees the whole causal prefix (Sec. 2.2, last paragraph)
        assert np.array_equal(windows.visible_mask(n_q, n_k, w_sink, max(w_near, 1), 0, 1), causal)
        # windows spanning the sequence: every head is dense causal
        for h in range(4):
            assert np.array_equal(windows.visible_mask(n_q, n_k, 0, n_k, h, 4), causal)
            assert np.array_equal(windows.visible_mask(n_q, n_k, n_k - n_k // 2, n_k // 2 + 1, h, 4), causal)


def test_three_constructions_agree():
    rng = np.random.default_rng(6)
    for n_q, n_k, w_sink, w_near, h_total in _shapes(rng, 60):
        for h in range(h_total):
            m = windows.visible_mask(n_q, n_k, w_sink, w_near, h, h_total)
            sizes = windows.support_sizes(n_q, n_k, w_sink, w_near, h, h_total)
            for i_q in range(n_q):
                s = windows.visible_set(i_q, n_q, n_k, w_sink, w_near, h, h_total)
                assert set(np.nonzero(m[i_q])[0].tolist()) == s
                runs = windows.visible_intervals(i_q, n_q, n_k, w_sink, w_near, h, h_total)
                from_runs = set()
                for a, b in runs:
                    from_runs |= set(range(a, b))
                assert from_runs == s
                # runs are disjoint and not touching
                assert all(runs[t][1] < runs[t + 1][0] for t in range(len(runs) - 1))
                assert sizes[i_q] == len(s)


def test_global_head_indexing():
    """A device holding KV heads [r*H_loc, (r+1)*H_loc) must use the global index
    and the global H_k in the breakpoints (Eq. fwa_global_head)."""
    n, w_sink, w_near, h_total = 300, 5, 20, 8
    for tp in (1, 2, 4, 8):
        h_loc = h_total // tp
        for r in range(tp):
            for hl in range(h_loc):
                hg = windows.global_kv_head(r, h_loc, hl)
                assert hg == r * h_loc + hl
                assert windows.window_tuple(n, w_sink, w_near, hg, h_total) == \
                    (w_sink, w_near, *[(hg * 275) // 8, ((hg + 1) * 275) // 8 - (hg * 275) // 8])
    # a local index with the local head count gives a different (wrong) partition
    assert windows.long_window_bounds(n, w_sink, w_near, 1, 2) != windows.long_window_bounds(n, w_sink, w_near, 1, 8)


def test_gqa_map():
    # Sec. 2.1: contiguous groups of H_q / H_k QO heads share a KV head
    assert [windows.kv_head_of(h, 4, 2) for h in range(4)] == [0, 0, 1, 1]
    assert [windows.kv_head_of(h, 32, 8) for h in range(32)] == [h // 4 for h in range(32)]
    assert [windows.kv_head_of(h, 8, 8) for h in range(8)] == list(range(8))
