"""Pins of the oracle's block schedule (Sec. 2.3: J_h(i), its inverse I_h(j),
FULL vs boundary blocks).

The two constructions share nothing but the window definitions: method A
reduces the element mask over each tile, method B marks tiles from each
query's merged key runs.  Regression values for the measured workloads were
computed independently (element-mask brute force) and are restated here.
"""

import numpy as np
import pytest

from oracle import schedule, windows

KEYS = ("fwd_row_ptr", "fwd_ent", "bwd_col_ptr", "bwd_ent")


def _same(a, b):
    return all(np.array_equal(a[k], b[k]) for k in KEYS)


def _random_cases(rng, count):
    cases = []
    for _ in range(count):
        n_k = int(rng.integers(1, 700))
        n_q = int(rng.integers(1, n_k + 1))
        tq = int(rng.choice([16, 32, 64, 128]))
        tk = int(rng.choice([16, 32, 64, 128]))
        h_total = int(rng.integers(1, 9))
        h_k = int(rng.integers(1, h_total + 1))
        h_off = int(rng.integers(0, h_total - h_k + 1))
        w_sink = int(rng.integers(0, 80))
        w_near = int(rng.integers(0, 300))
        cases.append((n_q, n_k, tq, tk, w_sink, w_near, h_k, h_total, h_off))
    return cases


def test_two_methods_agree_random():
    rng = np.random.default_rng(11)
    for c in _random_cases(rng, 120):
        a = schedule.build(*c, method="bruteforce")
        b = schedule.build(*c, method="intervals")
        assert _same(a, b), c


def test_two_methods_agree_workload_small():
    # 512 tokens, tile 32, sink 16, near 64, two KV heads; and the 8K workload
    for c in [(512, 512, 32, 32, 16, 64, 2, 2, 0), (8192, 8192, 64, 64, 64, 1024, 8, 8, 0)]:
        assert _same(schedule.build(*c, method="bruteforce"), schedule.build(*c, method="intervals"))


def test_listed_iff_a_legal_pair_and_full_iff_all_legal():
    rng = np.random.default_rng(12)
    for (n_q, n_k, tq, tk, w_sink, w_near, h_k, h_total, h_off) in _random_cases(rng, 40):
        s = schedule.build(n_q, n_k, tq, tk, w_sink, w_near, h_k, h_total, h_off, method="intervals")
        for h in range(h_k):
            m = windows.visible_mask(n_q, n_k, w_sink, w_near, h_off + h, h_total)
            for i in range(s["n_qt"]):
                row = s["fwd_ent"][s["fwd_row_ptr"][h * s["n_qt"] + i]:s["fwd_row_ptr"][h * s["n_qt"] + i + 1]]
                js = [int(e) >> 1 for e in row]
                assert js == sorted(js, reverse=True)
                for j in range(s["n_kt"]):
                    rect = m[i * tq:(i + 1) * tq, j * tk:(j + 1) * tk]
                    in_bounds = (i + 1) * tq <= n_q and (j + 1) * tk <= n_k
                    assert (j in js) == bool(rect.any())
                    if j in js:
                        partial = int(row[js.index(j)]) & 1
                        assert partial == int(not (in_bounds and rect.all()))


def test_bwd_is_transpose_of_fwd():
    rng = np.random.default_rng(13)
    for c in _random_cases(rng, 40):
        s = schedule.build(*c)
        h_k, n_qt, n_kt = c[6], s["n_qt"], s["n_kt"]
        pairs_f, pairs_b = set(), set()
        for h in range(h_k):
            for i in range(n_qt):
                r = h * n_qt + i
                for e in s["fwd_ent"][s["fwd_row_ptr"][r]:s["fwd_row_ptr"][r + 1]]:
                    pairs_f.add((h, i, int(e) >> 1, int(e) & 1))
            for j in range(n_kt):
                col = s["bwd_ent"][s["bwd_col_ptr"][h * n_kt + j]:s["bwd_col_ptr"][h * n_kt + j + 1]]
                is_ = [int(e) >> 1 for e in col]
                assert is_ == sorted(is_)
                for e in col:
                    pairs_b.add((h, int(e) >> 1, j, int(e) & 1))
        assert pairs_f == pairs_b
        assert len(s["fwd_ent"]) == len(s["bwd_ent"])


def _nnz_per_head(s, h_k):
    n = s["n_qt"]
    return [int(s["fwd_row_ptr"][n * (h + 1)] - s["fwd_row_ptr"][n * h]) for h in range(h_k)]


def test_regression_fwd_fp32_t512():
    s = schedule.build(512, 512, 32, 32, 16, 64, 2)
    assert _nnz_per_head(s, 2) == [121, 86]
    assert [int(s["full"][h].sum()) for h in range(2)] == [85, 36]


def test_regression_bf16_t8k():
    s = schedule.build(8192, 8192, 64, 64, 64, 1024, 8)
    assert _nnz_per_head(s, 8) == [3600, 3599, 3375, 3151, 2927, 2703, 2479, 2256]


@pytest.mark.slow
def test_regression_bf16_t128k():
    s = schedule.build(131072, 131072, 128, 128, 128, 4096, 8)
    assert _nnz_per_head(s, 8) == [149389, 135748, 120124, 104500, 88876, 73252, 57628, 42005]
    assert int(np.diff(s["fwd_row_ptr"]).max()) == 160


def test_global_offset_matches_full_device():
    """A device holding global KV head r alone builds the rows of head r of the
    all-heads schedule (Eq. fwa_global_head)."""
    full = schedule.build(1000, 1000, 64, 64, 7, 100, 4)
    n_qt = full["n_qt"]
    for r in range(4):
        one = schedule.build(1000, 1000, 64, 64, 7, 100, 1, h_total=4, h_offset=r)
        lo, hi = full["fwd_row_ptr"][r * n_qt], full["fwd_row_ptr"][(r + 1) * n_qt]
        assert np.array_equal(one["fwd_ent"], full["fwd_ent"][lo:hi])
        assert np.array_equal(one["fwd_row_ptr"], full["fwd_row_ptr"][r * n_qt:(r + 1) * n_qt + 1] - lo)
