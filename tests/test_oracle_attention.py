"""Pins of the oracle's attention forward, gradient and decode.

* reductions to dense causal attention (H_k = 1; windows spanning the
  sequence; Sec. 2.2) against torch's CPU float64 scaled_dot_product_attention
  and against a separately written dense softmax
* general CoWA against torch's CPU float64 SDPA with the boolean mask of the
  visible sets and torch's own GQA head map
* brute force: per-row pure-Python softmax over the explicit visible set
* invariants: a constant added to every key leaves O unchanged; V = 1 gives O = 1
* exact gradient (Sec. 2.3, backward execution): torch autograd in float64 and
  central finite differences
* decoding (Sec. 2.3) equals the last row of the full forward
* sampled-row helpers equal the full computation
* planted mistakes in copies of the oracle are caught
"""

import math

import numpy as np
import pytest
import torch

from oracle import attention, windows, counts


def _rand(rng, shape):
    return rng.standard_normal(shape)


def _case(rng, bsz, h_q, h_k, n_q, n_k, d):
    q = _rand(rng, (bsz, h_q, n_q, d))
    k = _rand(rng, (bsz, h_k, n_k, d))
    v = _rand(rng, (bsz, h_k, n_k, d))
    do = _rand(rng, (bsz, h_q, n_q, d))
    return q, k, v, do


def _sdpa(q, k, v, mask_per_kv_head, scale):
    """torch SDPA on CPU float64 with an explicit boolean mask per QO head
    (each QO head takes its KV head's mask via torch's own GQA expansion)."""
    h_q, h_k = q.shape[1], k.shape[1]
    m = torch.from_numpy(np.stack(mask_per_kv_head))            # [H_k, N_q, N_k]
    m = m.repeat_interleave(h_q // h_k, dim=0)[None]             # [1, H_q, N_q, N_k]
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), attn_mask=m, scale=scale,
        enable_gqa=True)


def _dense_causal(q, k, v, scale):
    """Dense bottom-right causal attention written out independently (GQA by
    repeating KV heads), returning O and LSE."""
    bsz, h_q, n_q, _ = q.shape
    h_k, n_k = k.shape[1], k.shape[2]
    o = np.zeros_like(q)
    lse = np.zeros((bsz, h_q, n_q))
    for b in range(bsz):
        for h in range(h_q):
            kk, vv = k[b, h // (h_q // h_k)], v[b, h // (h_q // h_k)]
            for i in range(n_q):
                last = i + n_k - n_q
                s = scale * (kk[:last + 1] @ q[b, h, i])
                mx = s.max()
                e = np.exp(s - mx)
                o[b, h, i] = e @ vv[:last + 1] / e.sum()
                lse[b, h, i] = mx + math.log(e.sum())
    return o, lse


@pytest.mark.parametrize("n_q,n_k", [(40, 40), (17, 53), (1, 9)])
def test_single_kv_head_is_dense_causal(n_q, n_k):
    rng = np.random.default_rng(21)
    q, k, v, _ = _case(rng, 2, 3, 1, n_q, n_k, 16)
    o, lse = attention.forward(q, k, v, w_sink=3, w_near=5, scale=0.3)
    od, ld = _dense_causal(q, k, v, 0.3)
    np.testing.assert_allclose(o, od, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse, ld, rtol=1e-12, atol=1e-12)
    if n_q == n_k:
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q), torch.from_numpy(k), torch.from_numpy(v), is_causal=True, scale=0.3,
            enable_gqa=True).numpy()
        np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)


def test_spanning_windows_are_dense_causal():
    rng = np.random.default_rng(22)
    q, k, v, _ = _case(rng, 1, 8, 4, 33, 33, 8)
    for w_sink, w_near in [(0, 33), (10, 23), (40, 40)]:
        o, lse = attention.forward(q, k, v, w_sink, w_near, scale=0.5)
        od, ld = _dense_causal(q, k, v, 0.5)
        np.testing.assert_allclose(o, od, rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse, ld, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("shape", [(1, 4, 2, 64, 64, 16, 3, 9), (2, 8, 4, 50, 77, 8, 5, 11),
                                   (1, 6, 3, 31, 31, 4, 0, 7), (1, 2, 2, 90, 90, 8, 12, 1)])
def test_general_pattern_vs_torch_sdpa(shape):
    bsz, h_q, h_k, n_q, n_k, d, w_sink, w_near = shape
    rng = np.random.default_rng(23)
    q, k, v, _ = _case(rng, bsz, h_q, h_k, n_q, n_k, d)
    o, _ = attention.forward(q, k, v, w_sink, w_near, scale=0.25)
    masks = [windows.visible_mask(n_q, n_k, w_sink, w_near, h, h_k) for h in range(h_k)]
    ref = _sdpa(q, k, v, masks, 0.25).numpy()
    np.testing.assert_allclose(o, ref, rtol=1e-12, atol=1e-12)


def test_bruteforce_rows():
    rng = np.random.default_rng(24)
    bsz, h_q, h_k, n_q, n_k, d = 1, 4, 2, 23, 29, 3
    q, k, v, _ = _case(rng, bsz, h_q, h_k, n_q, n_k, d)
    w_sink, w_near, scale = 2, 4, 0.7
    o, lse = attention.forward(q, k, v, w_sink, w_near, scale)
    for h in range(h_q):
        hk = (h * h_k) // h_q
        for i in range(n_q):
            keys = sorted(windows.visible_set(i, n_q, n_k, w_sink, w_near, hk, h_k))
            s = [scale * sum(q[0, h, i, t] * k[0, hk, j, t] for t in range(d)) for j in keys]
            mx = max(s)
            e = [math.exp(x - mx) for x in s]
            z = sum(e)
            for t in range(d):
                assert abs(o[0, h, i, t] - sum(e[n] * v[0, hk, j, t] for n, j in enumerate(keys)) / z) < 1e-12
            assert abs(lse[0, h, i] - (mx + math.log(z))) < 1e-12


def test_invariants():
    rng = np.random.default_rng(25)
    q, k, v, _ = _case(rng, 1, 4, 2, 40, 40, 8)
    o, lse = attention.forward(q, k, v, 3, 6, 0.4)
    shift = rng.standard_normal(8)
    o2, lse2 = attention.forward(q, k + shift, v, 3, 6, 0.4)
    np.testing.assert_allclose(o2, o, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(lse2 - lse, 0.4 * (q @ shift)[..., :], rtol=1e-10, atol=1e-10)
    o3, _ = attention.forward(q, k, np.ones_like(v), 3, 6, 0.4)
    np.testing.assert_allclose(o3, 1.0, rtol=1e-12, atol=1e-12)


def test_empty_rows_without_near_window():
    rng = np.random.default_rng(26)
    q, k, v, do = _case(rng, 1, 2, 2, 20, 20, 4)
    # w_near = 0, no sink: head 0's long window starts at distance 0, head 1's
    # at distance 10, so head 1's first ten queries see nothing
    o, lse = attention.forward(q, k, v, 0, 0, 1.0)
    assert np.all(o[0, 1, :10] == 0) and np.all(np.isneginf(lse[0, 1, :10]))
    assert np.all(np.isfinite(lse[0, 0]))
    dq, dk, dv, _, _ = attention.backward(q, k, v, do, 0, 0, 1.0)
    assert np.all(dq[0, 1, :10] == 0)


def _torch_grads(q, k, v, do, masks, scale):
    tq, tk, tv = (torch.from_numpy(x.copy()).requires_grad_(True) for x in (q, k, v))
    h_q, h_k = q.shape[1], k.shape[1]
    m = torch.from_numpy(np.stack(masks)).repeat_interleave(h_q // h_k, dim=0)[None]
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=m, scale=scale,
                                                           enable_gqa=True)
    out.backward(torch.from_numpy(do))
    return tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


@pytest.mark.parametrize("shape", [(1, 4, 2, 48, 48, 8, 4, 7), (2, 6, 3, 21, 37, 4, 0, 5),
                                   (1, 8, 8, 30, 30, 16, 2, 3)])
def test_gradient_vs_torch_autograd(shape):
    bsz, h_q, h_k, n_q, n_k, d, w_sink, w_near = shape
    rng = np.random.default_rng(27)
    q, k, v, do = _case(rng, bsz, h_q, h_k, n_q, n_k, d)
    dq, dk, dv, o, lse = attention.backward(q, k, v, do, w_sink, w_near, 0.35)
    masks = [windows.visible_mask(n_q, n_k, w_sink, w_near, h, h_k) for h in range(h_k)]
    rq, rk, rv = _torch_grads(q, k, v, do, masks, 0.35)
    np.testing.assert_allclose(dq, rq, rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dk, rk, rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dv, rv, rtol=1e-10, atol=1e-11)


def test_gradient_finite_differences():
    rng = np.random.default_rng(28)
    q, k, v, do = _case(rng, 1, 4, 2, 9, 11, 3)
    args = dict(w_sink=1, w_near=3, scale=0.6)
    dq, dk, dv, _, _ = attention.backward(q, k, v, do, **args)

    def loss(q_, k_, v_):
        return float((attention.forward(q_, k_, v_, **args)[0] * do).sum())

    eps = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for idx in [tuple(rng.integers(0, s) for s in x.shape) for _ in range(12)]:
            xp, xm = x.copy(), x.copy()
            xp[idx] += eps
            xm[idx] -= eps
            a = dict(q_=q, k_=k, v_=v)
            a[name + "_"] = xp
            lp = loss(**a)
            a[name + "_"] = xm
            lm = loss(**a)
            assert abs((lp - lm) / (2 * eps) - g[idx]) < 1e-6, (name, idx)


def test_gradient_sum_identities():
    """sum over keys of dV = sum over queries of dO per QO-head group (rows of P
    sum to one); sum over keys of dK = 0 (rows of dS sum to zero)."""
    rng = np.random.default_rng(29)
    q, k, v, do = _case(rng, 1, 8, 2, 64, 64, 8)
    dq, dk, dv, _, _ = attention.backward(q, k, v, do, 4, 8, 0.3)
    for hk in range(2):
        np.testing.assert_allclose(dv[0, hk].sum(0), do[0, 4 * hk:4 * hk + 4].sum((0, 1)), atol=1e-10)
        np.testing.assert_allclose(dk[0, hk].sum(0), 0.0, atol=1e-10)


@pytest.mark.parametrize("n_k", [1, 5, 40, 100, 257])
def test_decode_is_last_row_of_forward(n_k):
    rng = np.random.default_rng(30)
    h_q, h_k, d, n_max = 8, 4, 8, 300
    kc = _rand(rng, (3, h_k, n_max, d))
    vc = _rand(rng, (3, h_k, n_max, d))
    qd = _rand(rng, (3, h_q, d))
    seqlens = np.array([n_k, max(1, n_k // 2), n_max])
    o, lse = attention.decode(qd, kc, vc, seqlens, 6, 20, 0.5)
    for b in range(3):
        nk = int(seqlens[b])
        qfull = np.zeros((1, h_q, nk, d))
        qfull[0, :, -1] = qd[b]
        of, lf = attention.forward(qfull, kc[b:b + 1, :, :nk], vc[b:b + 1, :, :nk], 6, 20, 0.5)
        np.testing.assert_allclose(o[b], of[0, :, -1], rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(lse[b], lf[0, :, -1], rtol=1e-12, atol=1e-12)
        # and a single-query forward (N_q = 1, bottom-right aligned)
        o1, l1 = attention.forward(qd[b][None, :, None], kc[b:b + 1, :, :nk], vc[b:b + 1, :, :nk], 6, 20, 0.5)
        np.testing.assert_allclose(o[b], o1[0, :, 0], rtol=1e-12, atol=1e-12)


def test_sampled_helpers_match_full():
    rng = np.random.default_rng(31)
    q, k, v, do = _case(rng, 2, 4, 2, 70, 90, 8)
    args = dict(w_sink=5, w_near=12, scale=0.3)
    dq, dk, dv, o, lse = attention.backward(q, k, v, do, **args)
    rows = [(b, h, i) for b in range(2) for h in range(4) for i in (0, 1, 33, 69)]
    fo, fl = attention.forward_rows(q, k, v, rows, **args)
    gq, go, gl = attention.backward_q_rows(q, k, v, do, rows, **args)
    for n, (b, h, i) in enumerate(rows):
        np.testing.assert_allclose(fo[n], o[b, h, i], atol=1e-12)
        np.testing.assert_allclose(go[n], o[b, h, i], atol=1e-12)
        np.testing.assert_allclose(fl[n], lse[b, h, i], atol=1e-12)
        np.testing.assert_allclose(gq[n], dq[b, h, i], atol=1e-12)
    kv_rows = [(b, hk, i) for b in range(2) for hk in range(2) for i in (0, 4, 5, 50, 89)]
    gk, gv = attention.backward_kv_rows(q, k, v, do, kv_rows, **args)
    for n, (b, hk, i) in enumerate(kv_rows):
        np.testing.assert_allclose(gk[n], dk[b, hk, i], atol=1e-12)
        np.testing.assert_allclose(gv[n], dv[b, hk, i], atol=1e-12)


def test_full_forward_equals_global_offset_runs():
    rng = np.random.default_rng(32)
    q, k, v, _ = _case(rng, 1, 8, 4, 60, 60, 8)
    o, lse = attention.forward(q, k, v, 2, 9, 0.5)
    for r in range(4):
        o1, l1 = attention.forward(q[:, 2 * r:2 * r + 2], k[:, r:r + 1], v[:, r:r + 1], 2, 9, 0.5,
                                   h_total=4, h_offset=r)
        np.testing.assert_allclose(o1, o[:, 2 * r:2 * r + 2], atol=1e-12)


def test_legal_pair_counts():
    # counts from the per-query support sizes equal the element mask sums
    rng = np.random.default_rng(33)
    for _ in range(30):
        n_k = int(rng.integers(1, 200))
        n_q = int(rng.integers(1, n_k + 1))
        h_k = int(rng.integers(1, 5))
        ws, wn = int(rng.integers(0, 20)), int(rng.integers(0, 50))
        per = counts.legal_pairs_per_kv_head(n_q, n_k, ws, wn, h_k)
        for h in range(h_k):
            assert per[h] == windows.visible_mask(n_q, n_k, ws, wn, h, h_k).sum()
    # measured workloads (independently computed regression values)
    assert counts.legal_pairs(1, 512, 512, 4, 2, 16, 64) == 338256
    assert counts.legal_pairs(1, 8192, 8192, 32, 8, 64, 1024) == 367238016
    assert counts.legal_pairs(2, 32768, 32768, 32, 8, 64, 2048) == 8045799168
    assert counts.legal_pairs(1, 131072, 131072, 32, 8, 128, 4096) == 49612416768
    keys = counts.decode_visible_keys([131072] * 4, 128, 4096, 8)
    assert np.all(keys == 20080)
    assert counts.dense_causal_pairs(1, 4, 4, 1) == 10


# ---------------------------------------------------------------------------
# Planted mistakes: copies of oracle steps with one plausible error each must
# fail the pins above.

def test_planted_missing_d_term_is_caught():
    rng = np.random.default_rng(34)
    q, k, v, do = _case(rng, 1, 2, 1, 16, 16, 4)
    masks = [windows.visible_mask(16, 16, 1, 3, 0, 1)]
    rq, _, _ = _torch_grads(q, k, v, do, masks, 0.5)
    # dS = P * dP (dropped "- D")
    s = 0.5 * q[0] @ k[0, 0].T
    s = np.where(masks[0], s, -np.inf)
    p = np.exp(s - s.max(-1, keepdims=True))
    p /= p.sum(-1, keepdims=True)
    dq_bad = 0.5 * (p * (do[0] @ v[0, 0].T)) @ k[0, 0]
    assert not np.allclose(dq_bad, rq, atol=1e-6)


def test_planted_wrong_gqa_map_is_caught():
    rng = np.random.default_rng(35)
    q, k, v, _ = _case(rng, 1, 4, 2, 20, 20, 4)
    masks = [windows.visible_mask(20, 20, 1, 3, h, 2) for h in range(2)]
    ref = _sdpa(q, k, v, masks, 0.5).numpy()
    # h % H_k instead of floor(h * H_k / H_q)
    bad = np.zeros_like(q)
    for h in range(4):
        o1, _ = attention.forward(q[:, h:h + 1], k[:, h % 2:h % 2 + 1], v[:, h % 2:h % 2 + 1], 1, 3, 0.5,
                                  h_total=2, h_offset=h % 2)
        bad[:, h] = o1[:, 0]
    assert not np.allclose(bad, ref, atol=1e-6)


def test_planted_local_head_count_is_caught():
    """Breakpoints from the local head count on a one-head device differ from
    the all-heads run."""
    rng = np.random.default_rng(36)
    q, k, v, _ = _case(rng, 1, 4, 4, 50, 50, 4)
    o, _ = attention.forward(q, k, v, 2, 8, 0.5)
    o_bad, _ = attention.forward(q[:, 2:3], k[:, 2:3], v[:, 2:3], 2, 8, 0.5, h_total=1, h_offset=0)
    assert not np.allclose(o_bad, o[:, 2:3], atol=1e-6)
