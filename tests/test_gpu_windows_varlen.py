"""Explicit per-head window tuples (Sec. 2.1) and ragged batches
(Eq. fwa_distance per sequence) through the C ABI, against the fp64 oracle:
forward, backward and decoding.  Full outputs; outputs poisoned with NaN."""

import numpy as np
import pytest

import inputs
from oracle import attention as ref, windows as ow
from gpu_util import need_gpu, log, to_dev, to_host, compare, torch

pytestmark = pytest.mark.gpu


def _draw(key, shapes):
    return {n: inputs.normal_bf16(s, inputs.seed_sequence(inputs.key_of(*key), n)) for n, s in shapes.items()}


TUPLE_CASES = [
    # name, n_q, n_k, h_q, h_k, d, tile_q, tile_k, tuples (None: the m-window layout below)
    ("m2_layout", 3000, 3000, 8, 4, 128, 128, 128, "m2"),
    ("m1_layout_d64", 1500, 1500, 4, 4, 64, 64, 64, "m1"),
    ("head_specific", 2000, 2500, 8, 4, 128, 64, 128, [(0, 64, 0, 500), (32, 128, 300, 700), (8, 0, 100, 2000),
                                                       (200, 300, 1000, 0)]),
    ("huge_windows", 700, 700, 4, 2, 128, 128, 64, [(10 ** 9, 0, 0, 0), (0, 1, 0, 2 ** 30)]),
]


def _tuples(spec, n_k, h_k):
    if spec in ("m1", "m2"):
        return ow.m_window_layout(n_k, 16, 256, h_k, int(spec[1]))
    return spec


@pytest.mark.parametrize("case", TUPLE_CASES, ids=[c[0] for c in TUPLE_CASES])
def test_fwd_bwd_explicit_tuples(case):
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    name, n_q, n_k, h_q, h_k, d, tq, tk, spec = case
    tuples = _tuples(spec, n_k, h_k)
    log(f"tuples {name}: n_q={n_q} n_k={n_k} h={h_q}/{h_k} d={d} tiles={tq}x{tk} windows={tuples}")
    t = _draw(("tuples", name), {"q": (1, h_q, n_q, d), "k": (1, h_k, n_k, d), "v": (1, h_k, n_k, d),
                                 "do": (1, h_q, n_q, d)})
    q, k, v, do = (to_dev(t[n][0], dev) for n in ("q", "k", "v", "do"))
    scale = d ** -0.5
    o = torch.full_like(q, float("nan"))
    lse = torch.full((1, h_q, n_q), float("nan"), dtype=torch.float32, device=dev)
    cowa.fwd(q, k, v, 0, 0, tq, tk, scale, out=o, lse=lse, windows=tuples)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    cowa.bwd(q, k, v, o, lse, do, 0, 0, tq, tk, scale, dq=dq, dk=dk, dv=dv, windows=tuples)
    torch.cuda.synchronize()
    dq_r, dk_r, dv_r, o_r, l_r = ref.backward(t["q"][1], t["k"][1], t["v"][1], t["do"][1], 0, 0, scale,
                                              windows=tuples)
    compare("O", to_host(o), o_r)
    compare("LSE", to_host(lse), l_r)
    compare("dQ", to_host(dq), dq_r)
    compare("dK", to_host(dk), dk_r)
    compare("dV", to_host(dv), dv_r)


RAGGED_CASES = [
    # name, seqs [(n_q, n_k)], h_q, h_k, d, sink, near, tile_q, tile_k, tuples
    ("mixed", [(300, 1111), (1000, 1000), (0, 257), (1, 1), (777, 800)], 8, 2, 128, 16, 128, 128, 128, None),
    ("mixed_t64_d64", [(64, 64), (500, 900), (129, 129), (0, 0), (333, 1000)], 4, 1, 64, 3, 77, 64, 64, None),
    ("tuples", [(400, 400), (90, 1200), (1000, 1500)], 8, 4, 128, 0, 0, 64, 128,
     [(16, 128, 0, 300), (16, 128, 300, 300), (0, 64, 600, 900), (100, 0, 0, 50)]),
    ("tp_rank", [(1500, 2000), (2048, 2048)], 4, 1, 128, 32, 256, 128, 128, None),
    # split sink blocks (three per sequence) with a sequence shorter than three blocks
    ("wide_sink", [(200, 200), (1500, 1500), (600, 900)], 8, 2, 128, 300, 64, 128, 128, None),
]


def _cu(lens):
    out = [0]
    for x in lens:
        out.append(out[-1] + x)
    return out


@pytest.mark.parametrize("case", RAGGED_CASES, ids=[c[0] for c in RAGGED_CASES])
def test_fwd_bwd_ragged(case):
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    name, seqs, h_q, h_k, d, ws, wn, tq, tk, tuples = case
    ht, ho = (8, 3) if name == "tp_rank" else (None, 0)
    cu_q, cu_k = _cu([a for a, _ in seqs]), _cu([b for _, b in seqs])
    log(f"ragged {name}: seqs={seqs} h={h_q}/{h_k} d={d} sink={ws} near={wn} tiles={tq}x{tk} windows={tuples}")
    t = _draw(("ragged", name), {"q": (h_q, cu_q[-1], d), "k": (h_k, cu_k[-1], d), "v": (h_k, cu_k[-1], d),
                                 "do": (h_q, cu_q[-1], d)})
    q, k, v, do = (to_dev(t[n][0], dev) for n in ("q", "k", "v", "do"))
    scale = d ** -0.5
    o = torch.full_like(q, float("nan"))
    lse = torch.full((h_q, cu_q[-1]), float("nan"), dtype=torch.float32, device=dev)
    cowa.fwd_varlen(q, k, v, cu_q, cu_k, ws, wn, tq, tk, scale, h_k_total=ht, h_k_offset=ho, out=o, lse=lse,
                    windows=tuples)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    cowa.bwd_varlen(q, k, v, o, lse, do, cu_q, cu_k, ws, wn, tq, tk, scale, h_k_total=ht, h_k_offset=ho, dq=dq,
                    dk=dk, dv=dv, windows=tuples)
    torch.cuda.synchronize()
    dq_r, dk_r, dv_r, o_r, l_r = ref.backward_varlen(t["q"][1], t["k"][1], t["v"][1], t["do"][1], cu_q, cu_k, ws,
                                                     wn, scale, h_total=ht, h_offset=ho, windows=tuples)
    compare("O", to_host(o), o_r)
    compare("LSE", to_host(lse), l_r)
    compare("dQ", to_host(dq), dq_r)
    compare("dK", to_host(dk), dk_r)
    compare("dV", to_host(dv), dv_r)


def test_fwd_fp32_ragged_tuples():
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    seqs, h_q, h_k, d = [(100, 300), (257, 257), (0, 40)], 4, 2, 64
    tuples = [(3, 20, 10, 60), (0, 50, 0, 500)]
    cu_q, cu_k = _cu([a for a, _ in seqs]), _cu([b for _, b in seqs])
    rng = np.random.default_rng(inputs.key_of("fp32_ragged"))
    qf, kf, vf = (rng.standard_normal((h, n, d)).astype(np.float32)
                  for h, n in ((h_q, cu_q[-1]), (h_k, cu_k[-1]), (h_k, cu_k[-1])))
    q, k, v = (to_dev(x, dev) for x in (qf, kf, vf))
    o = torch.full_like(q, float("nan"))
    lse = torch.full((h_q, cu_q[-1]), float("nan"), dtype=torch.float32, device=dev)
    cowa.fwd_varlen(q, k, v, cu_q, cu_k, 0, 0, 32, 32, 0.125, out=o, lse=lse, windows=tuples)
    torch.cuda.synchronize()
    o_r, l_r = ref.forward_varlen(qf, kf, vf, cu_q, cu_k, 0, 0, 0.125, windows=tuples)
    compare("O", to_host(o), o_r, "fp32")
    compare("LSE", to_host(lse), l_r, "fp32")


def test_autograd_varlen():
    """attention_varlen: gradients of sum(O * dO) against the oracle."""
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    seqs, h_q, h_k, d = [(200, 600), (333, 333)], 8, 2, 128
    cu_q, cu_k = _cu([a for a, _ in seqs]), _cu([b for _, b in seqs])
    t = _draw(("autograd_varlen",), {"q": (h_q, cu_q[-1], d), "k": (h_k, cu_k[-1], d), "v": (h_k, cu_k[-1], d),
                                     "do": (h_q, cu_q[-1], d)})
    q, k, v = (to_dev(t[n][0], dev).requires_grad_(True) for n in ("q", "k", "v"))
    do = to_dev(t["do"][0], dev)
    o = cowa.attention_varlen(q, k, v, cu_q, cu_k, 8, 64, 128, 128, d ** -0.5)
    (o.float() * do.float()).sum().backward()
    torch.cuda.synchronize()
    dq_r, dk_r, dv_r, o_r, _ = ref.backward_varlen(t["q"][1], t["k"][1], t["v"][1], t["do"][1], cu_q, cu_k, 8, 64,
                                                   d ** -0.5)
    compare("O", to_host(o.detach()), o_r)
    compare("dQ", to_host(q.grad), dq_r)
    compare("dK", to_host(k.grad), dk_r)
    compare("dV", to_host(v.grad), dv_r)


@pytest.mark.parametrize("spec", ["m2", "custom"])
def test_decode_explicit_tuples(spec):
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    bsz, h_q, h_k, d, n_max = 3, 16, 4, 128, 6000
    tuples = ow.m_window_layout(n_max, 16, 256, h_k, 2) if spec == "m2" else \
        [(0, 100, 0, 3000), (64, 0, 500, 10 ** 9), (5, 5, 5, 5), (10 ** 9, 1, 0, 0)]
    seqlens = [6000, 2500, 77]
    t = _draw(("dec_tuples", spec), {"q": (bsz, h_q, d), "k_cache": (bsz, h_k, n_max, d),
                                     "v_cache": (bsz, h_k, n_max, d)})
    q, kc, vc = (to_dev(t[n][0], dev) for n in ("q", "k_cache", "v_cache"))
    sl = torch.tensor(seqlens, dtype=torch.int32, device=dev)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((bsz, h_q), float("nan"), dtype=torch.float32, device=dev)
    cowa.decode(q, kc, vc, sl, 0, 0, d ** -0.5, out=o, lse=lse, windows=tuples)
    torch.cuda.synchronize()
    o_r, l_r = ref.decode(t["q"][1], t["k_cache"][1], t["v_cache"][1], seqlens, 0, 0, d ** -0.5, windows=tuples)
    compare("O", to_host(o), o_r)
    compare("LSE", lse.cpu().numpy().astype(np.float64), l_r)
