"""Seeded random shapes against the fp64 oracle, full outputs, through the
C ABI: forward + backward (training path) and split-KV decoding.

The hand-picked edge cases elsewhere cover the named corners; this sweep
draws batch, lengths (N_q <= N_k, seldom multiples of the tiles), GQA group
sizes, head dimensions, tile shapes, sink and near widths (zero, small, wider
than the sequence) and a global KV-head offset at random, so that block-list
shapes, partial-block masks and window edges land where no one chose them.
Every draw is printed before its call; every output is poisoned with NaN.
"""

import numpy as np
import pytest

import inputs
from oracle import attention as ref
from gpu_util import need_gpu, log, to_dev, to_host, compare, torch
from test_gpu_decode import _check as _decode_check

pytestmark = pytest.mark.gpu

N_TRAIN, N_DECODE = 48, 16


def _width(rng, n):
    r = rng.random()
    if r < 0.15:
        return 0
    if r < 0.3:
        return int(rng.integers(n, 2 * n + 2))  # covers the whole sequence
    return int(rng.integers(1, 300))


def _heads(rng):
    h_k = int(rng.choice([1, 2, 4]))
    g = int(rng.choice([1, 2, 4, 8]))
    if rng.random() < 0.3:
        h_total = h_k * int(rng.integers(2, 5))
        return h_k * g, h_k, h_total, int(rng.integers(0, h_total - h_k + 1))
    return h_k * g, h_k, 0, 0


def _draw_train(case):
    rng = np.random.default_rng(inputs.key_of("random_train", case))
    n_k = int(rng.integers(1, 1600))
    n_q = int(rng.integers(1, n_k + 1)) if rng.random() < 0.4 else n_k
    h_q, h_k, ht, ho = _heads(rng)
    return dict(batch=int(rng.integers(1, 3)), n_q=n_q, n_k=n_k, h_q=h_q, h_k=h_k,
                head_dim=int(rng.choice([64, 128])), w_sink=_width(rng, n_k), w_near=_width(rng, n_k),
                h_total=ht, h_offset=ho), (int(rng.choice([64, 128])), int(rng.choice([64, 128])))


@pytest.mark.parametrize("case", range(N_TRAIN))
def test_random_fwd_bwd(case):
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    c, (tq, tk) = _draw_train(case)
    log(f"random train case {case}: {c} tiles={tq}x{tk}")
    w = inputs.custom(f"random_train_{case}", tile=tq, **c)
    t = inputs.train_tensors(w, key=inputs.key_of("random_train_t", case))
    q, k, v, do = (to_dev(t[n][0], dev) for n in ("q", "k", "v", "do"))
    o = torch.full_like(q, float("nan"))
    lse = torch.full((w.batch, w.h_q, w.n_q), float("nan"), dtype=torch.float32, device=dev)
    cowa.fwd(q, k, v, w.w_sink, w.w_near, tq, tk, w.scale, h_k_total=w.kv_total, h_k_offset=w.h_offset,
             out=o, lse=lse)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    cowa.bwd(q, k, v, o, lse, do, w.w_sink, w.w_near, tq, tk, w.scale, h_k_total=w.kv_total,
             h_k_offset=w.h_offset, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    dq_r, dk_r, dv_r, o_r, l_r = ref.backward(t["q"][1], t["k"][1], t["v"][1], t["do"][1], w.w_sink, w.w_near,
                                              w.scale, h_total=w.kv_total, h_offset=w.h_offset)
    compare("O", to_host(o), o_r)
    compare("LSE", lse.cpu().numpy().astype(np.float64), l_r)
    compare("dQ", to_host(dq), dq_r)
    compare("dK", to_host(dk), dk_r)
    compare("dV", to_host(dv), dv_r)


@pytest.mark.parametrize("case", range(N_DECODE))
def test_random_decode(case):
    rng = np.random.default_rng(inputs.key_of("random_decode", case))
    n_max = int(rng.integers(1, 20000))
    bsz = int(rng.integers(1, 6))
    h_q, h_k, ht, ho = _heads(rng)
    seqlens = [int(rng.integers(1, n_max + 1)) for _ in range(bsz)]
    if rng.random() < 0.5:
        seqlens[0] = n_max
    split = int(rng.choice([0, 64, 256, 1024]))
    w = inputs.custom(f"random_decode_{case}", batch=bsz, n_q=1, n_k=n_max, h_q=h_q, h_k=h_k,
                      head_dim=int(rng.choice([64, 128])), w_sink=_width(rng, n_max), w_near=_width(rng, n_max),
                      kind="decode", h_total=ht, h_offset=ho)
    log(f"random decode case {case}: seqlens={seqlens} split_keys={split}")
    _decode_check(w, seqlens, key=inputs.key_of("random_decode_t", case), split_keys=split)
