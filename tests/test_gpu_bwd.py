"""Backward parity (cowa_bwd through the C ABI) against the fp64 oracle.

Two paths: the device forward's own O and LSE fed to the backward (the
training path), and the oracle's O and LSE (rounded to the kernel's input
types) fed to it, which isolates the backward.  Full gradients at the 8K
workload and odd shapes; sampled query rows (dQ) and key rows (dK, dV) at the
32K and 128K workloads in the launch configuration the benchmark times.
Outputs are poisoned with NaN before each call.
"""

import numpy as np
import pytest

import inputs
from oracle import attention as ref
from gpu_util import need_gpu, log, to_dev, to_host, compare, torch

pytestmark = pytest.mark.gpu


def _bf16_of(x, dev):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev).to(torch.bfloat16)


def _run_bwd(w, t, dev, o=None, lse=None, tile_q=None, tile_k=None):
    import paper_2609_32704_amd as cowa
    tq, tk = tile_q or w.tile, tile_k or w.tile
    q, k, v, do = (to_dev(t[n][0], dev) for n in ("q", "k", "v", "do"))
    p = cowa.make_params(w.batch, w.n_q, w.n_k, w.h_q, w.h_k, w.head_dim, w.w_sink, w.w_near, tq, tk, w.scale,
                         h_k_total=w.kv_total, h_k_offset=w.h_offset)
    sched = cowa.Schedule(p, dev)
    if o is None:
        o, lse = cowa.fwd(q, k, v, w.w_sink, w.w_near, tq, tk, w.scale, h_k_total=w.kv_total,
                          h_k_offset=w.h_offset, schedule=sched)
    dq = torch.full_like(q, float("nan"))
    dk = torch.full_like(k, float("nan"))
    dv = torch.full_like(v, float("nan"))
    cowa.bwd(q, k, v, o, lse, do, w.w_sink, w.w_near, tq, tk, w.scale, h_k_total=w.kv_total,
             h_k_offset=w.h_offset, schedule=sched, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    return dq, dk, dv


def _full_check(w, key=None, tile_q=None, tile_k=None, isolated=False):
    dev = need_gpu()
    log(f"bwd {w.name}: B={w.batch} n_q={w.n_q} n_k={w.n_k} h={w.h_q}/{w.h_k} d={w.head_dim} sink={w.w_sink} "
        f"near={w.w_near} tiles={tile_q or w.tile}x{tile_k or w.tile} isolated={isolated}")
    t = inputs.train_tensors(w, key=key)
    dq_r, dk_r, dv_r, o_r, l_r = ref.backward(t["q"][1], t["k"][1], t["v"][1], t["do"][1], w.w_sink, w.w_near,
                                              w.scale, h_total=w.kv_total, h_offset=w.h_offset)
    o = lse = None
    if isolated:
        o = _bf16_of(o_r, dev)
        lse = torch.from_numpy(l_r.astype(np.float32)).to(dev)
    dq, dk, dv = _run_bwd(w, t, dev, o, lse, tile_q, tile_k)
    compare("dQ", to_host(dq), dq_r)
    compare("dK", to_host(dk), dk_r)
    compare("dV", to_host(dv), dv_r)


def test_bwd_bf16_t8k():
    _full_check(inputs.WORKLOADS["bf16_t8k"])


def test_bwd_bf16_t8k_isolated():
    _full_check(inputs.WORKLOADS["bf16_t8k"], isolated=True)


ODD = [
    # name, batch, n_q, n_k, h_q, h_k, d, sink, near, tile_q, tile_k, h_total, h_offset
    ("ragged", 2, 333, 333, 4, 2, 128, 5, 40, 64, 64, 0, 0),
    ("chunked_prefill", 1, 200, 1111, 8, 2, 128, 16, 100, 128, 128, 0, 0),
    ("gqa8_d64", 1, 1000, 1000, 8, 1, 64, 3, 77, 128, 64, 0, 0),
    ("mha", 1, 700, 700, 3, 3, 128, 0, 50, 64, 128, 0, 0),
    ("tp_rank", 1, 2048, 2048, 4, 1, 128, 32, 256, 128, 128, 8, 5),
    ("dense", 1, 777, 777, 4, 2, 128, 0, 777, 128, 128, 0, 0),
    ("wide_windows", 1, 500, 500, 2, 2, 64, 400, 400, 64, 128, 0, 0),
    ("no_near", 1, 300, 300, 2, 2, 64, 0, 0, 64, 64, 0, 0),
    ("tiny", 1, 5, 9, 2, 1, 128, 1, 2, 64, 64, 0, 0),
    # four-wave dQ workgroups of 64-row query blocks (4 QO heads each)
    ("gqa4_tq64", 1, 900, 900, 8, 2, 128, 8, 200, 64, 128, 0, 0),
    ("gqa4_d64_t64", 1, 650, 650, 4, 1, 64, 16, 130, 64, 64, 0, 0),
]


@pytest.mark.parametrize("case", ODD, ids=[c[0] for c in ODD])
def test_bwd_odd_shapes(case):
    name, bsz, n_q, n_k, h_q, h_k, d, ws, wn, tq, tk, ht, ho = case
    w = inputs.custom("bwd_" + name, batch=bsz, n_q=n_q, n_k=n_k, h_q=h_q, h_k=h_k, head_dim=d, w_sink=ws,
                      w_near=wn, tile=tq, h_total=ht, h_offset=ho)
    _full_check(w, key=inputs.key_of("bwd", name), tile_q=tq, tile_k=tk)


def _sampled_check(name, q_blocks, kv_heads, sink_head, seed):
    dev = need_gpu()
    w = inputs.WORKLOADS[name]
    log(f"bwd {name} sampled: generating inputs")
    t = inputs.train_tensors(w)
    dq, dk, dv = _run_bwd(w, t, dev)
    for x in (dq, dk, dv):
        assert not torch.isnan(x).any().item()
    rng = np.random.default_rng(seed)
    n_qt = -(-w.n_q // w.tile)
    blocks = sorted(set([0, n_qt - 1] + list(rng.choice(n_qt, size=q_blocks, replace=False))))
    rows = []
    for blk in blocks:
        b = int(rng.integers(0, w.batch))
        for h in range(w.h_q):
            for i in range(blk * w.tile, min((blk + 1) * w.tile, w.n_q), 7):
                rows.append((b, h, i))
    log(f" dQ on {len(rows)} sampled rows")
    dq_r, _, _ = ref.backward_q_rows(t["q"][1], t["k"][1], t["v"][1], t["do"][1], rows, w.w_sink, w.w_near,
                                     w.scale)
    got = np.stack([to_host(dq[b, h, i]) for b, h, i in rows])
    compare("dQ", got, dq_r)
    # key rows of the sampled KV heads: one random key and the last key; key 0 (in
    # the sink, seen by every query) for one head
    kv_rows = []
    for hk in kv_heads:
        b = int(rng.integers(0, w.batch))
        kv_rows += [(b, hk, int(rng.integers(w.w_sink, w.n_k))), (b, hk, w.n_k - 1)]
        if hk == sink_head:
            kv_rows.append((b, hk, 0))
    log(f" dK/dV on {len(kv_rows)} sampled key rows")
    dk_r, dv_r = ref.backward_kv_rows(t["q"][1], t["k"][1], t["v"][1], t["do"][1], kv_rows, w.w_sink, w.w_near,
                                      w.scale)
    compare("dK", np.stack([to_host(dk[b, h, i]) for b, h, i in kv_rows]), dk_r)
    compare("dV", np.stack([to_host(dv[b, h, i]) for b, h, i in kv_rows]), dv_r)


def test_bwd_bf16_t32k_sampled():
    _sampled_check("bf16_t32k_b2", 3, [0, 5], 5, 1)


def test_bwd_bf16_t128k_sampled():
    _sampled_check("bf16_t128k", 3, [0, 7], None, 2)
