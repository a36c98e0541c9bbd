"""Decode parity (cowa_decode through the C ABI) against the fp64 oracle.

The 64-sequence x 131072-token workload in the configuration the benchmark
times, split-count invariance, ragged per-sequence lengths (including lengths
shorter than the shared windows and invalid lengths), GQA groups and global
head offsets.
"""

import numpy as np
import pytest

import inputs
from oracle import attention as ref
from gpu_util import need_gpu, log, to_dev, to_host, compare, torch

pytestmark = pytest.mark.gpu


def _run(w, t, seqlens, dev, split_keys=0):
    import paper_2609_32704_amd as cowa
    q, kc, vc = (to_dev(t[n][0], dev) for n in ("q", "k_cache", "v_cache"))
    sl = torch.tensor(seqlens, dtype=torch.int32, device=dev)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((w.batch, w.h_q), float("nan"), dtype=torch.float32, device=dev)
    cowa.decode(q, kc, vc, sl, w.w_sink, w.w_near, w.scale, h_k_total=w.kv_total, h_k_offset=w.h_offset,
                split_keys=split_keys, out=o, lse=lse)
    torch.cuda.synchronize()
    return o, lse


def _check(w, seqlens, key=None, split_keys=0, n_max=None):
    dev = need_gpu()
    log(f"decode {w.name}: B={w.batch} h={w.h_q}/{w.h_k} d={w.head_dim} sink={w.w_sink} near={w.w_near} "
        f"n_max={n_max or w.n_k} split_keys={split_keys}")
    t = inputs.decode_tensors(w, n_max=n_max, key=key)
    o, lse = _run(w, t, seqlens, dev, split_keys)
    valid = [(1 <= s <= (n_max or w.n_k)) for s in seqlens]
    sl_ok = np.array([s if v else 1 for s, v in zip(seqlens, valid)])
    o_r, l_r = ref.decode(t["q"][1], t["k_cache"][1], t["v_cache"][1], sl_ok, w.w_sink, w.w_near, w.scale,
                          h_total=w.kv_total, h_offset=w.h_offset)
    for b, v in enumerate(valid):
        if not v:  # documented: an invalid length gives O = 0 and LSE = -inf
            o_r[b] = 0.0
            l_r[b] = -np.inf
    compare("O", to_host(o), o_r)
    compare("LSE", lse.cpu().numpy().astype(np.float64), l_r)
    return o, lse


def test_decode_64x128k_sampled():
    """The full 64 x 131072 workload runs on the device; the caches hold NaN
    everywhere except the visible rows, so a read of any other row poisons the
    output.  Sampled sequences get seeded host draws on their visible rows and
    are checked against the oracle for every QO head; the others get device
    draws (load only)."""
    import paper_2609_32704_amd as cowa
    from oracle import windows as ow
    dev = need_gpu()
    w = inputs.WORKLOADS["decode_64x128k"]
    sampled = [0, 21, 42, 63]
    log(f"decode {w.name}: filling caches")
    shape = (w.batch, w.h_k, w.n_k, w.head_dim)
    kc = torch.full(shape, float("nan"), dtype=torch.bfloat16, device=dev)
    vc = torch.full(shape, float("nan"), dtype=torch.bfloat16, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(42)
    t_q = inputs.normal_bf16((w.batch, w.h_q, w.head_dim), inputs.seed_sequence(w.name, "q"))
    q = to_dev(t_q[0], dev)
    host = {}
    for hk in range(w.h_k):
        runs = ow.visible_intervals(0, 1, w.n_k, w.w_sink, w.w_near, hk, w.h_k)
        rows = np.concatenate([np.arange(a, b) for a, b in runs])
        idx = torch.from_numpy(rows).to(dev)
        for b in range(w.batch):
            if b in sampled:
                kb = inputs.normal_bf16((len(rows), w.head_dim), inputs.seed_sequence(w.name, f"k{b}_{hk}"))
                vb = inputs.normal_bf16((len(rows), w.head_dim), inputs.seed_sequence(w.name, f"v{b}_{hk}"))
                host[(b, hk)] = (rows, kb[1], vb[1])
                kd, vd = to_dev(kb[0], dev), to_dev(vb[0], dev)
            else:
                kd = torch.randn((len(rows), w.head_dim), generator=gen, device=dev).to(torch.bfloat16)
                vd = torch.randn((len(rows), w.head_dim), generator=gen, device=dev).to(torch.bfloat16)
            kc[b, hk].index_copy_(0, idx, kd)
            vc[b, hk].index_copy_(0, idx, vd)
    sl = torch.full((w.batch,), w.n_k, dtype=torch.int32, device=dev)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((w.batch, w.h_q), float("nan"), dtype=torch.float32, device=dev)
    log("decode: running")
    cowa.decode(q, kc, vc, sl, w.w_sink, w.w_near, w.scale, out=o, lse=lse)
    torch.cuda.synchronize()
    assert not torch.isnan(o).any().item() and not torch.isnan(lse).any().item()
    for b in sampled:
        kfull = np.full((1, w.h_k, w.n_k, w.head_dim), np.nan)
        vfull = np.full((1, w.h_k, w.n_k, w.head_dim), np.nan)
        for hk in range(w.h_k):
            rows, kv, vv = host[(b, hk)]
            kfull[0, hk, rows] = kv
            vfull[0, hk, rows] = vv
        o_r, l_r = ref.decode(t_q[1][b:b + 1], kfull, vfull, [w.n_k], w.w_sink, w.w_near, w.scale)
        log(f" sequence {b}")
        compare("O", to_host(o[b:b + 1]), o_r)
        compare("LSE", lse[b:b + 1].cpu().numpy().astype(np.float64), l_r)


def test_decode_split_invariance():
    w = inputs.custom("dec_split", batch=3, n_q=1, n_k=20000, h_q=8, h_k=2, head_dim=128, w_sink=64, w_near=1024,
                      kind="decode")
    outs = [_check(w, [20000, 9999, 3000], key=inputs.key_of("dec_split"), split_keys=sk)[0]
            for sk in (64, 512, 4096, 0)]
    for o in outs[1:]:
        assert (o.float() - outs[0].float()).abs().max().item() < 2e-2


@pytest.mark.parametrize("case", [
    ("short", 4, 8, 2, 128, 16, 100, 300, [1, 2, 50, 116]),
    ("ragged", 5, 32, 8, 128, 128, 4096, 40000, [40000, 1, 4224, 4225, 12345]),
    ("gqa1_d64", 2, 4, 4, 64, 3, 33, 5000, [5000, 4097]),
    ("gqa8", 2, 8, 1, 128, 0, 200, 3000, [2999, 3000]),
    ("gqa2_d64", 3, 4, 2, 64, 7, 0, 2000, [2000, 1500, 9]),
    ("invalid_len", 3, 8, 2, 128, 16, 64, 1000, [0, 1001, 500]),
])
def test_decode_shapes(case):
    name, bsz, h_q, h_k, d, ws, wn, n_max, seqlens = case
    w = inputs.custom("dec_" + name, batch=bsz, n_q=1, n_k=n_max, h_q=h_q, h_k=h_k, head_dim=d, w_sink=ws,
                      w_near=wn, kind="decode")
    _check(w, seqlens, key=inputs.key_of("dec", name))


def test_decode_global_head_offset():
    for r in (0, 3, 7):
        w = inputs.custom("dec_tp", batch=2, n_q=1, n_k=9000, h_q=4, h_k=1, head_dim=128, w_sink=32, w_near=512,
                          kind="decode", h_total=8, h_offset=r)
        _check(w, [9000, 7777], key=inputs.key_of("dec_tp", r))
