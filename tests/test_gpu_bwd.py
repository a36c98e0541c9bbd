"""Backward parity (cowa_bwd through the C ABI) against the fp64 oracle.

Two paths: the device forward's own O and LSE fed to the backward (the
training path), and the oracle's O and LSE (rounded to the kernel's input
types) fed to it, which isolates the backward.  Full gradients at the 8K
workload and odd shapes (the 32K and 128K workloads are sampled against
stored oracle values in test_gpu_sampled.py).  Outputs are poisoned with NaN
before each call.
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
    # the pipelined dQ pass (128-key blocks) at head dimension 64
    ("gqa2_d64_t128", 1, 600, 600, 4, 2, 64, 8, 150, 128, 128, 0, 0),
    ("gqa4_d64_tq64_t128", 1, 700, 700, 8, 2, 64, 8, 150, 64, 128, 0, 0),
    # a sink of three 128-key blocks, each split into parts in the dK/dV pass
    ("wide_sink", 1, 1500, 1500, 8, 2, 128, 300, 64, 128, 128, 0, 0),
]


@pytest.mark.parametrize("case", ODD, ids=[c[0] for c in ODD])
def test_bwd_odd_shapes(case):
    name, bsz, n_q, n_k, h_q, h_k, d, ws, wn, tq, tk, ht, ho = case
    w = inputs.custom("bwd_" + name, batch=bsz, n_q=n_q, n_k=n_k, h_q=h_q, h_k=h_k, head_dim=d, w_sink=ws,
                      w_near=wn, tile=tq, h_total=ht, h_offset=ho)
    _full_check(w, key=inputs.key_of("bwd", name), tile_q=tq, tile_k=tk)


def test_autograd_function_and_determinism():
    """cowa.attention (torch.autograd.Function over cowa_fwd / cowa_bwd):
    gradients of sum(O * dO) match the oracle, and a second forward and
    backward on the same inputs give bitwise the same O, LSE and gradients (the
    backward has no atomics)."""
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    w = inputs.custom("autograd", batch=2, n_q=700, n_k=900, h_q=8, h_k=2, head_dim=128, w_sink=16, w_near=128,
                      tile=128)
    t = inputs.train_tensors(w, key=inputs.key_of("autograd"))
    dq_r, dk_r, dv_r, o_r, _ = ref.backward(t["q"][1], t["k"][1], t["v"][1], t["do"][1], w.w_sink, w.w_near,
                                            w.scale)
    do = to_dev(t["do"][0], dev)
    runs = []
    for _ in range(2):
        q, k, v = (to_dev(t[n][0], dev).requires_grad_(True) for n in ("q", "k", "v"))
        o, lse = cowa.attention(q, k, v, w.w_sink, w.w_near, 128, 128, w.scale, return_lse=True)
        (o.float() * do.float()).sum().backward()
        torch.cuda.synchronize()
        runs.append((o.detach(), lse.detach(), q.grad, k.grad, v.grad))
    compare("O", to_host(runs[0][0]), o_r)
    compare("dQ", to_host(runs[0][2]), dq_r)
    compare("dK", to_host(runs[0][3]), dk_r)
    compare("dV", to_host(runs[0][4]), dv_r)
    for a, b, n in zip(runs[0], runs[1], ("O", "LSE", "dQ", "dK", "dV")):
        assert torch.equal(a, b), f"{n} differs between two identical runs"


def test_bwd_bitwise_deterministic_8k():
    """The backward at the 8K workload, run twice on the same inputs, gives
    bitwise equal dQ, dK and dV."""
    dev = need_gpu()
    w = inputs.WORKLOADS["bf16_t8k"]
    t = inputs.train_tensors(w, values=False)
    first = _run_bwd(w, t, dev)
    second = _run_bwd(w, t, dev)
    for a, b, n in zip(first, second, ("dQ", "dK", "dV")):
        assert torch.equal(a, b), f"{n} differs between two identical runs"


def test_bwd_reads_no_rows_past_the_sequence():
    """Regression: with 128-row QO blocks and n_q % 128 <= 64, the last block's
    second 64-row step lies wholly past n_q.  Its copies of Q and dO must read
    nothing (they once read past the end of the tensors).  Q and dO sit at the
    start of NaN-filled buffers here, so a row read past the last QO head's end
    would turn dK and dV into NaN; the reads stay inside those buffers."""
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    n, h_q, h_k, d, sink, near, tile = 3000, 4, 2, 128, 16, 256, 128
    assert 0 < n % tile <= 64
    t = {nm: inputs.normal_bf16(s, inputs.seed_sequence(inputs.key_of("past_end", n), nm))
         for nm, s in (("q", (1, h_q, n, d)), ("k", (1, h_k, n, d)), ("v", (1, h_k, n, d)), ("do", (1, h_q, n, d)))}
    k, v = to_dev(t["k"][0], dev), to_dev(t["v"][0], dev)

    def padded(bits):  # the tensor at the start of a buffer with 256 NaN rows behind it
        buf = torch.full(((h_q * n + 256) * d,), float("nan"), dtype=torch.bfloat16, device=dev)
        view = buf[:h_q * n * d].view(1, h_q, n, d)
        view.copy_(to_dev(bits, dev))
        return buf, view

    qbuf, q = padded(t["q"][0])
    dobuf, do = padded(t["do"][0])
    scale = d ** -0.5
    o, lse = cowa.fwd(q, k, v, sink, near, tile, tile, scale)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    cowa.bwd(q, k, v, o, lse, do, sink, near, tile, tile, scale, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    dq_r, dk_r, dv_r, _, _ = ref.backward(t["q"][1], t["k"][1], t["v"][1], t["do"][1], sink, near, scale)
    compare("dQ", to_host(dq), dq_r)
    compare("dK", to_host(dk), dk_r)
    compare("dV", to_host(dv), dv_r)
    del qbuf, dobuf
