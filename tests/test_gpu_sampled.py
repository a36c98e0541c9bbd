"""Parity at the 32K (B=2) and 128K training workloads, in the launch
configuration the benchmark times (128 x 128 blocks), against stored values of
the fp64 oracle.

The kernels run the whole forward and backward on the full seeded inputs; a
sample of their outputs is compared element by element with the values that
``tests/golden/make_sampled.py`` computed with the oracle alone (no value there
comes from the HIP path):

* O, LSE and dQ of every QO head on 16 QO blocks -- the first and last
  blocks, the blocks where each KV head's long-range window first appears and
  where it stops being clipped at the start of the sequence, and random ones;
  10 rows of each block;
* dK and dV of every KV head on a sink key, a key seen only through the near
  window, a key inside the head's long-range window, and the last key.

Every output is poisoned with NaN before the call, and the test asserts that
none is left anywhere.
"""

import os

import numpy as np
import pytest

import inputs
from conftest import GOLDEN
from gpu_util import need_gpu, log, to_dev, to_host, compare, torch

pytestmark = pytest.mark.gpu


def _golden(name):
    path = os.path.join(GOLDEN, f"sampled_{name}.npz")
    assert os.path.exists(path), f"missing {path}: run tests/golden/make_sampled.py {name}"
    g = np.load(path, allow_pickle=False)
    assert str(g["workload"]) == name
    return g


def _sampled(name):
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    g = _golden(name)
    w = inputs.WORKLOADS[name]
    log(f"{name}: generating inputs")
    t = inputs.train_tensors(w, values=False)
    q, k, v, do = (to_dev(t[n][0], dev) for n in ("q", "k", "v", "do"))
    del t
    o = torch.full_like(q, float("nan"))
    lse = torch.full((w.batch, w.h_q, w.n_q), float("nan"), dtype=torch.float32, device=dev)
    dq, dk, dv = (torch.full_like(x, float("nan")) for x in (q, k, v))
    p = cowa.make_params(w.batch, w.n_q, w.n_k, w.h_q, w.h_k, w.head_dim, w.w_sink, w.w_near, w.tile, w.tile,
                         w.scale)
    sched = cowa.Schedule(p, dev)
    log(f"{name}: forward + backward on the device")
    cowa.fwd(q, k, v, w.w_sink, w.w_near, w.tile, w.tile, w.scale, schedule=sched, out=o, lse=lse)
    cowa.bwd(q, k, v, o, lse, do, w.w_sink, w.w_near, w.tile, w.tile, w.scale, schedule=sched, dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    for x, n in ((o, "O"), (lse, "LSE"), (dq, "dQ"), (dk, "dK"), (dv, "dV")):
        assert not torch.isnan(x).any().item(), f"{n} has unwritten (NaN) elements"
    rows = torch.from_numpy(g["q_rows"]).to(dev)
    b, h, i = rows[:, 0], rows[:, 1], rows[:, 2]
    log(f"{name}: {len(rows)} query rows on {len(g['q_blocks'])} QO blocks x {w.h_q} QO heads")
    compare("O", to_host(o[b, h, i]), g["o"])
    compare("LSE", lse[b, h, i].cpu().numpy().astype(np.float64), g["lse"])
    compare("dQ", to_host(dq[b, h, i]), g["dq"])
    kv = torch.from_numpy(g["kv_rows"]).to(dev)
    b, h, i = kv[:, 0], kv[:, 1], kv[:, 2]
    assert set(g["kv_rows"][:, 1].tolist()) == set(range(w.h_k))
    log(f"{name}: {len(kv)} key rows over all {w.h_k} KV heads")
    compare("dK", to_host(dk[b, h, i]), g["dk"])
    compare("dV", to_host(dv[b, h, i]), g["dv"])


def test_sampled_bf16_t32k_b2():
    _sampled("bf16_t32k_b2")


def test_sampled_bf16_t128k():
    _sampled("bf16_t128k")


def test_sampled_bf16_t128k_wide_scores():
    """The 128K forward with Q scaled by 32 (exact in bf16), against stored
    oracle O and LSE: most rows' scores climb far past the forward's starting
    exponent offset, so the offset moves at block ends (and in rare rows the
    row runs again); the fp64 oracle has no offset."""
    import paper_2609_32704_amd as cowa
    dev = need_gpu()
    g = _golden("bf16_t128k_wide")
    w = inputs.WORKLOADS[str(g["base"])]
    scale_q = float(g["q_scale"])
    log(f"bf16_t128k_wide: generating inputs (Q x {scale_q:g})")
    t = inputs.train_tensors(w, which=("q", "k", "v"), values=False)
    q, k, v = (to_dev(t[n][0], dev) for n in ("q", "k", "v"))
    del t
    q = (q.float() * scale_q).to(torch.bfloat16)  # exact: a power of two
    o = torch.full_like(q, float("nan"))
    lse = torch.full((w.batch, w.h_q, w.n_q), float("nan"), dtype=torch.float32, device=dev)
    log("bf16_t128k_wide: forward on the device")
    cowa.fwd(q, k, v, w.w_sink, w.w_near, w.tile, w.tile, w.scale, out=o, lse=lse)
    torch.cuda.synchronize()
    assert not torch.isnan(o).any().item() and not torch.isnan(lse).any().item()
    rows = torch.from_numpy(g["q_rows"]).to(dev)
    b, h, i = rows[:, 0], rows[:, 1], rows[:, 2]
    log(f"bf16_t128k_wide: {len(rows)} query rows on {len(g['q_blocks'])} QO blocks x {w.h_q} QO heads")
    assert float(g["lse"].max()) > 100.0  # the score range of the case (natural log)
    compare("O", to_host(o[b, h, i]), g["o"])
    compare("LSE", lse[b, h, i].cpu().numpy().astype(np.float64), g["lse"])
