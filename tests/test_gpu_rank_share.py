"""One rank's share of the 8-way KV-head split at 131072 tokens equals the
corresponding slice of the all-heads run, bit for bit.

Sec. 2.3 (global KV-head assignment): rank r of a tensor-parallel group owns KV
head r and the QO heads of its group, builds its windows from the global head
index (Eq. fwa_global_head), and needs nothing from the other ranks.  The
library takes the global index through h_k_offset / h_k_total, so the call
with h_k = 1, h_q = 4, h_k_offset = r, h_k_total = 8 on the slices of the
tensors must reproduce the all-heads call's O, LSE, dQ, dK and dV for those
heads exactly: every row and column is computed by the same steps in the same
order (the dK/dV split plan depends only on the column lengths, which are the
same).  This checks the full-size launch configuration of the benchmark at
every output element, without an oracle.
"""

import pytest

from gpu_util import need_gpu, log, torch

pytestmark = pytest.mark.gpu

N, HQ, HK, D, SINK, NEAR, TILE = 131072, 32, 8, 128, 128, 4096, 128


def _run(q, k, v, do, h_k_total, h_k_offset):
    import paper_2609_32704_amd as cowa
    o, lse = cowa.fwd(q, k, v, SINK, NEAR, TILE, TILE, h_k_total=h_k_total, h_k_offset=h_k_offset)
    dq, dk, dv = cowa.bwd(q, k, v, o, lse, do, SINK, NEAR, TILE, TILE, h_k_total=h_k_total, h_k_offset=h_k_offset)
    return o, lse, dq, dk, dv


def test_rank_share_equals_all_heads_slice():
    dev = need_gpu()
    gen = torch.Generator(device=dev)
    gen.manual_seed(2609)

    def randn(shape):
        return torch.randn(shape, generator=gen, device=dev, dtype=torch.float32).to(torch.bfloat16)

    q, k, v, do = randn((1, HQ, N, D)), randn((1, HK, N, D)), randn((1, HK, N, D)), randn((1, HQ, N, D))
    log("all 8 KV heads at 131072 tokens")
    full = _run(q, k, v, do, HK, 0)
    torch.cuda.synchronize()
    g = HQ // HK
    for r in (0, 3, 7):
        log(f"rank {r} of 8: KV head {r}, QO heads {g * r}..{g * r + g - 1}")
        qs, ks, vs, dos = (x[:, a:b].contiguous() for x, a, b in ((q, g * r, g * r + g), (k, r, r + 1),
                                                                  (v, r, r + 1), (do, g * r, g * r + g)))
        part = _run(qs, ks, vs, dos, HK, r)
        torch.cuda.synchronize()
        for name, a, b, sl in (("O", part[0], full[0], slice(g * r, g * r + g)),
                               ("LSE", part[1], full[1], slice(g * r, g * r + g)),
                               ("dQ", part[2], full[2], slice(g * r, g * r + g)),
                               ("dK", part[3], full[3], slice(r, r + 1)),
                               ("dV", part[4], full[4], slice(r, r + 1))):
            ref = b[:, sl]
            same = torch.equal(a, ref)
            if not same:
                diff = (a.float() - ref.float()).abs().max().item()
                log(f"  {name}: max |diff| {diff:.3e}")
            assert same, f"rank {r}: {name} differs from the all-heads run"
        log(f"  rank {r}: O, LSE, dQ, dK, dV bitwise equal")
