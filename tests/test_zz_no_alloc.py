"""cowa_decode_noalloc (the decoding step without a workspace: its split
partials live in a device array inside the library) against cowa_decode
with a caller workspace, through the C ABI, on two calls in a row, the second
with a smaller input: the outputs must be bitwise equal (same kernels, same
split sizes), which is within the parity bar of the tests."""

import numpy as np
import pytest

import inputs
from gpu_util import need_gpu, log, to_dev, torch

pytestmark = pytest.mark.gpu


def _run_both(abi, cowa, dev, bsz, h_q, h_k, d, n_max, seqlens, ws, wn, key):
    t = {n: inputs.normal_bf16(s, inputs.seed_sequence(inputs.key_of("noalloc", key), n))[0]
         for n, s in (("q", (bsz, h_q, d)), ("k", (bsz, h_k, n_max, d)), ("v", (bsz, h_k, n_max, d)))}
    q, kc, vc = (to_dev(t[n], dev) for n in ("q", "k", "v"))
    sl = torch.tensor(seqlens, dtype=torch.int32, device=dev)
    p = cowa.make_decode_params(bsz, h_q, h_k, d, n_max, ws, wn)
    stream = torch.cuda.current_stream().cuda_stream
    o_ref = torch.full_like(q, float("nan"))
    l_ref = torch.full((bsz, h_q), float("nan"), dtype=torch.float32, device=dev)
    need = abi.cowa_decode_workspace_size(p)
    work = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    abi.cowa_decode(p, q.data_ptr(), kc.data_ptr(), vc.data_ptr(), sl.data_ptr(), o_ref.data_ptr(), l_ref.data_ptr(),
                    work.data_ptr(), work.numel(), stream)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((bsz, h_q), float("nan"), dtype=torch.float32, device=dev)
    abi.cowa_decode_noalloc(p, q.data_ptr(), kc.data_ptr(), vc.data_ptr(), sl.data_ptr(), o.data_ptr(),
                            lse.data_ptr(), stream)
    torch.cuda.synchronize()
    log(f"noalloc decode B={bsz} h={h_q}/{h_k} d={d} n_max={n_max} workspace {need} bytes")
    assert not torch.isnan(o).any().item() and not torch.isnan(lse).any().item()
    assert torch.equal(o, o_ref), "O differs from cowa_decode"
    assert torch.equal(lse, l_ref), "LSE differs from cowa_decode"
    return need


def test_decode_noalloc_matches_decode_twice():
    import paper_2609_32704_amd as cowa
    from paper_2609_32704_amd import _abi as abi
    dev = need_gpu()
    big = _run_both(abi, cowa, dev, 8, 32, 8, 128, 40000, [40000, 1, 4225, 39999, 12345, 20000, 8, 40000], 128, 4096,
                    "first")
    small = _run_both(abi, cowa, dev, 2, 8, 2, 64, 3000, [3000, 777], 16, 256, "second")
    assert small < big
