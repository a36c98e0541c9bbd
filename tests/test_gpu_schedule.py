"""GPU schedule builder vs the oracle's schedule: bit-exact, every array."""

import numpy as np
import pytest

import inputs
from oracle import schedule as oracle_schedule
from gpu_util import need_gpu, log, torch

pytestmark = pytest.mark.gpu

KEYS = ("fwd_row_ptr", "fwd_ent", "bwd_col_ptr", "bwd_ent")


def _check(n_q, n_k, tq, tk, ws, wn, hk, ht=None, ho=0, h_q=None):
    import paper_2609_32704_amd as cowa
    need_gpu()
    ht = hk if ht is None else ht
    h_q = hk if h_q is None else h_q
    log(f"schedule n_q={n_q} n_k={n_k} tiles={tq}x{tk} sink={ws} near={wn} h_k={hk}/{ht}+{ho}")
    p = cowa.make_params(1, n_q, n_k, h_q, hk, 128, ws, wn, tq, tk, h_k_total=ht, h_k_offset=ho)
    s = cowa.Schedule(p)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in s.arrays().items()}
    ref = oracle_schedule.build(n_q, n_k, tq, tk, ws, wn, hk, ht, ho)
    assert s.nnz == len(ref["fwd_ent"])
    for key in KEYS:
        r = ref[key].astype(np.int64)
        g = got[key].astype(np.int64) & 0xFFFFFFFF
        assert np.array_equal(g, r), f"{key} differs"
    rl = np.diff(ref["fwd_row_ptr"])
    assert s.s.max_row == (rl.max() if rl.size else 0)


@pytest.mark.parametrize("name", ["fwd_fp32_t512", "bf16_t8k", "bf16_t32k_b2", "bf16_t128k"])
def test_schedule_workloads(name):
    w = inputs.WORKLOADS[name]
    _check(w.n_q, w.n_k, w.tile, w.tile, w.w_sink, w.w_near, w.h_k)


@pytest.mark.parametrize("case", [
    (1, 1, 32, 32, 0, 1, 1), (33, 77, 32, 64, 5, 9, 3), (100, 1000, 64, 32, 0, 0, 4),
    (999, 999, 128, 128, 130, 257, 8), (5000, 5003, 64, 128, 1, 1023, 8), (257, 4096, 32, 128, 64, 64, 2),
    (700, 700, 64, 64, 700, 0, 5), (640, 640, 128, 32, 0, 700, 2),
])
def test_schedule_odd_shapes(case):
    _check(*case)


def test_schedule_global_heads():
    for r in range(8):
        _check(4000, 4000, 128, 128, 16, 300, 1, ht=8, ho=r)
    _check(3000, 3100, 64, 64, 7, 100, 2, ht=8, ho=6)


def test_schedule_random_shapes():
    rng = np.random.default_rng(5)
    for _ in range(12):
        n_k = int(rng.integers(1, 3000))
        n_q = int(rng.integers(1, n_k + 1))
        ht = int(rng.integers(1, 9))
        hk = int(rng.integers(1, ht + 1))
        _check(n_q, n_k, int(rng.choice([32, 64, 128])), int(rng.choice([32, 64, 128])), int(rng.integers(0, 200)),
               int(rng.integers(0, 800)), hk, ht, int(rng.integers(0, ht - hk + 1)))


def _check_general(p, ref):
    import paper_2609_32704_amd as cowa
    s = cowa.Schedule(p)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in s.arrays().items()}
    assert s.nnz == len(ref["fwd_ent"])
    for key in KEYS:
        r = ref[key].astype(np.int64)
        g = got[key].astype(np.int64) & 0xFFFFFFFF
        assert np.array_equal(g, r), f"{key} differs"


@pytest.mark.parametrize("cu_q,cu_k", [([0, 70, 70, 200, 233], [0, 100, 131, 300, 500]),
                                       ([0, 1000, 1777, 2000], [0, 1000, 2000, 2500]),
                                       ([0, 0, 0, 5], [0, 0, 3, 9])])
@pytest.mark.parametrize("tuples", [None, [(1, 16, 5, 40), (0, 33, 0, 100), (50, 0, 3, 3)]])
def test_schedule_ragged(cu_q, cu_k, tuples):
    import paper_2609_32704_amd as cowa
    need_gpu()
    log(f"ragged schedule cu_q={cu_q} cu_k={cu_k} tuples={tuples}")
    for tq, tk in ((64, 32), (128, 128)):
        p = cowa.make_params(len(cu_q) - 1, cu_q[-1], cu_k[-1], 3, 3, 128, 4, 20, tq, tk, windows=tuples,
                             cu_seqlens_q=cu_q, cu_seqlens_k=cu_k)
        _check_general(p, oracle_schedule.build_varlen(cu_q, cu_k, tq, tk, 4, 20, 3, windows=tuples))


@pytest.mark.parametrize("tuples", [[(1, 16, 5, 40), (0, 33, 0, 100), (50, 0, 3, 3)],
                                    [(0, 1, 0, 10 ** 9), (7, 7, 10 ** 9, 10 ** 9), (2 ** 30, 0, 0, 0)]])
def test_schedule_tuples(tuples):
    import paper_2609_32704_amd as cowa
    need_gpu()
    for n_q, n_k, tq, tk in ((333, 1000, 64, 128), (1000, 1000, 128, 32)):
        p = cowa.make_params(1, n_q, n_k, 3, 3, 128, 4, 20, tq, tk, windows=tuples)
        _check_general(p, oracle_schedule.build(n_q, n_k, tq, tk, 4, 20, 3, windows=tuples))
