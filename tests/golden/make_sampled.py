#!/usr/bin/env python3
"""Write the sampled fp64-oracle values of the 32K and 128K training workloads.

The GPU parity tests at these sizes run the kernels on the full seeded inputs
and compare a sample of their outputs, element by element, with the values
this script stores.  It calls only ``oracle/`` (the float64 reference) and
``inputs/`` (the seeded draws); nothing here comes from the HIP path.

Sample (per workload):

* query rows -- O, LSE and dQ for every QO head on 16 QO blocks: the first
  and the last block, every block where some KV head's long-range window
  starts (query i_q = lo_h, its first visible distance) or stops being
  clipped by the start of the sequence (i_q = hi_h - 1), and random blocks to
  make up 16; in each block 8 rows at a seeded offset and stride 16, plus the
  block's first and last rows.  lo_h = w_near + b_h and hi_h = w_near + b_{h+1}
  are the long-window distance bounds of Eq. fwa_long_range_span.
* key rows -- dK and dV for every KV head: a sink key (i_k < w_sink, seen by
  every later query of the group), a key seen only through the near window
  (i_k > N_k - lo_h - 1), a key inside that head's long-range window
  (w_sink <= i_k < N_k - lo_h), and the last key.  Each key row is exact: every
  query that sees it is evaluated over its whole visible set (Alg. 2).

A third sample, ``bf16_t128k_wide``, takes the 128K workload with Q scaled
by 32 (exact in bf16: a power of two), so that the softmax of most rows spans
far more than the forward's exponent headroom; it stores O and LSE of the same
kind of query sample (forward only).

Usage: python tests/golden/make_sampled.py [bf16_t32k_b2] [bf16_t128k] [bf16_t128k_wide]
Writes tests/golden/sampled_<workload>.npz (float32 values, int64 indices).
"""

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import inputs  # noqa: E402
from oracle import attention as ref, windows as ow  # noqa: E402

N_BLOCKS = 16


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def sample_query_rows(w, rng):
    """(b, h, i_q) rows of the query sample and the block list."""
    tile = w.tile
    n_qt = -(-w.n_q // tile)
    blocks = {0, n_qt - 1}
    for hk in range(w.h_k):
        lo, hi = ow.long_window_bounds(w.n_k, w.w_sink, w.w_near, hk, w.h_k)
        off = w.n_k - w.n_q
        # the first query whose long window is non-empty, and the first whose
        # long window is no longer clipped at key 0
        for pos in (lo - off, hi - 1 - off):
            if 0 <= pos < w.n_q:
                blocks.add(pos // tile)
    extra = [int(x) for x in rng.permutation(n_qt)]
    for x in extra:
        if len(blocks) >= N_BLOCKS:
            break
        blocks.add(x)
    blocks = sorted(blocks)
    rows = []
    for blk in blocks:
        b = int(rng.integers(0, w.batch))
        for h in range(w.h_q):
            off = int(rng.integers(0, 16))
            first, last = blk * tile, min((blk + 1) * tile, w.n_q) - 1
            picks = {first, last} | {first + off + 16 * t for t in range(8)}
            rows += [(b, h, i) for i in sorted(picks) if i <= last]
    return blocks, rows


def sample_key_rows(w, rng):
    """(b, h_k, i_k) rows of the key sample."""
    rows = []
    for hk in range(w.h_k):
        b = int(rng.integers(0, w.batch))
        lo, _ = ow.long_window_bounds(w.n_k, w.w_sink, w.w_near, hk, w.h_k)
        sink = int(rng.integers(0, w.w_sink))
        near_only = int(rng.integers(max(w.n_k - lo, w.w_sink), w.n_k - 1))
        long_key = int(rng.integers(w.w_sink, max(w.n_k - lo, w.w_sink + 1)))
        for i in (sink, near_only, long_key, w.n_k - 1):
            if (b, hk, i) not in rows:
                rows.append((b, hk, i))
    return rows


def make(name):
    w = inputs.WORKLOADS[name]
    rng = np.random.default_rng(inputs.key_of("golden", name))
    blocks, q_rows = sample_query_rows(w, rng)
    kv_rows = sample_key_rows(w, rng)
    log(f"{name}: {len(blocks)} QO blocks {blocks}, {len(q_rows)} query rows, {len(kv_rows)} key rows")
    t0 = time.perf_counter()
    t = inputs.train_tensors(w)
    q, k, v, do = (t[n][1] for n in ("q", "k", "v", "do"))
    del t
    log(f"  inputs: {time.perf_counter() - t0:.1f} s")
    t0 = time.perf_counter()
    dq, o, lse = ref.backward_q_rows(q, k, v, do, q_rows, w.w_sink, w.w_near, w.scale)
    log(f"  query rows: {time.perf_counter() - t0:.1f} s")
    dk = np.zeros((len(kv_rows), w.head_dim))
    dv = np.zeros((len(kv_rows), w.head_dim))
    for hk in range(w.h_k):
        sel = [n for n, r in enumerate(kv_rows) if r[1] == hk]
        t0 = time.perf_counter()
        a, c = ref.backward_kv_rows(q, k, v, do, [kv_rows[n] for n in sel], w.w_sink, w.w_near, w.scale)
        dk[sel], dv[sel] = a, c
        log(f"  key rows of KV head {hk}: {time.perf_counter() - t0:.1f} s")
    out = os.path.join(HERE, f"sampled_{name}.npz")
    np.savez(out, workload=np.array(name), q_rows=np.array(q_rows, dtype=np.int64),
             o=o.astype(np.float32), lse=lse.astype(np.float32), dq=dq.astype(np.float32),
             kv_rows=np.array(kv_rows, dtype=np.int64), dk=dk.astype(np.float32), dv=dv.astype(np.float32),
             q_blocks=np.array(blocks, dtype=np.int64))
    log(f"  wrote {out} ({os.path.getsize(out) / 1e6:.1f} MB)")


WIDE_SCALE = 32.0  # Q multiplier of the wide-score sample


def make_wide(name="bf16_t128k_wide", base="bf16_t128k"):
    w = inputs.WORKLOADS[base]
    rng = np.random.default_rng(inputs.key_of("golden", name))
    blocks, q_rows = sample_query_rows(w, rng)
    log(f"{name}: {len(blocks)} QO blocks {blocks}, {len(q_rows)} query rows")
    t0 = time.perf_counter()
    t = inputs.train_tensors(w, which=("q", "k", "v"))
    q, k, v = (t[n][1] for n in ("q", "k", "v"))
    del t
    q = q * WIDE_SCALE
    log(f"  inputs: {time.perf_counter() - t0:.1f} s")
    t0 = time.perf_counter()
    o, lse = ref.forward_rows(q, k, v, q_rows, w.w_sink, w.w_near, w.scale)
    log(f"  query rows: {time.perf_counter() - t0:.1f} s")
    out = os.path.join(HERE, f"sampled_{name}.npz")
    np.savez(out, workload=np.array(name), base=np.array(base), q_scale=np.array(WIDE_SCALE),
             q_rows=np.array(q_rows, dtype=np.int64), o=o.astype(np.float32), lse=lse.astype(np.float32),
             q_blocks=np.array(blocks, dtype=np.int64))
    log(f"  wrote {out} ({os.path.getsize(out) / 1e6:.1f} MB)")


if __name__ == "__main__":
    names = sys.argv[1:] or ["bf16_t32k_b2", "bf16_t128k", "bf16_t128k_wide"]
    for n in names:
        make_wide(n) if n == "bf16_t128k_wide" else make(n)
