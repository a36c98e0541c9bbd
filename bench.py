#!/usr/bin/env python3
"""Benchmark of the CoWA hot path on one MI355X.

One step is one pass of the whole hot path over one batch of synthetic input:

  window tuples (host) -> schedule build -> forward -> backward (prepare, dK/dV
  pass, dQ pass) at 131072 tokens, bf16, B=1, H_q=32, H_k=8, d=128, sink 128, near
  4096, 128x128 blocks; then one decoding step over 64 sequences x 131072
  cached tokens with the same heads and windows.

``value`` is the effective TFLOP/s of the training path (forward + backward):
algorithmic FLOPs (4d per legal query-key pair forward, 10d backward, summed
over every QO head) divided by the mean time of schedule + forward + backward
per step.  Every kernel is timed with HIP events on the stream it runs on.
The decoding step is reported as ms and effective HBM GB/s (visible K/V rows,
q, O and LSE bytes).  Inputs are N(0, 1) bf16 drawn on the device from a
generator seeded with 42, resident in HBM before timing starts.

Extra blocks in the JSON line:
  roofline      the dominant kernel (backward main pass) against the bf16
                MFMA peak; traffic from committed rocprofv3 counter summaries
  kernels       every kernel's time, work and roofline fraction (decode with
                its counter bytes over the algorithmic bytes)
  workloads     forward / backward times and fractions at 8192 tokens and at
                2 x 32768 tokens, and one rank's share of the 131072-token
                step in the paper's 8-way KV-head tensor parallelism (1 KV
                head, 4 QO heads, global KV head 0 = heaviest and 7 = lightest)
  dense         the same kernels in dense causal mode (w_sink = 0,
                w_near = N), the in-house FullAttn twin, and CoWA/dense ratios
  cpu_baseline  the fp64 CPU oracle timed on a bounded sample of the same
                workload on this host (with the host's CPU model and memory)
  ceilings      what the device sustains outside this library: a 16384^3
                bf16 GEMM through torch.matmul (hipBLASLt) and a 4 GiB device
                copy and a read-only sum over it (torch's own kernels, which
                reach less than the decoding kernel here); each matrix kernel
                also reports its rate as a fraction of the GEMM

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
"""

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E
PAPER_RATIOS = {"fwd": 7.4, "bwd": 8.6, "decode": 3.0,
                "hardware": "8x NVIDIA H100 (SM90), TP=8, BF16, batch 1, 64 QO / 8 KV heads, d=128, 128K"}

TRAIN = dict(batch=1, n=131072, h_q=32, h_k=8, d=128, w_sink=128, w_near=4096, tile=128)
DECODE = dict(batch=64, n=131072, h_q=32, h_k=8, d=128, w_sink=128, w_near=4096)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_digest(path):
    """What a kernel's code object depends on: its source, its per-file compile
    options and the shared headers of the sources' directory."""
    from paper_2609_32704_amd.build import FILE_FLAGS
    h = hashlib.sha256()
    with open(path, "rb") as f:
        h.update(f.read())
    h.update(b"\0" + " ".join(FILE_FLAGS.get(os.path.basename(path), [])).encode())
    folder = os.path.dirname(path)
    for name in sorted(os.listdir(folder)):
        if name.endswith(".h"):
            with open(os.path.join(folder, name), "rb") as f:
                h.update(b"\0" + name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


def read_traffic(kernel):
    """HBM bytes per launch from the committed counter summary
    (profiles/hbm_traffic.txt), or None when missing or when the kernel's
    source changed after the counters were taken."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.txt")
    if not os.path.exists(path):
        return None
    for line in open(path):
        parts = line.split()
        if len(parts) >= 4 and parts[0] == kernel and not line.startswith("#"):
            src, digest, nbytes = parts[1], parts[2], parts[3]
            try:
                if source_digest(os.path.join(ROOT, src)) != digest:
                    return None
            except OSError:
                return None
            return float(nbytes)
    return None


def host_info():
    """CPU model, logical CPUs and memory of this host."""
    model, mem_gb = "unknown", None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal"):
                mem_gb = round(int(line.split()[1]) / 1024 ** 2, 1)
                break
    except OSError:
        pass
    return {"cpu_model": model, "logical_cpus": os.cpu_count(), "ram_gib": mem_gb}


def cpu_baseline(target_s=12.0):
    """The fp64 oracle (as it stands) on a bounded sample of the 128K training
    workload: every QO-head row of a few 128-row query blocks, full forward
    and backward work of those rows (their dK/dV contributions included)."""
    import numpy as np
    import inputs
    from oracle import attention as ref, counts
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count() or 1])
    except Exception:  # noqa: BLE001
        threads = os.cpu_count() or 1
    w = inputs.WORKLOADS["bf16_t128k"]
    rng = np.random.default_rng(7)
    # inputs: the rows the sample touches come from the same seeded streams (full tensors)
    log("cpu_baseline: generating inputs")
    t = inputs.train_tensors(w)
    q, k, v, do = (t[n][1] for n in ("q", "k", "v", "do"))
    sizes = {hk: counts.support_table(w.n_q, w.n_k, w.w_sink, w.w_near, w.h_k)[hk] for hk in range(w.h_k)}
    done_pairs, elapsed, blocks = 0, 0.0, []
    n_qt = w.n_q // w.tile
    while elapsed < target_s and len(blocks) < 64:
        blk = int(rng.integers(0, n_qt))
        h = int(rng.integers(0, w.h_q))
        rows = np.arange(blk * w.tile, (blk + 1) * w.tile)
        t0 = time.perf_counter()
        ref.backward(q, k, v, do, w.w_sink, w.w_near, w.scale, rows=rows, heads=[h])
        elapsed += time.perf_counter() - t0
        done_pairs += int(sizes[(h * w.h_k) // w.h_q][rows].sum())
        blocks.append((h, blk))
    flops = 14 * w.head_dim * done_pairs
    return {"value": flops / elapsed / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "seconds": round(elapsed, 3), "host": host_info(),
            "sample": f"{len(blocks)} (QO head, 128-row query block) pairs of the 131072-token workload, "
                      f"full fp64 forward+backward of those rows ({done_pairs} legal pairs, 14d FLOPs each)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--dense-iters", type=int, default=2)
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-workloads", action="store_true", help="skip the 8K / 32K / per-rank timings")
    ap.add_argument("--no-ceiling", action="store_true", help="skip the vendor GEMM / copy reference timings")
    ap.add_argument("--only", choices=["all", "train", "decode", "copy", "ceiling"], default="all",
                    help="profiling aid: run only part of the step (the JSON line is printed for 'all' only)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on exactly one GPU: the CoWA path shards by KV head with no exchange, "
              "and this build measures one device's share (--gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_32704_amd as cowa
    from paper_2609_32704_amd import _abi

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream().cuda_stream
    gen = torch.Generator(device=dev)
    gen.manual_seed(42)

    def randn(shape):
        """N(0, 1) bf16 drawn on the device, one leading slice at a time."""
        out = torch.empty(shape, dtype=torch.bfloat16, device=dev)
        for s in range(shape[0]):
            out[s].copy_(torch.randn(shape[1:], generator=gen, device=dev, dtype=torch.float32))
        return out

    def ceilings():
        """What the device sustains outside this library: a bf16 GEMM through
        torch.matmul (hipBLASLt) and a device-to-device copy, timed with HIP
        events.  Under sustained matrix-core load the shader clock drops well
        below its 2.4 GHz peak, so the vendor GEMM bounds what any bf16 kernel
        reaches in practice."""
        n = 16384
        a = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
        b = torch.randn(n, n, device=dev, dtype=torch.bfloat16)
        for _ in range(6):  # the shader clock settles over the first launches
            c = a @ b
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(10):
            c = a @ b
        e1.record()
        torch.cuda.synchronize()
        gemm_ms = e0.elapsed_time(e1) / 10
        del a, b, c
        src = torch.empty(4 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(5):
            dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        copy_ms = e0.elapsed_time(e1) / 5
        del dst
        x = src.view(torch.float32)
        tot = x.sum()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(5):
            tot = x.sum()
        e1.record()
        torch.cuda.synchronize()
        read_ms = e0.elapsed_time(e1) / 5
        del src, x, tot
        return {"gemm_bf16_tflops": 2 * n ** 3 / (gemm_ms * 1e-3) / 1e12, "gemm_shape": f"{n}x{n}x{n}",
                "copy_gbps": 2 * (4 << 30) / (copy_ms * 1e-3) / 1e9, "read_gbps": (4 << 30) / (read_ms * 1e-3) / 1e9,
                "hbm_bytes": 4 << 30,
                "note": "torch.matmul (hipBLASLt) bf16 GEMM (6 warm-up + 10 timed); a 4 GiB device copy (read + "
                        "write bytes) and a float32 sum over the same 4 GiB (read bytes), 5 runs each"}

    if args.only == "ceiling":
        log("ceilings:", ceilings())
        return

    if args.only == "copy":
        # plain device copy of a known size: the reference for HBM byte counters
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst2 = torch.empty_like(src)
        for _ in range(3):
            dst2.copy_(src)
        torch.cuda.synchronize()
        log("copied 3 x 1 GiB")
        return

    ceil = None
    if args.only == "all" and not args.no_ceiling:
        log("vendor GEMM and copy reference timings")
        ceil = ceilings()
    do_train = args.only in ("all", "train")
    do_decode = args.only in ("all", "decode")
    T = TRAIN
    log("allocating training inputs")
    tq = (T["batch"], T["h_q"], T["n"], T["d"]) if do_train else (1, 1, 1, T["d"])
    tk = (T["batch"], T["h_k"], T["n"], T["d"]) if do_train else (1, 1, 1, T["d"])
    q = randn(tq)
    k = randn(tk)
    v = randn(tk)
    do = randn(tq)
    o = torch.empty_like(q)
    lse = torch.empty((T["batch"], T["h_q"], T["n"]), dtype=torch.float32, device=dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)

    def params(w_sink, w_near):
        return cowa.make_params(T["batch"], T["n"], T["n"], T["h_q"], T["h_k"], T["d"], w_sink, w_near,
                                T["tile"], T["tile"])

    p = params(T["w_sink"], T["w_near"])
    sched = cowa.Schedule(p, dev, build=False)
    ws_bytes = _abi.cowa_bwd_workspace_size(p)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    pairs = _abi.cowa_legal_pairs(p)
    fwd_flops = 4 * T["d"] * pairs
    bwd_flops = 10 * T["d"] * pairs

    D = DECODE
    log("allocating decode inputs (2 x 17 GB KV cache)")
    dq_in = randn((D["batch"], D["h_q"], D["d"]))
    kc = randn((D["batch"], D["h_k"], D["n"], D["d"]) if do_decode else (1, 1, 1, D["d"]))
    vc = randn((D["batch"], D["h_k"], D["n"], D["d"]) if do_decode else (1, 1, 1, D["d"]))
    seqlens_host = [D["n"]] * D["batch"]
    seqlens = torch.tensor(seqlens_host, dtype=torch.int32, device=dev)
    dpar = cowa.make_decode_params(D["batch"], D["h_q"], D["h_k"], D["d"], D["n"], D["w_sink"], D["w_near"])
    dws = torch.empty(_abi.cowa_decode_workspace_size(dpar), dtype=torch.uint8, device=dev)
    od = torch.empty_like(dq_in)
    lsed = torch.empty((D["batch"], D["h_q"]), dtype=torch.float32, device=dev)
    vis_keys = _abi.cowa_decode_visible_keys(dpar, seqlens_host)
    dec_bytes = 2 * vis_keys * D["d"] * 2 + D["batch"] * D["h_q"] * (2 * D["d"] * 2 + 4)

    names = ["schedule", "fwd", "bwd_prepare", "bwd_main", "bwd_dq", "decode"]

    def step(evs):
        evs[0].record()
        if not do_train:
            for e in evs[1:6]:
                e.record()
            _abi.cowa_decode(dpar, dq_in.data_ptr(), kc.data_ptr(), vc.data_ptr(), seqlens.data_ptr(),
                             od.data_ptr(), lsed.data_ptr(), dws.data_ptr(), dws.numel(), stream)
            evs[6].record()
            return
        _abi.cowa_windows(p)
        _abi.cowa_schedule(sched.s, stream)
        evs[1].record()
        _abi.cowa_fwd(p, sched.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), stream)
        evs[2].record()
        _abi.cowa_bwd_prepare(p, o.data_ptr(), do.data_ptr(), lse.data_ptr(), ws.data_ptr(), ws_bytes, stream)
        evs[3].record()
        _abi.cowa_bwd_main(p, sched.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), do.data_ptr(), dk.data_ptr(),
                           dv.data_ptr(), ws.data_ptr(), ws_bytes, stream)
        evs[4].record()
        _abi.cowa_bwd_dq(p, sched.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), do.data_ptr(), dq.data_ptr(),
                         ws.data_ptr(), ws_bytes, stream)
        evs[5].record()
        if do_decode:
            _abi.cowa_decode(dpar, dq_in.data_ptr(), kc.data_ptr(), vc.data_ptr(), seqlens.data_ptr(),
                             od.data_ptr(), lsed.data_ptr(), dws.data_ptr(), dws.numel(), stream)
        evs[6].record()

    def new_events():
        return [torch.cuda.Event(enable_timing=True) for _ in range(7)]

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        step(new_events())
    torch.cuda.synchronize()
    log(f"timing {args.steps} steps")
    all_evs = [new_events() for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for evs in all_evs:
        step(evs)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    samples = {n: [evs[idx].elapsed_time(evs[idx + 1]) for evs in all_evs] for idx, n in enumerate(names)}
    per = {n: sum(x) / args.steps for n, x in samples.items()}
    if args.only != "all":
        log("per-kernel ms:", {n: round(x, 3) for n, x in per.items()})
        return
    bwd_ms = per["bwd_prepare"] + per["bwd_main"] + per["bwd_dq"]
    train_ms = per["schedule"] + per["fwd"] + bwd_ms
    value = (fwd_flops + bwd_flops) / (train_ms * 1e-3) / 1e12

    rows_q = T["batch"] * T["h_q"] * T["n"]
    elem_q = rows_q * T["d"]
    kernels = {
        "schedule": {"ms": per["schedule"], "bound": "launch", "note": "three small kernels"},
        "fwd": {"ms": per["fwd"], "bound": "mfma", "work": fwd_flops, "unit": "TFLOP/s",
                "achieved": fwd_flops / (per["fwd"] * 1e-3) / 1e12},
        # reads O, dO and LSE, writes -D and -LSE log2(e)
        "bwd_prepare": {"ms": per["bwd_prepare"], "bound": "hbm", "unit": "GB/s", "work": 2 * elem_q * 2 + rows_q * 12,
                        "achieved": (2 * elem_q * 2 + rows_q * 12) / (per["bwd_prepare"] * 1e-3) / 1e9},
        # algorithmic share of the backward's 10d per pair: the dK/dV pass does the
        # recompute of S and dP plus dV and dK (8d); the dQ pass adds dQ (2d) and
        # recomputes S and dP again (4d executed on top, not counted)
        "bwd_main": {"ms": per["bwd_main"], "bound": "mfma", "work": 8 * T["d"] * pairs, "unit": "TFLOP/s",
                     "achieved": 8 * T["d"] * pairs / (per["bwd_main"] * 1e-3) / 1e12},
        "bwd_dq": {"ms": per["bwd_dq"], "bound": "mfma", "work": 2 * T["d"] * pairs, "unit": "TFLOP/s",
                   "achieved": 2 * T["d"] * pairs / (per["bwd_dq"] * 1e-3) / 1e12,
                   "executed_tflops": 6 * T["d"] * pairs / (per["bwd_dq"] * 1e-3) / 1e12},
        "decode": {"ms": per["decode"], "bound": "hbm", "unit": "GB/s", "work": dec_bytes,
                   "achieved": dec_bytes / (per["decode"] * 1e-3) / 1e9},
    }
    for n, kn in kernels.items():
        kn["ms_median"] = statistics.median(samples[n])
        kn["ms_min"] = min(samples[n])
        if kn["bound"] == "mfma":
            kn["frac"] = kn["achieved"] / PEAK_BF16_TFLOPS
        elif kn["bound"] == "hbm":
            kn["frac"] = kn["achieved"] / PEAK_HBM_GBPS
    # tile-FLOP rates: every listed tile (schedule entry x QO heads of its group x
    # sequences) at its full B_q x B_k size, i.e. the work the matrix cores see
    # including the masked part of partial tiles
    tile_pairs = sched.nnz * (T["h_q"] // T["h_k"]) * T["batch"] * T["tile"] * T["tile"]
    for n, per_pair in (("fwd", 4), ("bwd_main", 8), ("bwd_dq", 6)):
        kernels[n]["tile_tflops"] = per_pair * T["d"] * tile_pairs / (per[n] * 1e-3) / 1e12
    kernels["fwd"]["tile_fill"] = pairs / tile_pairs
    # the split partials (m, l and float32 O per split and QO head): written by
    # the split kernel, read by the combine kernel; not in the algorithmic bytes
    kernels["decode"]["partial_state_bytes"] = 2 * dws.numel()

    if ceil:
        for kn in kernels.values():
            if kn["bound"] == "mfma":
                kn["frac_of_gemm"] = kn["achieved"] / ceil["gemm_bf16_tflops"]

    main_k = kernels["bwd_main"]
    traffic = read_traffic("bwd_main")
    roofline = {"kernel": "bwd_main (backward dK/dV pass, 131072 tokens)", "bound": "mfma",
                "achieved": main_k["achieved"], "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": main_k["frac"], "traffic": traffic,
                "frac_of_gemm_ceiling": main_k.get("frac_of_gemm"),
                "work_per_launch": f"{8 * T['d'] * pairs:.4e} FLOP = 8 d x {pairs} legal pairs"}

    # decode: counter bytes (both kernels) over the algorithmic bytes
    t_split, t_comb = read_traffic("decode_split"), read_traffic("decode_combine")
    if t_split is not None and t_comb is not None:
        kernels["decode"]["traffic"] = t_split + t_comb
        kernels["decode"]["traffic_over_algorithmic"] = (t_split + t_comb) / dec_bytes

    workloads = None
    if not args.no_workloads:
        log("other workloads: 8192 tokens, 2 x 32768 tokens, per-rank shares of the 131072-token step")
        workloads = {}

        def time_train(par, tq, tk, tv, tdo, iters):
            """Mean ms of schedule+forward and of the backward, HIP events on the launch stream."""
            sch = cowa.Schedule(par, dev, build=False)
            o_ = torch.empty_like(tq)
            lse_ = torch.empty(tq.shape[:3], dtype=torch.float32, device=dev)
            dq_, dk_, dv_ = torch.empty_like(tq), torch.empty_like(tk), torch.empty_like(tv)
            wsb = _abi.cowa_bwd_workspace_size(par)
            ws_ = torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
            tf = tb = 0.0
            stages = [0.0, 0.0, 0.0]  # backward prepare, dK/dV pass, dQ pass
            for it in range(iters + 1):
                e = [torch.cuda.Event(enable_timing=True) for _ in range(5)]
                e[0].record()
                _abi.cowa_schedule(sch.s, stream)
                _abi.cowa_fwd(par, sch.s, tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), o_.data_ptr(),
                              lse_.data_ptr(), stream)
                e[1].record()
                _abi.cowa_bwd_prepare(par, o_.data_ptr(), tdo.data_ptr(), lse_.data_ptr(), ws_.data_ptr(), wsb, stream)
                e[2].record()
                _abi.cowa_bwd_main(par, sch.s, tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), tdo.data_ptr(),
                                   dk_.data_ptr(), dv_.data_ptr(), ws_.data_ptr(), wsb, stream)
                e[3].record()
                _abi.cowa_bwd_dq(par, sch.s, tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), tdo.data_ptr(),
                                 dq_.data_ptr(), ws_.data_ptr(), wsb, stream)
                e[4].record()
                torch.cuda.synchronize()
                if it:
                    tf += e[0].elapsed_time(e[1]) / iters
                    tb += e[1].elapsed_time(e[4]) / iters
                    for x in range(3):
                        stages[x] += e[x + 1].elapsed_time(e[x + 2]) / iters
            pr = _abi.cowa_legal_pairs(par)
            d_ = par.head_dim
            return {"fwd_ms": tf, "bwd_ms": tb, "legal_pairs": pr,
                    "bwd_prepare_ms": stages[0], "bwd_main_ms": stages[1], "bwd_dq_ms": stages[2],
                    "fwd_tflops": 4 * d_ * pr / (tf * 1e-3) / 1e12, "bwd_tflops": 10 * d_ * pr / (tb * 1e-3) / 1e12,
                    "fwd_frac": 4 * d_ * pr / (tf * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                    "bwd_frac": 10 * d_ * pr / (tb * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}

        for name, (bsz, n, ws_w, wn_w, tile) in (("bf16_t8k", (1, 8192, 64, 1024, 64)),
                                                ("bf16_t32k_b2", (2, 32768, 64, 2048, 128))):
            tq2, tk2 = randn((bsz, 32, n, 128)), randn((bsz, 8, n, 128))
            tv2, tdo2 = randn((bsz, 8, n, 128)), randn((bsz, 32, n, 128))
            par = cowa.make_params(bsz, n, n, 32, 8, 128, ws_w, wn_w, tile, tile)
            workloads[name] = dict(time_train(par, tq2, tk2, tv2, tdo2, 10),
                                   shape=f"B={bsz}, T={n}, 32 QO / 8 KV heads, d=128, sink {ws_w}, near {wn_w}, "
                                         f"{tile}x{tile} blocks")
            del tq2, tk2, tv2, tdo2
        if do_train:
            # one rank of the 8-way KV-head split: its KV head (global index r) and the 4 QO heads
            # of that head's group (contiguous leading heads of the 131072-token tensors)
            for r in (0, 7):
                par = cowa.make_params(1, T["n"], T["n"], 4, 1, T["d"], T["w_sink"], T["w_near"], T["tile"],
                                       T["tile"], h_k_total=8, h_k_offset=r)
                workloads[f"tp8_rank{r}"] = dict(
                    time_train(par, q[:, :4], k[:, :1], v[:, :1], do[:, :4], 5),
                    shape=f"131072 tokens, one rank of 8: global KV head {r}, 4 QO heads")
            # the forward with a wide score range: Q scaled by 40, so that in most rows later
            # scores climb far past the row's first 32 keys: the exponent offset moves at block
            # ends several times per row, and rows whose maximum jumps past the headroom within
            # one block run a second pass (the worst case of the forward's softmax offset)
            qw = (q.float() * 40.0).to(torch.bfloat16)
            ow = torch.empty_like(qw)
            tw = 0.0
            for it in range(4):
                e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                e[0].record()
                _abi.cowa_fwd(p, sched.s, qw.data_ptr(), k.data_ptr(), v.data_ptr(), ow.data_ptr(), lse.data_ptr(),
                              stream)
                e[1].record()
                torch.cuda.synchronize()
                if it:
                    tw += e[0].elapsed_time(e[1]) / 3
            workloads["fwd_wide_scores"] = {
                "fwd_ms": tw, "fwd_ms_normal_scores": per["fwd"], "slowdown": tw / per["fwd"],
                "shape": "the 131072-token forward with Q scaled by 40 (the softmax offset moves often; "
                         "a few rows run the second pass)"}
            del qw, ow

    dense = None
    if not args.no_dense and args.dense_iters > 0:
        log("dense causal twin")
        pd = params(0, T["n"])
        sd = cowa.Schedule(pd, dev)
        dpairs = _abi.cowa_legal_pairs(pd)
        ddp = cowa.make_decode_params(D["batch"], D["h_q"], D["h_k"], D["d"], D["n"], 0, D["n"])
        dws2 = torch.empty(_abi.cowa_decode_workspace_size(ddp), dtype=torch.uint8, device=dev)
        times = {"fwd": 0.0, "bwd": 0.0, "decode": 0.0}
        for it in range(args.dense_iters + 1):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            e[0].record()
            _abi.cowa_fwd(pd, sd.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(), stream)
            e[1].record()
            _abi.cowa_bwd(pd, sd.s, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), lse.data_ptr(),
                          do.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), ws.data_ptr(), ws_bytes,
                          stream)
            e[2].record()
            _abi.cowa_decode(ddp, dq_in.data_ptr(), kc.data_ptr(), vc.data_ptr(), seqlens.data_ptr(),
                             od.data_ptr(), lsed.data_ptr(), dws2.data_ptr(), dws2.numel(), stream)
            e[3].record()
            torch.cuda.synchronize()
            if it > 0:
                times["fwd"] += e[0].elapsed_time(e[1])
                times["bwd"] += e[1].elapsed_time(e[2])
                times["decode"] += e[2].elapsed_time(e[3])
        times = {kk: vv / args.dense_iters for kk, vv in times.items()}
        cowa_fwd_ms = per["schedule"] + per["fwd"]
        dense = {"fwd_ms": times["fwd"], "bwd_ms": times["bwd"], "decode_ms": times["decode"],
                 "fwd_tflops": 4 * T["d"] * dpairs / (times["fwd"] * 1e-3) / 1e12,
                 "bwd_tflops": 10 * T["d"] * dpairs / (times["bwd"] * 1e-3) / 1e12,
                 "ratio_fwd": times["fwd"] / cowa_fwd_ms, "ratio_bwd": times["bwd"] / bwd_ms,
                 "ratio_decode": times["decode"] / per["decode"],
                 "work_ratio_train": dpairs / pairs,
                 "paper_ratios": PAPER_RATIOS, "iters": args.dense_iters}

    cpu = None
    if not args.no_cpu:
        log("cpu baseline (fp64 oracle on a bounded sample)")
        cpu = cpu_baseline()

    out = {
        "metric": "fwd/bwd ms + effective TFLOP/s at 128K bf16; decode ms/step and HBM GB/s",
        "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "CoWA fwd+bwd at 131072 tokens + decode of 64 x 131072-token caches",
                   "batch": T["batch"], "seq_len": T["n"], "h_q": T["h_q"], "h_k": T["h_k"],
                   "head_dim": T["d"], "w_sink": T["w_sink"], "w_near": T["w_near"], "tile": T["tile"],
                   "decode_batch": D["batch"], "decode_cache_len": D["n"],
                   "parallelism": "one GPU holding all 8 KV heads (the 8 KV-head TP shares)"},
        "fwd_ms": per["schedule"] + per["fwd"], "bwd_ms": bwd_ms,
        "fwd_tflops": fwd_flops / ((per["schedule"] + per["fwd"]) * 1e-3) / 1e12,
        "bwd_tflops": bwd_flops / (bwd_ms * 1e-3) / 1e12,
        "decode_ms": per["decode"], "decode_gbps": dec_bytes / (per["decode"] * 1e-3) / 1e9,
        "legal_pairs": pairs, "decode_visible_keys": vis_keys,
        "roofline": roofline, "kernels": kernels, "workloads": workloads, "dense": dense, "cpu_baseline": cpu,
        "ceilings": ceil,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
