"""Seeded synthetic inputs and the workload registry.

This module is shared by the tests, the benchmark and the smoke check.  It
holds no arithmetic of the attention method: only shapes, window sizes,
seeded normal draws and the bf16 rounding of those draws.

Input recipe: every tensor is drawn i.i.d. N(0, 1) as float32 from its own
PCG64 stream, seeded by ``SeedSequence(42, spawn_key=(workload, tensor))``
(42 is the fixed seed of the paper's training runs, App. A.3), and rounded to
bfloat16 with round-to-nearest-even for the bf16 workloads.  The kernels get
the bf16 bits; the oracle gets the same rounded values widened to float64.
The softmax scale is 1/sqrt(d) for every workload.  The paper's operator
benchmark runs on random tensors of these shapes (App. A.2); it names no
dataset, so there is none to stand in for.
"""

from dataclasses import dataclass, asdict
import math

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    n_q: int
    n_k: int
    h_q: int
    h_k: int
    head_dim: int
    w_sink: int
    w_near: int
    tile: int
    dtype: str            # "bf16" | "fp32"
    kind: str             # "train" (fwd+bwd) | "fwd" | "decode"
    h_total: int = 0      # 0: all KV heads are local
    h_offset: int = 0
    note: str = ""

    @property
    def scale(self):
        return 1.0 / math.sqrt(self.head_dim)

    @property
    def kv_total(self):
        return self.h_total or self.h_k

    def as_dict(self):
        return asdict(self)


# The five workloads the method is measured and checked on, plus tiny ones.
WORKLOADS = {
    "fwd_fp32_t512": Workload("fwd_fp32_t512", 1, 512, 512, 4, 2, 64, 16, 64, 32, "fp32", "fwd",
                              note="forward only, fp32, GQA 2"),
    "bf16_t8k": Workload("bf16_t8k", 1, 8192, 8192, 32, 8, 128, 64, 1024, 64, "bf16", "train"),
    "bf16_t32k_b2": Workload("bf16_t32k_b2", 2, 32768, 32768, 32, 8, 128, 64, 2048, 128, "bf16", "train",
                             note="training shape"),
    "bf16_t128k": Workload("bf16_t128k", 1, 131072, 131072, 32, 8, 128, 128, 4096, 128, "bf16", "train",
                           note="all 8 KV heads of the 8-way KV-head TP setup on one GPU"),
    "decode_64x128k": Workload("decode_64x128k", 64, 1, 131072, 32, 8, 128, 128, 4096, 128, "bf16",
                               "decode", note="64 sequences, contiguous KV cache of 131072 tokens"),
}

_WORKLOAD_KEYS = {name: i for i, name in enumerate(WORKLOADS)}
_TENSOR_KEYS = {"q": 0, "k": 1, "v": 2, "do": 3, "k_cache": 4, "v_cache": 5}


def seed_sequence(workload_key, tensor):
    """The SeedSequence of one tensor of one workload (or of a free-form test key)."""
    if isinstance(workload_key, str):
        workload_key = _WORKLOAD_KEYS.get(workload_key, None) if workload_key in _WORKLOAD_KEYS \
            else key_of(workload_key)
    return np.random.SeedSequence(42, spawn_key=(int(workload_key), _TENSOR_KEYS.get(tensor, key_of(tensor))))


def f32_to_bf16_bits(x):
    """Round float32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns as uint16.  NaN stays NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = rounded.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f64(bits):
    """Widen bfloat16 bit patterns (uint16) to float64 exactly."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def normal(shape, seq):
    """i.i.d. N(0, 1) float32 draws from the stream of ``seq``."""
    return np.random.Generator(np.random.PCG64(seq)).standard_normal(size=shape, dtype=np.float32)


def normal_bf16(shape, seq):
    """N(0, 1) draws rounded to bf16: returns (bits uint16, values float64)."""
    bits = f32_to_bf16_bits(normal(shape, seq))
    return bits, bf16_bits_to_f64(bits)


def train_tensors(w, which=("q", "k", "v", "do"), key=None, values=True):
    """Inputs of a forward/backward workload.  Returns {name: (device_payload,
    float64 values)} where the payload is uint16 bf16 bits or float32
    (values=False: the float64 values are None, which saves their memory)."""
    key = w.name if key is None else key
    shapes = {"q": (w.batch, w.h_q, w.n_q, w.head_dim), "k": (w.batch, w.h_k, w.n_k, w.head_dim),
              "v": (w.batch, w.h_k, w.n_k, w.head_dim), "do": (w.batch, w.h_q, w.n_q, w.head_dim)}
    out = {}
    for name in which:
        seq = seed_sequence(key, name)
        if w.dtype == "bf16":
            if values:
                out[name] = normal_bf16(shapes[name], seq)
            else:
                out[name] = (f32_to_bf16_bits(normal(shapes[name], seq)), None)
        else:
            x = normal(shapes[name], seq)
            out[name] = (x, x.astype(np.float64) if values else None)
    return out


def decode_tensors(w, n_max=None, key=None):
    """Inputs of a decode workload: q [B, H_q, d], caches [B, H_k, n_max, d]."""
    key = w.name if key is None else key
    n_max = w.n_k if n_max is None else n_max
    out = {}
    for name, shape in (("q", (w.batch, w.h_q, w.head_dim)),
                        ("k_cache", (w.batch, w.h_k, n_max, w.head_dim)),
                        ("v_cache", (w.batch, w.h_k, n_max, w.head_dim))):
        seq = seed_sequence(key, name)
        if w.dtype == "bf16":
            out[name] = normal_bf16(shape, seq)
        else:
            x = normal(shape, seq)
            out[name] = (x, x.astype(np.float64))
    return out


def custom(name, **kw):
    """A free-form workload for tests (tiny, ragged or odd shapes)."""
    base = dict(batch=1, n_q=128, n_k=128, h_q=2, h_k=1, head_dim=64, w_sink=4, w_near=16, tile=32,
                dtype="bf16", kind="train")
    base.update(kw)
    return Workload(name=name, **base)


def key_of(*parts):
    """A deterministic integer key for a free-form test workload."""
    h = 1000
    for p in parts:
        for ch in str(p):
            h = (h * 131 + ord(ch)) % (1 << 31)
    return h
