"""Helpers shared by the GPU parity tests (no test functions here)."""

import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

# Parity bar, per output tensor (atol, rtol): every element must satisfy
# |x - ref| <= atol + rtol * |ref| (max-abs 2e-2 with relative 1e-2 for bf16;
# 1e-5 / 1e-5 for fp32), and ||x - ref||_F / ||ref||_F <= rtol.  A pure
# max-abs bound cannot hold for bf16 outputs of magnitude >= 8, whose
# rounding alone (half a bf16 ulp, 2^-5 there) exceeds 2e-2.
TOL = {"bf16": (2e-2, 1e-2), "fp32": (1e-5, 1e-5)}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def to_dev(payload, dev):
    """uint16 bf16 bits -> torch.bfloat16; float32 -> torch.float32."""
    if payload.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(payload).view(np.int16)).view(torch.bfloat16).to(dev)
    return torch.from_numpy(np.ascontiguousarray(payload)).to(dev)


def to_host(t):
    return t.float().cpu().numpy().astype(np.float64)


# Kernel error beyond the rounding of a bf16 output (O, dQ, dK, dV): with
# e = max(0, |x - ref| - |bf16(ref) - ref|) per element, what the kernel adds
# to the unavoidable rounding of the exact result to bf16, the test asserts
# ||e||_F / ||ref||_F <= 5e-3 (half of the relative bar) and logs the largest
# e / (2e-2 + 1e-2 |ref|).  (LSE is written in float32: its error is all the
# kernel's own.)
EXCESS_REL = 5e-3


def _bf16_round(x):
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float64).numpy()


def compare(name, got, ref, dtype="bf16"):
    """Assert the parity bar; returns (max_abs, rel_fro)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(got), fin), f"{name}: non-finite pattern differs"
    # -inf entries (empty rows) must match exactly
    assert np.array_equal(got[~fin], ref[~fin]), f"{name}: non-finite values differ"
    diff = np.abs(got[fin] - ref[fin])
    a_tol, r_tol = TOL[dtype]
    max_abs = float(diff.max(initial=0.0))
    bound = a_tol + r_tol * np.abs(ref[fin])
    worst = float((diff / bound).max(initial=0.0))
    denom = float(np.sqrt((ref[fin] ** 2).sum()))
    rel = float(np.sqrt((diff ** 2).sum()) / denom) if denom > 0 else max_abs
    excess_worst = excess_rel = 0.0
    if dtype == "bf16" and not name.startswith("LSE"):
        rounding = np.abs(_bf16_round(ref[fin]) - ref[fin])
        excess = np.maximum(diff - rounding, 0.0)
        excess_worst = float((excess / bound).max(initial=0.0))
        excess_rel = float(np.sqrt((excess ** 2).sum()) / denom) if denom > 0 else 0.0
    log(f"  {name}: max_abs={max_abs:.3e} worst(|d|/(atol+rtol|ref|))={worst:.3f} rel_fro={rel:.3e} "
        f"beyond bf16 output rounding: worst={excess_worst:.3f} rel_fro={excess_rel:.3e}")
    assert worst <= 1.0, f"{name}: |x - ref| exceeds {a_tol} + {r_tol}|ref| (worst ratio {worst:.3f})"
    assert rel <= r_tol, f"{name}: relative Frobenius error {rel:.3e} > {r_tol}"
    assert excess_rel <= EXCESS_REL, (f"{name}: error beyond the output's bf16 rounding, relative Frobenius "
                                      f"{excess_rel:.3e} > {EXCESS_REL}")
    return max_abs, rel
