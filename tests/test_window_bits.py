"""The bit-mask forms of the window rule that the kernels use for partial
blocks (csrc/window_rule.h: legal_keys32 over 32 keys of one query,
legal_queries32 over 32 queries of one key) against the per-pair rule
legal32, on random windows and positions around every boundary (host build of
the kernels' own header, tests/probes/legal_bits_check.cpp).  legal32 itself
is what every GPU parity test checks against the oracle's element mask."""

import os
import shutil
import subprocess

import pytest

from conftest import ROOT

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def test_bit_masks_match_pair_rule(tmp_path):
    if not os.path.exists(HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "legal_bits_check")
    src = os.path.join(ROOT, "tests", "probes", "legal_bits_check.cpp")
    subprocess.run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-I", os.path.join(ROOT, "include"), src,
                    "-o", exe], check=True, capture_output=True)
    out = subprocess.run([exe], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    assert "mismatches 0" in out.stdout
