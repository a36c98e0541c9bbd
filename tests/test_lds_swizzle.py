"""The LDS tile swizzle of the matrix kernels against the gfx950 bank model.

The model was measured on the device with the probes in ``tests/probes``
(bank-conflict counters per dispatch): the LDS has 64 four-byte banks;
ds_read_b128 serves 16 lanes per clock, namely the lanes with equal lane / 32
and equal parity of bits 2..4 of the lane ({0-3, 12-15, 20-23, 24-27},
{4-11, 16-19, 28-31}, and the same + 32); ds_read_b64 and ds_read_b64_tr_b16
serve lanes 0-31, then 32-63.  A read is conflict-free iff the lanes served
together touch distinct banks.

The test builds the kernels' own swizzle function (host build of
``csrc/mfma_tiles.h``), checks that every LDS read pattern of the forward, the
dK/dV pass and the dQ pass is conflict-free under the model for head
dimensions 128 and 64, and that the model reproduces the measured counters:
the earlier swizzle gave two-way conflicts on the backward's row fragments
and on the forward's V^T reads, and none elsewhere.
"""

import os
import shutil
import subprocess

import pytest

from conftest import ROOT

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def group_b128(lane):
    return (lane >> 5, bin((lane >> 2) & 7).count("1") & 1)


def ways(kind, addrs):
    """Largest number of lanes served in one clock that hit the same bank."""
    groups = {}
    for lane, a in enumerate(addrs):
        if kind == "b128":
            groups.setdefault(group_b128(lane), []).append((a // 16) % 16)  # four banks per lane
        else:
            groups.setdefault(lane >> 5, []).append((a // 8) % 32)         # two banks per lane
    return max(max(g.count(x) for x in g) for g in groups.values())


def read_patterns(D):
    """(kind, [(row, chunk, half) per lane]) for every read pattern of the kernels."""
    pats = {}
    for ks in range(D // 32):   # dK/dV and dQ passes: row fragments (row8_off)
        pats[f"row8_ks{ks}"] = ("b128", [(l & 15, 4 * ks + (l >> 4), 0) for l in range(64)])
    for md in range(D // 16):   # dK/dV and dQ passes: transposing reads (tr8_off), both 16-row halves
        for hi in (0, 16):
            pats[f"tr8_md{md}_{hi}"] = ("b64", [(4 * (l >> 4) + ((l & 15) >> 2) + hi, (16 * md + 4 * (l & 3)) >> 3,
                                                  (l & 3) & 1) for l in range(64)])
    for ks in range(D // 16):   # forward: K rows
        pats[f"fwd_k_ks{ks}"] = ("b128", [(l & 31, 2 * ks + (l >> 5), 0) for l in range(64)])
    for md in range(D // 32):   # forward: V^T reads
        for hf in range(2):
            pats[f"fwd_v_md{md}_hf{hf}"] = ("b64", [(4 * (l >> 5) + ((l & 15) >> 2) + 8 * hf,
                                                     (32 * md + 16 * ((l >> 4) & 1) + 4 * (l & 3)) >> 3,
                                                     (l & 3) & 1) for l in range(64)])
    return pats


def conflicts(D, masks):
    pitch = 2 * D
    out = {}
    for name, (kind, lanes) in read_patterns(D).items():
        addrs = [row * pitch + ((ch ^ masks[row % 16]) << 4) + 8 * half for row, ch, half in lanes]
        out[name] = ways(kind, addrs)
    return out


@pytest.fixture(scope="module")
def kernel_masks(tmp_path_factory):
    if not os.path.exists(HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("hipcc not available")
    exe = str(tmp_path_factory.mktemp("swz") / "swz_dump")
    src = os.path.join(ROOT, "tests", "probes", "swz_dump.cpp")
    subprocess.run([HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-I", os.path.join(ROOT, "include"), src,
                    "-o", exe], check=True, capture_output=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True).stdout.split("\n")
    masks = {}
    for line in out:
        parts = line.split()
        if parts:
            masks[int(parts[0])] = [int(x) for x in parts[1:]]
    return masks


@pytest.mark.parametrize("D", [128, 64])
def test_kernel_swizzle_conflict_free(kernel_masks, D):
    masks = kernel_masks[D]
    assert len(masks) == 16
    for r0 in range(0, 16, 4):  # XOR masks keep a row's chunks a permutation
        assert all(0 <= m < D // 8 for m in masks[r0:r0 + 4])
    res = conflicts(D, masks)
    assert max(res.values()) == 1, {k: v for k, v in res.items() if v > 1}


def test_model_reproduces_measured_counters():
    # measured on the device (tests/probes/lds_patterns.hip): plain strides
    linear = [16 * l for l in range(64)]
    assert ways("b128", linear) == 1
    assert ways("b128", [16 * (l % 8) + 256 * (l // 8) for l in range(64)]) == 2
    assert ways("b128", [16 * (l % 16) + 512 * (l // 16) for l in range(64)]) == 1
    assert ways("b64", [8 * (l % 16) + 256 * (l // 16) for l in range(64)]) == 2
    assert ways("b64", [8 * (l % 32) + 512 * (l // 32) for l in range(64)]) == 1
    # the earlier swizzle: two-way conflicts on the backward's row fragments and
    # the forward's V^T reads, none on the other patterns (as the counters showed)
    old = [((r & 7) << 1) | (((r >> 2) ^ (r >> 3)) & 1) for r in range(16)]
    res = conflicts(128, old)
    for name, w in res.items():
        expect = 2 if name.startswith(("row8", "fwd_v")) else 1
        assert w == expect, (name, w)
