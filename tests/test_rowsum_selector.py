"""The forward's row sums on the matrix cores (csrc/fwd_bf16.hip): a model of
the register layouts involved, checked on the host.

The forward holds P^T of a 16-key k-step as the B operand of a 32x32x16
product: lane L holds query column L % 32 and eight of the sixteen keys,
which half depending on L / 32 (keys 4 h .. 4 h + 3 and 8 + 4 h .. 8 + 4 h + 3
for h = L / 32, the same permutation as the V^T operand it meets).  The row
sum reads that register unchanged as the B operand of a 16x16x32 product (lane
L: column L % 16, k-group L / 16, eight k values each) against a 0/1 selector
A (lane L: row L % 16, k-group L / 16), whose lanes hold ones where
(L & 4) == 0 equals (k-group even).  The result (lane L: rows 4 (L / 16) ..
+ 3, column L % 16) must then hold, in all four slots of every lane, the sum
of P over the sixteen keys for lane L's own query column L % 32.

The operand layouts are the ones the kernels are built on (the dK/dV pass
uses the same 16x16x32 layout, the forward and the dQ pass the 32x32x16 one);
the GPU parity tests check the kernel itself.  A selector that is off by one
k-group or row block, or that mixes the two 16-column halves, fails here."""

import numpy as np


def _selector(lane):
    return ((lane & 4) == 0) == (((lane >> 4) & 1) == 0)


def _keys_of_half(h):
    return [4 * h + i for i in range(4)] + [8 + 4 * h + i for i in range(4)]


def test_selector_leaves_own_column_sum_in_every_lane():
    rng = np.random.default_rng(2609)
    p = rng.random((16, 32))  # P of one k-step: 16 keys x 32 query columns
    # P^T fragment as the forward holds it (B of 32x32x16)
    reg = np.array([[p[k, lane % 32] for k in _keys_of_half(lane // 32)] for lane in range(64)])
    # the same registers read as B of 16x16x32: B[8 g + j][n] from lane 16 g + n
    b = np.zeros((32, 16))
    for lane in range(64):
        g, n = lane // 16, lane % 16
        b[8 * g:8 * g + 8, n] = reg[lane]
    # selector A of 16x16x32: A[m][8 g + j] from lane 16 g + m
    a = np.zeros((16, 32))
    for lane in range(64):
        g, m = lane // 16, lane % 16
        a[m, 8 * g:8 * g + 8] = 1.0 if _selector(lane) else 0.0
    d = a @ b  # 16 x 16 result
    for lane in range(64):
        g, n = lane // 16, lane % 16
        want = p[:, lane % 32].sum()
        got = d[4 * g:4 * g + 4, n]
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=0)


def test_other_selectors_fail():
    """The model is sharp: the selector that leaves the sums in other lanes
    (row < 8 instead of row & 4) and an all-ones selector both fail."""
    rng = np.random.default_rng(7)
    p = rng.random((16, 32))
    reg = np.array([[p[k, lane % 32] for k in _keys_of_half(lane // 32)] for lane in range(64)])
    b = np.zeros((32, 16))
    for lane in range(64):
        b[8 * (lane // 16):8 * (lane // 16) + 8, lane % 16] = reg[lane]
    for sel in (lambda lane: ((lane & 15) < 8) == (((lane >> 4) & 1) == 0), lambda lane: True):
        a = np.zeros((16, 32))
        for lane in range(64):
            a[lane % 16, 8 * (lane // 16):8 * (lane // 16) + 8] = 1.0 if sel(lane) else 0.0
        d = a @ b
        ok = all(np.allclose(d[4 * (lane // 16):4 * (lane // 16) + 4, lane % 16], p[:, lane % 32].sum())
                 for lane in range(64))
        assert not ok
