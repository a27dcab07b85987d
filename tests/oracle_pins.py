"""Pins for the CPU oracle: checks against facts that do not come from the oracle.

Each pin takes a bound oracle library (so the same checks can be run against a
deliberately broken build of the oracle) and raises AssertionError on failure.
What the pins rest on:

* hand-computed cases of the definition (orientation, padding, stride, bias,
  channel contraction), each derived in its docstring;
* closed forms: box sums from a summed-area table, border tap counts, a
  centred delta filter reproducing its input, the output-size formula;
* library routines the definition reduces to: 1x1 conv = matrix product
  (numpy), single image plane = scipy.signal.correlate2d, the whole
  multi-channel sum = scipy.signal.correlate over (ci, kh, kw);
* invariants: linearity in the input and in the weights, a bias shift,
  |out - b| <= S, S = correlation of |x| with |w|, the point variant and the
  thread count not changing a bit.

The operation is the one ILP-M evaluates (Section 4, Algorithm 2): taps
(r, s) index the input at (y + r, x + s), i.e. cross-correlation without a
filter flip.
"""
from __future__ import annotations

import numpy as np
import scipy.signal

import oracle
import workloads


def _conv(lib, x, w, b=None, stride=1, pad=0):
    return oracle.conv2d_f64(x, w, b, stride, pad, lib=lib)


X33 = np.arange(1, 10, dtype=np.float32).reshape(1, 1, 3, 3)  # [[1,2,3],[4,5,6],[7,8,9]]


def pin_orientation_delta(lib):
    """A delta filter at (kh, kw) = (1, 2) with pad 1 picks x[oh][ow + 1]:
    row i of the output is (x[i][1], x[i][2], 0).  A flipped (true) convolution
    would pick x[oh][ow - 1] and give (0, x[i][0], x[i][1])."""
    w = np.zeros((1, 1, 3, 3), np.float32)
    w[0, 0, 1, 2] = 1.0
    out, _ = _conv(lib, X33, w, None, 1, 1)
    expect = np.array([[2, 3, 0], [5, 6, 0], [8, 9, 0]], np.float64)
    np.testing.assert_array_equal(out[0, 0], expect)


def pin_box_sums_hand(lib):
    """All-ones 3x3 filter, pad 1: each output is the sum of the in-bounds 3x3
    neighbourhood.  Corner (0,0): 1+2+4+5 = 12; centre: 45; (0,1): 1+2+3+4+5+6 = 21."""
    w = np.ones((1, 1, 3, 3), np.float32)
    out, _ = _conv(lib, X33, w, None, 1, 1)
    expect = np.array([[12, 21, 16], [27, 45, 33], [24, 39, 28]], np.float64)
    np.testing.assert_array_equal(out[0, 0], expect)


def pin_stride2_hand(lib):
    """Same all-ones case with stride 2: the stride-1 result sampled at even
    rows and columns, [[12, 16], [24, 28]]."""
    w = np.ones((1, 1, 3, 3), np.float32)
    out, _ = _conv(lib, X33, w, None, 2, 1)
    np.testing.assert_array_equal(out[0, 0], np.array([[12, 16], [24, 28]], np.float64))


def pin_1x1_bias_hand(lib):
    """1x1 conv with bias: out[co] = b[co] + sum_ci w[co][ci] * x[ci].
    x0 = [[1,2],[3,4]], x1 = [[5,6],[7,8]], w = [[1,-1],[0.5,2]], b = [10, 0]:
    out0 = 10 + x0 - x1 = all 6;  out1 = 0.5*x0 + 2*x1 = [[10.5,13],[15.5,18]]."""
    x = np.array([[[1, 2], [3, 4]], [[5, 6], [7, 8]]], np.float32)[None]
    w = np.array([[1, -1], [0.5, 2]], np.float32).reshape(2, 2, 1, 1)
    b = np.array([10, 0], np.float32)
    out, _ = _conv(lib, x, w, b, 1, 0)
    np.testing.assert_array_equal(out[0, 0], np.full((2, 2), 6.0))
    np.testing.assert_array_equal(out[0, 1], np.array([[10.5, 13], [15.5, 18]]))


def pin_k2_valid_hand(lib):
    """K = 2, pad 0 on a 2x2 input: one output, 1*1 + 0*2 + 0*3 + (-1)*4 = -3."""
    x = np.array([[1, 2], [3, 4]], np.float32).reshape(1, 1, 2, 2)
    w = np.array([[1, 0], [0, -1]], np.float32).reshape(1, 1, 2, 2)
    out, sab = _conv(lib, x, w, None, 1, 0)
    assert out.shape == (1, 1, 1, 1)
    assert out[0, 0, 0, 0] == -3.0
    assert sab[0, 0, 0, 0] == 5.0  # |1*1| + |(-1)*4|


def pin_out_size(lib):
    """H_out = floor((H + 2p - K)/s) + 1 on hand cases; 0 when no window fits."""
    cases = [((224, 3, 1, 1), 224), ((28, 3, 2, 1), 14), ((7, 5, 1, 2), 7), ((7, 1, 1, 0), 7),
             ((5, 3, 2, 0), 2), ((6, 3, 2, 0), 2), ((7, 3, 3, 1), 3), ((2, 3, 1, 0), 0),
             ((1, 7, 3, 3), 1), ((23, 4, 3, 4), 10)]
    for (n, k, s, p), want in cases:
        got = oracle.out_size(n, k, s, p, lib=lib)
        assert got == want, ((n, k, s, p), got, want)


def pin_centered_delta_identity(lib):
    """w[co][ci] = delta(co, ci) at the centre tap with pad K//2 reproduces the
    input exactly (every other term is an exact 0)."""
    rng = np.random.default_rng(7)
    for k in (1, 3, 5):
        c = 4
        x = rng.standard_normal((1, c, 9, 11)).astype(np.float32)
        w = np.zeros((c, c, k, k), np.float32)
        for i in range(c):
            w[i, i, k // 2, k // 2] = 1.0
        out, _ = _conv(lib, x, w, None, 1, k // 2)
        np.testing.assert_array_equal(out, x.astype(np.float64))


def _sat_box(xpad, k):
    """Box sums of every k x k window (valid) from a summed-area table."""
    sat = np.zeros((xpad.shape[0] + 1, xpad.shape[1] + 1), np.float64)
    sat[1:, 1:] = xpad.cumsum(0).cumsum(1)
    return sat[k:, k:] - sat[:-k, k:] - sat[k:, :-k] + sat[:-k, :-k]


def pin_box_sums_sat(lib):
    """All-ones K x K filter over C_in channels = sum over channels of the
    windowed box sums, computed independently from a summed-area table, then
    subsampled by the stride."""
    rng = np.random.default_rng(11)
    for (c_in, h, wd, k, s, p) in [(3, 13, 17, 3, 1, 1), (2, 10, 9, 5, 2, 2), (4, 8, 12, 4, 3, 3)]:
        x = rng.integers(-8, 9, size=(1, c_in, h, wd)).astype(np.float32)
        w = np.ones((1, c_in, k, k), np.float32)
        out, _ = _conv(lib, x, w, None, s, p)
        want = sum(_sat_box(np.pad(x[0, ci].astype(np.float64), p), k) for ci in range(c_in))
        np.testing.assert_array_equal(out[0, 0], want[::s, ::s])


def pin_tap_counts(lib):
    """All-ones input and filter: each output counts its in-bounds taps times C_in.
    3x3/pad 1: corner 4, edge 6, interior 9.  5x5/pad 2 on 7x7: row 0 is
    [9,12,15,15,15,12,9], row 3 is [15,20,25,25,25,20,15]."""
    c_in = 3
    x = np.ones((1, c_in, 6, 6), np.float32)
    out, _ = _conv(lib, x, np.ones((1, c_in, 3, 3), np.float32), None, 1, 1)
    o = out[0, 0] / c_in
    assert o[0, 0] == 4 and o[0, 5] == 4 and o[5, 0] == 4 and o[5, 5] == 4
    assert o[0, 2] == 6 and o[3, 0] == 6 and o[2, 2] == 9
    x = np.ones((1, c_in, 7, 7), np.float32)
    out, _ = _conv(lib, x, np.ones((1, c_in, 5, 5), np.float32), None, 1, 2)
    o = out[0, 0] / c_in
    np.testing.assert_array_equal(o[0], [9, 12, 15, 15, 15, 12, 9])
    np.testing.assert_array_equal(o[3], [15, 20, 25, 25, 25, 20, 15])


def pin_1x1_matmul(lib):
    """A 1x1 stride-1 conv is W [C_out x C_in] times X [C_in x H*W], plus b."""
    rng = np.random.default_rng(3)
    c_in, c_out, h, wd = 7, 5, 6, 9
    x = rng.standard_normal((1, c_in, h, wd)).astype(np.float32)
    w = rng.standard_normal((c_out, c_in, 1, 1)).astype(np.float32)
    b = rng.standard_normal(c_out).astype(np.float32)
    out, _ = _conv(lib, x, w, b, 1, 0)
    want = (w[:, :, 0, 0].astype(np.float64) @ x[0].reshape(c_in, -1).astype(np.float64)
            + b.astype(np.float64)[:, None])
    np.testing.assert_allclose(out[0].reshape(c_out, -1), want, rtol=1e-12, atol=1e-12)


def _scipy_conv(x, w, b, s, p):
    """scipy.signal.correlate over (ci, kh, kw) of the zero-padded input, 'valid'
    mode, subsampled by the stride, plus the bias."""
    xp = np.pad(x[0].astype(np.float64), ((0, 0), (p, p), (p, p)))
    outs = []
    for co in range(w.shape[0]):
        r = scipy.signal.correlate(xp, w[co].astype(np.float64), mode="valid", method="direct")[0]
        r = r[::s, ::s]
        if b is not None:
            r = r + float(b[co])
        outs.append(r)
    return np.stack(outs)[None]


def pin_single_plane_correlate2d(lib):
    """C_in = C_out = 1: the output is scipy.signal.correlate2d of the padded
    plane with the filter ('valid'), subsampled by the stride."""
    rng = np.random.default_rng(5)
    for (h, wd, k, s, p) in [(9, 7, 3, 1, 1), (12, 10, 5, 2, 2), (8, 8, 2, 1, 0),
                             (11, 6, 4, 3, 1), (5, 5, 7, 1, 3), (6, 9, 1, 2, 0)]:
        x = rng.standard_normal((1, 1, h, wd)).astype(np.float32)
        w = rng.standard_normal((1, 1, k, k)).astype(np.float32)
        out, _ = _conv(lib, x, w, None, s, p)
        xp = np.pad(x[0, 0].astype(np.float64), p)
        want = scipy.signal.correlate2d(xp, w[0, 0].astype(np.float64), mode="valid")[::s, ::s]
        np.testing.assert_allclose(out[0, 0], want, rtol=1e-12, atol=1e-12)


def pin_multichannel_correlate(lib):
    """C_in != C_out, every K/stride/pad mix: equals scipy.signal.correlate over
    (ci, kh, kw) per output channel plus the bias."""
    rng = np.random.default_rng(9)
    for (c_in, h, wd, c_out, k, s, p) in [(3, 9, 11, 5, 3, 1, 1), (5, 10, 7, 2, 5, 2, 2),
                                          (2, 12, 12, 3, 4, 3, 2), (4, 6, 8, 6, 1, 2, 0),
                                          (6, 7, 5, 4, 2, 1, 1)]:
        x = rng.standard_normal((1, c_in, h, wd)).astype(np.float32)
        w = rng.standard_normal((c_out, c_in, k, k)).astype(np.float32)
        b = rng.standard_normal(c_out).astype(np.float32)
        out, _ = _conv(lib, x, w, b, s, p)
        np.testing.assert_allclose(out, _scipy_conv(x, w, b, s, p), rtol=1e-12, atol=1e-12)


def pin_sumabs(lib):
    """S is the correlation of |x| with |w| (|w*x| = |w|*|x|), excludes the bias,
    and bounds |out - b|."""
    rng = np.random.default_rng(13)
    c_in, h, wd, c_out, k, s, p = 3, 8, 9, 4, 3, 2, 1
    x = rng.standard_normal((1, c_in, h, wd)).astype(np.float32)
    w = rng.standard_normal((c_out, c_in, k, k)).astype(np.float32)
    b = (100 + rng.standard_normal(c_out)).astype(np.float32)
    out, sab = _conv(lib, x, w, b, s, p)
    want = _scipy_conv(np.abs(x), np.abs(w), None, s, p)
    np.testing.assert_allclose(sab, want, rtol=1e-12, atol=1e-12)
    assert np.all(np.abs(out - b.astype(np.float64)[None, :, None, None]) <= sab * (1 + 1e-12))


def pin_linearity(lib):
    """conv(a*x1 + c*x2, w) = a*conv(x1, w) + c*conv(x2, w) and the same in w.
    Values are small dyadic numbers, so every input, product and sum is exact and
    the identities hold bit for bit."""
    rng = np.random.default_rng(17)
    c_in, h, wd, c_out, k, s, p = 3, 7, 8, 2, 3, 1, 1
    x1 = (rng.integers(-100, 101, (1, c_in, h, wd)) / 64).astype(np.float32)
    x2 = (rng.integers(-100, 101, (1, c_in, h, wd)) / 64).astype(np.float32)
    w1 = (rng.integers(-50, 51, (c_out, c_in, k, k)) / 32).astype(np.float32)
    w2 = (rng.integers(-50, 51, (c_out, c_in, k, k)) / 32).astype(np.float32)
    a, c = 2.0, -0.5
    lhs, _ = _conv(lib, (a * x1 + c * x2).astype(np.float32), w1, None, s, p)
    r1, _ = _conv(lib, x1, w1, None, s, p)
    r2, _ = _conv(lib, x2, w1, None, s, p)
    np.testing.assert_array_equal(lhs, a * r1 + c * r2)
    lhs, _ = _conv(lib, x1, (a * w1 + c * w2).astype(np.float32), None, s, p)
    r3, _ = _conv(lib, x1, w2, None, s, p)
    np.testing.assert_array_equal(lhs, a * r1 + c * r3)


def pin_bias_shift(lib):
    """Adding a bias shifts output channel co by exactly b[co] (small dyadic
    values keep every sum exact) and leaves S unchanged."""
    rng = np.random.default_rng(19)
    x = (rng.integers(-30, 31, (1, 2, 6, 5)) / 16).astype(np.float32)
    w = (rng.integers(-30, 31, (3, 2, 3, 3)) / 16).astype(np.float32)
    b = np.array([1.5, -2.25, 1024.0], np.float32)
    o0, s0 = _conv(lib, x, w, None, 1, 1)
    o1, s1 = _conv(lib, x, w, b, 1, 1)
    np.testing.assert_array_equal(o1 - o0, np.broadcast_to(b.astype(np.float64)[None, :, None, None], o0.shape))
    np.testing.assert_array_equal(s0, s1)


def pin_points_and_threads(lib):
    """The point variant returns the same bits as the full output, and the
    full output does not change with the thread count."""
    rng = np.random.default_rng(23)
    x = rng.standard_normal((1, 5, 13, 9)).astype(np.float32)
    w = rng.standard_normal((6, 5, 3, 3)).astype(np.float32)
    b = rng.standard_normal(6).astype(np.float32)
    oracle.set_threads(1, lib=lib)
    o1, s1 = _conv(lib, x, w, b, 2, 1)
    oracle.set_threads(4, lib=lib)
    o4, s4 = _conv(lib, x, w, b, 2, 1)
    np.testing.assert_array_equal(o1, o4)
    np.testing.assert_array_equal(s1, s4)
    idx = np.array([0, 1, 17, o1.size // 2, o1.size - 1], np.int64)
    pv, ps = oracle.conv2d_f64_points(x, w, b, 2, 1, idx, lib=lib)
    np.testing.assert_array_equal(pv, o1.reshape(-1)[idx])
    np.testing.assert_array_equal(ps, s1.reshape(-1)[idx])


def pin_relu_maxpool(lib):
    """relu = max(x, 0); 2x2/stride-2 max-pool = max over each 2x2 block
    (numpy reshape-max), including odd sizes (last row/column dropped)."""
    rng = np.random.default_rng(29)
    x = rng.standard_normal((1, 3, 7, 10)).astype(np.float32)
    np.testing.assert_array_equal(oracle.relu(x, lib=lib), np.maximum(x, 0))
    y = oracle.maxpool2x2(x, lib=lib)
    want = x[:, :, :6, :10].reshape(1, 3, 3, 2, 5, 2).max(axis=(3, 5))
    np.testing.assert_array_equal(y, want)


def pin_workload_conv4x_scale(lib):
    """The conv4.x layer the paper profiles (256 -> 256 channels, 14x14, 3x3,
    Section 5.2): with pad 1 the output keeps 14x14."""
    assert oracle.out_size(14, 3, 1, 1, lib=lib) == 14
    c = workloads.RESNET_CONV4
    assert (c.c_in, c.c_out, c.h, c.k) == (256, 256, 14, 3)


ALL_PINS = [pin_orientation_delta, pin_box_sums_hand, pin_stride2_hand, pin_1x1_bias_hand,
            pin_k2_valid_hand, pin_out_size, pin_centered_delta_identity, pin_box_sums_sat,
            pin_tap_counts, pin_1x1_matmul, pin_single_plane_correlate2d,
            pin_multichannel_correlate, pin_sumabs, pin_linearity, pin_bias_shift,
            pin_points_and_threads, pin_relu_maxpool, pin_workload_conv4x_scale]
