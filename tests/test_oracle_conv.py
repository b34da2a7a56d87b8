"""Pins of the oracle's 3x3 convolution (stride 1, zero padding 1, channels last) that the
UNet path's shortcut-fed conv layers use (Sec. 4.6; their inputs are routed to MXFP8)."""
import numpy as np

import oracle


def test_center_tap_is_the_linear_layer():
    g = np.random.default_rng(0)
    B, H, W, C, Co = 2, 5, 4, 16, 7
    X = g.normal(size=(B, H, W, C)).astype(np.float32)
    Wc = g.normal(size=(Co, C)).astype(np.float32)
    Wt = np.zeros((Co, 9 * C), np.float32)
    Wt[:, 4 * C:5 * C] = Wc  # tap (1, 1)
    Y, _ = oracle.conv3x3(X, Wt)
    Yl, _ = oracle.linear(X.reshape(-1, C), Wc)
    assert np.allclose(Y.reshape(-1, Co), Yl, rtol=1e-12, atol=0)


def test_matches_numpy_im2col_and_padding():
    """Against an independent numpy construction: zero-padded input, the 9 shifted views
    stacked tap-major, one matrix product."""
    g = np.random.default_rng(1)
    B, H, W, C, Co = 2, 6, 7, 8, 5
    X = g.normal(size=(B, H, W, C)).astype(np.float32)
    Wt = g.normal(size=(Co, 9 * C)).astype(np.float32)
    Y, Bm = oracle.conv3x3(X, Wt)
    Xp = np.zeros((B, H + 2, W + 2, C))
    Xp[:, 1:-1, 1:-1] = X
    cols = np.concatenate([Xp[:, ky:ky + H, kx:kx + W] for ky in range(3) for kx in range(3)], axis=-1)
    Yr = cols.reshape(-1, 9 * C) @ Wt.astype(np.float64).T
    assert np.allclose(Y.reshape(-1, Co), Yr, rtol=1e-11, atol=1e-12)
    assert np.allclose(Bm.reshape(-1, Co), np.abs(cols.reshape(-1, 9 * C)) @ np.abs(Wt.astype(np.float64)).T,
                       rtol=1e-11)


def test_single_pixel_gives_the_flipped_kernel():
    """One nonzero input pixel: the output around it is the kernel's spatially flipped
    taps (a correlation), and nothing reaches beyond the 3 x 3 neighbourhood."""
    C, Co = 4, 3
    X = np.zeros((1, 5, 5, C), np.float32)
    X[0, 2, 2, 1] = 1.0
    g = np.random.default_rng(2)
    Wt = g.normal(size=(Co, 9 * C)).astype(np.float32)
    Y, _ = oracle.conv3x3(X, Wt)
    for y in range(5):
        for x in range(5):
            ky, kx = 2 - y + 1, 2 - x + 1
            if 0 <= ky < 3 and 0 <= kx < 3:
                assert np.array_equal(Y[0, y, x], Wt[:, (ky * 3 + kx) * C + 1].astype(np.float64))
            else:
                assert not Y[0, y, x].any()
