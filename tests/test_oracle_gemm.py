"""Pins of the oracle's linear-layer reference: numpy's binary64 matmul (a library routine),
exact equality on exact-arithmetic inputs, the column-permutation property, and the
end-to-end quantized layer built from the oracle's own codes."""
import numpy as np

import oracle
from paper_2609_33496_amd import synth


def test_linear_matches_numpy_float64():
    g = np.random.default_rng(0)
    X = g.normal(size=(17, 96)).astype(np.float32)
    W = g.normal(size=(23, 96)).astype(np.float32)
    Y, Bm = oracle.linear(X, W)
    ref = X.astype(np.float64) @ W.astype(np.float64).T
    assert np.allclose(Y, ref, rtol=1e-13, atol=1e-13)
    assert np.allclose(Bm, np.abs(X.astype(np.float64)) @ np.abs(W.astype(np.float64)).T, rtol=1e-13)


def test_linear_exact_on_grid_values():
    g = np.random.default_rng(1)
    X = (g.integers(-255, 256, size=(9, 64)) * 2.0 ** -7).astype(np.float32)
    W = (g.integers(-7, 8, size=(11, 64)) * 2.0 ** -3).astype(np.float32)
    Y, _ = oracle.linear(X, W)
    ref = (X.astype(np.float64) @ W.astype(np.float64).T)
    assert np.array_equal(Y, ref)


def test_permuting_weight_rows_permutes_columns():
    g = np.random.default_rng(2)
    X = g.normal(size=(5, 32)).astype(np.float32)
    W = g.normal(size=(12, 32)).astype(np.float32)
    p = g.permutation(12)
    Y, _ = oracle.linear(X, W)
    Yp, _ = oracle.linear(X, W[p])
    assert np.array_equal(Yp, Y[:, p])


def test_pairs_agree_with_full():
    g = np.random.default_rng(3)
    X = g.normal(size=(8, 64)).astype(np.float32)
    W = g.normal(size=(10, 64)).astype(np.float32)
    Y, Bm = oracle.linear(X, W)
    mm = g.integers(0, 8, 30)
    nn = g.integers(0, 10, 30)
    y, b = oracle.linear_pairs(X, W, mm, nn)
    assert np.array_equal(y, Y[mm, nn]) and np.array_equal(b, Bm[mm, nn])


def test_quantized_layer_error_is_small_vs_float():
    """End to end on the single-layer workload: W4 per-channel formats and A8 activations
    (INT8-asym and E4M3, dynamic per-tensor) reproduce the float layer to a few percent."""
    X, W = synth.single_layer(0, M=64, K=640, N=96)
    wq = oracle.select_weight_formats(W, oracle.MASK_W4)
    Wh = oracle.dequant_weights(wq, 640)
    Yf = X.astype(np.float64) @ W.astype(np.float64).T
    for fmt in (oracle.A_INT8_ASYM, oracle.A_FP8_E4M3):
        codes, e8, xh, s, z = oracle.quantize_act_dynamic(X, fmt, want_xhat=True)
        assert np.array_equal(oracle.dequant_act(codes, e8, fmt, s, z), xh)
        Y, _ = oracle.linear(xh, Wh)
        rel = np.linalg.norm(Y - Yf) / np.linalg.norm(Yf)
        assert rel < 0.2, (fmt, rel)
