"""Pins of the oracle's DiT joint (group size, format) search (Sec. 4.6 (i)): groups of g
input channels with their own scales, the input-aware error sum_k E[x_k^2] (w - w^)^2,
argmin over (g, f) with ties to the lowest tuple index, and its reductions to the
per-channel search."""
import numpy as np
import pytest

import oracle
from paper_2609_33496_amd import synth

W4 = oracle.MASK_DIT_W4
W8 = oracle.MASK_DIT_W8


def test_group_equal_to_row_reduces_to_per_channel_quantizer():
    """g = K (K = 288 or 192): one group per row, so every group quantizer is the
    per-channel quantizer of the per-channel search."""
    g = np.random.default_rng(1)
    for K in (192, 288):
        gi = oracle.GROUP_SIZES.index(K)
        W = (g.normal(size=(6, K)) * np.exp(g.normal(0, 1, (6, 1)))).astype(np.float32)
        for f in (oracle.W_INT4_ASYM, oracle.W_FP4, oracle.W_INT8_SYM, oracle.W_INT8_ASYM):
            for n in range(6):
                c1, wh1, gs, gz, _ = oracle.gq_row(f, K, W[n])
                c2, wh2, s, z, _, _ = oracle.wq_row(f, W[n])
                assert np.array_equal(c1, c2) and np.array_equal(wh1, wh2) and gs[0] == s and gz[0] == z
        # layer errors with unit energy are the per-channel search's error sums of that format
        m = (1 << oracle.W_INT4_ASYM) | (1 << oracle.W_FP4) | (1 << oracle.W_INT8_SYM) | (1 << oracle.W_INT8_ASYM)
        out = oracle.select_group_formats(W, m, np.ones(K, np.float32), gmask=1 << gi)
        ref = oracle.select_weight_formats(W, m)
        for f in (oracle.W_INT4_ASYM, oracle.W_FP4, oracle.W_INT8_SYM, oracle.W_INT8_ASYM):
            assert np.isclose(out["err"][gi * 9 + f], ref["err"][:, f].sum(), rtol=1e-12)


def test_groups_are_consecutive_input_channels_with_own_scales():
    """Each group of g consecutive elements (the last one ragged) is quantized as a row of
    its own; the NF4 group scale is the group absmax."""
    g = np.random.default_rng(2)
    K = 320  # 320 = 288 + 32: a ragged last group at g = 288, 192 (192 + 128), 128 (2 x 128 + 64)
    w = (g.normal(size=K) * np.repeat(np.exp(g.normal(0, 2, K // 32)), 32)).astype(np.float32)
    for gsz in oracle.GROUP_SIZES:
        for f in (oracle.W_INT4_ASYM, oracle.W_NF4, oracle.W_FP4):
            c, wh, gs, gz, _ = oracle.gq_row(f, gsz, w)
            for j in range(-(-K // gsz)):
                sl = slice(j * gsz, min((j + 1) * gsz, K))
                if f == oracle.W_NF4:
                    assert gs[j] == np.max(np.abs(w[sl]))
                elif f == oracle.W_FP4:
                    assert gs[j] == np.float32(np.max(np.abs(w[sl])) / np.float32(6))
                else:
                    lo, hi = w[sl].min(), w[sl].max()
                    levels = (np.arange(16) - float(gz[j])) * float(gs[j])
                    assert abs(levels[0] - lo) <= 0.51 * gs[j] and abs(levels[-1] - hi) <= 0.51 * gs[j]
            assert not np.any(gs[-(-K // gsz):])  # nothing past the last group


def test_known_winner_nf4_at_group_64():
    """NF4 levels times one absmax per 64 input channels, the absmax met once per group
    (so no 32-half reaches it on both sides): NF4 at g = 64 is exact and the unique winner."""
    g = np.random.default_rng(3)
    N, K = 8, 256
    v = oracle.nf4_table()
    W = v[g.integers(1, 15, (N, K))].astype(np.float32)  # levels strictly inside (-1, 1)
    a = np.exp(g.normal(0, 1, (N, K // 64))).astype(np.float32)
    W[:, ::64] = 1.0
    W = (W * np.repeat(a, 64, axis=1)).astype(np.float32)
    out = oracle.select_group_formats(W, W4, np.ones(K, np.float32))
    assert (out["g"], out["fmt_id"]) == (64, oracle.W_NF4)
    assert out["err"][1 * 9 + oracle.W_NF4] == 0.0
    others = [e for t, e in enumerate(out["err"]) if e >= 0 and t != 1 * 9 + oracle.W_NF4]
    assert min(others) > 0


def test_energy_weights_decide():
    """All activation energy on the first 32 input channels, which hold 16 evenly spaced
    values: INT4-asym at g = 32 has zero weighted error there and wins; with unit energy the
    remainder (NF4 levels times 10, every 32-group meeting +-10) decides for NF4."""
    g = np.random.default_rng(4)
    N, K = 6, 128
    v = oracle.nf4_table()
    W = (v[g.integers(0, 16, (N, K))] * np.float32(10)).astype(np.float32)
    W[:, ::32] = 10.0
    q = g.integers(0, 16, (N, 32))
    q[:, 0], q[:, 1] = 0, 15
    W[:, :32] = ((q - 6) * 0.125).astype(np.float32)
    e = np.zeros(K, np.float32)
    e[:32] = 1.0
    out = oracle.select_group_formats(W, W4, e)
    assert (out["g"], out["fmt_id"]) == (32, oracle.W_INT4_ASYM) and out["err"][oracle.W_INT4_ASYM] == 0.0
    out1 = oracle.select_group_formats(W, W4, np.ones(K, np.float32))
    assert (out1["g"], out1["fmt_id"]) == (32, oracle.W_NF4)


def test_errors_recomputed_independently_and_argmin():
    """Every tuple's layer error equals the energy-weighted sum over rows of the squared
    differences of gq_row's round trip (numpy sums), the choice is their argmin with ties to
    the lowest index, and the emitted codes / group metadata are the chosen tuple's."""
    g = np.random.default_rng(5)
    W, _ = synth.hetero_weights(6, 12, 576)
    e = np.exp(g.normal(0, 1, 576)).astype(np.float32)
    for mask in (W4, W8):
        out = oracle.select_group_formats(W, mask, e)
        for gi, gsz in enumerate(oracle.GROUP_SIZES):
            for f in range(9):
                t = gi * 9 + f
                if not (mask >> f) & 1 or (f in (oracle.W_MXINT8, oracle.W_MXINT4, oracle.W_MXFP4) and gsz != 32):
                    assert out["err"][t] == -1.0
                    continue
                tot = 0.0
                for n in range(W.shape[0]):
                    _, wh, *_ = oracle.gq_row(f, gsz, W[n])
                    d = (W[n] - wh).astype(np.float64)
                    tot += np.sum(e.astype(np.float64) * d * d)
                assert np.isclose(out["err"][t], tot, rtol=1e-12), (gi, f)
        valid = [(err, t) for t, err in enumerate(out["err"]) if err >= 0]
        best = min(valid)[1]
        assert (out["g"], out["fmt_id"]) == (oracle.GROUP_SIZES[best // 9], best % 9)
        Wh = oracle.dequant_grouped(out, 576)
        for n in range(W.shape[0]):
            _, wh, gs, gz, e8 = oracle.gq_row(out["fmt_id"], out["g"], W[n])
            assert np.array_equal(Wh[n], wh)
            assert np.array_equal(out["gscale"][n], gs) and np.array_equal(out["gzero"][n], gz)


def test_all_zero_layer_and_mx_only_at_32():
    K = 192
    out = oracle.select_group_formats(np.zeros((3, K), np.float32), W4, np.ones(K, np.float32))
    assert (out["g"], out["fmt_id"]) == (32, oracle.W_INT4_ASYM)  # every tuple exact: the lowest index
    out = oracle.select_group_formats(np.zeros((3, K), np.float32), W8, np.ones(K, np.float32))
    assert (out["g"], out["fmt_id"]) == (32, oracle.W_INT8_SYM)
    assert out["err"][1 * 9 + oracle.W_MXINT8] == -1.0 and out["err"][oracle.W_MXINT8] == 0.0
    with pytest.raises(ValueError):
        oracle.select_group_formats(np.zeros((3, K), np.float32), 1 << oracle.W_MXINT8, np.ones(K, np.float32),
                                    gmask=0b10)
