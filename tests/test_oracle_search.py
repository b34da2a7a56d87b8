"""Pins of the oracle's per-channel weight-format search (Sec. 4.5, Eq. weight-argmax):
constructed rows with a known exact winner, independent recomputation of each format's
error and the SQNR argmax, tie rule, packing layout, grouping and degenerate rows."""
import numpy as np
import pytest

import oracle
from paper_2609_33496_amd import synth

M4 = oracle.MASK_W4


def _nf4_row(K, g, scale):
    v = oracle.nf4_table()
    row = v[g.integers(0, 16, size=K)].astype(np.float32)
    for b in range(K // 64):  # every 64-block contains +1 so its absmax is exactly `scale`
        row[64 * b] = 1.0
    return (row * np.float32(scale)).astype(np.float32)


def _e2m1_pos():
    return np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6], np.float32)


def test_known_winners():
    K = 128
    g = np.random.default_rng(0)
    rows, expect = [], []
    # 1. NF4 levels times a power of two per 64-block: NF4 is exact
    rows.append(_nf4_row(K, g, 2.0 ** -5)); expect.append(oracle.W_NF4)
    # 2. 16 evenly spaced values with an integral zero point: INT4-asym is exact
    q = g.integers(0, 16, size=K); q[0], q[1] = 0, 15
    rows.append(((q - 5).astype(np.float32) * np.float32(0.0625)).astype(np.float32)); expect.append(oracle.W_INT4_ASYM)
    # 3. E2M1 grid times one scale (row max 6*2^-6): FP4 and MXFP4 exact -> tie -> lower id (FP4)
    r = _e2m1_pos()[g.integers(0, 8, size=K)] * g.choice([-1, 1], size=K)
    for b in range(K // 32):
        r[32 * b] = 6.0
    rows.append((r * 2.0 ** -6).astype(np.float32)); expect.append(oracle.W_FP4)
    # 4. E2M1 grid with a different power of two per 32-block: only MXFP4 is exact
    r = _e2m1_pos()[g.integers(0, 8, size=K)] * g.choice([-1, 1], size=K)
    for b in range(K // 32):
        r[32 * b] = 6.0
        r[32 * b:32 * b + 32] *= 2.0 ** (-3 * b)
    rows.append(r.astype(np.float32)); expect.append(oracle.W_MXFP4)
    # 5. integers k in [-7, 7] (block max 5 or 7) with a power of two per 32-block: MXINT4 exact
    k = g.integers(-7, 8, size=K).astype(np.float32)
    for b in range(K // 32):
        k[32 * b] = 7.0
        k[32 * b + 1] = 5.0
        k[32 * b:32 * b + 32] *= 2.0 ** (-4 * b - 2 - 2)  # value k * 2^(E-2) with E = -4b-2
    rows.append(k.astype(np.float32)); expect.append(oracle.W_MXINT4)
    # 6. all-zero row: every format is exact -> the lowest enabled id
    rows.append(np.zeros(K, np.float32)); expect.append(oracle.W_INT4_ASYM)
    W = np.stack(rows)
    out = oracle.select_weight_formats(W, M4)
    assert list(out["fmt"]) == expect, (list(out["fmt"]), out["err"])
    for n, f in enumerate(expect):
        assert out["err"][n, f] == 0.0


def test_errors_recomputed_independently_and_sqnr_argmax():
    """err_f equals sum((w - wq_row(f).w_hat)^2) summed by numpy, and the choice is the
    argmax of the SQNR in dB of Eq. weight-argmax (the row energy is common to all f)."""
    W, _ = synth.hetero_weights(5, 48, 256)
    for mask in (M4, oracle.MASK_W8, oracle.MASK_W4_FULL):
        out = oracle.select_weight_formats(W, mask)
        for n in range(W.shape[0]):
            sq = {}
            for f in range(9):
                if not (mask >> f) & 1:
                    assert out["err"][n, f] == -1.0
                    continue
                _, wh, *_ = oracle.wq_row(f, W[n])
                d = (W[n] - wh).astype(np.float64)  # binary32 differences, binary64 squares
                e = np.sum(d * d)
                assert np.isclose(out["err"][n, f], e, rtol=1e-12, atol=0)
                sq[f] = 10 * np.log10(np.mean(W[n].astype(np.float64) ** 2) / (e / W.shape[1]))
            best = max(sq, key=lambda f: (sq[f], -f))
            assert out["fmt"][n] == best


def test_codes_packing_and_metadata_match_row_round_trip():
    W, _ = synth.hetero_weights(7, 40, 192)
    for mask in (M4, oracle.MASK_W8):
        out = oracle.select_weight_formats(W, mask)
        cb = out["code_bits"]
        assert cb == (4 if mask == M4 else 8)
        for n in range(W.shape[0]):
            f = int(out["fmt"][n])
            c, wh, s, z, nf, e8 = oracle.wq_row(f, W[n])
            if cb == 4:
                packed = out["codes"][n]
                unpacked = np.empty(192, np.uint8)
                unpacked[0::2] = packed & 15
                unpacked[1::2] = packed >> 4
                assert np.array_equal(unpacked, c & 15)
            else:
                assert np.array_equal(out["codes"][n], c)
            assert out["scale"][n] == np.float32(s) and out["zero"][n] == z
            assert np.array_equal(out["nf4_absmax"][n], nf)
            assert np.array_equal(out["e8m0"][n], e8)
        # dequantizing the emitted representation reproduces each row's round trip
        Wh = oracle.dequant_weights(out, 192)
        for n in range(W.shape[0]):
            _, wh, *_ = oracle.wq_row(int(out["fmt"][n]), W[n])
            assert np.array_equal(Wh[n], wh)


def test_perm_is_stable_sort_by_format():
    W, _ = synth.hetero_weights(3, 300, 128)
    out = oracle.select_weight_formats(W, M4)
    ref = np.argsort(out["fmt"], kind="stable")
    assert np.array_equal(out["perm"], ref)
    cnt = np.bincount(out["fmt"], minlength=9)
    assert np.array_equal(out["group_off"], np.concatenate([[0], np.cumsum(cnt)]))


def test_single_layer_workload_format_mix():
    """The Gaussian-per-row single-layer workload: NF4 has the best mean SQNR, and the
    mean SQNR ordering is NF4 > FP4 > MXFP4 > INT4-asym > MXINT4 (a soft sanity check)."""
    X, W = synth.single_layer(0)
    out = oracle.select_weight_formats(W[:128], M4)
    e = out["err"]
    energy = np.sum(W[:128].astype(np.float64) ** 2, axis=1)
    mean_sqnr = {f: np.mean(10 * np.log10(energy / e[:, f])) for f in range(9) if (M4 >> f) & 1}
    order = sorted(mean_sqnr, key=lambda f: -mean_sqnr[f])
    assert order[0] == oracle.W_NF4
    assert np.all(out["fmt"] == oracle.W_NF4)


def test_w8_split_is_mixed_on_hetero_rows():
    """App. A.12: with E8M0 exponents the W8 choice spreads over INT8-asym, MXINT8 and
    INT8-sym instead of collapsing onto MXINT8 (soft check, synthetic weights)."""
    W, _ = synth.hetero_weights(1, 400, 256)
    out = oracle.select_weight_formats(W, oracle.MASK_W8)
    cnt = np.bincount(out["fmt"], minlength=9)
    assert cnt[oracle.W_INT8_ASYM] > 0 and cnt[oracle.W_MXINT8] > 0
    assert cnt[oracle.W_MXINT8] < 400


def test_bad_arguments_rejected():
    W = np.zeros((4, 96), np.float32)
    with pytest.raises(ValueError):
        oracle.select_weight_formats(W, M4)  # NF4 needs K % 64 == 0
    with pytest.raises(ValueError):
        oracle.select_weight_formats(W, 0)
    with pytest.raises(ValueError):
        oracle.select_weight_formats(W, 1 << 12)
    out = oracle.select_weight_formats(W, (1 << oracle.W_MXFP4) | (1 << oracle.W_FP4))
    assert np.all(out["fmt"] == oracle.W_FP4)
