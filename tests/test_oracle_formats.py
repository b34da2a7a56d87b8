"""Pins of the oracle's number formats (App. A.11) against things other than itself:
the paper's printed constants, torch's float8 casts, scipy's normal quantiles, an
independent scale-and-round E2M1 rounder, and grid/round-trip invariants."""
import os

import numpy as np
import pytest
import torch

import oracle

GOLD = os.path.join(os.path.dirname(__file__), "golden", "format_constants.txt")


def _golden():
    d = {}
    for line in open(GOLD):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        k, *v = line.split()
        d[k] = v
    return d


def test_e2m1_value_set_matches_paper():
    g = _golden()
    printed = sorted(float(v) for v in g["e2m1_values"])
    vals = [oracle.mf_decode(oracle.MF_E2M1, c) for c in range(16)]
    pos = sorted(set(abs(v) for v in vals))
    assert pos == printed
    # codes 8..15 are the negatives of 0..7 (sign bit), -0 included
    for c in range(8):
        assert vals[c + 8] == -vals[c]
    assert np.signbit(vals[8])


def test_fp8_constants_match_paper():
    g = _golden()
    e4 = dict(zip(g["e4m3"][0::2], g["e4m3"][1::2]))
    e5 = dict(zip(g["e5m2"][0::2], g["e5m2"][1::2]))
    # max finite: E4M3 code 0x7E, E5M2 code 0x7B; smallest normal: exponent field 1, mantissa 0
    assert oracle.mf_decode(oracle.MF_E4M3, 0x7E) == float(e4["max"])
    assert oracle.mf_decode(oracle.MF_E5M2, 0x7B) == float(e5["max"])
    assert oracle.mf_decode(oracle.MF_E4M3, 1 << 3) == float(e4["min_normal"])
    assert oracle.mf_decode(oracle.MF_E5M2, 1 << 2) == float(e5["min_normal"])
    # one exponent step doubles the value: bias consistent with min_normal = 2^(1-bias)
    assert float(e4["min_normal"]) == 2.0 ** (1 - int(e4["bias"]))
    assert float(e5["min_normal"]) == 2.0 ** (1 - int(e5["bias"]))


@pytest.mark.parametrize("which,tdtype,maxcode", [(oracle.MF_E4M3, torch.float8_e4m3fn, 0x7E),
                                                  (oracle.MF_E5M2, torch.float8_e5m2, 0x7B)])
def test_fp8_decode_matches_torch(which, tdtype, maxcode):
    codes = [c for c in range(256) if (c & 0x7F) <= maxcode]
    ref = torch.tensor(codes, dtype=torch.uint8).view(tdtype).float().numpy()
    ours = np.array([oracle.mf_decode(which, c) for c in codes], np.float32)
    assert np.array_equal(ref.view(np.uint32), ours.view(np.uint32))  # sign of zero included


@pytest.mark.parametrize("which,tdtype,mx", [(oracle.MF_E4M3, torch.float8_e4m3fn, 448.0),
                                             (oracle.MF_E5M2, torch.float8_e5m2, 57344.0)])
def test_fp8_encode_matches_torch_cast(which, tdtype, mx):
    g = np.random.default_rng(7)
    # random magnitudes over the whole range, plus every midpoint between adjacent codes and
    # the floats on either side of it (the RNE tie cases)
    ys = list(g.uniform(-mx, mx, 2000)) + list(np.exp(g.uniform(-30, np.log(mx), 3000)) * g.choice([-1, 1], 3000))
    vals = sorted(set(oracle.mf_decode(which, c) for c in range(0x80) if (c & 0x7F) <= (0x7E if mx == 448 else 0x7B)))
    for a, b in zip(vals[:-1], vals[1:]):
        m = np.float32((a + b) / 2)
        ys += [m, np.nextafter(m, np.float32(0)), np.nextafter(m, np.float32(1e9)), -m]
    ys = np.array(ys, np.float32)
    ys = np.clip(ys, -mx, mx)
    ref = torch.from_numpy(ys).to(tdtype).view(torch.uint8).numpy()
    ours = np.array([oracle.mf_encode(which, y) for y in ys], np.uint8)
    bad = np.nonzero(ref != ours)[0]
    assert bad.size == 0, (ys[bad[:5]], ref[bad[:5]], ours[bad[:5]])


def _e2m1_round_independent(y):
    """E2M1 rounding by scaling to the binade's step and rounding half to even
    (binade [2^e, 2^(e+1)) has step 2^(e-1), e >= 0; below 1 the step is 0.5)."""
    a = abs(float(y))
    e = 0 if a < 1 else int(np.floor(np.log2(a)))
    step = 2.0 ** (e - 1)
    v = float(np.round(a / step)) * step
    return -v if np.signbit(y) else v


def test_e2m1_encode_against_independent_rounder():
    g = np.random.default_rng(3)
    ys = list(g.uniform(-6, 6, 5000))
    ys += [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0, -0.25, -5.0, 0.0, -0.0, 6.0, -6.0]
    for y in ys:
        y = np.float32(y)
        c = oracle.mf_encode(oracle.MF_E2M1, y)
        v = oracle.mf_decode(oracle.MF_E2M1, c)
        assert v == _e2m1_round_independent(y), (y, c, v)
        assert np.signbit(v) == np.signbit(y)


def test_e2m1_ties_go_to_even_code():
    expect = {0.25: 0.0, 0.75: 1.0, 1.25: 1.0, 1.75: 2.0, 2.5: 2.0, 3.5: 4.0, 5.0: 4.0}
    for y, v in expect.items():
        c = oracle.mf_encode(oracle.MF_E2M1, y)
        assert oracle.mf_decode(oracle.MF_E2M1, c) == v
        assert c % 2 == 0


def test_nf4_table_matches_scipy_construction():
    from scipy.special import ndtri
    d = 1 - 0.5 * (1 / 30 + 1 / 32)
    pos = [ndtri(d + (0.5 - d) * i / 8) for i in range(8)]
    neg = [-ndtri(d + (0.5 - d) * j / 7) for j in range(7)]
    ref = np.array(sorted(neg + [0.0] + pos), np.float64) / ndtri(d)
    ours = oracle.nf4_table()
    assert np.array_equal(ours, ref.astype(np.float32))


def test_nf4_table_structure():
    v = oracle.nf4_table()
    assert v[0] == -1.0 and v[7] == 0.0 and v[15] == 1.0
    assert np.all(np.diff(v) > 0)
    assert (v < 0).sum() == 7 and (v > 0).sum() == 8


# ---------------------------------------------------------------------------------------
# weight quantizers: grid-nearest property, round-trip idempotence, degenerate groups
# ---------------------------------------------------------------------------------------
W4 = [oracle.W_INT4_SYM, oracle.W_INT4_ASYM, oracle.W_NF4, oracle.W_FP4, oracle.W_MXINT4, oracle.W_MXFP4]
W8 = [oracle.W_INT8_SYM, oracle.W_INT8_ASYM, oracle.W_MXINT8]


def _grid(fmt, s, z, nf4a, e8, K):
    """All representable values of each element's scale group (as a [K, G] array)."""
    if fmt in (oracle.W_INT8_SYM, oracle.W_INT4_SYM):
        Q = 127 if fmt == oracle.W_INT8_SYM else 7
        g = np.arange(-Q, Q + 1, dtype=np.float32) * np.float32(s)
        return np.tile(g, (K, 1))
    if fmt in (oracle.W_INT8_ASYM, oracle.W_INT4_ASYM):
        L = 255 if fmt == oracle.W_INT8_ASYM else 15
        g = (np.arange(0, L + 1, dtype=np.float32) - np.float32(z)) * np.float32(s)
        return np.tile(g, (K, 1))
    if fmt == oracle.W_FP4:
        vals = np.array([oracle.mf_decode(0, c) for c in range(16)], np.float32)
        return np.tile(vals * np.float32(s), (K, 1))
    if fmt == oracle.W_NF4:
        v = oracle.nf4_table()
        return np.stack([v * nf4a[k // 64] for k in range(K)])
    if fmt in (oracle.W_MXINT8, oracle.W_MXINT4):
        Q, F = (127, 6) if fmt == oracle.W_MXINT8 else (7, 2)
        ks = np.arange(-Q, Q + 1, dtype=np.float64)
        return np.stack([np.ldexp(ks, int(e8[k // 32]) - 127 - F) for k in range(K)])
    vals = np.array([oracle.mf_decode(0, c) for c in range(16)], np.float64)
    return np.stack([np.ldexp(vals, int(e8[k // 32]) - 127) for k in range(K)])


@pytest.mark.parametrize("fmt", W4 + W8)
def test_weight_round_trip_is_grid_nearest(fmt):
    """Each reconstructed value is a nearest point of its group's grid (brute force over the
    whole grid; a rounding inside x*(1/s) may move an exact tie by one ulp, hence the slack)."""
    g = np.random.default_rng(11 + fmt)
    w = (g.standard_t(5, 128) * 0.03).astype(np.float32)
    w[:32] *= 8  # one block of larger magnitude
    codes, wh, s, z, nf, e8 = oracle.wq_row(fmt, w)
    grid = _grid(fmt, s, z, nf, e8, w.shape[0])
    dmin = np.min(np.abs(grid - w.astype(np.float64)[:, None]), axis=1)
    d = np.abs(wh.astype(np.float64) - w)
    sat = np.zeros_like(d, bool)
    if fmt in (oracle.W_MXINT4, oracle.W_MXINT8, oracle.W_MXFP4):
        sat = np.abs(wh) == np.max(np.abs(grid), axis=1)  # saturated block maxima
    assert np.all((d <= dmin + 6e-8 * np.abs(w) + 1e-12) | sat)


@pytest.mark.parametrize("fmt", W4 + W8)
def test_weight_requantize_idempotent(fmt):
    """Re-quantizing the dequantized row (metadata re-derived from it) gives the same codes.
    The values are identical too, except for INT-asym, whose re-derived scale
    (hi' - lo')/L can differ from s by one ulp."""
    g = np.random.default_rng(100 + fmt)
    for trial in range(40):
        w = (g.normal(size=256) * np.exp(g.normal(0, 2))).astype(np.float32)
        c1, wh1, s1, z1, *_ = oracle.wq_row(fmt, w)
        c2, wh2, s2, z2, *_ = oracle.wq_row(fmt, wh1)
        assert np.array_equal(c1, c2), (fmt, trial)
        if fmt in (oracle.W_INT4_ASYM, oracle.W_INT8_ASYM):
            assert z1 == z2 and abs(np.float32(s1).view(np.int32) - np.float32(s2).view(np.int32)) <= 1
        else:
            assert np.array_equal(wh1, wh2), (fmt, trial)


def test_degenerate_rows():
    K = 64
    for fmt in W4 + W8:
        codes, wh, s, z, nf, e8 = oracle.wq_row(fmt, np.zeros(K, np.float32))
        assert np.all(wh == 0)
        c = np.float32(0.37)
        codes, wh, s, z, nf, e8 = oracle.wq_row(fmt, np.full(K, c, np.float32))
        # a constant row reconstructs to within one grid step of the constant
        assert np.all(np.abs(wh - c) <= 0.5 * c), fmt
    # INT-asym on a constant row (hi == lo): s = |c|, z = -sign(c), exact reconstruction
    for fmt in (oracle.W_INT4_ASYM, oracle.W_INT8_ASYM):
        for c, zexp in ((np.float32(0.37), -1.0), (np.float32(-2.5), 1.0), (np.float32(0.0), 0.0)):
            codes, wh, s, z, nf, e8 = oracle.wq_row(fmt, np.full(K, c, np.float32))
            assert np.array_equal(wh, np.full(K, c, np.float32)), (fmt, c)
            assert z == zexp and s == (abs(c) if c != 0 else 1.0), (fmt, c, s, z)


# INT-asym (App. A.7 ScaleZP, App. A.11): L + 1 evenly spaced levels from min to max, the
# zero point round(-lo/s) not clamped.  Ranges whose every step is exact in binary32, with
# their scale, zero point and the codes of the range ends worked out by hand.
INT_ASYM_HAND = [
    # (L, lo, hi, s, z): one-sided positive, one-sided negative, crossing zero
    (15, 1.0, 16.0, 1.0, -1.0),
    (15, -16.0, -1.0, 1.0, 16.0),
    (15, -5.0, 10.0, 1.0, 5.0),
    (255, 2.0, 257.0, 1.0, -2.0),
    (255, -0.5, -0.5 + 255 * 0.125, 0.125, 4.0),
    (255, 64.0, 64.0 + 255 * 0.25, 0.25, -256.0),
]


@pytest.mark.parametrize("L,lo,hi,s_exp,z_exp", INT_ASYM_HAND)
def test_int_asym_scale_zp_hand_computed(L, lo, hi, s_exp, z_exp):
    fmt = oracle.W_INT4_ASYM if L == 15 else oracle.W_INT8_ASYM
    K = 64
    w = np.linspace(lo, hi, K).astype(np.float32)
    w[0], w[-1] = lo, hi
    codes, wh, s, z, *_ = oracle.wq_row(fmt, w)
    assert s == s_exp and z == z_exp
    assert codes[0] == 0 and codes[-1] == L  # the range ends are the first and last level
    assert wh[0] == np.float32(lo) and wh[-1] == np.float32(hi)
    if L == 255:  # the activation ScaleZP is the same helper
        sa, za = oracle.scale_zp(oracle.A_INT8_ASYM, lo, hi)
        assert sa == s_exp and za == z_exp


@pytest.mark.parametrize("L", [15, 255])
def test_int_asym_one_sided_levels_span_the_range(L):
    """For one-sided rows the L + 1 levels (q - z) s run from min to max (App. A.11), every
    element lands on its nearest level (brute force over the grid), and the zero point is
    outside [0, L] -- a range widened to contain zero, or a clamped z, fails these."""
    fmt = oracle.W_INT4_ASYM if L == 15 else oracle.W_INT8_ASYM
    g = np.random.default_rng(21 + L)
    for trial in range(30):
        sign = 1 if trial % 2 == 0 else -1
        base = np.float32(np.exp(g.normal(0, 2)))
        w = (sign * (base * (1.0 + g.uniform(0.01, 2.0) * g.random(256)))).astype(np.float32)
        lo, hi = np.float64(w.min()), np.float64(w.max())
        codes, wh, s, z, *_ = oracle.wq_row(fmt, w)
        assert (z < 0) if sign > 0 else (z > L), (trial, z)
        step = (hi - lo) / L
        assert abs(s - step) <= 2 ** -22 * step
        levels = (np.arange(L + 1, dtype=np.float64) - z) * s
        assert abs(levels[0] - lo) <= 0.5 * s * (1 + 1e-5) and abs(levels[-1] - hi) <= 0.5 * s * (1 + 1e-5)
        near = np.min(np.abs(levels[None, :] - w.astype(np.float64)[:, None]), axis=1)
        err = np.abs(wh.astype(np.float64) - w)
        assert np.all(err <= near + 4e-7 * np.abs(w)), trial
        assert np.max(err) <= 0.5 * step * (1 + 1e-4) + 4e-7 * np.max(np.abs(w))


def test_nf4_exact_midpoint_goes_to_lower_level():
    """An input exactly on the midpoint of two NF4 levels (representable in binary32 for
    four of the fifteen pairs) is assigned the lower level (the stated tie rule)."""
    v = oracle.nf4_table().astype(np.float64)
    ties = [i for i in range(15) if np.float32((v[i] + v[i + 1]) / 2) == (v[i] + v[i + 1]) / 2]
    assert ties == [2, 6, 7, 14]
    for i in ties:
        w = np.zeros(64, np.float32)
        w[0] = 1.0  # block absmax exactly 1, so w * fl(1/a) = w
        w[1] = np.float32((v[i] + v[i + 1]) / 2)
        w[2] = np.nextafter(w[1], np.float32(2))  # just above: the upper level
        codes, wh, *_ = oracle.wq_row(oracle.W_NF4, w)
        assert codes[1] == i and codes[2] == i + 1, (i, codes[:3])


def test_mx_exponents():
    w = np.zeros(64, np.float32)
    w[:32] = 3.0  # floor(log2 3) = 1
    w[32:] = 0.0
    _, wh, _, _, _, e8 = oracle.wq_row(oracle.W_MXINT8, w)
    assert e8[0] == 127 + 1 and e8[1] == 0  # all-zero block: E = -127
    _, wh, _, _, _, e8 = oracle.wq_row(oracle.W_MXFP4, w)
    assert e8[0] == 127 + 1 - 2  # OCP: minus emax(E2M1) = 2
    assert np.all(wh[:32] == 3.0)  # 3 = 1.5 * 2^1 is on the E2M1 grid at scale 2^-1 ... exact
    # subnormal block maximum: exponent read exactly from the binary32 number
    w2 = np.full(32, np.float32(3e-40))
    _, _, _, _, _, e8 = oracle.wq_row(oracle.W_MXINT8, w2)
    assert int(e8[0]) - 127 == max(int(np.floor(np.log2(3e-40))), -127)


# ---------------------------------------------------------------------------------------
# activation quantizers (Alg. 2 / Alg. 3, ScaleZP of App. A.7)
# ---------------------------------------------------------------------------------------
def test_scale_zp_printed_formulas():
    s, z = oracle.scale_zp(oracle.A_INT8_ASYM, -1.0, 1.0)
    assert s == np.float32(np.float32(2.0) / np.float32(255.0))
    # z = round(-lo/s) with -lo/s = 1/fl(2/255) = 127.4999.. in binary32
    assert z == np.rint(np.float32(1.0) / s) == 127.0
    # one-sided ranges keep their own end points: X in [0.5, 1.5] puts z near -127.5
    s, z = oracle.scale_zp(oracle.A_INT8_ASYM, 0.5, 1.5)
    assert s == np.float32(np.float32(1.0) / np.float32(255.0)) and z in (-127.0, -128.0)
    s, z = oracle.scale_zp(oracle.A_INT8_ASYM, -3.0, -1.0)
    assert s == np.float32(np.float32(2.0) / np.float32(255.0)) and z in (382.0, 383.0)
    s, z = oracle.scale_zp(oracle.A_FP8_E4M3, -3.0, 2.0)
    assert s == np.float32(np.float32(3.0) / np.float32(448.0)) and z == 0
    s, z = oracle.scale_zp(oracle.A_FP8_E5M2, -3.0, 2.0)
    assert s == np.float32(np.float32(3.0) / np.float32(57344.0)) and z == 0
    for f in (oracle.A_MXFP8, oracle.A_MXINT8):
        assert oracle.scale_zp(f, -3.0, 2.0) == (1.0, 0.0)


@pytest.mark.parametrize("fmt,tdtype,mx", [(oracle.A_FP8_E4M3, torch.float8_e4m3fn, 448.0),
                                           (oracle.A_FP8_E5M2, torch.float8_e5m2, 57344.0)])
def test_fp8_act_quant_matches_torch(fmt, tdtype, mx):
    g = np.random.default_rng(5)
    X = (g.standard_t(3, size=(16, 96)) * 0.7).astype(np.float32)
    codes, _, xh, s, z = oracle.quantize_act_dynamic(X, fmt, want_xhat=True)
    r = np.float32(1.0) / s
    y = np.clip(X * r, -mx, mx).astype(np.float32)
    ref = torch.from_numpy(y).to(tdtype).view(torch.uint8).numpy()
    assert np.array_equal(ref, codes)
    # static scale below the tensor's range: values above the range saturate instead of NaN
    codes2, _, xh2 = oracle.quantize_act(X, fmt, s * np.float32(0.25), 0.0, want_xhat=True)
    assert np.all(np.isfinite(xh2))


def test_int8_asym_act_is_grid_nearest():
    g = np.random.default_rng(9)
    X = g.normal(size=(8, 64)).astype(np.float32)
    codes, _, xh, s, z = oracle.quantize_act_dynamic(X, oracle.A_INT8_ASYM, want_xhat=True)
    grid = (np.arange(256, dtype=np.float64) - float(z)) * float(s)
    dmin = np.min(np.abs(grid[None, None, :] - X.astype(np.float64)[..., None]), axis=-1)
    # grid points are rounded to binary32 in the reconstruction: half an ulp of slack
    assert np.all(np.abs(xh.astype(np.float64) - X) <= dmin + 6e-8 * np.abs(X) + 1e-12)
    assert codes.min() == 0 or codes.max() == 255


def test_mxfp8_act_block_values_in_open_interval():
    """Paper's activation MX exponent E = floor(log2 amax): normalized values in (-2, 2)."""
    g = np.random.default_rng(2)
    X = (g.standard_t(3, size=(4, 128)) * np.exp(g.normal(0, 3, size=(4, 1)))).astype(np.float32)
    codes, e8, xh = oracle.quantize_act(X, oracle.A_MXFP8, want_xhat=True)
    for m in range(4):
        for b in range(4):
            blk = X[m, 32 * b:32 * b + 32].astype(np.float64)
            E = int(e8[m, b]) - 127
            assert E == int(np.floor(np.log2(np.max(np.abs(blk)))))
            y = blk / 2.0 ** E
            assert np.all(np.abs(y) < 2)
    # dequantized equals the E4M3 decode of the codes times 2^E
    for m in range(4):
        for k in range(128):
            v = oracle.mf_decode(oracle.MF_E4M3, int(codes[m, k])) * 2.0 ** (int(e8[m, k // 32]) - 127)
            assert np.float32(v) == xh[m, k]


def test_act_dequant_inverts_codes():
    g = np.random.default_rng(4)
    X = g.normal(size=(6, 64)).astype(np.float32)
    for fmt in range(5):
        codes, e8, xh, s, z = oracle.quantize_act_dynamic(X, fmt, want_xhat=True)
        assert np.array_equal(oracle.dequant_act(codes, e8, fmt, s, z), xh)
        # re-quantizing the reconstruction with the same scale is idempotent
        c2, e82, xh2 = oracle.quantize_act(xh, fmt, s, z, want_xhat=True)
        if fmt != oracle.A_MXFP8:
            assert np.array_equal(xh2, xh), fmt


# ---------------------------------------------------------------------------------------
# per-sample dynamic scaling (Alg. 3: lo, hi = min, max per sample and forward; Sec. 4.6 (ii))
# ---------------------------------------------------------------------------------------
def test_per_sample_scaling_hand_computed():
    """Two samples whose ranges give exact scales: INT8-asym [-128, 127] -> s = 1, z = 128 and
    [2, 257] -> s = 1, z = -2; E4M3 amax 448 -> s = 1 and amax 896 -> s = 2."""
    K = 64
    X = np.zeros((4, K), np.float32)
    X[0:2] = np.linspace(-128, 127, 2 * K).reshape(2, K)
    X[2:4] = np.linspace(2, 257, 2 * K).reshape(2, K)
    codes, _, xh, s, z = oracle.quantize_act_per_sample(X, oracle.A_INT8_ASYM, 2, want_xhat=True)
    assert list(s) == [1.0, 1.0] and list(z) == [128.0, -2.0]
    assert codes[0, 0] == 0 and codes[1, -1] == 255 and codes[2, 0] == 0 and codes[3, -1] == 255
    assert xh[0, 0] == -128 and xh[1, -1] == 127 and xh[2, 0] == 2 and xh[3, -1] == 257
    Y = np.zeros((4, K), np.float32)
    Y[0:2, 0], Y[0:2, 1] = 448.0, -3.0
    Y[2:4, 0], Y[2:4, 1] = -896.0, 3.0
    codes, _, _, s, z = oracle.quantize_act_per_sample(Y, oracle.A_FP8_E4M3, 2)
    assert list(s) == [1.0, 2.0] and list(z) == [0.0, 0.0]
    assert codes[0, 0] == 0x7E and codes[2, 0] == 0xFE       # +-448: the largest finite code
    assert codes[0, 1] == 0xC4 and codes[2, 1] == 0x3C       # -3 at s = 1; 3/2 = 1.5 at s = 2


def test_per_sample_scaling_properties():
    """One sample is the per-tensor path; samples are independent (reordering the samples
    reorders scales and codes and changes nothing else); MX formats carry no scale."""
    g = np.random.default_rng(30)
    X = np.concatenate([g.normal(0, 1, (6, 96)), 40 + 5 * g.standard_t(3, (6, 96)),
                        -0.01 * g.random((6, 96))]).astype(np.float32)
    for fmt in range(5):
        c1, e1, h1, s1, z1 = oracle.quantize_act_per_sample(X, fmt, 1, want_xhat=True)
        c0, e0, h0, s0, z0 = oracle.quantize_act_dynamic(X, fmt, want_xhat=True)
        assert np.array_equal(c1, c0) and np.array_equal(h1, h0) and s1[0] == s0 and z1[0] == z0
        c, e, h, s, z = oracle.quantize_act_per_sample(X, fmt, 3, want_xhat=True)
        Xp = np.concatenate([X[12:18], X[0:6], X[6:12]])
        cp, ep, hp, sp, zp = oracle.quantize_act_per_sample(Xp, fmt, 3, want_xhat=True)
        assert np.array_equal(cp, np.concatenate([c[12:18], c[0:6], c[6:12]]))
        assert list(sp) == [s[2], s[0], s[1]] and list(zp) == [z[2], z[0], z[1]]
        if fmt >= oracle.A_MXFP8:
            assert np.all(s == 1) and np.all(z == 0) and np.array_equal(c, c0)
        else:
            assert len(set(s.tolist())) == 3  # three different ranges, three scales
