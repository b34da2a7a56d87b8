"""GPU parity on the edges of the method's definitions: INT-asym ScaleZP on one-sided and
constant ranges (App. A.7, App. A.11: levels from min to max, the zero point not clamped),
the NF4 tie rule, zero points beyond the half-precision decode in the linear layer, block
scales spanning many binades, the calibration LUT at the full sizes of the 70-block stack
(L = 280 instrumented layers, B = 10 buckets, both schedules; B = 1 kurtosis-only), and
the correctly rounded reciprocal of the quantizers over every binary32 input."""
import ctypes
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2609_33496_amd import cham, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DIAG = os.path.join(ROOT, "tests", "native", "_build", "libcham_diag.so")


def case(msg):
    print(f"[case] {msg}", flush=True)


def _np(t):
    return t.detach().cpu().numpy()


def _one_sided_rows(K, g):
    """Rows whose range does not contain zero, of every width: wide and narrow, positive
    and negative, and narrow rows far from zero whose zero points reach 2^23 and beyond
    (INT8-asym) or 2^11 and beyond (INT4-asym); constant rows; NF4 exact-midpoint rows."""
    rows = []
    for sign in (1.0, -1.0):
        rows.append(sign * (0.5 + g.random(K)))                       # [0.5, 1.5]
        rows.append(sign * (3.0 + 0.01 * g.random(K)))                # z ~ 300 L
        rows.append(sign * (1000.0 + 1e-3 * g.random(K)))             # z ~ 2.5e8 at L = 255
        rows.append(sign * np.exp(g.normal(0, 1, K)) * 1e-3)          # one-sided, wide
        rows.append(sign * (7.0 + 1e-5 * np.arange(K)))               # steps of 1e-5
    rows.append(np.full(K, 0.37))
    rows.append(np.full(K, -2.5e-3))
    rows.append(np.full(K, 1000.0))
    v = oracle.nf4_table().astype(np.float64)
    r = g.normal(0, 0.3, K).clip(-1, 1)
    r[::64] = 1.0
    for j, i in enumerate((2, 6, 7, 14)):  # exact midpoints between levels: the lower level
        r[1 + 64 * (j % (K // 64)) + 2 * j] = (v[i] + v[i + 1]) / 2
    rows.append(r)
    return np.stack(rows).astype(np.float32)


@pytest.mark.parametrize("K", [256, 1024])  # 1024: rows split over four wavefronts
def test_search_one_sided_and_constant_rows(K):
    W = _one_sided_rows(K, np.random.default_rng(K))
    for mask in (oracle.MASK_W4, oracle.MASK_W8, 0x1FF, 1 << oracle.W_INT4_ASYM, 1 << oracle.W_INT8_ASYM):
        case(f"select_weight_formats one-sided rows K={K} mask={mask:#x}")
        wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), mask, want_err=True)
        torch.cuda.synchronize()
        ref = oracle.select_weight_formats(W, mask)
        assert np.array_equal(_np(wq.fmt), ref["fmt"]), (_np(wq.fmt), ref["fmt"])
        assert np.array_equal(_np(wq.codes), ref["codes"])
        assert np.array_equal(_np(wq.scale).view(np.uint32), ref["scale"].view(np.uint32))
        assert np.array_equal(_np(wq.zero), ref["zero"])
        if mask & (1 << oracle.W_INT8_ASYM):  # the narrow rows far from zero are in the test
            assert np.abs(ref["zero"]).max() > 2 ** 23 or not np.any(ref["fmt"] == oracle.W_INT8_ASYM)
    one = oracle.select_weight_formats(W, 1 << oracle.W_INT8_ASYM)
    assert np.abs(one["zero"]).max() > 2 ** 23 and one["zero"].min() < 0 < one["zero"].max()


def test_quantize_act_one_sided_and_far_zero_points():
    """Dynamic INT8-asym on tensors whose range excludes zero (z outside [0, 255], up to
    |z| > 2^23), and static quantization with such calibrated (s, z)."""
    g = np.random.default_rng(3)
    Xs = [(0.5 + g.random((64, 128))), -(2.0 + g.random((64, 128))), 100.0 + 0.05 * g.random((64, 128)),
          -(1000.0 + 1e-3 * g.random((64, 128)))]
    for i, X in enumerate(Xs):
        X = X.astype(np.float32)
        case(f"quantize_act INT8-asym one-sided tensor {i}")
        aq = cham.quantize_act(torch.from_numpy(X).to(DEV), cham.A_INT8_ASYM, dynamic=True)
        torch.cuda.synchronize()
        codes, _, _, s, z = oracle.quantize_act_dynamic(X, oracle.A_INT8_ASYM)
        assert not (0 <= z <= 255)
        assert np.array_equal(_np(aq.codes), codes) and _np(aq.scale)[0] == s and _np(aq.zero)[0] == z
        lo, hi = oracle.minmax(X)
        s2, z2 = oracle.scale_zp(oracle.A_INT8_ASYM, lo * 0.999, hi * 1.001)  # a calibrated range
        aq2 = cham.quantize_act(torch.from_numpy(X).to(DEV), cham.A_INT8_ASYM, dynamic=False,
                                s=torch.tensor([s2], device=DEV), z=torch.tensor([z2], device=DEV))
        torch.cuda.synchronize()
        assert np.array_equal(_np(aq2.codes), oracle.quantize_act(X, oracle.A_INT8_ASYM, s2, z2)[0])


def _linear_check(X, W, mask, afmt, name):
    M, K = X.shape
    case(f"mixed_linear {name} M={M} N={W.shape[0]} K={K} mask={mask:#x} afmt={afmt}")
    wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), mask)
    xq = cham.quantize_act(torch.from_numpy(X).to(DEV), afmt, dynamic=True)
    Y = _np(cham.mixed_linear(xq, wq)).astype(np.float64)
    wp = cham.select_weight_formats(torch.from_numpy(W).to(DEV), mask, want_packed=True)
    Yp = _np(cham.mixed_linear(xq, wp)).astype(np.float64)
    ref = oracle.select_weight_formats(W, mask, want_err=False, want_perm=False)
    codes, e8, xh, s, z = oracle.quantize_act_dynamic(X, afmt, want_xhat=True)
    assert np.array_equal(_np(wq.fmt), ref["fmt"]) and np.array_equal(_np(xq.codes), codes)
    Yr, Bm = oracle.linear(xh, oracle.dequant_weights(ref, K))
    rel = np.abs(Y - Yr) / np.maximum(Bm, 1e-300)
    assert rel.max() <= 1e-3, (name, rel.max(), np.unravel_index(np.argmax(rel), rel.shape))
    assert np.array_equal(Y, Yp)  # packed layout and pre-pass: the same operands
    return ref, z


def test_linear_int8_act_zero_point_beyond_half_precision():
    """INT8-asym activations with |z| > 1024 (narrow one-sided tensors): the decode keeps
    z clamped to +-1024 and the epilogue adds the rest through the weights' column sums."""
    g = np.random.default_rng(5)
    W, _ = synth.hetero_weights(6, 200, 640)
    for lo, width in ((30.0, 1.0), (-1000.0, 0.05), (0.5, 1.0)):
        X = (lo + width * g.random((96, 640))).astype(np.float32)
        for mask in (oracle.MASK_W4, oracle.MASK_W8):
            _, z = _linear_check(X, W, mask, cham.A_INT8_ASYM, f"act z beyond half ({lo}, {width})")
            assert (abs(z) > 1024) == (lo != 0.5)


def test_linear_int_asym_weights_far_zero_points():
    """INT-asym weight channels whose levels q - z exceed 2^11 (and 2^15: scaled by a power
    of two) in magnitude, alone and mixed with the other formats."""
    g = np.random.default_rng(8)
    K = 640
    W = _one_sided_rows(K, g)
    W = np.concatenate([W, synth.hetero_weights(9, 40, K)[0]])
    X = synth.diffusion_acts(0, 1, 300, 80, K)
    for mask in (1 << oracle.W_INT4_ASYM, 1 << oracle.W_INT8_ASYM, oracle.MASK_W4, oracle.MASK_W8):
        for afmt in (cham.A_FP8_E4M3, cham.A_INT8_ASYM, cham.A_MXFP8):
            ref, _ = _linear_check(X, W, mask, afmt, "far weight zero points")
    assert np.abs(ref["zero"]).max() > 2 ** 15


def test_linear_block_scales_spanning_many_binades():
    """NF4 and MX weight blocks spanning 2^24 within a channel against MXFP8 / MXINT8
    activation rows spanning 2^20, arranged so the large weight blocks meet the small
    activation blocks: every block is held to half precision relative to its channel's or
    row's largest block, and blocks down to 2^-28 of it stay normal numbers."""
    g = np.random.default_rng(12)
    M, N, K = 64, 96, 512
    wspan = 2.0 ** (-24 * np.arange(K // 64) / (K // 64 - 1))          # per 64-block
    W = (g.normal(0, 1, (N, K)) * np.repeat(wspan, 64)[None, :]).astype(np.float32)
    xspan = 2.0 ** (-20 * np.arange(K // 32)[::-1] / (K // 32 - 1))    # reversed: small x meets large w
    X = (g.normal(0, 1, (M, K)) * np.repeat(xspan, 32)[None, :]).astype(np.float32)
    for mask in (1 << oracle.W_NF4, 1 << oracle.W_MXFP4, 1 << oracle.W_MXINT4, 1 << oracle.W_MXINT8):
        for afmt in (cham.A_MXFP8, cham.A_MXINT8):
            _linear_check(X, W, mask, afmt, "block scales over 2^24")


def _c5_calibration(L, B, M=16, K=64, T=1000):
    """One tensor per (layer, bucket) from the sweep's activation generator at the bucket's
    middle timestep, accumulated on the GPU in one batched call and in the oracle."""
    Xs, layers, buckets = [], [], []
    for l in range(L):
        for b in range(B):
            t = min(T - 1, (b * T) // B + T // (2 * B))
            Xs.append(synth.diffusion_acts(40, l, t, M, K))
            layers.append(l)
            buckets.append(b)
    st = cham.alloc_stats(L, B, DEV)
    cham.act_stats_reset(st)
    case(f"act_stats_accumulate_batch L={L} B={B} ({len(Xs)} tensors)")
    cham.act_stats_accumulate_batch([torch.from_numpy(x).to(DEV) for x in Xs], layers, buckets, st)
    ost = oracle.Stats(L, B)
    for x, l, b in zip(Xs, layers, buckets):
        ost.accumulate(x, l, b)
    torch.cuda.synchronize()
    assert np.allclose(_np(st.nS), ost.nS, rtol=1e-12, atol=0)
    assert np.array_equal(_np(st.lohi), ost.lohi)
    return st, ost


def _check_lut(lut, F, S, Z, kap):
    kg = _np(lut.kappa)
    assert np.allclose(kg, kap, rtol=1e-4)
    near_gate = np.any(np.abs(kap[:, None] - np.array([3.0, 5.0])[None, :]) < 1e-9 * np.abs(kap[:, None]), axis=1)
    assert ((_np(lut.F) == F) | near_gate).all()
    assert np.array_equal(_np(lut.S).view(np.uint32), S.view(np.uint32))
    assert np.array_equal(_np(lut.Z), Z)


def test_lut_full_stack_ten_buckets():
    """The sweep's LUT: 280 layers (70 blocks x 4 linears) x 10 buckets, SDXL's scaled-linear
    and PixArt's linear schedules, with a shortcut mask."""
    L, B = 280, 10
    st, ost = _c5_calibration(L, B)
    sc = (np.arange(L) % 37 == 5).astype(np.uint8)
    for sched, name in ((oracle.BETAS_SDXL, "sdxl"), (oracle.BETAS_PIXART, "pixart")):
        T, b0, b1, kind = sched
        case(f"build_act_lut {name} L={L} B={B}")
        lut = cham.build_act_lut(st, cham.Schedule(T=T, beta0=b0, beta1=b1, kind=kind),
                                 is_shortcut=torch.from_numpy(sc).to(DEV))
        torch.cuda.synchronize()
        F, S, Z, kap = oracle.build_lut(ost, sched, is_shortcut=sc)
        _check_lut(lut, F, S, Z, kap)
        assert len(set(F.tolist())) >= 3  # the gates route buckets to several formats


def test_lut_full_stack_kurtosis_only_one_bucket():
    """The single-step stack's fixed per-layer format: B = 1, SNR gate off (kurtosis only),
    statistics at t = 999, 280 layers."""
    L = 280
    Xs = [synth.diffusion_acts(41, l, 999, 16, 64) for l in range(L)]
    st = cham.alloc_stats(L, 1, DEV)
    cham.act_stats_reset(st)
    cham.act_stats_accumulate_batch([torch.from_numpy(x).to(DEV) for x in Xs], list(range(L)), [0] * L, st)
    ost = oracle.Stats(L, 1)
    for l, x in enumerate(Xs):
        ost.accumulate(x, l, 0)
    case(f"build_act_lut kurtosis-only L={L} B=1")
    lut = cham.build_act_lut(st, cham.Schedule(snr_gate_on=0))
    torch.cuda.synchronize()
    F, S, Z, kap = oracle.build_lut(ost, snr_gate_on=0)
    _check_lut(lut, F, S, Z, kap)


def _diag():
    if not os.path.exists(DIAG):
        from tests.native import build_diag
        build_diag.build()
    L = ctypes.CDLL(DIAG)
    L.cham_diag_rcp_sweep.argtypes = [ctypes.c_uint32, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p]
    L.cham_diag_rcp_values.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    return L


def test_rcp_rn_equals_ieee_quotient_everywhere():
    """rcp_rn (hardware estimate + one Newton step, division from 2^126 up) equals the
    correctly rounded 1.0f / a for every binary32 a in [2^-126, 2^128); and, against numpy's
    binary32 division on the CPU, for every mantissa at several exponents and around the
    2^126 switch."""
    L = _diag()
    out = torch.zeros(2, dtype=torch.int32, device=DEV)
    out[1] = -1  # 0xFFFFFFFF
    case("rcp_rn sweep over [2^-126, 2^128)")
    assert L.cham_diag_rcp_sweep(0x00800000, 0x7F800000, out.data_ptr(), None) == 0
    torch.cuda.synchronize()
    o = _np(out).view(np.uint32)
    assert o[0] == 0, f"{o[0]} mismatches, first at bits {o[1]:#010x}"
    mant = np.arange(1 << 23, dtype=np.uint32)
    for e in (-126, -1, 0, 63, 125, 126, 127):
        a = ((np.uint32(e + 127) << np.uint32(23)) | mant).view(np.float32)
        ad = torch.from_numpy(a).to(DEV)
        rd = torch.empty_like(ad)
        case(f"rcp_rn values at exponent {e}")
        assert L.cham_diag_rcp_values(ad.data_ptr(), rd.data_ptr(), a.size, None) == 0
        torch.cuda.synchronize()
        ref = np.float32(1.0) / a
        assert np.array_equal(_np(rd).view(np.uint32), ref.view(np.uint32)), e


@pytest.mark.parametrize("afmt,packed,M,N,K", [(cham.A_FP8_E5M2, True, 2048, 3840, 1280),
                                                (cham.A_MXFP8, False, 2048, 1280, 5120),
                                                (cham.A_INT8_ASYM, False, 300, 200, 640)])
def test_linear_exact_workspace(afmt, packed, M, N, K):
    """The workspace query names exactly what the call uses: the half-precision copy and
    row scales only for MX activations, the weight layout only without a packed layout, the
    partials only when the plan splits K; one byte less is refused before any launch, and
    the output equals the one computed with the CHAM_OP_LINEAR upper bound."""
    W = synth.hetero_weights_dev(77, N, K, DEV)
    X = synth.diffusion_acts_dev(0, 3, 379, M, K, DEV)
    case(f"exact workspace afmt={afmt} packed={packed} M={M} N={N} K={K}")
    wq = cham.select_weight_formats(W, cham.MASK_W4, want_packed=packed)
    xq = cham.quantize_act(X, afmt, dynamic=True)
    need = cham.linear_workspace_query(xq, wq)
    plan = cham.linear_plan(M, N, K, 4)
    exp = 0
    if afmt in (cham.A_MXFP8, cham.A_MXINT8):
        exp += -(-M * K * 2 // 256) * 256 + -(-M * 4 // 256) * 256
    if not packed:
        exp += -(-int(cham.lib().cham_packed_bytes(N, K)) // 256) * 256
    if plan["splits"] > 1:
        exp += plan["splits"] * M * N * 4
    assert need == exp, (need, exp, plan)
    assert need <= cham.workspace_bytes(cham.OP_LINEAR, M, N, K)
    full = torch.empty(cham.workspace_bytes(cham.OP_LINEAR, M, N, K), dtype=torch.uint8, device=DEV)
    Y_full = cham.mixed_linear(xq, wq, ws=full)
    Y_exact = cham.mixed_linear(xq, wq, ws=torch.empty(max(need, 1), dtype=torch.uint8, device=DEV)[:need]
                                if need else None)
    torch.cuda.synchronize()
    assert torch.equal(Y_full, Y_exact)
    if need:
        short = torch.empty(need, dtype=torch.uint8, device=DEV)[: need - 1]
        with pytest.raises(cham.ChamError) as ei:
            cham.mixed_linear(xq, wq, ws=short)
        assert ei.value.status == cham.EWORKSPACE
