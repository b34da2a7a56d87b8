"""GPU parity of the DiT path's activation side (Sec. 4.6 (ii), Alg. 3): per-sample,
per-forward dynamic scaling -- each sample of the CFG-doubled batch takes ScaleZP of its own
range -- through quantization and the mixed-format linear layer, at the PixArt-like
block's shapes (2 x 4096 tokens, width 1152; cross-attention KV over 2 x 120 tokens)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_33496_amd import cham, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def case(msg):
    print(f"[case] {msg}", flush=True)


def _np(t):
    return t.detach().cpu().numpy()


def _cfg_batch(M, K, seed, far=False):
    """Two samples of M/2 rows with different ranges (the second shifted and scaled, or, with
    far=True, narrow and far from zero so its INT8-asym zero point is beyond +-1024)."""
    h = M // 2
    a = synth.diffusion_acts(seed, 0, 300, h, K)
    b = synth.diffusion_acts(seed, 1, 700, h, K) * np.float32(6.0) + np.float32(2.0)
    if far:
        b = (np.float32(50.0) + np.float32(0.5) * np.abs(b) / np.abs(b).max()).astype(np.float32)
    return np.concatenate([a, b]).astype(np.float32)


@pytest.mark.parametrize("M,K,ns", [(8192, 1152, 2), (240, 4096, 2), (8192, 1152, 1), (256, 640, 4)])
def test_quantize_act_per_sample(M, K, ns):
    X = _cfg_batch(M, K, M + K)
    for fmt in range(5):
        case(f"quantize_act per-sample M={M} K={K} nsamples={ns} fmt={fmt}")
        aq = cham.quantize_act(torch.from_numpy(X).to(DEV), fmt, dynamic=True, nsamples=ns)
        torch.cuda.synchronize()
        codes, e8, _, s, z = oracle.quantize_act_per_sample(X, fmt, ns)
        assert np.array_equal(_np(aq.codes), codes), fmt
        assert np.array_equal(_np(aq.scale).view(np.uint32), s.view(np.uint32)), fmt
        assert np.array_equal(_np(aq.zero), z), fmt
        if fmt >= 3:
            assert np.array_equal(_np(aq.e8m0), e8)


@pytest.mark.parametrize("far", [False, True])
def test_linear_per_sample_dynamic(far):
    """A PixArt-like fc1 (1152 -> 4608) at 2 x 4096 tokens with W4 per-channel formats and
    per-sample A8 scales; sampled outputs of both samples against the oracle."""
    M, K, N = 8192, 1152, 4608
    X = _cfg_batch(M, K, 5, far=far)
    W, _ = synth.hetero_weights(71, N, K)
    wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), oracle.MASK_W4, want_packed=True)
    g = np.random.default_rng(9)
    mm = g.integers(0, M, 3000)
    nn = g.integers(0, N, 3000)
    rows = np.unique(mm)
    chans = np.unique(nn)
    ref = oracle.select_weight_formats(W[chans], oracle.MASK_W4, want_err=False, want_perm=False)
    Wh = np.zeros((N, K), np.float32)
    Wh[chans] = oracle.dequant_weights(ref, K)
    for fmt in (cham.A_INT8_ASYM, cham.A_FP8_E4M3, cham.A_FP8_E5M2):
        case(f"mixed_linear per-sample M={M} N={N} K={K} fmt={fmt} far={far}")
        xq = cham.quantize_act(torch.from_numpy(X).to(DEV), fmt, dynamic=True, nsamples=2)
        Y = _np(cham.mixed_linear(xq, wq))
        _, _, xh, s, z = oracle.quantize_act_per_sample(X, fmt, 2, want_xhat=True)
        if fmt == cham.A_INT8_ASYM and far:
            assert abs(z[1]) > 1024 and abs(z[0]) <= 255
        Yr, Bm = oracle.linear_pairs(xh, Wh, mm, nn)
        rel = np.abs(Y[mm, nn].astype(np.float64) - Yr) / np.maximum(Bm, 1e-300)
        assert rel.max() <= 1e-3, (fmt, rel.max())
        assert np.array_equal(_np(wq.fmt)[chans], ref["fmt"])
        assert rows.size > 1000


# ---------------------------------------------------------------------------------------
# joint (group size, format) search and the group-scaled GEMM (Sec. 4.6 (i))
# ---------------------------------------------------------------------------------------
def _gsearch_both(W, e, mask, gmask=cham.GMASK_ALL, packed=False):
    case(f"select_group_formats N={W.shape[0]} K={W.shape[1]} mask={mask:#x} gmask={gmask:#x} packed={packed}")
    gq = cham.select_group_formats(torch.from_numpy(W).to(DEV), torch.from_numpy(e).to(DEV), mask, gmask,
                                   want_packed=packed)
    torch.cuda.synchronize()
    ref = oracle.select_group_formats(W, mask, e, gmask)
    return gq, ref


def _assert_gsearch_equal(gq, ref):
    ch = _np(gq.choice)
    eg, er = _np(gq.err), ref["err"]
    assert np.array_equal(eg < 0, er < 0)
    assert np.allclose(eg[er >= 0], er[er >= 0], rtol=1e-10, atol=0), np.max(np.abs(eg - er) / np.maximum(er, 1e-300))
    if (ch[0], ch[1]) != (ref["g"], ref["fmt_id"]):
        v = np.sort(er[er >= 0])
        assert (v[1] - v[0]) <= 1e-12 * v[0], (ch, ref["g"], ref["fmt_id"], v[:2])  # a near tie only
        return False
    assert np.array_equal(_np(gq.fmt), ref["fmt"])
    assert np.array_equal(_np(gq.codes), ref["codes"])
    assert np.array_equal(_np(gq.gscale).view(np.uint32), ref["gscale"].view(np.uint32))
    assert np.array_equal(_np(gq.gzero), ref["gzero"])
    if gq.e8m0 is not None:
        assert np.array_equal(_np(gq.e8m0), ref["e8m0"])
    return True


@pytest.mark.parametrize("mask", [cham.MASK_DIT_W4, cham.MASK_W8, 0x1FF])
@pytest.mark.parametrize("N,K", [(37, 320), (9, 1152), (64, 4096), (5, 8192)])
def test_group_search_small(mask, N, K):
    W, _ = synth.hetero_weights(N + K, N, K)
    e = np.exp(np.random.default_rng(K).normal(0, 1, K)).astype(np.float32)
    for gmask in (cham.GMASK_ALL, 0b11000, 0b00010):
        gq, ref = _gsearch_both(W, e, mask, gmask)
        _assert_gsearch_equal(gq, ref)


def test_group_search_known_winner_and_zero_layer():
    g = np.random.default_rng(3)
    N, K = 12, 512
    v = oracle.nf4_table()
    W = v[g.integers(1, 15, (N, K))].astype(np.float32)
    W[:, ::64] = 1.0
    W = (W * np.repeat(np.exp(g.normal(0, 1, (N, K // 64))), 64, axis=1)).astype(np.float32)
    gq, ref = _gsearch_both(W, np.ones(K, np.float32), cham.MASK_DIT_W4)
    assert _assert_gsearch_equal(gq, ref) and tuple(_np(gq.choice)) == (64, cham.W_NF4)
    gq, ref = _gsearch_both(np.zeros((3, 192), np.float32), np.ones(192, np.float32), cham.MASK_W8)
    assert _assert_gsearch_equal(gq, ref) and tuple(_np(gq.choice)) == (32, cham.W_INT8_SYM)


def test_colsq_accumulate():
    g = np.random.default_rng(4)
    colsq = torch.zeros(1152, dtype=torch.float64, device=DEV)
    ref = np.zeros(1152)
    for M in (240, 8192, 7):
        X = (g.standard_t(3, (M, 1152)) * np.exp(g.normal(0, 1, 1152))).astype(np.float32)
        case(f"act_colsq_accumulate M={M}")
        cham.act_colsq_accumulate(torch.from_numpy(X).to(DEV), colsq)
        ref += np.sum(X.astype(np.float64) ** 2, axis=0)
    torch.cuda.synchronize()
    assert np.allclose(_np(colsq), ref, rtol=1e-12, atol=0)


@pytest.mark.parametrize("mask", [cham.MASK_DIT_W4, cham.MASK_W8])
def test_group_search_pixart_layers_and_gemm(mask):
    """PixArt-like proj (1152 -> 1152) and cross-attention KV (4096 -> 1152: K not a
    multiple of 192 or 288) with input-aware weights E[x_k^2] from the activations' column
    sums of squares: the search against the oracle, then (4-bit) the group-scaled GEMM with
    per-sample dynamic A8 scales on sampled outputs."""
    for name, K, N, M in (("proj", 1152, 1152, 8192), ("cross_kv", 4096, 1152, 240)):
        X = _cfg_batch(M, K, K)
        colsq = torch.zeros(K, dtype=torch.float64, device=DEV)
        cham.act_colsq_accumulate(torch.from_numpy(X).to(DEV), colsq)
        e = (_np(colsq) / M).astype(np.float32)
        W, _ = synth.hetero_weights(80 + K, N, K)
        gq, ref = _gsearch_both(W, e, mask, packed=mask == cham.MASK_DIT_W4)
        if not _assert_gsearch_equal(gq, ref) or mask != cham.MASK_DIT_W4:
            continue
        Wh = oracle.dequant_grouped(ref, K)
        g = np.random.default_rng(K)
        mm, nn = g.integers(0, M, 3000), g.integers(0, N, 3000)
        for fmt in (cham.A_INT8_ASYM, cham.A_FP8_E5M2, cham.A_MXFP8):
            case(f"mixed_linear_grouped {name} M={M} fmt={fmt} choice={tuple(_np(gq.choice))}")
            xq = cham.quantize_act(torch.from_numpy(X).to(DEV), fmt, dynamic=True, nsamples=2)
            Y = _np(cham.mixed_linear_grouped(xq, gq))
            gq_np = cham.GWQ(**{**gq.__dict__, "packed": None})  # the same weights through the pre-pass
            Y2 = _np(cham.mixed_linear_grouped(xq, gq_np))
            _, _, xh, _, _ = oracle.quantize_act_per_sample(X, fmt, 2, want_xhat=True)
            Yr, Bm = oracle.linear_pairs(xh, Wh, mm, nn)
            rel = np.abs(Y[mm, nn].astype(np.float64) - Yr) / np.maximum(Bm, 1e-300)
            assert rel.max() <= 1e-3, (name, fmt, rel.max())
            assert np.array_equal(Y, Y2)


def test_group_gemm_every_choice():
    """The group-scaled GEMM for every (g, f) of the 4-bit DiT set, forced one tuple at a
    time (single-group, single-format masks), K = 320 (ragged groups) and 1152."""
    g = np.random.default_rng(6)
    for K in (320, 1152):
        W, _ = synth.hetero_weights(90 + K, 200, K)
        X = (g.standard_t(4, (130, K)) * 0.7).astype(np.float32)
        e = np.ones(K, np.float32)
        for gi, gsz in enumerate(cham.GROUP_SIZES):
            for f in (cham.W_INT4_ASYM, cham.W_NF4, cham.W_FP4):
                if K % 64 and f == cham.W_NF4:
                    pass  # NF4 groups follow g, not 64: any K % 32 == 0 works
                gq, ref = _gsearch_both(W, e, 1 << f, 1 << gi)
                assert _assert_gsearch_equal(gq, ref)
                if K % 64:
                    continue  # the GEMM takes 64-wide k-steps
                Wh = oracle.dequant_grouped(ref, K)
                xq = cham.quantize_act(torch.from_numpy(X).to(DEV), cham.A_FP8_E4M3, dynamic=True)
                Y = _np(cham.mixed_linear_grouped(xq, gq)).astype(np.float64)
                _, _, xh, _, _ = oracle.quantize_act_dynamic(X, cham.A_FP8_E4M3, want_xhat=True)
                Yr, Bm = oracle.linear(xh, Wh)
                rel = np.abs(Y - Yr) / np.maximum(Bm, 1e-300)
                assert rel.max() <= 1e-3, (gsz, f, rel.max())
