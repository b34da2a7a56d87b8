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
