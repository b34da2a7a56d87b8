"""GPU parity of the UNet path's 3x3 convolution on quantized activations (implicit GEMM,
stride 1, zero padding 1, channels last): every activation format, W4 and W8 weights,
ragged rows and channels, against the oracle's convolution; and an SDXL-like up-block
resnet conv1 fed by a shortcut concatenation, whose LUT entry is pinned to MXFP8 (Sec. 4.6),
on sampled outputs."""
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


@pytest.mark.parametrize("mask", [oracle.MASK_W4, oracle.MASK_W8])
def test_conv3x3_small_every_format(mask):
    B, H, W, C, Co = 2, 5, 7, 64, 96
    g = np.random.default_rng(1)
    X = (g.standard_t(4, (B, H, W, C)) * np.exp(g.normal(0, 1, (1, 1, 1, C)))).astype(np.float32)
    Wt, _ = synth.hetero_weights(2, Co, 9 * C)
    wq = cham.select_weight_formats(torch.from_numpy(Wt).to(DEV), mask)
    wp = cham.select_weight_formats(torch.from_numpy(Wt).to(DEV), mask, want_packed=True)
    ref = oracle.select_weight_formats(Wt, mask, want_err=False, want_perm=False)
    Wh = oracle.dequant_weights(ref, 9 * C)
    for fmt in range(5):
        for ns in (1, B):
            case(f"conv3x3 B={B} H={H} W={W} C={C} Co={Co} mask={mask:#x} fmt={fmt} nsamples={ns}")
            xq = cham.quantize_act(torch.from_numpy(X.reshape(-1, C)).to(DEV), fmt, dynamic=True, nsamples=ns)
            Y = _np(cham.conv3x3_mixed(xq, B, H, W, wq)).astype(np.float64)
            Yp = _np(cham.conv3x3_mixed(xq, B, H, W, wp)).astype(np.float64)
            _, _, xh, _, _ = oracle.quantize_act_per_sample(X.reshape(-1, C), fmt, ns, want_xhat=True)
            Yr, Bm = oracle.conv3x3(xh.reshape(B, H, W, C), Wh)
            rel = np.abs(Y - Yr.reshape(-1, Co)) / np.maximum(Bm.reshape(-1, Co), 1e-300)
            assert rel.max() <= 1e-3, (fmt, ns, rel.max())
            assert np.array_equal(Y, Yp)


def test_conv3x3_shortcut_conv1_mxfp8_sampled():
    """An SDXL-like up-block resnet conv1 on a shortcut concatenation (1280 + 640 -> 640
    channels at 32 x 32, CFG batch 2): the LUT routes its input to MXFP8 in every bucket,
    the W4 weights are searched per channel, and sampled outputs match the oracle."""
    B, H, W, C, Co = 2, 32, 32, 1920, 640
    L, Bk = 2, 4
    st = cham.alloc_stats(L, Bk, DEV)
    cham.act_stats_reset(st)
    for b in range(Bk):
        for l in range(L):
            cham.act_stats_accumulate(torch.from_numpy(synth.diffusion_acts(3, l, 125 + 250 * b, 64, C)).to(DEV), l, b, st)
    lut = cham.build_act_lut(st, is_shortcut=torch.tensor([0, 1], dtype=torch.uint8, device=DEV)).mirror()
    assert np.all(lut.F_host.numpy().reshape(L, Bk)[1] == cham.A_MXFP8)
    X = synth.diffusion_acts(4, 1, 600, B * H * W, C)
    X[:, 1280:] *= np.float32(8.0)  # the concatenated skip half on another scale: wide tails
    xq = cham.quantize_act_lut(torch.from_numpy(X).to(DEV), lut, 1, 600)
    assert xq.fmt == cham.A_MXFP8
    Wt, _ = synth.hetero_weights(5, Co, 9 * C)
    wq = cham.select_weight_formats(torch.from_numpy(Wt).to(DEV), cham.MASK_W4, want_packed=True)
    case(f"conv3x3 shortcut conv1 B={B} H={H} W={W} C={C} Co={Co} MXFP8")
    Y = _np(cham.conv3x3_mixed(xq, B, H, W, wq))
    codes, e8, xh = oracle.quantize_act(X, oracle.A_MXFP8, want_xhat=True)
    assert np.array_equal(_np(xq.codes), codes)
    g = np.random.default_rng(6)
    S = 1500
    pix = g.integers(0, B * H * W, S)
    pix[:4] = [0, W - 1, H * W - 1, B * H * W - W]  # corners: padding on two sides
    nn = g.integers(0, Co, S)
    chans = np.unique(nn)
    ref = oracle.select_weight_formats(Wt[chans], cham.MASK_W4, want_err=False, want_perm=False)
    Wh = np.zeros((Co, 9 * C), np.float32)
    Wh[chans] = oracle.dequant_weights(ref, 9 * C)
    xp = np.zeros((B, H + 2, W + 2, C), np.float32)
    xp[:, 1:-1, 1:-1] = xh.reshape(B, H, W, C)
    b, rem = pix // (H * W), pix % (H * W)
    y, x = rem // W, rem % W
    cols = np.concatenate([xp[b, y + ky, x + kx] for ky in range(3) for kx in range(3)], axis=1)
    Yr, Bm = oracle.linear_pairs(cols, Wh, np.arange(S), nn)
    rel = np.abs(Y[pix, nn].astype(np.float64) - Yr) / np.maximum(Bm, 1e-300)
    assert rel.max() <= 1e-3, rel.max()
