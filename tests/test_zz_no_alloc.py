"""The allocation-free quantization entry point (cham_quantize_act_noalloc) against
cham_quantize_act on the same inputs: bit-identical codes, block exponents, scales and zero
points, over two calls in a row on the shared device array, the second with a smaller input
(per-tensor and per-sample dynamic scales, a static scale, an MX format)."""
import numpy as np
import pytest
import torch

from paper_2609_33496_amd import cham, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _same(a, b):
    for name in ("codes", "scale", "zero"):
        assert torch.equal(getattr(a, name), getattr(b, name)), name
    if a.fmt >= cham.A_MXFP8:
        assert torch.equal(a.e8m0, b.e8m0)


@pytest.mark.parametrize("fmt,ns", [(cham.A_INT8_ASYM, 1), (cham.A_INT8_ASYM, 2), (cham.A_FP8_E4M3, 2),
                                    (cham.A_FP8_E5M2, 1), (cham.A_MXFP8, 1)])
def test_noalloc_matches_workspace_entry_point(fmt, ns):
    big = synth.diffusion_acts(3, 1, 400, 4096, 1280)
    big[2048:] = big[2048:] * np.float32(4.0) + np.float32(1.5)  # the second sample: another range
    small = synth.diffusion_acts(4, 2, 800, 96, 640)
    for X in (big, small):  # the second call is smaller: leftover partials must not leak in
        M, K = X.shape
        print(f"[case] quantize_act_noalloc fmt={fmt} nsamples={ns} M={M} K={K}", flush=True)
        Xd = torch.from_numpy(X).to(DEV)
        ref = cham.quantize_act(Xd, fmt, dynamic=True, nsamples=ns)
        out = cham.alloc_aq(M, K, DEV, nsamples=ns)
        cham.quantize_act_noalloc(Xd, fmt, True, None, None, out)
        torch.cuda.synchronize()
        _same(out, ref)
    # static scales through the same entry point
    Xd = torch.from_numpy(small).to(DEV)
    sd, zd = torch.tensor([0.05], device=DEV), torch.tensor([-3.0], device=DEV)
    ref = cham.quantize_act(Xd, fmt, dynamic=False, s=sd, z=zd)
    out = cham.alloc_aq(*small.shape, DEV)
    cham.quantize_act_noalloc(Xd, fmt, False, sd, zd, out)
    torch.cuda.synchronize()
    _same(out, ref)
