"""GPU parity: the HIP library (through the C ABI) against the CPU oracle on the same seeded
inputs.  Bit-exact for formats, codes, scales, zero points, block metadata, perm and the LUT;
kurtosis within 1e-4 relative; the linear layer within 1e-3 * sum|x^ w^| per element."""
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


def _search_both(W, mask, want_err=True):
    case(f"select_weight_formats N={W.shape[0]} K={W.shape[1]} mask={mask:#x}")
    wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), mask, want_err=want_err)
    torch.cuda.synchronize()
    ref = oracle.select_weight_formats(W, mask, want_err=want_err)
    return wq, ref


def _assert_search_equal(wq, ref, check_perm=True):
    f = _np(wq.fmt)
    bad = np.nonzero(f != ref["fmt"])[0]
    if bad.size and ref["err"] is not None:
        # report near-ties (errors equal to ~1e-12) separately from real mismatches
        e = ref["err"][bad]
        ties = [np.sort(r[r >= 0])[:2] for r in e]
        rel = [abs(t[1] - t[0]) / max(t[0], 1e-300) for t in ties]
        assert all(r < 1e-12 for r in rel), (bad[:10], f[bad[:10]], ref["fmt"][bad[:10]], rel[:10])
    assert bad.size == 0, bad[:10]
    assert np.array_equal(_np(wq.codes), ref["codes"])
    assert np.array_equal(_np(wq.scale).view(np.uint32), ref["scale"].view(np.uint32))
    assert np.array_equal(_np(wq.zero), ref["zero"])
    if wq.nf4_absmax is not None:
        assert np.array_equal(_np(wq.nf4_absmax).view(np.uint32), ref["nf4_absmax"].view(np.uint32))
    if wq.e8m0 is not None:
        assert np.array_equal(_np(wq.e8m0), ref["e8m0"])
    if check_perm and wq.perm is not None:
        assert np.array_equal(_np(wq.perm), ref["perm"])
        assert np.array_equal(_np(wq.group_off), ref["group_off"])
    if wq.err is not None and ref["err"] is not None:
        g, r = _np(wq.err), ref["err"]
        # binary32 sums unless a near tie forced the binary64 re-check (documented accuracy 1e-5)
        assert np.allclose(g, r, rtol=1e-5, atol=1e-30), np.max(np.abs(g - r) / np.maximum(np.abs(r), 1e-300))


# ---------------------------------------------------------------------------------------
# weight-format search
# ---------------------------------------------------------------------------------------
def test_search_single_layer_w4():
    X, W = synth.single_layer(0)
    wq, ref = _search_both(W, oracle.MASK_W4)
    _assert_search_equal(wq, ref)
    assert np.all(ref["fmt"] == oracle.W_NF4)


@pytest.mark.parametrize("mask", [oracle.MASK_W4, oracle.MASK_W8, oracle.MASK_W4_FULL,
                                  (1 << oracle.W_INT4_SYM) | (1 << oracle.W_FP4) | (1 << oracle.W_MXFP4),
                                  0x1FF])
@pytest.mark.parametrize("N,K", [(37, 640), (300, 1280), (20, 1152), (24, 4608), (9, 5120), (5, 8192), (3, 64)])
def test_search_hetero_rows(mask, N, K):
    if (mask >> oracle.W_NF4) & 1 and K % 64:
        pytest.skip("NF4 needs K % 64 == 0")
    W, fam = synth.hetero_weights(N * 7 + K, N, K)
    wq, ref = _search_both(W, mask)
    _assert_search_equal(wq, ref)


def _special_rows(K, g):
    """Rows with known winners (NF4 levels, INT4 grid, E2M1 grid with one block scale --
    an exact FP4 / MXFP4 tie --, E2M1 with a scale per block) and degenerate rows."""
    rows = []
    v = oracle.nf4_table()
    r = v[g.integers(0, 16, K)]
    r[::64] = 1.0
    rows.append(r * 2.0 ** -5)
    q = g.integers(0, 16, K); q[:2] = (0, 15)
    rows.append((q - 5) * 0.0625)
    e2 = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6])
    r = e2[g.integers(0, 8, K)] * g.choice([-1, 1], K); r[::32] = 6
    rows.append(r * 2.0 ** -6)
    r = e2[g.integers(0, 8, K)] * g.choice([-1, 1], K); r[::32] = 6
    rows.append(r * np.repeat(2.0 ** (-3.0 * np.arange(K // 32)), 32))
    rows.append(np.zeros(K))                                   # all zero
    rows.append(np.full(K, 0.37))                              # constant positive
    rows.append(np.full(K, -2.5e-3))                           # constant negative
    rows.append(g.normal(size=K) * 1e-39)                      # subnormal
    rows.append(g.normal(size=K) * 1e30)                       # huge
    rr = g.normal(size=K) * 0.02; rr[17] = 3.0                 # one outlier
    rows.append(rr)
    rr = g.normal(size=K); rr[:128] = 0                        # half zero (all-zero blocks)
    rows.append(rr)
    rows.append(np.where(g.random(K) < 0.5, -0.0, 0.0))       # signed zeros
    return rows


@pytest.mark.parametrize("K", [256, 1024])  # 1024: each row split over four wavefronts
def test_search_known_winners_and_degenerate_rows(K):
    W = np.stack(_special_rows(K, np.random.default_rng(0))).astype(np.float32)
    for mask in (oracle.MASK_W4, oracle.MASK_W8, 0x1FF):
        wq, ref = _search_both(W, mask)
        _assert_search_equal(wq, ref)


@pytest.mark.parametrize("mask", [oracle.MASK_W4, oracle.MASK_W8, 0x1FF,
                                  (1 << oracle.W_INT4_SYM) | (1 << oracle.W_FP4) | (1 << oracle.W_MXFP4)])
@pytest.mark.parametrize("K", [64, 640, 1152, 2560, 3200, 5120])
def test_search_several_channels_per_wavefront(mask, K):
    """Layers of >= 1024 channels with rows up to 5120 elements: 4, 2 or 1 channels per
    wavefront, 8 consecutive elements per lane (ragged last chunk at K = 1152, 3200 and 64).  The
    special rows (exact ties take the binary64 re-check) sit at every offset within a
    wavefront's channel groups; the rest are heterogeneous rows."""
    g = np.random.default_rng(K)
    sp = _special_rows(K, g) if K >= 256 else []
    H, _ = synth.hetero_weights(K + 5, 1031, K)
    rows = list(H)
    for i, r in enumerate(sp):  # row 3 i + (0, 1, 2): different lane groups and wavefronts
        rows[3 * i + i % 3] = r
    W = np.stack(rows).astype(np.float32)
    wq, ref = _search_both(W, mask)
    _assert_search_equal(wq, ref)


def test_search_full_size_sampled():
    """SDXL-like GEGLU weight (N = 10240, K = 1280) and FF-out (N = 1280, K = 5120): the
    whole matrix is searched on the GPU; sampled channels are checked against the oracle."""
    for name, K, N in (("geglu", 1280, 10240), ("ff_out", 5120, 1280)):
        W, _ = synth.hetero_weights(11, N, K)
        case(f"select_weight_formats full-size {name} N={N} K={K}")
        wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), oracle.MASK_W4)
        torch.cuda.synchronize()
        rows = np.sort(np.random.default_rng(1).choice(N, 256, replace=False))
        ref = oracle.select_weight_formats(W[rows], oracle.MASK_W4)
        f = _np(wq.fmt)
        assert np.array_equal(f[rows], ref["fmt"])
        assert np.array_equal(_np(wq.codes)[rows], ref["codes"])
        assert np.array_equal(_np(wq.scale)[rows], ref["scale"])
        assert np.array_equal(_np(wq.nf4_absmax)[rows], ref["nf4_absmax"])
        assert np.array_equal(_np(wq.e8m0)[rows], ref["e8m0"])
        # perm is a stable sort of the GPU's own format vector, group_off its group starts
        assert np.array_equal(_np(wq.perm), np.argsort(f, kind="stable"))
        counts = np.bincount(f, minlength=9)
        assert np.array_equal(_np(wq.group_off), np.concatenate([[0], np.cumsum(counts)]))


@pytest.mark.parametrize("mask", [oracle.MASK_W4, oracle.MASK_W8])
def test_search_pixart_block_sampled(mask):
    """One PixArt-like DiT block (QKV 1152->3456, proj 1152->1152, MLP 1152->4608->1152,
    cross-attn KV 4096->1152) searched in one batched call, at W4 and at W8 {INT8, MXINT8}:
    sampled channels of every layer against the oracle (formats, codes, metadata), and the
    grouping of each layer's own format vector."""
    layers = synth.pixart_block_layers()
    Ws = [synth.hetero_weights(70 + i, N, K)[0] for i, (_, K, N, _) in enumerate(layers)]
    case(f"select_weight_formats_batch PixArt-like block mask={mask:#x}")
    outs = cham.select_weight_formats_batch([torch.from_numpy(W).to(DEV) for W in Ws], mask)
    torch.cuda.synchronize()
    g = np.random.default_rng(mask)
    for (name, K, N, _), W, wq in zip(layers, Ws, outs):
        rows = np.sort(g.choice(N, 96, replace=False))
        ref = oracle.select_weight_formats(W[rows], mask)
        f = _np(wq.fmt)
        assert np.array_equal(f[rows], ref["fmt"]), name
        assert np.array_equal(_np(wq.codes)[rows], ref["codes"]), name
        assert np.array_equal(_np(wq.scale)[rows], ref["scale"]), name
        assert np.array_equal(_np(wq.zero)[rows], ref["zero"]), name
        for meta in ("nf4_absmax", "e8m0"):  # a palette without the kind allocates no buffer
            buf = getattr(wq, meta)
            if buf is None:
                assert not np.any(ref[meta]), (name, meta)
            else:
                assert np.array_equal(_np(buf)[rows], ref[meta]), (name, meta)
        assert np.array_equal(_np(wq.perm), np.argsort(f, kind="stable")), name
        counts = np.bincount(f, minlength=9)
        assert np.array_equal(_np(wq.group_off), np.concatenate([[0], np.cumsum(counts)])), name


def test_search_batch_matches_single_calls():
    """The batched search over 19 layers of mixed shapes, kernel variants and palettes (more
    layers than one launch takes) equals one call per layer, bit for bit."""
    shapes = [(37, 640), (300, 1280), (20, 1152), (24, 4608), (9, 5120), (5, 8192), (3, 64), (4100, 256),
              (1280, 1280), (64, 5120), (7, 2048)] * 2
    masks = [oracle.MASK_W4, oracle.MASK_W8, 0x1FF, (1 << oracle.W_INT4_SYM) | (1 << oracle.W_FP4)]
    Ws, outs, singles = [], [], []
    for i, (N, K) in enumerate(shapes[:19]):
        m = masks[i % len(masks)]
        W, _ = synth.hetero_weights(500 + i, N, K)
        Wd = torch.from_numpy(W).to(DEV)
        Ws.append(Wd)
        pk = K % 64 == 0 and i % 2 == 0
        o, o1 = [cham.alloc_wq(N, K, m, DEV, want_perm=(i % 3 != 2), want_err=(i % 5 == 0), want_packed=pk)
                 for _ in range(2)]
        if pk:  # the layout leaves alignment padding unwritten: start both from zeros
            o.packed.zero_()
            o1.packed.zero_()
        outs.append(o)
        singles.append(cham.select_weight_formats(Wd, m, out=o1))
    case("select_weight_formats_batch 19 layers")
    cham.select_weight_formats_batch(Ws, outs=outs)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(outs, singles)):
        assert a.code_bits == b.code_bits, i
        for name in ("fmt", "codes", "scale", "zero", "nf4_absmax", "e8m0", "perm", "group_off", "err", "packed"):
            x, y = getattr(a, name), getattr(b, name)
            assert (x is None) == (y is None), (i, name)
            if x is not None:
                assert torch.equal(x, y), (i, name)


def test_pack_batch_matches_packing_search():
    """Packing on its own after a search that wrote no layout (in chunks, on a second stream
    that waits for the search) gives the bytes the packing search writes, for 40 layers of
    mixed shapes and palettes (more than one packing launch takes)."""
    shapes = [(37, 640), (300, 1280), (24, 4608), (9, 5120), (5, 8192), (3, 64), (4100, 256), (1280, 1280),
              (64, 5120), (130, 2048)]
    masks = [oracle.MASK_W4, oracle.MASK_W8, 0x1FF, (1 << oracle.W_NF4) | (1 << oracle.W_MXFP4),
             (1 << oracle.W_INT8_ASYM) | (1 << oracle.W_MXINT8)]
    Ws, plain, packing = [], [], []
    for i in range(40):
        N, K = shapes[i % len(shapes)]
        m = masks[i % len(masks)]
        W, _ = synth.hetero_weights(900 + i, N, K)
        Ws.append(torch.from_numpy(W).to(DEV))
        a = cham.alloc_wq(N, K, m, DEV, want_perm=(i % 2 == 0))
        a.packed = torch.zeros(cham.packed_bytes(N, K), dtype=torch.uint8, device=DEV)
        b = cham.alloc_wq(N, K, m, DEV, want_perm=(i % 2 == 0), want_packed=True)
        b.packed.zero_()
        plain.append(a)
        packing.append(b)
    case("select_weight_formats_batch 40 layers, packing alone in chunks on a second stream")
    bufs = [a.packed for a in plain]
    for a in plain:
        a.packed = None
    cham.SearchBatch(Ws, plain).run()
    for a, buf in zip(plain, bufs):
        a.packed = buf
    done = torch.cuda.Event()
    done.record()
    side = torch.cuda.Stream()
    side.wait_event(done)
    for c in range(0, 40, 13):
        cham.PackBatch(plain[c:c + 13], bufs[c:c + 13]).run(side)
    cham.select_weight_formats_batch(Ws, outs=packing)
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(plain, packing)):
        for name in ("fmt", "codes", "scale", "zero", "nf4_absmax", "e8m0", "perm", "group_off", "packed"):
            x, y = getattr(a, name), getattr(b, name)
            assert (x is None) == (y is None), (i, name)
            if x is not None:
                assert torch.equal(x, y), (i, name)


def test_search_grouping_repeated_and_partial_outputs():
    """Repeated calls on one output object, a different matrix in between, and calls that
    request only perm or only group_off all give the stable sort of the formats."""
    Wa, _ = synth.hetero_weights(21, 3000, 640)   # 750 workgroups, ragged last one
    Wb, _ = synth.hetero_weights(22, 3000, 640)
    wq = cham.alloc_wq(3000, 640, oracle.MASK_W4, DEV)
    wp = cham.alloc_wq(3000, 640, oracle.MASK_W4, DEV, want_packed=True)  # grouping in the packing launch
    for it, (W, w) in enumerate(((Wa, wq), (Wb, wq), (Wa, wq), (Wb, wp), (Wa, wp))):
        wq = w
        case(f"select_weight_formats grouping call {it} N=3000 K=640 packed={w.packed is not None}")
        cham.select_weight_formats(torch.from_numpy(W).to(DEV), oracle.MASK_W4, out=wq)
        torch.cuda.synchronize()
        f = _np(wq.fmt)
        assert np.array_equal(_np(wq.perm), np.argsort(f, kind="stable"))
        assert np.array_equal(_np(wq.group_off), np.concatenate([[0], np.cumsum(np.bincount(f, minlength=9))]))
    for keep, pk in (("perm", False), ("group_off", False), ("perm", True), ("group_off", True)):
        case(f"select_weight_formats grouping with only {keep} packed={pk}")
        w2 = cham.alloc_wq(3000, 640, oracle.MASK_W4, DEV, want_packed=pk)
        setattr(w2, "group_off" if keep == "perm" else "perm", None)
        cham.select_weight_formats(torch.from_numpy(Wa).to(DEV), oracle.MASK_W4, out=w2)
        torch.cuda.synchronize()
        f = _np(w2.fmt)
        if keep == "perm":
            assert np.array_equal(_np(w2.perm), np.argsort(f, kind="stable"))
        else:
            assert np.array_equal(_np(w2.group_off), np.concatenate([[0], np.cumsum(np.bincount(f, minlength=9))]))


# ---------------------------------------------------------------------------------------
# activation statistics and LUT
# ---------------------------------------------------------------------------------------
def _calibrate(L, B, M, K, seed=0, T=1000, steps_per_bucket=2):
    st = cham.alloc_stats(L, B, DEV)
    cham.act_stats_reset(st)
    ost = oracle.Stats(L, B)
    for b in range(B):
        for i in range(steps_per_bucket):
            t = (b * T) // B + (i * T) // (B * steps_per_bucket) + 3
            for l in range(L):
                x = synth.diffusion_acts(seed, l, t, M, K)
                case(f"act_stats_accumulate layer={l} bucket={b} t={t} numel={x.size}")
                cham.act_stats_accumulate(torch.from_numpy(x).to(DEV), l, b, st)
                ost.accumulate(x, l, b)
    return st, ost


def test_stats_and_lut_match_oracle():
    L, B = 6, 4
    st, ost = _calibrate(L, B, 96, 320)
    torch.cuda.synchronize()
    nS = _np(st.nS)
    assert np.allclose(nS, ost.nS, rtol=1e-12, atol=0)
    assert np.array_equal(_np(st.lohi), ost.lohi)
    for sched, name in ((oracle.BETAS_SDXL, "sdxl"), (oracle.BETAS_PIXART, "pixart")):
        T, b0, b1, kind = sched
        s = cham.Schedule(T=T, beta0=b0, beta1=b1, kind=kind)
        shortcut = torch.tensor([0, 0, 1, 0, 0, 0], dtype=torch.uint8, device=DEV)
        case(f"build_act_lut {name} L={L} B={B}")
        lut = cham.build_act_lut(st, s, is_shortcut=shortcut)
        torch.cuda.synchronize()
        F, S, Z, kap = oracle.build_lut(ost, sched, is_shortcut=np.array([0, 0, 1, 0, 0, 0], np.uint8))
        kg = _np(lut.kappa)
        assert np.allclose(kg, kap, rtol=1e-4)
        near_gate = np.any(np.abs(kap[:, None] - np.array([3.0, 5.0])[None, :]) < 1e-9 * np.abs(kap[:, None]), axis=1)
        ok = (_np(lut.F) == F) | near_gate
        assert ok.all(), (_np(lut.F), F)
        assert np.array_equal(_np(lut.S).view(np.uint32), S.view(np.uint32))
        assert np.array_equal(_np(lut.Z), Z)
    # the kurtosis-only arm (SNR gate off) and an empty bucket
    st2 = cham.alloc_stats(2, 3, DEV)
    cham.act_stats_reset(st2)
    ost2 = oracle.Stats(2, 3)
    for l in range(2):
        x = synth.diffusion_acts(1, l, 900, 64, 128)
        cham.act_stats_accumulate(torch.from_numpy(x).to(DEV), l, 0, st2)
        ost2.accumulate(x, l, 0)
    lut2 = cham.build_act_lut(st2, cham.Schedule(snr_gate_on=0))
    torch.cuda.synchronize()
    F2, S2, Z2, _ = oracle.build_lut(ost2, snr_gate_on=0)
    assert np.array_equal(_np(lut2.F), F2) and np.array_equal(_np(lut2.S), S2) and np.array_equal(_np(lut2.Z), Z2)


def test_stats_batch_matches_single_calls():
    """The batched accumulate over 21 tensors (two launches' worth; ragged sizes; several
    tensors of the same (layer, bucket), interleaved with others) gives the bits of one
    call per tensor in array order, and matches the oracle."""
    L, B = 3, 2
    g = np.random.default_rng(7)
    sizes = [int(v) for v in g.integers(1, 300_000, 21)] + [5, 2_000_003]
    Xs = [g.standard_t(4, n).astype(np.float32) * (1 + i % 3) for i, n in enumerate(sizes)]
    layers = [i % L for i in range(len(Xs))]
    buckets = [(i // L) % B for i in range(len(Xs))]
    sa, sb = cham.alloc_stats(L, B, DEV), cham.alloc_stats(L, B, DEV)
    cham.act_stats_reset(sa)
    cham.act_stats_reset(sb)
    ost = oracle.Stats(L, B)
    Xd = [torch.from_numpy(x).to(DEV) for x in Xs]
    case(f"act_stats_accumulate_batch {len(Xs)} tensors")
    cham.act_stats_accumulate_batch(Xd, layers, buckets, sa)
    for x, xd, l, b in zip(Xs, Xd, layers, buckets):
        cham.act_stats_accumulate(xd, l, b, sb)
        ost.accumulate(x, l, b)
    torch.cuda.synchronize()
    assert np.array_equal(_np(sa.nS), _np(sb.nS))
    assert np.array_equal(_np(sa.lohi), _np(sb.lohi))
    assert np.allclose(_np(sa.nS), ost.nS, rtol=1e-12, atol=0)
    assert np.array_equal(_np(sa.lohi), ost.lohi)


def test_stats_ragged_and_tiny():
    for n in (1, 3, 5, 1023, 4097, 1_000_003):
        x = np.random.default_rng(n).standard_t(4, n).astype(np.float32)
        st = cham.alloc_stats(1, 1, DEV)
        cham.act_stats_reset(st)
        case(f"act_stats_accumulate ragged numel={n}")
        cham.act_stats_accumulate(torch.from_numpy(x).to(DEV), 0, 0, st)
        torch.cuda.synchronize()
        ost = oracle.Stats(1, 1)
        ost.accumulate(x, 0, 0)
        assert np.allclose(_np(st.nS), ost.nS, rtol=1e-12)
        assert np.array_equal(_np(st.lohi), ost.lohi)


# ---------------------------------------------------------------------------------------
# activation quantization
# ---------------------------------------------------------------------------------------
def _check_aq(aq, X, fmt, s=None, z=None, dynamic=True):
    if dynamic:
        codes, e8, xh, s_ref, z_ref = oracle.quantize_act_dynamic(X, fmt)
    else:
        codes, e8, xh = oracle.quantize_act(X, fmt, s, z)
        s_ref, z_ref = (np.float32(s), np.float32(z)) if fmt < 3 else (np.float32(1), np.float32(0))
    gc = _np(aq.codes)
    bad = np.argwhere(gc != codes)
    assert bad.shape[0] == 0, (fmt, bad[:5], gc[tuple(bad[:5].T)], codes[tuple(bad[:5].T)], X[tuple(bad[:5].T)])
    assert _np(aq.scale)[0] == s_ref and _np(aq.zero)[0] == z_ref
    if fmt >= 3:
        assert np.array_equal(_np(aq.e8m0), e8)


@pytest.mark.parametrize("fmt", range(5))
def test_quantize_act_dynamic(fmt):
    X, _ = synth.single_layer(0)
    case(f"quantize_act dynamic fmt={fmt} M={X.shape[0]} K={X.shape[1]}")
    aq = cham.quantize_act(torch.from_numpy(X).to(DEV), fmt, dynamic=True)
    torch.cuda.synchronize()
    _check_aq(aq, X, fmt)


@pytest.mark.parametrize("fmt", range(5))
def test_quantize_act_static_with_saturation(fmt):
    X = synth.diffusion_acts(0, 1, 500, 200, 384)
    lo, hi = oracle.minmax(X)
    s, z = oracle.scale_zp(fmt, lo * 0.5, hi * 0.5)  # calibrated range narrower than X: saturation
    sd = torch.tensor([s], dtype=torch.float32, device=DEV)
    zd = torch.tensor([z], dtype=torch.float32, device=DEV)
    case(f"quantize_act static fmt={fmt}")
    aq = cham.quantize_act(torch.from_numpy(X).to(DEV), fmt, dynamic=False, s=sd, z=zd)
    torch.cuda.synchronize()
    _check_aq(aq, X, fmt, s, z, dynamic=False)


def test_fp8_conversion_on_every_tie_and_boundary():
    """Every midpoint between neighbouring E4M3 / E5M2 values, the floats next to it, the
    subnormal range and the saturation edge, quantized with s = 1 (static)."""
    for fmt, which, mx in ((cham.A_FP8_E4M3, oracle.MF_E4M3, 448.0), (cham.A_FP8_E5M2, oracle.MF_E5M2, 57344.0)):
        maxc = 0x7E if which == oracle.MF_E4M3 else 0x7B
        vals = sorted(set(oracle.mf_decode(which, c) for c in range(maxc + 1)))
        xs = []
        for a_, b_ in zip(vals[:-1], vals[1:]):
            m = np.float32((a_ + b_) / 2)
            xs += [a_, m, np.nextafter(m, np.float32(0)), np.nextafter(m, np.float32(1e30))]
        xs += [mx, mx * 1.01, 1e30, 1e-45, 0.0]
        xs = np.array(xs + [-x for x in xs], np.float32)
        xs = np.concatenate([xs, np.zeros((-xs.size) % 64, np.float32)]).reshape(-1, 64)
        sd = torch.ones(1, device=DEV)
        zd = torch.zeros(1, device=DEV)
        case(f"quantize_act fp8 boundaries fmt={fmt}")
        aq = cham.quantize_act(torch.from_numpy(xs).to(DEV), fmt, dynamic=False, s=sd, z=zd)
        torch.cuda.synchronize()
        _check_aq(aq, xs, fmt, 1.0, 0.0, dynamic=False)


def test_mxfp8_conversion_on_every_tie():
    """MXFP8: every E4M3 midpoint (and its neighbours) times the block scale 2^E, in
    32-element blocks whose largest element fixes E, for several E (subnormal, clamped)."""
    vals = sorted(set(oracle.mf_decode(oracle.MF_E4M3, c) for c in range(0x7F)))
    xs = []
    for a_, b_ in zip(vals[:-1], vals[1:]):
        m = np.float32((a_ + b_) / 2)
        xs += [m, np.nextafter(m, np.float32(0)), np.nextafter(m, np.float32(1e30))]
    xs = np.array(xs + [-x for x in xs], np.float32)
    xs = np.concatenate([xs, np.zeros((-xs.size) % 31, np.float32)]).reshape(-1, 31)
    rows = []
    for E in (-20, -3, 0, 7, 40):
        blk = np.concatenate([np.full((xs.shape[0], 1), 256.0, np.float32), xs], axis=1) * np.float32(2.0 ** E)
        rows.append(blk.reshape(-1))
    X = np.concatenate(rows)
    X = np.concatenate([X, np.zeros((-X.size) % 256, np.float32)]).reshape(-1, 256)
    case(f"quantize_act MXFP8 ties M={X.shape[0]}")
    aq = cham.quantize_act(torch.from_numpy(X).to(DEV), cham.A_MXFP8, dynamic=True)
    torch.cuda.synchronize()
    _check_aq(aq, X, cham.A_MXFP8)


@pytest.mark.parametrize("dynamic", [False, True])
def test_quantize_act_lut_lookup(dynamic):
    """Alg. runtime (static: the bucket's calibrated S, Z) and Alg. runtime_dit (dynamic:
    the LUT's format with ScaleZP of this tensor's own min / max)."""
    L, B = 3, 4
    st, ost = _calibrate(L, B, 64, 256, seed=2, steps_per_bucket=1)
    lut = cham.build_act_lut(st).mirror()
    F, S, Z, _ = oracle.build_lut(ost)
    for l in range(L):
        for t in (0, 260, 600, 999):
            X = synth.diffusion_acts(5, l, t, 64, 256)
            case(f"quantize_act_lut layer={l} t={t} dynamic={dynamic}")
            aq = cham.quantize_act_lut(torch.from_numpy(X).to(DEV), lut, l, t, dynamic=dynamic)
            torch.cuda.synchronize()
            i = l * B + oracle.bucket(t, 1000, B)
            assert aq.fmt == F[i]
            if dynamic:
                _check_aq(aq, X, int(F[i]))
            else:
                _check_aq(aq, X, int(F[i]), S[i], Z[i], dynamic=False)


def test_quantize_accumulate_matches_separate_calls():
    """The fused pass (quantize with the LUT's static scales while adding the moments) gives
    the bits of quantize_act_lut per tensor followed by act_stats_accumulate_batch: every
    activation format (a host format mirror set per layer), ragged row counts, two samples,
    K a multiple of 32 only, a layer seen twice, and more tensors than one launch takes;
    the codes also against the oracle."""
    L, B, t = 7, 4, 600
    st0, _ = _calibrate(L, B, 64, 256, seed=4, steps_per_bucket=1)
    lut = cham.build_act_lut(st0).mirror()
    b = oracle.bucket(t, 1000, B)
    F = lut.F_host.clone()
    for l in range(L):  # every format, whatever the gates chose
        F[l * B + b] = l % 5
    lut.F_host = F
    shapes = [(37 + 13 * i, 32 * (1 + i % 5)) for i in range(40)]
    layers = [i % L for i in range(40)]
    Xs = [torch.from_numpy(synth.diffusion_acts(6, l, t, M, K)).to(DEV) for (M, K), l in zip(shapes, layers)]
    nsamp = [2 if M % 2 == 0 else 1 for (M, _) in shapes]
    # separate calls on a copy of the accumulators
    st_a = cham.alloc_stats(L, B, DEV)
    st_a.nS.copy_(st0.nS)
    st_a.lohi.copy_(st0.lohi)
    st_b = cham.alloc_stats(L, B, DEV)
    st_b.nS.copy_(st0.nS)
    st_b.lohi.copy_(st0.lohi)
    case("quantize_act_lut x 40 then act_stats_accumulate_batch")
    ref = [cham.quantize_act_lut(X, lut, l, t, dynamic=False, nsamples=ns) for X, l, ns in zip(Xs, layers, nsamp)]
    cham.act_stats_accumulate_batch(Xs, layers, [b] * len(Xs), st_a)
    case("quantize_act_lut_accumulate_batch x 40")
    outs = [cham.alloc_aq(X.shape[0], X.shape[1], DEV, nsamples=ns) for X, ns in zip(Xs, nsamp)]
    cham.quantize_act_lut_accumulate_batch(Xs, layers, t, lut, st_b, outs=outs)
    torch.cuda.synchronize()
    assert np.array_equal(_np(st_a.nS).view(np.uint64), _np(st_b.nS).view(np.uint64))
    assert np.array_equal(_np(st_a.lohi).view(np.uint32), _np(st_b.lohi).view(np.uint32))
    S, Z = _np(lut.S), _np(lut.Z)
    for i, (r, o, X, l) in enumerate(zip(ref, outs, Xs, layers)):
        fmt = int(F[l * B + b])
        assert o.fmt == r.fmt == fmt
        assert np.array_equal(_np(o.codes), _np(r.codes)), i
        assert np.array_equal(_np(o.scale).view(np.uint32), _np(r.scale).view(np.uint32)), i
        assert np.array_equal(_np(o.zero).view(np.uint32), _np(r.zero).view(np.uint32)), i
        if fmt >= 3:
            assert np.array_equal(_np(o.e8m0), _np(r.e8m0)), i
        if i < 10:
            _check_aq(o, _np(X), fmt, S[l * B + b], Z[l * B + b], dynamic=False)


# ---------------------------------------------------------------------------------------
# mixed-format linear layer
# ---------------------------------------------------------------------------------------
def _linear_case(X, W, mask, afmt, dynamic=True):
    M, K = X.shape
    N = W.shape[0]
    case(f"mixed_linear M={M} N={N} K={K} mask={mask:#x} afmt={afmt}")
    wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), mask)
    xq = cham.quantize_act(torch.from_numpy(X).to(DEV), afmt, dynamic=True)
    Y = _np(cham.mixed_linear(xq, wq)).astype(np.float64)
    ref = oracle.select_weight_formats(W, mask, want_err=False, want_perm=False)
    Wh = oracle.dequant_weights(ref, K)
    codes, e8, xh, s, z = oracle.quantize_act_dynamic(X, afmt, want_xhat=True)
    assert np.array_equal(_np(wq.fmt), ref["fmt"])
    assert np.array_equal(_np(xq.codes), codes)
    Yr, Bm = oracle.linear(xh, Wh)
    err = np.abs(Y - Yr)
    bad = err > 1e-3 * Bm
    assert not bad.any(), (np.argwhere(bad)[:5], (err / np.maximum(Bm, 1e-300)).max())
    # the search's packed layout gives the same kernels the same operands: identical Y
    wp = cham.select_weight_formats(torch.from_numpy(W).to(DEV), mask, want_packed=True)
    assert np.array_equal(_np(cham.mixed_linear(xq, wp)).astype(np.float64), Y)
    return (err / np.maximum(Bm, 1e-300)).max()


@pytest.mark.parametrize("afmt", range(5))
def test_linear_single_layer(afmt):
    X, W = synth.single_layer(0)
    _linear_case(X, W, oracle.MASK_W4, afmt)


@pytest.mark.parametrize("wf", range(9))
def test_linear_each_weight_format(wf):
    """Every GEMM decode path, one weight format at a time (ragged M and N)."""
    X, _ = synth.single_layer(3, M=200, K=640, N=8)
    W, _ = synth.hetero_weights(4, 300, 640)
    for afmt in (cham.A_INT8_ASYM, cham.A_FP8_E4M3, cham.A_FP8_E5M2, cham.A_MXFP8):
        _linear_case(X, W, 1 << wf, afmt)


@pytest.mark.parametrize("mask", [oracle.MASK_W4, oracle.MASK_W8, 0x1FF])
def test_linear_hetero_mixed(mask):
    X = synth.diffusion_acts(0, 2, 400, 130, 1280)
    W, _ = synth.hetero_weights(8, 333, 1280)
    for afmt in range(5):
        _linear_case(X, W, mask, afmt)


def test_linear_exact_grid_inputs():
    """Activations and weights on exact grids with power-of-two scales: every product and
    partial sum is exact in binary32, so Y equals the binary64 reference exactly."""
    g = np.random.default_rng(0)
    M, N, K = 64, 96, 256
    X = (g.integers(-6, 7, (M, K)) * 0.25).astype(np.float32)   # E4M3-exact values
    e2 = np.array([0, 0.5, 1, 1.5, 2, 3, 4, 6], np.float32)
    W = (e2[g.integers(0, 8, (N, K))] * g.choice([-1, 1], (N, K))).astype(np.float32)
    W[:, 0] = 6.0
    sd = torch.tensor([2.0 ** -4], device=DEV)  # static power-of-two scale: x/s = 4k, exact in E4M3
    zd = torch.zeros(1, device=DEV)
    case("mixed_linear exact-grid inputs")
    xq = cham.quantize_act(torch.from_numpy(X).to(DEV), cham.A_FP8_E4M3, dynamic=False, s=sd, z=zd)
    wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), 1 << cham.W_MXFP4)
    Y = _np(cham.mixed_linear(xq, wq)).astype(np.float64)
    Yr = X.astype(np.float64) @ W.astype(np.float64).T
    assert np.array_equal(Y, Yr)


def test_linear_full_size_sampled():
    """SDXL-like out-proj and GEGLU at M = 2048 tokens (CFG batch 2 x 1024): sampled
    outputs against the oracle computed one by one."""
    for name, K, N in (("out", 1280, 1280), ("geglu", 1280, 10240), ("ff_out", 5120, 1280)):
        M = 2048
        X = synth.diffusion_acts(0, 1, 375, M, K)
        W, _ = synth.hetero_weights(21, N, K)
        case(f"mixed_linear full-size {name} M={M} N={N} K={K}")
        wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), oracle.MASK_W4)
        for afmt in (cham.A_FP8_E4M3, cham.A_INT8_ASYM):
            xq = cham.quantize_act(torch.from_numpy(X).to(DEV), afmt, dynamic=True)
            Y = _np(cham.mixed_linear(xq, wq)).astype(np.float64)
            g = np.random.default_rng(afmt)
            mm = g.integers(0, M, 2048)
            nn = g.integers(0, N, 2048)
            rows = np.unique(nn)
            ref = oracle.select_weight_formats(W[rows], oracle.MASK_W4, want_err=False, want_perm=False)
            Wh = np.zeros((N, K), np.float32)
            Wh[rows] = oracle.dequant_weights(ref, K)
            lo, hi = oracle.minmax(X)
            s, z = oracle.scale_zp(afmt, lo, hi)
            mrows = np.unique(mm)
            xh = np.zeros_like(X)
            xh[mrows] = oracle.quantize_act(X[mrows], afmt, s, z, want_xhat=True)[2]
            yr, bm = oracle.linear_pairs(xh, Wh, mm, nn)
            err = np.abs(Y[mm, nn] - yr)
            assert np.all(err <= 1e-3 * bm), (name, afmt, (err / bm).max())


@pytest.mark.parametrize("M,N,K,mask,afmt", [
    (1500, 3000, 2560, oracle.MASK_W4, cham.A_FP8_E5M2),   # 128-row tiles, 3 k-splits, ragged M
    (1500, 3000, 2560, oracle.MASK_W8, cham.A_INT8_ASYM),  # 8-bit codes, 256-row tiles, 3 k-splits
    (3000, 4000, 1280, oracle.MASK_W8, cham.A_MXFP8),      # 8-bit codes, 256-row tiles, MX activations
    (3000, 4000, 1280, oracle.MASK_W4, cham.A_MXINT8),     # 128-row tiles, MX activations
    (8192, 4608, 1152, oracle.MASK_W8, cham.A_FP8_E4M3),   # two launches: 256-row then 128-row tiles
    (1000, 1000, 1280, oracle.MASK_W4, cham.A_FP8_E4M3),   # 64 x 128 tiles, ragged M and N
    (1024, 1280, 1280, oracle.MASK_W4, cham.A_FP8_E5M2),   # 64 x 128 tiles: the single-step out-projection
    (1040, 1200, 1216, oracle.MASK_W4, cham.A_MXINT8),     # 64 x 128 tiles, MX activations, ragged M and N
    (700, 777, 1280, oracle.MASK_W8, cham.A_INT8_ASYM),    # half-width tiles, 8-bit codes, 5 k-splits
    (240, 1152, 4096, oracle.MASK_W4, cham.A_FP8_E4M3),    # PixArt-like cross-attn KV: 240 rows, 8 k-splits
    (4096, 5120, 640, oracle.MASK_W4, cham.A_INT8_ASYM),   # 640-wide GEGLU at 4096 tokens
    (1024, 1280, 5120, oracle.MASK_W4, cham.A_FP8_E5M2),   # 1280-wide FF-out at 1024 tokens
    (2048, 1280, 5120, oracle.MASK_W4, cham.A_INT8_ASYM),  # the sweep's FF-out: 3 k-splits, XCD-aware order
    (1300, 2000, 4096, oracle.MASK_W8, cham.A_INT8_ASYM),  # XCD-aware order over 11 x 16 tiles, ragged M and N
    (1300, 2000, 4096, oracle.MASK_W4, cham.A_MXFP8),      # the same with MX activations
])
def test_linear_plans_sampled(M, N, K, mask, afmt):
    """Tile heights, k-splits and two-launch plans the sizes above select (each code width,
    per-tensor and MX activations): sampled outputs against the oracle one by one."""
    X = synth.diffusion_acts(5, 2, 600, M, K)
    W, _ = synth.hetero_weights(31, N, K)
    case(f"mixed_linear plan M={M} N={N} K={K} mask={mask:#x} afmt={afmt}")
    wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), mask, want_packed=True)
    xq = cham.quantize_act(torch.from_numpy(X).to(DEV), afmt, dynamic=True)
    Y = _np(cham.mixed_linear(xq, wq)).astype(np.float64)
    wq.packed = None  # the same call deriving the layout from the codes in its pre-pass
    assert np.array_equal(_np(cham.mixed_linear(xq, wq)).astype(np.float64), Y)
    g = np.random.default_rng(M + N + K + afmt)
    mm = np.concatenate([g.integers(0, M, 1500), [M - 1, 0]])
    nn = np.concatenate([g.integers(0, N, 1500), [N - 1, 0]])
    rows = np.unique(nn)
    ref = oracle.select_weight_formats(W[rows], mask, want_err=False, want_perm=False)
    assert np.array_equal(_np(wq.fmt)[rows], ref["fmt"])
    Wh = np.zeros((N, K), np.float32)
    Wh[rows] = oracle.dequant_weights(ref, K)
    mrows = np.unique(mm)
    lo, hi = oracle.minmax(X)  # the whole tensor's range (MX formats: s = 1, z = 0)
    s, z = oracle.scale_zp(afmt, lo, hi)
    xh = np.zeros_like(X)
    xh[mrows] = oracle.quantize_act(X[mrows], afmt, s, z, want_xhat=True)[2]
    yr, bm = oracle.linear_pairs(xh, Wh, mm, nn)
    err = np.abs(Y[mm, nn] - yr)
    assert np.all(err <= 1e-3 * bm), (err / bm).max()


# ---------------------------------------------------------------------------------------
# the benchmark's two-stream step
def test_two_streams_match_one_stream():
    """The weight search on a second stream, concurrent with the activation statistics, LUT
    and quantization on the launch stream (which waits for it before the GEMMs; the next
    search waits for those GEMMs), gives the bits of the same calls on one stream."""
    layers = [("a", 640, 384), ("b", 1280, 256), ("c", 2560, 320)]
    M, T, B, t = 300, 1000, 4, 375
    Ws = [torch.from_numpy(synth.hetero_weights(50 + i, N, K)[0]).to(DEV) for i, (_, K, N) in enumerate(layers)]
    Xs = [torch.from_numpy(synth.diffusion_acts(3, i, t, M, K)).to(DEV) for i, (_, K, _) in enumerate(layers)]
    sched = cham.Schedule(T=T)
    b = cham.bucket(t, T, B)

    def alloc():
        wqs = [cham.alloc_wq(N, K, cham.MASK_W4, DEV, want_perm=True, want_packed=True) for (_, K, N) in layers]
        for w in wqs:
            w.packed.zero_()
        st = cham.alloc_stats(len(layers), B, DEV)
        aqs = [cham.alloc_aq(M, K, DEV) for (_, K, _) in layers]
        Ys = [torch.empty((M, N), dtype=torch.float32, device=DEV) for (_, _, N) in layers]
        return wqs, st, aqs, Ys

    def run(wqs, st, aqs, Ys, side, main):
        sb = cham.SearchBatch(Ws, wqs)
        cham.act_stats_reset(st, stream=main)
        end = None
        for _ in range(2):  # two steps: the second search waits for the first step's GEMMs
            if end is not None:
                side.wait_event(end)
            sb.run(stream=side)
            searched = torch.cuda.Event()
            searched.record(side)
            cham.act_stats_accumulate_batch(Xs, list(range(len(layers))), [b] * len(layers), st, stream=main)
            lut = cham.build_act_lut(st, sched, stream=main)
            lut.mirror()  # a copy on the launch stream (the current one in both runs)
            main.wait_event(searched)
            for i in range(len(layers)):
                cham.quantize_act_lut(Xs[i], lut, i, t, out=aqs[i], stream=main)
                cham.mixed_linear(aqs[i], wqs[i], Ys[i], stream=main)
            end = torch.cuda.Event()
            end.record(main)
        torch.cuda.synchronize()

    cur = torch.cuda.current_stream()
    case("one stream")
    ref = alloc()
    torch.cuda.synchronize()
    run(*ref, cur, cur)
    case("two streams")
    two = alloc()
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    run(*two, side, cur)
    for wa, wb in zip(ref[0], two[0]):
        assert np.array_equal(_np(wa.fmt), _np(wb.fmt))
        assert np.array_equal(_np(wa.codes), _np(wb.codes))
        assert np.array_equal(_np(wa.perm), _np(wb.perm))
        assert np.array_equal(_np(wa.packed), _np(wb.packed))
    assert np.array_equal(_np(ref[1].nS), _np(two[1].nS))
    for ya, yb in zip(ref[3], two[3]):
        assert np.array_equal(_np(ya).view(np.uint32), _np(yb).view(np.uint32))


def test_chunked_step_schedule_matches_one_stream():
    """The benchmark's step schedule: the search in chunks of layers on a second stream; on
    the launch stream the fused quantize-and-moments pass with the LUT built before it, the
    LUT rebuilt and its formats copied to the host mirror, then each chunk's GEMMs once that
    chunk is searched; the next step's search of a chunk waits for this step's GEMMs of that
    chunk.  New weights and inputs every step (a search that overtook the GEMMs still reading
    its packed layout would show), three steps, the bits of the same calls on one stream."""
    layers = [(640, 384), (1280, 256), (2560, 320), (640, 512), (1280, 384), (640, 256)]
    chunks = [(0, 2), (2, 4), (4, 6)]
    M, T, B, t, steps = 512, 1000, 4, 375, 3
    nl = len(layers)
    Ws = [[torch.from_numpy(synth.hetero_weights(70 + 10 * s + i, N, K)[0]).to(DEV) for i, (K, N) in enumerate(layers)]
          for s in range(steps)]
    Xs = [[torch.from_numpy(synth.diffusion_acts(4 + s, i, t, M, K)).to(DEV) for i, (K, _) in enumerate(layers)]
          for s in range(steps)]
    cal = [torch.from_numpy(synth.diffusion_acts(1, i, 100 + 250 * b, 64, K)).to(DEV)
           for b in range(B) for i, (K, _) in enumerate(layers)]
    sched = cham.Schedule(T=T)

    def run(side, main):
        wqs = [cham.alloc_wq(N, K, cham.MASK_W4, DEV, want_perm=True, want_packed=True) for (K, N) in layers]
        for w in wqs:
            w.packed.zero_()
        st = cham.alloc_stats(nl, B, DEV)
        cham.act_stats_reset(st, stream=main)
        cham.act_stats_accumulate_batch(cal, [i for _ in range(B) for i in range(nl)],
                                        [b for b in range(B) for _ in range(nl)], st, stream=main)
        lut = cham.build_act_lut(st, sched, stream=main)
        torch.cuda.synchronize()
        lut.F_host = torch.empty(lut.F.numel(), dtype=torch.uint8, pin_memory=True)
        lut.F_host.copy_(lut.F)
        aqs = [cham.alloc_aq(M, K, DEV) for (K, _) in layers]
        Ys = [[torch.empty((M, N), dtype=torch.float32, device=DEV) for (_, N) in layers] for _ in range(steps)]
        done = [None] * len(chunks)
        copied = None
        for s in range(steps):
            searched = []
            for c, (a, b) in enumerate(chunks):
                if done[c] is not None:
                    side.wait_event(done[c])
                cham.SearchBatch(Ws[s][a:b], wqs[a:b]).run(stream=side)
                searched.append(torch.cuda.Event())
                searched[-1].record(side)
            if copied is not None:
                copied.synchronize()
            with torch.cuda.stream(main):
                cham.QuantStatsBatch(Xs[s], list(range(nl)), aqs, lut, st).run(t, stream=main)
                cham.build_act_lut(st, sched, out=lut, stream=main)
                lut.F_host.copy_(lut.F, non_blocking=True)
                copied = torch.cuda.Event()
                copied.record(main)
            for c, (a, b) in enumerate(chunks):
                main.wait_event(searched[c])
                for i in range(a, b):
                    cham.mixed_linear(aqs[i], wqs[i], Ys[s][i], stream=main)
                done[c] = torch.cuda.Event()
                done[c].record(main)
        torch.cuda.synchronize()
        return wqs, st, Ys

    cur = torch.cuda.current_stream()
    case("chunked step schedule on one stream")
    ref = run(cur, cur)
    case("chunked step schedule on two streams")
    two = run(torch.cuda.Stream(), cur)
    for wa, wb in zip(ref[0], two[0]):
        assert np.array_equal(_np(wa.fmt), _np(wb.fmt))
        assert np.array_equal(_np(wa.packed), _np(wb.packed))
    assert np.array_equal(_np(ref[1].nS), _np(two[1].nS))
    for s in range(steps):
        for ya, yb in zip(ref[2][s], two[2][s]):
            assert np.array_equal(_np(ya).view(np.uint32), _np(yb).view(np.uint32)), s


@pytest.mark.parametrize("mask", [oracle.MASK_W4, oracle.MASK_W8])
@pytest.mark.parametrize("N,K", [(12, 17280), (6, 23040), (5, 32768), (3, 8256)])
def test_search_long_rows(mask, N, K):
    """Rows longer than one wavefront holds (3x3 conv weights, K = 9 C_in): split over the
    four wavefronts of a workgroup at 64-element block boundaries (unequal quarters)."""
    W, _ = synth.hetero_weights(N + K, N, K)
    wq, ref = _search_both(W, mask)
    _assert_search_equal(wq, ref)


# ---------------------------------------------------------------------------------------
# seeded random shapes and palettes
@pytest.mark.parametrize("seed", range(16))
def test_search_random_shapes(seed):
    """A random non-empty palette, K (a multiple of 32, of 64 with NF4) and channel count
    (below and above the several-channels-per-wavefront threshold): every output bit-exact."""
    g = np.random.default_rng(1000 + seed)
    mask = int(g.integers(1, 512))
    step = 64 if (mask >> oracle.W_NF4) & 1 else 32
    K = step * int(g.integers(1, 5120 // step + 1))
    N = int(g.integers(1, 200)) if seed % 2 else int(g.integers(1024, 1600))
    W, _ = synth.hetero_weights(2000 + seed, N, K)
    wq, ref = _search_both(W, mask)
    _assert_search_equal(wq, ref)


@pytest.mark.parametrize("seed", range(24))
def test_linear_random_shapes(seed):
    """Random M, N, K, palette, activation format, sample count and weight layout (packed
    by the search or derived per call): activation codes bit-exact, sampled outputs within
    1e-3 * sum|x^ w^| of the oracle."""
    g = np.random.default_rng(3000 + seed)
    masks = [oracle.MASK_W4, oracle.MASK_W8, 0x1FF] + [1 << f for f in range(9)]
    mask = int(masks[int(g.integers(0, len(masks)))])
    K = 64 * int(g.integers(1, 41))
    M, N = int(g.integers(1, 2500)), int(g.integers(1, 2500))
    afmt = int(g.integers(0, 5))
    ns = int(g.choice([d for d in (1, 2, 3, 4) if M % d == 0]))
    packed = bool(g.integers(0, 2))
    X = synth.diffusion_acts(seed, 3, int(g.integers(0, 1000)), M, K)
    W, _ = synth.hetero_weights(4000 + seed, N, K)
    case(f"mixed_linear random M={M} N={N} K={K} mask={mask:#x} afmt={afmt} nsamples={ns} packed={packed}")
    wq = cham.select_weight_formats(torch.from_numpy(W).to(DEV), mask, want_packed=packed)
    xq = cham.quantize_act(torch.from_numpy(X).to(DEV), afmt, dynamic=True, nsamples=ns)
    Y = _np(cham.mixed_linear(xq, wq)).astype(np.float64)
    if packed:  # the per-call pre-pass gives the kernels the same operands
        wq.packed = None
        assert np.array_equal(_np(cham.mixed_linear(xq, wq)).astype(np.float64), Y)
    codes, e8, xh, s, z = oracle.quantize_act_per_sample(X, afmt, ns, want_xhat=True)
    assert np.array_equal(_np(xq.codes), codes)
    assert np.array_equal(_np(xq.scale).view(np.uint32), s.view(np.uint32))
    mm = np.concatenate([g.integers(0, M, 1200), [M - 1, 0]])
    nn = np.concatenate([g.integers(0, N, 1200), [N - 1, 0]])
    rows = np.unique(nn)
    ref = oracle.select_weight_formats(W[rows], mask, want_err=False, want_perm=False)
    assert np.array_equal(_np(wq.fmt)[rows], ref["fmt"])
    Wh = np.zeros((N, K), np.float32)
    Wh[rows] = oracle.dequant_weights(ref, K)
    yr, bm = oracle.linear_pairs(xh, Wh, mm, nn)
    err = np.abs(Y[mm, nn] - yr)
    assert np.all(err <= 1e-3 * bm), (err / np.maximum(bm, 1e-300)).max()
