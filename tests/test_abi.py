"""CPU checks of the C ABI: the HIP library loads, exports every function the header
declares, and validates arguments on the host (no kernel is launched by these calls)."""
import ctypes
import os
import re

import pytest

from paper_2609_33496_amd import cham

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "chameleon.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cham_[a-z0-9_]+)\s*\(", text)))


def test_library_loads_and_exports_every_declared_symbol():
    L = cham.lib()
    names = _declared_functions()
    assert len(names) >= 12
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing


def test_host_only_helpers():
    L = cham.lib()
    assert L.cham_version() >= (0 << 16) | (1 << 8)
    for s in (0, -1, -2, -3, -4, -5, 7):
        assert L.cham_status_string(s)
    assert [cham.bucket(t, 1000, 10) for t in (0, 99, 100, 999, 5000)] == [0, 0, 1, 9, 9]
    assert cham.bucket(-1, 1000, 10) == -1
    s = cham._Sched()
    L.cham_schedule_default(ctypes.byref(s))
    assert (s.T, s.beta0, s.beta1, s.kind) == (1000, 0.00085, 0.012, 0)
    assert (s.kappa_lo, s.kappa_hi, s.snr_lo, s.snr_hi, s.snr_gate_on) == (3.0, 5.0, 0.2, 2.0, 1)
    assert cham.workspace_bytes(cham.OP_STATS, 1 << 20, 0, 0) > 0
    assert cham.workspace_bytes(cham.OP_QUANT_ACT, 2048, 0, 1280) > 0
    assert cham.workspace_bytes(cham.OP_SELECT, 10, 10, 64) == 0
    assert cham.workspace_bytes(cham.OP_LINEAR, 2048, 1280, 1280) >= 2048 * 1280 * 2 + 2048 * 4
    # per channel: parameters and column-sum partials; per (k-step, channel, half) a record slot
    assert 1280 * 16 + 1280 * 4 + 1280 * 20 * 2 * 64 <= cham.packed_bytes(1280, 1280) <= 1280 * 16 + 1280 * 20 * 4 + 1280 * 20 * 2 * 64 + 512
    assert cham.packed_bytes(0, 64) == 0


def _wq(**kw):
    d = dict(N=4, K=64, palette_mask=cham.MASK_W4, code_bits=0, fmt=16, codes=16, scale=16, zero=16,
             nf4_absmax=16, e8m0=16, perm=None, group_off=None, err=None, packed=None)
    d.update(kw)
    return cham._WQ(d["N"], d["K"], d["palette_mask"], d["code_bits"], *[d[k] for k in (
        "fmt", "codes", "scale", "zero", "nf4_absmax", "e8m0", "perm", "group_off", "err", "packed")])


@pytest.mark.parametrize("kw,status", [
    (dict(palette_mask=0), cham.EFORMAT),
    (dict(palette_mask=1 << 9), cham.EFORMAT),
    (dict(N=0), cham.EINVAL),
    (dict(K=48), cham.ESHAPE),            # not a multiple of 32
    (dict(K=96), cham.ESHAPE),            # NF4 enabled: multiple of 64 needed
    (dict(nf4_absmax=None), cham.EINVAL),
    (dict(e8m0=None), cham.EINVAL),
    (dict(fmt=None), cham.EINVAL),
    (dict(K=96, palette_mask=1 << cham.W_FP4, packed=256), cham.ESHAPE),  # packed layout: K % 64
    (dict(packed=16), cham.EINVAL),                                      # packed layout: 256-byte aligned
])
def test_select_weight_formats_argument_errors(kw, status):
    w = _wq(**kw)
    rc = cham.lib().cham_select_weight_formats(ctypes.c_void_p(16), ctypes.byref(w), None)
    assert rc == status


def test_select_weight_formats_batch_argument_errors():
    L = cham.lib()
    good, bad = _wq(), _wq(K=48)
    arr = (cham._WQ * 2)(good, bad)
    ptrs = (ctypes.c_void_p * 2)(16, 16)
    assert L.cham_select_weight_formats_batch(ptrs, arr, 2, None) == cham.ESHAPE  # checked before any launch
    assert L.cham_select_weight_formats_batch(ptrs, arr, 0, None) == cham.EINVAL
    assert L.cham_select_weight_formats_batch(None, arr, 1, None) == cham.EINVAL
    nullw = (ctypes.c_void_p * 1)(None)
    assert L.cham_select_weight_formats_batch(nullw, (cham._WQ * 1)(good), 1, None) == cham.EINVAL


@pytest.mark.parametrize("kw,status", [
    (dict(packed=None), cham.EINVAL),
    (dict(packed=272), cham.EINVAL),          # 256-byte aligned
    (dict(code_bits=0), cham.EINVAL),         # the searched code width
    (dict(code_bits=8), cham.EINVAL),
    (dict(K=96), cham.ESHAPE),
    (dict(K=(1 << 20) + 64), cham.ESHAPE),
    (dict(palette_mask=0), cham.EFORMAT),
    (dict(nf4_absmax=None), cham.EINVAL),
    (dict(palette_mask=1 << cham.W_MXFP4, e8m0=None), cham.EINVAL),
    (dict(scale=None), cham.EINVAL),
])
def test_pack_weights_batch_argument_errors(kw, status):
    """Every descriptor is checked before the packing launch: a bad one anywhere in the array
    fails the call with nothing launched."""
    L = cham.lib()
    good = _wq(code_bits=4, packed=256)
    bad = _wq(**{"code_bits": 4, "packed": 256, **kw})
    assert L.cham_pack_weights_batch((cham._WQ * 2)(good, bad), 2, None) == status
    assert L.cham_pack_weights_batch((cham._WQ * 1)(bad), 1, None) == status
    assert L.cham_pack_weights_batch((cham._WQ * 1)(good), 0, None) == cham.EINVAL
    assert L.cham_pack_weights_batch(None, 1, None) == cham.EINVAL


def test_other_argument_errors():
    L = cham.lib()
    st = cham._Stats(2, 3, ctypes.c_void_p(16), ctypes.c_void_p(16))
    P = ctypes.c_void_p
    assert L.cham_act_stats_accumulate(P(16), 100, 2, 0, ctypes.byref(st), P(256), 1 << 20, None) == cham.EINVAL
    assert L.cham_act_stats_accumulate(P(16), 100, 0, 3, ctypes.byref(st), P(256), 1 << 20, None) == cham.EINVAL
    assert L.cham_act_stats_accumulate(P(16), 1 << 20, 0, 0, ctypes.byref(st), None, 0, None) == cham.EWORKSPACE
    xs = (ctypes.c_void_p * 2)(16, 16)
    ne = (ctypes.c_int64 * 2)(100, 1 << 20)
    ly = (ctypes.c_int32 * 2)(0, 1)
    bk = (ctypes.c_int32 * 2)(0, 2)
    bk_bad = (ctypes.c_int32 * 2)(0, 3)  # B = 3: bucket 3 is out of range
    assert L.cham_act_stats_accumulate_batch(xs, ne, ly, bk_bad, 2, ctypes.byref(st), P(256), 1 << 30, None) == cham.EINVAL
    assert L.cham_act_stats_accumulate_batch(xs, ne, ly, bk, 0, ctypes.byref(st), P(256), 1 << 30, None) == cham.EINVAL
    assert L.cham_act_stats_accumulate_batch(xs, ne, ly, bk, 2, ctypes.byref(st), P(256), 64, None) == cham.EWORKSPACE
    aq = cham._AQ(4, 64, 0, 1, P(16), P(16), P(16), P(16))
    assert L.cham_quantize_act(P(16), 7, 1, None, None, ctypes.byref(aq), P(256), 1 << 20, None) == cham.EFORMAT
    aq48 = cham._AQ(4, 48, 0, 1, P(16), P(16), P(16), P(16))
    assert L.cham_quantize_act(P(16), 1, 1, None, None, ctypes.byref(aq48), P(256), 1 << 20, None) == cham.ESHAPE
    assert L.cham_quantize_act(P(16), 1, 0, None, None, ctypes.byref(aq), None, 0, None) == cham.EINVAL
    assert L.cham_quantize_act(P(16), 1, 1, None, None, ctypes.byref(aq), None, 0, None) == cham.EWORKSPACE
    for ns in (0, 3, 1025):  # samples: at least one, dividing M, at most 1024
        aqs = cham._AQ(4 if ns != 1025 else 2050, 64, 0, ns, P(16), P(16), P(16), P(16))
        assert L.cham_quantize_act(P(16), 1, 1, None, None, ctypes.byref(aqs), P(256), 1 << 20, None) == cham.EINVAL
    w = _wq(code_bits=4)
    aqk = cham._AQ(4, 128, 1, 1, P(16), P(16), P(16), P(16))  # K = 128 vs wq K = 64
    assert L.cham_mixed_linear(ctypes.byref(aqk), ctypes.byref(w), P(16), None, 0, None) == cham.EINVAL  # K mismatch
    aqf = cham._AQ(4, 64, 9, 1, P(16), P(16), P(16), P(16))
    assert L.cham_mixed_linear(ctypes.byref(aqf), ctypes.byref(w), P(16), None, 0, None) == cham.EFORMAT
    w8 = _wq(code_bits=4, palette_mask=cham.MASK_W8)
    assert L.cham_mixed_linear(ctypes.byref(aq), ctypes.byref(w8), P(16), None, 0, None) == cham.EFORMAT
    sch = cham.Schedule().struct()
    lut = cham._LUT(2, 4, 0, P(16), P(16), P(16))
    assert L.cham_build_act_lut(ctypes.byref(st), ctypes.byref(sch), None, ctypes.byref(lut), None, None) == cham.EINVAL


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(cham, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(cham, "_lib", None)
    with pytest.raises(RuntimeError):
        cham.lib()


def test_linear_plans_are_valid():
    """The GEMM planner on the host (no GPU: 256 CUs assumed): for a grid of shapes the
    launches tile the rows in order with shapes the kernels exist for, every k-split holds
    at least one k-step, only single launches split k, and the workspace the library asks
    for holds the split partial outputs."""
    for M in (1, 7, 64, 240, 1000, 2048, 4096, 8192):
        for N in (32, 640, 777, 1280, 3840, 10240):
            for K in (64, 640, 1280, 5120):
                for bits in (4, 8):
                    p = cham.linear_plan(M, N, K, bits)
                    ls = p["launches"]
                    assert 1 <= len(ls) <= 2, (M, N, K, bits, p)
                    assert ls[0]["rows"][0] == 0 and ls[-1]["rows"][1] == M, p
                    if len(ls) == 2:
                        assert ls[0]["rows"][1] == ls[1]["rows"][0] and p["splits"] == 1, p
                    for l in ls:
                        assert l["rows"][0] < l["rows"][1], p
                        assert l["tile"] in ((256, 256), (128, 256), (128, 128), (64, 256), (64, 128)), p
                    steps, sp = K // 64, p["splits"]
                    assert 1 <= sp <= 8, p
                    chunk = -(-steps // sp)
                    assert sp == 1 or (sp - 1) * chunk < steps, p
                    if sp > 1:
                        assert cham.workspace_bytes(cham.OP_LINEAR, M, N, K) >= sp * M * N * 4, p
    with pytest.raises(cham.ChamError):
        cham.linear_plan(0, 64, 64, 4)
    with pytest.raises(cham.ChamError):
        cham.linear_plan(64, 64, 64, 6)


def test_linear_workspace_query_on_the_host():
    """The exact-workspace query checks the operands like mixed_linear, launches nothing and
    reads no device memory: the decode layout without a packed one, nothing with it (FP8
    activations, no split at these sizes), the half-precision copy and row scales for MX."""
    L = cham.lib()
    P = ctypes.c_void_p
    nb = ctypes.c_size_t(12345)
    aq = cham._AQ(4, 64, cham.A_FP8_E4M3, 1, P(16), P(16), P(16), P(16))
    w = _wq(code_bits=4)
    assert L.cham_mixed_linear_workspace_query(ctypes.byref(aq), ctypes.byref(w), None) == cham.EINVAL
    assert L.cham_mixed_linear_workspace_query(ctypes.byref(aq), ctypes.byref(w), ctypes.byref(nb)) == cham.OK
    rec = (int(L.cham_packed_bytes(4, 64)) + 255) // 256 * 256
    assert nb.value == rec
    wp = _wq(code_bits=4, packed=256)
    assert L.cham_mixed_linear_workspace_query(ctypes.byref(aq), ctypes.byref(wp), ctypes.byref(nb)) == cham.OK
    assert nb.value == 0
    aqm = cham._AQ(4, 64, cham.A_MXFP8, 1, P(16), P(16), P(16), P(16))
    assert L.cham_mixed_linear_workspace_query(ctypes.byref(aqm), ctypes.byref(wp), ctypes.byref(nb)) == cham.OK
    assert nb.value == 512 + 256  # 4 x 64 halves (512 B) and 4 row scales, each rounded up to 256 bytes
    assert nb.value <= cham.workspace_bytes(cham.OP_LINEAR, 4, 4, 64)
    aqk = cham._AQ(4, 128, cham.A_FP8_E4M3, 1, P(16), P(16), P(16), P(16))  # K mismatch
    assert L.cham_mixed_linear_workspace_query(ctypes.byref(aqk), ctypes.byref(w), ctypes.byref(nb)) == cham.EINVAL


def test_linear_size_limits_on_the_host():
    """The kernels address operands with 32-bit offsets: N of 2^21 channels (a 256-row output
    tile past 2^31 bytes) and K beyond 2^20 are rejected before any launch; N just below
    the limit passes the checks."""
    L = cham.lib()
    P = ctypes.c_void_p
    nb = ctypes.c_size_t(0)
    aq = cham._AQ(4, 64, cham.A_FP8_E4M3, 1, P(16), P(16), P(16), P(16))
    big = _wq(N=1 << 21, code_bits=4, packed=256)
    assert L.cham_mixed_linear_workspace_query(ctypes.byref(aq), ctypes.byref(big), ctypes.byref(nb)) == cham.ESHAPE
    ok = _wq(N=(1 << 21) - 1, code_bits=4, packed=256)
    assert L.cham_mixed_linear_workspace_query(ctypes.byref(aq), ctypes.byref(ok), ctypes.byref(nb)) == cham.OK
    aqk = cham._AQ(4, (1 << 20) + 64, cham.A_FP8_E4M3, 1, P(16), P(16), P(16), P(16))
    wk = _wq(K=(1 << 20) + 64, code_bits=4, packed=256)
    assert L.cham_mixed_linear_workspace_query(ctypes.byref(aqk), ctypes.byref(wk), ctypes.byref(nb)) == cham.ESHAPE
