"""CPU oracle for the Chameleon quantized-linear path -- TEST INFRASTRUCTURE ONLY.

A thin numpy/ctypes wrapper around ``cham_oracle.c``, a plain scalar C implementation of
what the method computes (arXiv 2609.33496: Sec. 4.2-4.5, App. A.7, App. A.11-A.12).
Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this package.  It shares no code with the HIP library and never calls it.

Parity unpinned: none of the functions; every function is pinned by
``tests/test_oracle_*.py`` (code tables from bits, brute force, closed forms, paper
invariants, printed SNR values).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cham_oracle.c")
_BUILD_DIR = os.path.join(_HERE, "_build")
_LIB_PATH = os.path.join(_BUILD_DIR, "libcham_oracle.so")

# weight format ids (palette order of Sec. 4.2) and their names
W_INT8_SYM, W_INT8_ASYM, W_MXINT8, W_INT4_SYM, W_INT4_ASYM, W_NF4, W_FP4, W_MXINT4, W_MXFP4 = range(9)
W_NAMES = ["INT8-sym", "INT8-asym", "MXINT8", "INT4-sym", "INT4-asym", "NF4", "FP4", "MXINT4", "MXFP4"]
W_BITS = [8, 8, 8, 4, 4, 4, 4, 4, 4]
# activation codes of the runtime LUT (Sec. 4.2)
A_INT8_ASYM, A_FP8_E4M3, A_FP8_E5M2, A_MXFP8, A_MXINT8 = range(5)
A_NAMES = ["INT8-asym", "FP8-E4M3", "FP8-E5M2", "MXFP8-E4M3", "MXINT8"]

# palettes used by the workloads: the few-step W4 subset and F_w^(8) (Sec. 4.2, Sec. 4.6)
MASK_W4 = (1 << W_INT4_ASYM) | (1 << W_NF4) | (1 << W_FP4) | (1 << W_MXINT4) | (1 << W_MXFP4)
MASK_W4_FULL = MASK_W4 | (1 << W_INT4_SYM)
MASK_W8 = (1 << W_INT8_SYM) | (1 << W_INT8_ASYM) | (1 << W_MXINT8)

_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with plain IEEE semantics (no FMA contraction, no fast-math)."""
    os.makedirs(_BUILD_DIR, exist_ok=True)
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
               "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i64, i32, u32, f32, f64 = ctypes.c_int64, ctypes.c_int, ctypes.c_uint32, ctypes.c_float, ctypes.c_double
    lib.orc_rounding_ok.restype = i32
    lib.orc_mf_decode.argtypes = [i32, ctypes.c_uint]
    lib.orc_mf_decode.restype = f64
    lib.orc_mf_encode.argtypes = [i32, f32]
    lib.orc_mf_encode.restype = ctypes.c_uint
    lib.orc_nf4_table.argtypes = [P]
    lib.orc_select_weight_formats.argtypes = [P, i64, i64, u32, P, P, P, P, P, P, P, P, P]
    lib.orc_select_weight_formats.restype = i32
    lib.orc_dequant_weights.argtypes = [i64, i64, i32, P, P, P, P, P, P, P]
    lib.orc_dequant_weights.restype = i32
    lib.orc_wq_row.argtypes = [i32, P, i64, P, P, P, P, P, P]
    lib.orc_minmax.argtypes = [P, i64, P, P]
    lib.orc_scale_zp.argtypes = [i32, f32, f32, P, P]
    lib.orc_quantize_act.argtypes = [P, i64, i64, i32, f32, f32, P, P, P]
    lib.orc_quantize_act.restype = i32
    lib.orc_dequant_act.argtypes = [i64, i64, i32, P, P, f32, f32, P]
    lib.orc_dequant_act.restype = i32
    lib.orc_stats_accumulate.argtypes = [P, i64, P, P]
    lib.orc_kurtosis.argtypes = [P]
    lib.orc_kurtosis.restype = f64
    lib.orc_snr_table.argtypes = [i32, f64, f64, i32, P]
    lib.orc_bucket.argtypes = [i32, i32, i32]
    lib.orc_bucket.restype = i32
    lib.orc_bucket_mid.argtypes = [i32, i32, i32]
    lib.orc_bucket_mid.restype = i32
    lib.orc_route.argtypes = [f64, f64, i32, f64, f64, f64, f64, i32]
    lib.orc_route.restype = i32
    lib.orc_build_lut.argtypes = [i32, i32, P, P, i32, f64, f64, i32, f64, f64, f64, f64, i32, P, P, P,
                                  P, P]
    lib.orc_select_group_formats.argtypes = [P, i64, i64, u32, u32, P, P, P, P, P, P, P, P]
    lib.orc_select_group_formats.restype = i32
    lib.orc_dequant_grouped.argtypes = [i64, i64, i32, i32, i32, P, P, P, P, P]
    lib.orc_dequant_grouped.restype = i32
    lib.orc_gq_row.argtypes = [i32, i32, P, i64, P, P, P, P, P]
    lib.orc_linear.argtypes = [i64, i64, i64, P, P, P, P]
    lib.orc_linear_pairs.argtypes = [i64, i64, P, P, P, P, P, P]
    lib.orc_conv3x3.argtypes = [i64, i64, i64, i64, i64, P, P, P, P]
    if not lib.orc_rounding_ok():
        raise RuntimeError("oracle requires round-to-nearest-even")
    _lib = lib
    return lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


# ---------------------------------------------------------------------------------------------
# number formats (App. A.11)
# ---------------------------------------------------------------------------------------------
MF_E2M1, MF_E4M3, MF_E5M2 = 0, 1, 2


def mf_decode(which: int, code: int) -> float:
    """Value of a minifloat code (E2M1 / E4M3 / E5M2) from its bit fields."""
    return _load().orc_mf_decode(which, code)


def mf_encode(which: int, y: float) -> int:
    """Nearest code to y (|y| within range), ties to the even code, sign bit kept."""
    return _load().orc_mf_encode(which, float(np.float32(y)))


def nf4_table() -> np.ndarray:
    out = np.zeros(16, np.float32)
    _load().orc_nf4_table(_p(out))
    return out


def code_bits(mask: int) -> int:
    return 8 if any((mask >> f) & 1 and W_BITS[f] == 8 for f in range(9)) else 4


# ---------------------------------------------------------------------------------------------
# weight search (Sec. 4.5)
# ---------------------------------------------------------------------------------------------
def wq_row(fmt: int, w: np.ndarray):
    """Round trip one row through one weight format: (codes, w_hat, scale, zero, nf4_absmax, e8m0)."""
    w = _f32(w)
    K = w.shape[0]
    codes = np.zeros(K, np.uint8)
    wh = np.zeros(K, np.float32)
    s = np.zeros(1, np.float32)
    z = np.zeros(1, np.float32)
    nf = np.zeros(max(K // 64, 1), np.float32)
    e8 = np.zeros(max(K // 32, 1), np.uint8)
    _load().orc_wq_row(fmt, _p(w), K, _p(codes), _p(wh), _p(s), _p(z), _p(nf), _p(e8))
    return codes, wh, float(s[0]), float(z[0]), nf[:K // 64], e8[:K // 32]


def select_weight_formats(W: np.ndarray, mask: int, want_err: bool = True, want_perm: bool = True):
    """Per-output-channel format search.  Returns a dict of numpy arrays:
    fmt [N] u8, codes [N, K*bits/8] u8, scale [N] f32, zero [N] f32 (integral), nf4_absmax [N, K/64] f32,
    e8m0 [N, K/32] u8, perm [N] i32, group_off [10] i32, err [N, 9] f64."""
    W = _f32(W)
    N, K = W.shape
    cb = code_bits(mask)
    out = dict(
        fmt=np.zeros(N, np.uint8),
        codes=np.zeros((N, K * cb // 8), np.uint8),
        scale=np.zeros(N, np.float32),
        zero=np.zeros(N, np.float32),
        nf4_absmax=np.zeros((N, K // 64), np.float32),
        e8m0=np.zeros((N, K // 32), np.uint8),
        perm=np.zeros(N, np.int32) if want_perm else None,
        group_off=np.zeros(10, np.int32) if want_perm else None,
        err=np.zeros((N, 9), np.float64) if want_err else None,
    )
    rc = _load().orc_select_weight_formats(
        _p(W), N, K, mask, _p(out["fmt"]), _p(out["codes"]), _p(out["scale"]), _p(out["zero"]),
        _p(out["nf4_absmax"]), _p(out["e8m0"]), _p(out["perm"]), _p(out["group_off"]), _p(out["err"]))
    if rc != 0:
        raise ValueError("oracle: bad palette mask or shape")
    out["code_bits"] = cb
    return out


def dequant_weights(wq: dict, K: int) -> np.ndarray:
    N = wq["fmt"].shape[0]
    Wh = np.zeros((N, K), np.float32)
    rc = _load().orc_dequant_weights(N, K, wq["code_bits"], _p(wq["fmt"]), _p(np.ascontiguousarray(wq["codes"])),
                                     _p(wq["scale"]), _p(wq["zero"]), _p(np.ascontiguousarray(wq["nf4_absmax"])),
                                     _p(np.ascontiguousarray(wq["e8m0"])), _p(Wh))
    if rc != 0:
        raise ValueError("oracle: K too large")
    return Wh


# ---------------------------------------------------------------------------------------------
# DiT joint (group size, format) search (Sec. 4.6 (i))
# ---------------------------------------------------------------------------------------------
GROUP_SIZES = (32, 64, 128, 192, 288)
GMASK_ALL = 0x1F
MASK_DIT_W4 = (1 << W_INT4_ASYM) | (1 << W_NF4) | (1 << W_FP4)      # the DiT fork's 4-bit set
MASK_DIT_W8 = MASK_W8                                                 # {INT8-sym, INT8-asym, MXINT8}


def gq_row(fmt: int, g: int, w: np.ndarray):
    """Round trip one row in groups of g: (codes, w_hat, group scales, group zeros, e8m0)."""
    w = _f32(w)
    K = w.shape[0]
    codes = np.zeros(K, np.uint8)
    wh = np.zeros(K, np.float32)
    gs = np.zeros(K // 32, np.float32)
    gz = np.zeros(K // 32, np.float32)
    e8 = np.zeros(K // 32, np.uint8)
    _load().orc_gq_row(fmt, g, _p(w), K, _p(codes), _p(wh), _p(gs), _p(gz), _p(e8))
    return codes, wh, gs, gz, e8


def select_group_formats(W: np.ndarray, mask: int, energy: np.ndarray, gmask: int = GMASK_ALL):
    """Per-layer (g, f) search with input-aware error weights energy[K].  Returns a dict:
    g, fmt_id, err [45] (tuple t = group index * 9 + format; -1 not evaluated), fmt [N],
    codes, gscale / gzero [N, K/32], e8m0 [N, K/32], code_bits."""
    W = _f32(W)
    N, K = W.shape
    e = _f32(energy)
    cb = code_bits(mask)
    out = dict(choice=np.zeros(2, np.int32), err=np.zeros(45, np.float64), fmt=np.zeros(N, np.uint8),
               codes=np.zeros((N, K * cb // 8), np.uint8), gscale=np.zeros((N, K // 32), np.float32),
               gzero=np.zeros((N, K // 32), np.float32), e8m0=np.zeros((N, K // 32), np.uint8))
    rc = _load().orc_select_group_formats(_p(W), N, K, mask, gmask, _p(e), _p(out["choice"]), _p(out["err"]),
                                          _p(out["fmt"]), _p(out["codes"]), _p(out["gscale"]), _p(out["gzero"]),
                                          _p(out["e8m0"]))
    if rc != 0:
        raise ValueError("oracle: bad arguments to the group search")
    out["g"], out["fmt_id"], out["code_bits"] = int(out["choice"][0]), int(out["choice"][1]), cb
    return out


def dequant_grouped(gq: dict, K: int) -> np.ndarray:
    N = gq["fmt"].shape[0]
    Wh = np.zeros((N, K), np.float32)
    rc = _load().orc_dequant_grouped(N, K, gq["code_bits"], gq["g"], gq["fmt_id"], _p(np.ascontiguousarray(gq["codes"])),
                                     _p(gq["gscale"]), _p(gq["gzero"]), _p(gq["e8m0"]), _p(Wh))
    if rc != 0:
        raise ValueError("oracle: bad grouped weight")
    return Wh


# ---------------------------------------------------------------------------------------------
# activations (App. A.7: ScaleZP, Alg. 2, Alg. 3)
# ---------------------------------------------------------------------------------------------
def minmax(X: np.ndarray):
    X = _f32(X)
    lo = np.zeros(1, np.float32)
    hi = np.zeros(1, np.float32)
    _load().orc_minmax(_p(X), X.size, _p(lo), _p(hi))
    return float(lo[0]), float(hi[0])


def scale_zp(fmt: int, lo: float, hi: float):
    s = np.zeros(1, np.float32)
    z = np.zeros(1, np.float32)
    _load().orc_scale_zp(fmt, np.float32(lo), np.float32(hi), _p(s), _p(z))
    return np.float32(s[0]), np.float32(z[0])


def quantize_act(X: np.ndarray, fmt: int, s=1.0, z=0.0, want_xhat: bool = False):
    """Quantize X [M, K]; returns (codes [M,K] u8, e8m0 [M,K/32] u8, xhat or None)."""
    X = _f32(X)
    M, K = X.shape
    codes = np.zeros((M, K), np.uint8)
    e8 = np.zeros((M, max(K // 32, 1)), np.uint8)
    xh = np.zeros((M, K), np.float32) if want_xhat else None
    rc = _load().orc_quantize_act(_p(X), M, K, fmt, np.float32(s), np.float32(z), _p(codes), _p(e8), _p(xh))
    if rc != 0:
        raise ValueError("oracle: K must be a multiple of 32 for MX formats")
    return codes, e8[:, :K // 32], xh


def quantize_act_dynamic(X: np.ndarray, fmt: int, want_xhat: bool = False):
    """Alg. 3: (s, z) from this tensor's own min/max, then quantize."""
    lo, hi = minmax(X)
    s, z = scale_zp(fmt, lo, hi)
    codes, e8, xh = quantize_act(X, fmt, s, z, want_xhat)
    return codes, e8, xh, s, z


def quantize_act_per_sample(X: np.ndarray, fmt: int, nsamples: int, want_xhat: bool = False):
    """Alg. 3 with per-sample micro-scaling (Sec. 4.6 (ii)): X [M, K] holds nsamples samples of
    M / nsamples consecutive rows; each sample's (s, z) is ScaleZP of its own min / max, and its
    rows are quantized with them.  Returns (codes, e8m0, xhat or None, s [S], z [S])."""
    X = _f32(X)
    M, K = X.shape
    if nsamples < 1 or M % nsamples:
        raise ValueError("oracle: nsamples must divide M")
    rows = M // nsamples
    codes = np.zeros((M, K), np.uint8)
    e8 = np.zeros((M, K // 32), np.uint8)
    xh = np.zeros((M, K), np.float32) if want_xhat else None
    s_all = np.zeros(nsamples, np.float32)
    z_all = np.zeros(nsamples, np.float32)
    for b in range(nsamples):
        sl = slice(b * rows, (b + 1) * rows)
        c, e, h, s, z = quantize_act_dynamic(X[sl], fmt, want_xhat)
        codes[sl], e8[sl] = c, e
        if want_xhat:
            xh[sl] = h
        s_all[b], z_all[b] = s, z
    return codes, e8, xh, s_all, z_all


def dequant_act(codes: np.ndarray, e8: np.ndarray, fmt: int, s=1.0, z=0.0) -> np.ndarray:
    codes = np.ascontiguousarray(codes, np.uint8)
    M, K = codes.shape
    e8 = np.ascontiguousarray(e8 if e8 is not None and e8.size else np.zeros((M, 1), np.uint8), np.uint8)
    xh = np.zeros((M, K), np.float32)
    _load().orc_dequant_act(M, K, fmt, _p(codes), _p(e8), np.float32(s), np.float32(z), _p(xh))
    return xh


# ---------------------------------------------------------------------------------------------
# statistics and LUT (Sec. 4.3, Sec. 4.4, Alg. 1)
# ---------------------------------------------------------------------------------------------
class Stats:
    """Per-(layer, bucket) accumulator: n, S1..S4 (binary64) and lo/hi (binary32)."""

    def __init__(self, L: int, B: int):
        self.L, self.B = L, B
        self.nS = np.zeros((L * B, 5), np.float64)
        self.lohi = np.zeros((L * B, 2), np.float32)
        self.lohi[:, 0] = np.inf
        self.lohi[:, 1] = -np.inf

    def accumulate(self, X: np.ndarray, layer: int, bucket: int):
        X = _f32(X)
        i = layer * self.B + bucket
        nS = np.ascontiguousarray(self.nS[i])
        lohi = np.ascontiguousarray(self.lohi[i])
        _load().orc_stats_accumulate(_p(X), X.size, _p(nS), _p(lohi))
        self.nS[i] = nS
        self.lohi[i] = lohi


def kurtosis(nS) -> float:
    nS = np.ascontiguousarray(nS, np.float64)
    return _load().orc_kurtosis(_p(nS))


SCALED_LINEAR, LINEAR = 0, 1
# noise schedules: SDXL's scaled-linear 0.00085 -> 0.012 over T = 1000 (BETAS_SDXL) and the
# linear 1e-4 -> 0.02 read for PixArt-alpha (BETAS_PIXART)
BETAS_SDXL = (1000, 0.00085, 0.012, SCALED_LINEAR)
BETAS_PIXART = (1000, 1e-4, 0.02, LINEAR)


def snr_table(T: int, b0: float, b1: float, kind: int) -> np.ndarray:
    out = np.zeros(T, np.float64)
    _load().orc_snr_table(T, b0, b1, kind, _p(out))
    return out


def bucket(t: int, T: int, B: int) -> int:
    return _load().orc_bucket(t, T, B)


def bucket_mid(b: int, T: int, B: int) -> int:
    return _load().orc_bucket_mid(b, T, B)


def route(kappa, snr, is_shortcut=0, gates=(3.0, 5.0, 0.2, 2.0), snr_gate_on=1) -> int:
    return _load().orc_route(kappa, snr, int(is_shortcut), *gates, int(snr_gate_on))


def build_lut(stats: Stats, sched=BETAS_SDXL, gates=(3.0, 5.0, 0.2, 2.0), snr_gate_on=1, is_shortcut=None):
    L, B = stats.L, stats.B
    T, b0, b1, kind = sched
    F = np.zeros(L * B, np.uint8)
    S = np.zeros(L * B, np.float32)
    Z = np.zeros(L * B, np.float32)
    kap = np.zeros(L * B, np.float64)
    sc = None if is_shortcut is None else np.ascontiguousarray(is_shortcut, np.uint8)
    _load().orc_build_lut(L, B, _p(np.ascontiguousarray(stats.nS)), _p(np.ascontiguousarray(stats.lohi)), T, b0, b1,
                          kind, *gates, int(snr_gate_on), _p(sc), _p(F), _p(S), _p(Z), _p(kap))
    return F, S, Z, kap


# ---------------------------------------------------------------------------------------------
# the linear layer on dequantized operands (binary64)
# ---------------------------------------------------------------------------------------------
def linear(Xh: np.ndarray, Wh: np.ndarray):
    Xh, Wh = _f32(Xh), _f32(Wh)
    M, K = Xh.shape
    N = Wh.shape[0]
    Y = np.zeros((M, N), np.float64)
    Bm = np.zeros((M, N), np.float64)
    _load().orc_linear(M, N, K, _p(Xh), _p(Wh), _p(Y), _p(Bm))
    return Y, Bm


def linear_pairs(Xh: np.ndarray, Wh: np.ndarray, mm: np.ndarray, nn: np.ndarray):
    Xh, Wh = _f32(Xh), _f32(Wh)
    K = Xh.shape[1]
    mm = np.ascontiguousarray(mm, np.int64)
    nn = np.ascontiguousarray(nn, np.int64)
    Y = np.zeros(mm.shape[0], np.float64)
    Bm = np.zeros(mm.shape[0], np.float64)
    _load().orc_linear_pairs(K, mm.shape[0], _p(mm), _p(nn), _p(Xh), _p(Wh), _p(Y), _p(Bm))
    return Y, Bm


def conv3x3(Xh: np.ndarray, Wh: np.ndarray):
    """3x3 convolution, stride 1, zero padding 1, on dequantized operands (binary64):
    Xh [B, H, W, C] channels last, Wh [Co, 9C] with k = (ky * 3 + kx) * C + c.
    Returns (Y [B, H, W, Co], sum of |products| [B, H, W, Co])."""
    Xh, Wh = _f32(Xh), _f32(Wh)
    B, H, W, C = Xh.shape
    Co = Wh.shape[0]
    assert Wh.shape[1] == 9 * C
    Y = np.zeros((B, H, W, Co), np.float64)
    Bm = np.zeros((B, H, W, Co), np.float64)
    _load().orc_conv3x3(B, H, W, C, Co, _p(Xh), _p(Wh), _p(Y), _p(Bm))
    return Y, Bm

