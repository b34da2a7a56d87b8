"""Thin Python binding of the HIP library's C ABI (``include/chameleon.h``).

Argument marshalling only: torch tensors supply device memory and the current HIP stream;
every step of the computation runs in the library's kernels.  There is no fallback: if the
shared library is missing or a call fails, an exception is raised.

Functions keep the C names without the ``cham_`` prefix:
``select_weight_formats``, ``act_stats_reset``, ``act_stats_accumulate``,
``build_act_lut``, ``quantize_act``, ``quantize_act_lut``, ``mixed_linear``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libchameleon.so")

# status codes
OK, EINVAL, ESHAPE, EFORMAT, EHIP, EWORKSPACE = 0, -1, -2, -3, -4, -5
# weight formats (palette order) and masks
W_INT8_SYM, W_INT8_ASYM, W_MXINT8, W_INT4_SYM, W_INT4_ASYM, W_NF4, W_FP4, W_MXINT4, W_MXFP4 = range(9)
W_NAMES = ["INT8-sym", "INT8-asym", "MXINT8", "INT4-sym", "INT4-asym", "NF4", "FP4", "MXINT4", "MXFP4"]
MASK_W4 = 0x1F0
MASK_W8 = 0x007
# activation formats (LUT codes)
A_INT8_ASYM, A_FP8_E4M3, A_FP8_E5M2, A_MXFP8, A_MXINT8 = range(5)
A_NAMES = ["INT8-asym", "FP8-E4M3", "FP8-E5M2", "MXFP8-E4M3", "MXINT8"]
# workspace ops
OP_SELECT, OP_STATS, OP_QUANT_ACT, OP_LINEAR, OP_GSELECT, OP_COLSQ = range(6)
GROUP_SIZES = (32, 64, 128, 192, 288)
GMASK_ALL = 0x1F
MASK_DIT_W4 = 0x070  # {INT4-asym, NF4, FP4}
SCHED_SCALED_LINEAR, SCHED_LINEAR = 0, 1

_P = ctypes.c_void_p


class _WQ(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("K", ctypes.c_int64), ("palette_mask", ctypes.c_uint32),
                ("code_bits", ctypes.c_int32), ("fmt", _P), ("codes", _P), ("scale", _P), ("zero", _P),
                ("nf4_absmax", _P), ("e8m0", _P), ("perm", _P), ("group_off", _P), ("err", _P), ("packed", _P)]


class _Stats(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("B", ctypes.c_int32), ("nS", _P), ("lohi", _P)]


class _Sched(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("beta0", ctypes.c_double), ("beta1", ctypes.c_double),
                ("kind", ctypes.c_int32), ("kappa_lo", ctypes.c_double), ("kappa_hi", ctypes.c_double),
                ("snr_lo", ctypes.c_double), ("snr_hi", ctypes.c_double), ("snr_gate_on", ctypes.c_int32)]


class _LUT(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("B", ctypes.c_int32), ("T", ctypes.c_int32), ("F", _P), ("S", _P),
                ("Z", _P)]


class _GWQ(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("K", ctypes.c_int64), ("palette_mask", ctypes.c_uint32),
                ("group_mask", ctypes.c_uint32), ("code_bits", ctypes.c_int32), ("choice", _P), ("fmt", _P),
                ("codes", _P), ("gscale", _P), ("gzero", _P), ("e8m0", _P), ("err", _P), ("packed", _P)]


class _AQ(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("K", ctypes.c_int64), ("fmt", ctypes.c_int32), ("nsamples", ctypes.c_int32),
                ("codes", _P), ("e8m0", _P), ("scale", _P), ("zero", _P)]


_lib = None


def lib():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library {LIB_PATH} is not built; run __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    L.cham_status_string.argtypes = [ctypes.c_int]
    L.cham_status_string.restype = ctypes.c_char_p
    L.cham_version.restype = ctypes.c_int
    L.cham_select_weight_formats.argtypes = [_P, ctypes.POINTER(_WQ), _P]
    L.cham_select_weight_formats_batch.argtypes = [ctypes.POINTER(_P), ctypes.POINTER(_WQ), i32, _P]
    L.cham_pack_weights_batch.argtypes = [ctypes.POINTER(_WQ), i32, _P]
    L.cham_act_stats_reset.argtypes = [ctypes.POINTER(_Stats), _P]
    L.cham_act_stats_accumulate.argtypes = [_P, i64, i32, i32, ctypes.POINTER(_Stats), _P, sz, _P]
    L.cham_act_stats_accumulate_batch.argtypes = [ctypes.POINTER(_P), ctypes.POINTER(i64), ctypes.POINTER(i32),
                                                  ctypes.POINTER(i32), i32, ctypes.POINTER(_Stats), _P, sz, _P]
    L.cham_schedule_default.argtypes = [ctypes.POINTER(_Sched)]
    L.cham_schedule_default.restype = None
    L.cham_build_act_lut.argtypes = [ctypes.POINTER(_Stats), ctypes.POINTER(_Sched), _P, ctypes.POINTER(_LUT), _P,
                                     _P]
    L.cham_bucket.argtypes = [i32, i32, i32]
    L.cham_bucket.restype = i32
    L.cham_quantize_act.argtypes = [_P, i32, i32, _P, _P, ctypes.POINTER(_AQ), _P, sz, _P]
    L.cham_quantize_act_lut.argtypes = [_P, ctypes.POINTER(_LUT), _P, i32, i32, i32, ctypes.POINTER(_AQ), _P, sz,
                                        _P]
    L.cham_quantize_act_noalloc.argtypes = [_P, i32, i32, _P, _P, ctypes.POINTER(_AQ), _P]
    L.cham_quantize_act_lut_accumulate_batch.argtypes = [ctypes.POINTER(_P), ctypes.POINTER(i32), i32, i32,
                                                         ctypes.POINTER(_LUT), _P, ctypes.POINTER(_AQ),
                                                         ctypes.POINTER(_Stats), _P, sz, _P]
    L.cham_mixed_linear.argtypes = [ctypes.POINTER(_AQ), ctypes.POINTER(_WQ), _P, _P, sz, _P]
    L.cham_mixed_linear_grouped.argtypes = [ctypes.POINTER(_AQ), ctypes.POINTER(_GWQ), _P, _P, sz, _P]
    L.cham_mixed_linear_workspace_query.argtypes = [ctypes.POINTER(_AQ), ctypes.POINTER(_WQ), ctypes.POINTER(sz)]
    L.cham_mixed_linear_grouped_workspace_query.argtypes = [ctypes.POINTER(_AQ), ctypes.POINTER(_GWQ),
                                                            ctypes.POINTER(sz)]
    L.cham_conv3x3_mixed.argtypes = [ctypes.POINTER(_AQ), i32, i32, i32, ctypes.POINTER(_WQ), _P, _P, sz, _P]
    L.cham_conv3x3_workspace_bytes.argtypes = [i64, i64, i64, i64, i64]
    L.cham_conv3x3_workspace_bytes.restype = sz
    L.cham_select_group_formats.argtypes = [_P, _P, ctypes.POINTER(_GWQ), _P, sz, _P]
    L.cham_act_colsq_accumulate.argtypes = [_P, i64, i64, _P, _P, sz, _P]
    L.cham_workspace_bytes.argtypes = [i32, i64, i64, i64]
    L.cham_workspace_bytes.restype = sz
    L.cham_packed_bytes.argtypes = [i64, i64]
    L.cham_packed_bytes.restype = sz
    L.cham_linear_plan.argtypes = [i64, i64, i64, i32, ctypes.POINTER(ctypes.c_int32), i32]
    for name in ("cham_select_weight_formats", "cham_select_weight_formats_batch", "cham_pack_weights_batch",
                 "cham_act_stats_reset", "cham_act_stats_accumulate",
                 "cham_act_stats_accumulate_batch",
                 "cham_build_act_lut", "cham_quantize_act", "cham_quantize_act_lut", "cham_quantize_act_noalloc",
                 "cham_quantize_act_lut_accumulate_batch",
                 "cham_mixed_linear", "cham_mixed_linear_grouped", "cham_select_group_formats", "cham_conv3x3_mixed",
                 "cham_act_colsq_accumulate",
                 "cham_linear_plan"):
        getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


class ChamError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lib().cham_status_string(status).decode()} (status {status})")


def _check(rc: int, where: str):
    if rc != OK:
        raise ChamError(rc, where)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _dev_tensor(t: torch.Tensor, dtype, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def workspace_bytes(op: int, M: int, N: int, K: int) -> int:
    return int(lib().cham_workspace_bytes(op, M, N, K))


def linear_plan(M: int, N: int, K: int, code_bits: int) -> dict:
    """The launch plan mixed_linear takes for these sizes (host only)."""
    out = (ctypes.c_int32 * 10)()
    _check(lib().cham_linear_plan(M, N, K, code_bits, out, 10), "cham_linear_plan")
    launches = [{"rows": (out[2 + 4 * i], out[3 + 4 * i]), "tile": (out[4 + 4 * i], out[5 + 4 * i])}
                for i in range(out[0])]
    return {"splits": out[1], "launches": launches}


def _exact_workspace(ws, device, query, a, w):
    """The caller's workspace, else one of the exact size the query reports for these
    operands (None when it is 0)."""
    if ws is not None:
        return ws, ws.numel()
    nb = ctypes.c_size_t(0)
    _check(query(ctypes.byref(a), ctypes.byref(w), ctypes.byref(nb)), "workspace query")
    if nb.value == 0:
        return None, 0
    return torch.empty(nb.value, dtype=torch.uint8, device=device), nb.value


def linear_workspace_query(xq: "AQ", wq: "WQ") -> int:
    """Exact workspace bytes mixed_linear needs for these operands (host only)."""
    a, w = xq.struct(), wq.struct()
    nb = ctypes.c_size_t(0)
    _check(lib().cham_mixed_linear_workspace_query(ctypes.byref(a), ctypes.byref(w), ctypes.byref(nb)),
           "cham_mixed_linear_workspace_query")
    return nb.value


def _workspace(op, M, N, K, device, ws):
    nb = workspace_bytes(op, M, N, K)
    if ws is not None:
        return ws, ws.numel()
    if nb == 0:
        return None, 0
    return torch.empty(nb, dtype=torch.uint8, device=device), nb


# -------------------------------------------------------------------------------------------
# weight search
# -------------------------------------------------------------------------------------------
def code_bits(mask: int) -> int:
    return 8 if mask & 0x7 else 4


@dataclass
class WQ:
    """Packed per-channel weights (device tensors, see cham_wq)."""
    N: int
    K: int
    mask: int
    code_bits: int
    fmt: torch.Tensor
    codes: torch.Tensor
    scale: torch.Tensor
    zero: torch.Tensor
    nf4_absmax: Optional[torch.Tensor]
    e8m0: Optional[torch.Tensor]
    perm: Optional[torch.Tensor]
    group_off: Optional[torch.Tensor]
    err: Optional[torch.Tensor]
    packed: Optional[torch.Tensor] = None  # GEMM-ready layout written by the search (cham_wq.packed)

    def struct(self) -> _WQ:
        return _WQ(self.N, self.K, self.mask, self.code_bits, _ptr(self.fmt), _ptr(self.codes), _ptr(self.scale),
                   _ptr(self.zero), _ptr(self.nf4_absmax), _ptr(self.e8m0), _ptr(self.perm), _ptr(self.group_off),
                   _ptr(self.err), _ptr(self.packed))


def packed_bytes(N: int, K: int) -> int:
    return int(lib().cham_packed_bytes(N, K))


def alloc_wq(N: int, K: int, mask: int, device="cuda", want_perm=True, want_err=False, want_packed=False) -> WQ:
    cb = code_bits(mask)
    u8, f32, i32 = torch.uint8, torch.float32, torch.int32
    nf4 = bool(mask >> W_NF4 & 1)
    mx = bool(mask & ((1 << W_MXINT8) | (1 << W_MXINT4) | (1 << W_MXFP4)))
    return WQ(N, K, mask, cb,
              fmt=torch.empty(N, dtype=u8, device=device),
              codes=torch.empty((N, K * cb // 8), dtype=u8, device=device),
              scale=torch.empty(N, dtype=f32, device=device),
              zero=torch.empty(N, dtype=torch.float32, device=device),
              nf4_absmax=torch.empty((N, K // 64), dtype=f32, device=device) if nf4 else None,
              e8m0=torch.empty((N, K // 32), dtype=u8, device=device) if mx else None,
              perm=torch.empty(N, dtype=i32, device=device) if want_perm else None,
              group_off=torch.empty(10, dtype=i32, device=device) if want_perm else None,
              err=torch.empty((N, 9), dtype=torch.float64, device=device) if want_err else None,
              packed=torch.empty(packed_bytes(N, K), dtype=u8, device=device) if want_packed else None)


def select_weight_formats(W: torch.Tensor, mask: int = MASK_W4, out: Optional[WQ] = None, want_perm=True,
                          want_err=False, want_packed=False, stream=None) -> WQ:
    """Per-output-channel format search of W [N, K] (fp32, device); with want_packed the
    search also writes the GEMM-ready layout that mixed_linear then uses."""
    _dev_tensor(W, torch.float32, "W")
    N, K = W.shape
    if out is None:
        out = alloc_wq(N, K, mask, W.device, want_perm, want_err, want_packed)
    st = out.struct()
    _check(lib().cham_select_weight_formats(_ptr(W), ctypes.byref(st), _stream(stream)), "select_weight_formats")
    out.code_bits = st.code_bits
    return out


class SearchBatch:
    """Prepared C arguments of a batched search over several layers (host arrays of the
    weight pointers and descriptors), reusable across calls."""

    def __init__(self, Ws, outs):
        assert len(Ws) == len(outs) and len(Ws) > 0
        for W in Ws:
            _dev_tensor(W, torch.float32, "W")
        self.Ws, self.outs = list(Ws), list(outs)
        self.ptrs = (_P * len(Ws))(*[W.data_ptr() for W in Ws])
        self.structs = (_WQ * len(outs))(*[o.struct() for o in outs])

    def run(self, stream=None):
        _check(lib().cham_select_weight_formats_batch(self.ptrs, self.structs, len(self.Ws), _stream(stream)),
               "select_weight_formats_batch")
        for o, st in zip(self.outs, self.structs):
            o.code_bits = st.code_bits


class PackBatch:
    """Prepared C arguments of the packing step on its own for several searched weights
    (their descriptors, each with a packed buffer), reusable across calls."""

    def __init__(self, wqs, packed):
        assert len(wqs) == len(packed) and len(wqs) > 0
        self.wqs = list(wqs)
        structs = []
        for w, buf in zip(wqs, packed):
            st = w.struct()
            st.packed = _ptr(buf)
            st.perm = st.group_off = st.err = None
            structs.append(st)
        self.packed = list(packed)
        self.structs = (_WQ * len(structs))(*structs)

    def run(self, stream=None):
        _check(lib().cham_pack_weights_batch(self.structs, len(self.wqs), _stream(stream)), "pack_weights_batch")


def pack_weights_batch(wqs, stream=None):
    """Write the packed layout of searched weights (each wq.packed set) on its own."""
    PackBatch(wqs, [w.packed for w in wqs]).run(stream)


def select_weight_formats_batch(Ws, mask: int = MASK_W4, outs=None, want_perm=True, want_err=False,
                                want_packed=False, stream=None):
    """Format search of several layers' weights (each [N_i, K_i] fp32, device) in one call."""
    if outs is None:
        outs = [alloc_wq(W.shape[0], W.shape[1], mask, W.device, want_perm, want_err, want_packed) for W in Ws]
    SearchBatch(Ws, outs).run(stream)
    return outs


# -------------------------------------------------------------------------------------------
# statistics and LUT
# -------------------------------------------------------------------------------------------
@dataclass
class Stats:
    L: int
    B: int
    nS: torch.Tensor    # [L*B, 5] f64
    lohi: torch.Tensor  # [L*B, 2] f32

    def struct(self):
        return _Stats(self.L, self.B, _ptr(self.nS), _ptr(self.lohi))


def alloc_stats(L: int, B: int, device="cuda") -> Stats:
    return Stats(L, B, torch.empty((L * B, 5), dtype=torch.float64, device=device),
                 torch.empty((L * B, 2), dtype=torch.float32, device=device))


def act_stats_reset(st: Stats, stream=None):
    s = st.struct()
    _check(lib().cham_act_stats_reset(ctypes.byref(s), _stream(stream)), "act_stats_reset")


class StatsBatch:
    """Prepared C arguments of a batched statistics accumulation (several layer inputs),
    reusable across calls with the same tensors."""

    def __init__(self, Xs, layers, buckets, st: Stats, ws=None):
        n = len(Xs)
        assert n > 0 and len(layers) == n and len(buckets) == n
        for X in Xs:
            _dev_tensor(X, torch.float32, "X")
        self.Xs, self.st = list(Xs), st
        self.ptrs = (_P * n)(*[X.data_ptr() for X in Xs])
        self.numel = (ctypes.c_int64 * n)(*[X.numel() for X in Xs])
        self.layer = (ctypes.c_int32 * n)(*layers)
        self.bucket = (ctypes.c_int32 * n)(*buckets)
        nb = sum(workspace_bytes(OP_STATS, X.numel(), 0, 0) for X in Xs)
        self.ws = ws if ws is not None else torch.empty(max(nb, 256), dtype=torch.uint8, device=Xs[0].device)
        self.ws_bytes = self.ws.numel()
        self.s = st.struct()

    def run(self, stream=None):
        _check(lib().cham_act_stats_accumulate_batch(self.ptrs, self.numel, self.layer, self.bucket, len(self.Xs),
                                                     ctypes.byref(self.s), _ptr(self.ws), self.ws_bytes,
                                                     _stream(stream)), "act_stats_accumulate_batch")


def act_stats_accumulate_batch(Xs, layers, buckets, st: Stats, stream=None):
    StatsBatch(Xs, layers, buckets, st).run(stream)


def act_stats_accumulate(X: torch.Tensor, layer: int, bucket: int, st: Stats, ws=None, stream=None):
    _dev_tensor(X, torch.float32, "X")
    n = X.numel()
    ws, nb = _workspace(OP_STATS, n, 0, 0, X.device, ws)
    s = st.struct()
    _check(lib().cham_act_stats_accumulate(_ptr(X), n, layer, bucket, ctypes.byref(s), _ptr(ws), nb,
                                           _stream(stream)), "act_stats_accumulate")


@dataclass
class Schedule:
    T: int = 1000
    beta0: float = 0.00085
    beta1: float = 0.012
    kind: int = SCHED_SCALED_LINEAR
    kappa_lo: float = 3.0
    kappa_hi: float = 5.0
    snr_lo: float = 0.2
    snr_hi: float = 2.0
    snr_gate_on: int = 1

    def struct(self):
        return _Sched(self.T, self.beta0, self.beta1, self.kind, self.kappa_lo, self.kappa_hi, self.snr_lo,
                      self.snr_hi, self.snr_gate_on)


@dataclass
class LUT:
    L: int
    B: int
    T: int
    F: torch.Tensor       # [L*B] u8 (device)
    S: torch.Tensor       # [L*B] f32
    Z: torch.Tensor       # [L*B] f32
    kappa: Optional[torch.Tensor] = None
    F_host: Optional[torch.Tensor] = None  # host mirror of F

    def struct(self):
        return _LUT(self.L, self.B, self.T, _ptr(self.F), _ptr(self.S), _ptr(self.Z))

    def mirror(self):
        """Copy F to the host once (after calibration); the per-step lookup then needs no sync."""
        self.F_host = self.F.cpu().contiguous()
        return self


def build_act_lut(st: Stats, sched: Optional[Schedule] = None, is_shortcut: Optional[torch.Tensor] = None,
                  want_kappa=True, out: Optional[LUT] = None, stream=None) -> LUT:
    sched = sched or Schedule()
    dev = st.nS.device
    n = st.L * st.B
    if out is None:
        out = LUT(st.L, st.B, sched.T, torch.empty(n, dtype=torch.uint8, device=dev),
                  torch.empty(n, dtype=torch.float32, device=dev), torch.empty(n, dtype=torch.float32, device=dev),
                  torch.empty(n, dtype=torch.float64, device=dev) if want_kappa else None)
    if is_shortcut is not None:
        _dev_tensor(is_shortcut, torch.uint8, "is_shortcut")
    s, sc, l = st.struct(), sched.struct(), out.struct()
    _check(lib().cham_build_act_lut(ctypes.byref(s), ctypes.byref(sc), _ptr(is_shortcut), ctypes.byref(l),
                                    _ptr(out.kappa), _stream(stream)), "build_act_lut")
    out.T = l.T
    return out


def bucket(t: int, T: int, B: int) -> int:
    return int(lib().cham_bucket(t, T, B))


# -------------------------------------------------------------------------------------------
# activation quantization
# -------------------------------------------------------------------------------------------
@dataclass
class AQ:
    M: int
    K: int
    fmt: int
    codes: torch.Tensor              # [M, K] u8
    e8m0: Optional[torch.Tensor]     # [M, K/32] u8
    scale: torch.Tensor              # [nsamples] f32
    zero: torch.Tensor               # [nsamples] f32
    nsamples: int = 1                # samples of M / nsamples consecutive rows

    def struct(self):
        return _AQ(self.M, self.K, self.fmt, self.nsamples, _ptr(self.codes), _ptr(self.e8m0), _ptr(self.scale),
                   _ptr(self.zero))


def alloc_aq(M: int, K: int, device="cuda", with_e8m0=True, nsamples: int = 1) -> AQ:
    return AQ(M, K, -1, torch.empty((M, K), dtype=torch.uint8, device=device),
              torch.empty((M, K // 32), dtype=torch.uint8, device=device) if with_e8m0 else None,
              torch.empty(nsamples, dtype=torch.float32, device=device),
              torch.empty(nsamples, dtype=torch.float32, device=device), nsamples)


def quantize_act(X: torch.Tensor, fmt: int, dynamic: bool = True, s: Optional[torch.Tensor] = None,
                 z: Optional[torch.Tensor] = None, out: Optional[AQ] = None, ws=None, stream=None,
                 nsamples: int = 1) -> AQ:
    """Quantize X [M, K]; static mode reads the scale/zero from device tensors s, z; dynamic
    mode takes each of the nsamples row blocks' own range (per-sample scaling)."""
    _dev_tensor(X, torch.float32, "X")
    M, K = X.shape
    if out is None:
        out = alloc_aq(M, K, X.device, nsamples=nsamples)
    ws, nb = _workspace(OP_QUANT_ACT, M, 0, K, X.device, ws)
    a = out.struct()
    _check(lib().cham_quantize_act(_ptr(X), fmt, int(dynamic), _ptr(s), _ptr(z), ctypes.byref(a), _ptr(ws), nb,
                                   _stream(stream)), "quantize_act")
    out.fmt = a.fmt
    return out


def quantize_act_noalloc(X: torch.Tensor, fmt: int, dynamic: bool, s: Optional[torch.Tensor], z: Optional[torch.Tensor],
                         out: AQ, stream=None) -> AQ:
    """cham_quantize_act_noalloc: the caller passes the output buffers; no workspace."""
    _dev_tensor(X, torch.float32, "X")
    a = out.struct()
    _check(lib().cham_quantize_act_noalloc(_ptr(X), fmt, int(dynamic), _ptr(s), _ptr(z), ctypes.byref(a),
                                           _stream(stream)), "quantize_act_noalloc")
    out.fmt = a.fmt
    return out


def quantize_act_lut(X: torch.Tensor, lut: LUT, layer: int, t: int, dynamic: bool = False,
                     out: Optional[AQ] = None, ws=None, stream=None, nsamples: int = 1) -> AQ:
    _dev_tensor(X, torch.float32, "X")
    if lut.F_host is None:
        lut.mirror()
    M, K = X.shape
    if out is None:
        out = alloc_aq(M, K, X.device, nsamples=nsamples)
    ws, nb = _workspace(OP_QUANT_ACT, M, 0, K, X.device, ws)
    a, l = out.struct(), lut.struct()
    _check(lib().cham_quantize_act_lut(_ptr(X), ctypes.byref(l), ctypes.c_void_p(lut.F_host.data_ptr()), layer, t,
                                       int(dynamic), ctypes.byref(a), _ptr(ws), nb, _stream(stream)),
           "quantize_act_lut")
    out.fmt = a.fmt
    return out


class QuantStatsBatch:
    """Prepared C arguments of a fused quantize-and-accumulate call: inputs Xs[i] of
    layers[i] quantized into outs[i] with the LUT's static scales at timestep t while their
    moments are added into st (reusable across calls with the same tensors)."""

    def __init__(self, Xs, layers, outs, lut: "LUT", st: Stats, ws=None):
        n = len(Xs)
        assert n > 0 and len(layers) == n and len(outs) == n
        for X, o in zip(Xs, outs):
            _dev_tensor(X, torch.float32, "X")
            assert X.shape == (o.M, o.K), "X and its AQ differ in shape"
        if lut.F_host is None:
            lut.mirror()
        self.Xs, self.outs, self.lut, self.st = list(Xs), list(outs), lut, st
        self.ptrs = (_P * n)(*[X.data_ptr() for X in Xs])
        self.layer = (ctypes.c_int32 * n)(*layers)
        self.aq = (_AQ * n)(*[o.struct() for o in outs])
        nb = sum(workspace_bytes(OP_STATS, X.numel(), 0, 0) for X in Xs)
        self.ws = ws if ws is not None else torch.empty(max(nb, 256), dtype=torch.uint8, device=Xs[0].device)
        self.ws_bytes = self.ws.numel()
        self.s = st.struct()
        self.l = lut.struct()

    def run(self, t: int, stream=None):
        _check(lib().cham_quantize_act_lut_accumulate_batch(
            self.ptrs, self.layer, len(self.Xs), t, ctypes.byref(self.l), ctypes.c_void_p(self.lut.F_host.data_ptr()),
            self.aq, ctypes.byref(self.s), _ptr(self.ws), self.ws_bytes, _stream(stream)),
            "quantize_act_lut_accumulate_batch")
        for o, a in zip(self.outs, self.aq):
            o.fmt = a.fmt


def quantize_act_lut_accumulate_batch(Xs, layers, t: int, lut: "LUT", st: Stats, outs=None, stream=None):
    """Quantize each Xs[i] as quantize_act_lut(Xs[i], lut, layers[i], t) does (static scales)
    and add its moments into st at (layers[i], bucket of t), in one pass; returns the AQs."""
    if outs is None:
        outs = [alloc_aq(X.shape[0], X.shape[1], X.device) for X in Xs]
    QuantStatsBatch(Xs, layers, outs, lut, st).run(t, stream)
    return outs


# -------------------------------------------------------------------------------------------
# DiT joint (group size, format) search (Sec. 4.6 (i))
# -------------------------------------------------------------------------------------------
@dataclass
class GWQ:
    """Group-scaled weights of one format (device tensors, see cham_gwq)."""
    N: int
    K: int
    mask: int
    gmask: int
    code_bits: int
    choice: torch.Tensor             # [2] i32: group size, format
    fmt: torch.Tensor
    codes: torch.Tensor
    gscale: torch.Tensor             # [N, K/32]
    gzero: torch.Tensor              # [N, K/32]
    e8m0: Optional[torch.Tensor]
    err: Optional[torch.Tensor]      # [45] f64
    packed: Optional[torch.Tensor] = None

    def struct(self) -> _GWQ:
        return _GWQ(self.N, self.K, self.mask, self.gmask, self.code_bits, _ptr(self.choice), _ptr(self.fmt),
                    _ptr(self.codes), _ptr(self.gscale), _ptr(self.gzero), _ptr(self.e8m0), _ptr(self.err),
                    _ptr(self.packed))


def alloc_gwq(N: int, K: int, mask: int, gmask: int = GMASK_ALL, device="cuda", want_err=True,
              want_packed=False) -> GWQ:
    cb = code_bits(mask)
    mx = bool(mask & ((1 << W_MXINT8) | (1 << W_MXINT4) | (1 << W_MXFP4)))
    f32 = torch.float32
    return GWQ(N, K, mask, gmask, cb, torch.zeros(2, dtype=torch.int32, device=device),
               torch.empty(N, dtype=torch.uint8, device=device),
               torch.empty((N, K * cb // 8), dtype=torch.uint8, device=device),
               torch.empty((N, K // 32), dtype=f32, device=device), torch.empty((N, K // 32), dtype=f32, device=device),
               torch.empty((N, K // 32), dtype=torch.uint8, device=device) if mx else None,
               torch.empty(45, dtype=torch.float64, device=device) if want_err else None,
               torch.empty(packed_bytes(N, K), dtype=torch.uint8, device=device) if want_packed else None)


def select_group_formats(W: torch.Tensor, energy: torch.Tensor, mask: int = MASK_DIT_W4, gmask: int = GMASK_ALL,
                         out: Optional[GWQ] = None, want_packed=False, ws=None, stream=None) -> GWQ:
    _dev_tensor(W, torch.float32, "W")
    _dev_tensor(energy, torch.float32, "energy")
    N, K = W.shape
    if out is None:
        out = alloc_gwq(N, K, mask, gmask, W.device, want_packed=want_packed)
    ws, nb = _workspace(OP_GSELECT, 0, N, K, W.device, ws)
    g = out.struct()
    _check(lib().cham_select_group_formats(_ptr(W), _ptr(energy), ctypes.byref(g), _ptr(ws), nb, _stream(stream)),
           "select_group_formats")
    out.code_bits = g.code_bits
    return out


def act_colsq_accumulate(X: torch.Tensor, colsq: torch.Tensor, ws=None, stream=None):
    """colsq[k] += sum_m X[m, k]^2 (binary64, fixed order)."""
    _dev_tensor(X, torch.float32, "X")
    _dev_tensor(colsq, torch.float64, "colsq")
    M, K = X.shape
    ws, nb = _workspace(OP_COLSQ, M, 0, K, X.device, ws)
    _check(lib().cham_act_colsq_accumulate(_ptr(X), M, K, _ptr(colsq), _ptr(ws), nb, _stream(stream)),
           "act_colsq_accumulate")


def mixed_linear_grouped(xq: "AQ", gq: GWQ, Y: Optional[torch.Tensor] = None, ws=None, stream=None) -> torch.Tensor:
    if Y is None:
        Y = torch.empty((xq.M, gq.N), dtype=torch.float32, device=xq.codes.device)
    _dev_tensor(Y, torch.float32, "Y")
    a, g = xq.struct(), gq.struct()
    ws, nb = _exact_workspace(ws, Y.device, lib().cham_mixed_linear_grouped_workspace_query, a, g)
    _check(lib().cham_mixed_linear_grouped(ctypes.byref(a), ctypes.byref(g), _ptr(Y), _ptr(ws), nb, _stream(stream)),
           "mixed_linear_grouped")
    return Y


# -------------------------------------------------------------------------------------------
# mixed-format linear layer
# -------------------------------------------------------------------------------------------
def mixed_linear(xq: AQ, wq: WQ, Y: Optional[torch.Tensor] = None, ws=None, stream=None) -> torch.Tensor:
    if Y is None:
        Y = torch.empty((xq.M, wq.N), dtype=torch.float32, device=xq.codes.device)
    _dev_tensor(Y, torch.float32, "Y")
    a, w = xq.struct(), wq.struct()
    ws, nb = _exact_workspace(ws, Y.device, lib().cham_mixed_linear_workspace_query, a, w)
    _check(lib().cham_mixed_linear(ctypes.byref(a), ctypes.byref(w), _ptr(Y), _ptr(ws), nb, _stream(stream)),
           "mixed_linear")
    return Y


def conv3x3_mixed(xq: AQ, B: int, H: int, W: int, wq: WQ, Y: Optional[torch.Tensor] = None, ws=None,
                  stream=None) -> torch.Tensor:
    """3x3 convolution (stride 1, zero padding 1) of channels-last activation codes xq
    (M = B H W rows, K = C) with weights wq [Co][9 C]; returns Y [B H W, Co]."""
    if Y is None:
        Y = torch.empty((xq.M, wq.N), dtype=torch.float32, device=xq.codes.device)
    _dev_tensor(Y, torch.float32, "Y")
    if ws is None:
        nb = int(lib().cham_conv3x3_workspace_bytes(B, H, W, xq.K, wq.N))
        ws = torch.empty(max(nb, 256), dtype=torch.uint8, device=Y.device)
    a, w = xq.struct(), wq.struct()
    _check(lib().cham_conv3x3_mixed(ctypes.byref(a), B, H, W, ctypes.byref(w), _ptr(Y), _ptr(ws), ws.numel(),
                                    _stream(stream)), "conv3x3_mixed")
    return Y

