"""Benchmark of the whole Chameleon quantized-linear hot path on one MI355X.

Workload: the multi-step SDXL-like sweep -- the 70-block linear stack (10 transformer blocks
at width 640 on 4096 latent tokens, 60 at width 1280 on 1024 tokens, each block QKV d->3d,
out-proj d->d, GEGLU d->8d and FF-out 4d->d: 280 linears, 1.64 G weights) at CFG batch 2
(M = 8192 / 2048 rows), W4 per-channel weight formats, A8 activation formats from a lookup
table over B = 10 timestep buckets (scaled-linear schedule 0.00085 -> 0.012, T = 1000).

One step = one pass of every step of the path over one batch (one sampler step), all inputs
resident in HBM:
  select_weight_formats_batch (the 280 layers, writing each layer's packed GEMM layout) ->
  quantize_act_lut_accumulate_batch (the 280 layer inputs quantized with the LUT's static
  scales while their moments are added into the step's bucket: one read of each input) ->
  build_act_lut (280 x 10, from the moments so far) -> mixed_linear (280).
As a deployed model does, a step quantizes with the LUT calibrated before it (the setup's
calibration plus the steps already run) and gathers its own inputs' moments for the LUT the
next step uses; the formats' host mirror is refreshed from each step's LUT (a 2.8 KB copy
that the next step's launch waits for).  The weight side runs on a second stream (default
priority) beside the activation side on the launch stream, in three chunks of consecutive
layers (about equal weight counts): the GEMMs of a chunk wait only for that chunk's search,
so the later chunks' searches share the chip with the earlier chunks' GEMMs, and the next
step's search of a chunk waits for this step's GEMMs of that chunk (they read the packed
weights it rewrites).

Printed: one JSON line.  `value` = the step's GEMM flops / step time (everything else in the
step counts against it).  `roofline` is for the dominant kernel, the mixed-format GEMM: its
280 calls timed with HIP events on the launch stream inside the timed steps (where a search
chunk runs beside them), and the same calls alone after the timed steps; per layer kind
(width x linear) from untimed steps with an event between calls.  Beside it: the weight
search of the whole stack timed as its own call (no packing; the search's own algorithmic
bytes), the packing pass by difference, the PixArt-like 28-block search at W4 and W8, the single-step (batch 1)
stack's quantize + GEMM pass with one fixed A8 format per layer, and `cpu_baseline`: the CPU
oracle on a bounded sample of the step, single-threaded and on all host cores.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
F16_PEAK_TFLOPS = 2500.0   # dense f16/bf16 MFMA
T_SCHED = 1000
B_BUCKETS = 10
ROWS = {640: 8192, 1280: 2048}   # CFG batch 2 x (4096 | 1024) tokens


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=5)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--t", type=int, default=379, help="timestep of the benchmarked sampler step (999 - 20 i)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-budget-s", type=float, default=12.0, help="seconds of oracle work per baseline run")
    p.add_argument("--no-extras", action="store_true",
                   help="skip the C3 search, the single-step stack and the dense f16 comparison")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="first run one device-to-device copy of this many MiB (the known-size "
                        "kernel that scales the profiler's HBM byte counters; 0: none)")
    p.add_argument("--search-chunks", type=int, default=3,
                   help="split the stack's search into this many chunks of consecutive layers (about equal "
                        "weight counts); the GEMMs of a chunk wait only for its search")
    p.add_argument("--layer-steps", type=int, default=2,
                   help="untimed steps after the timed ones for the per-layer GEMM breakdown (0: none)")
    return p.parse_args()


def committed_traffic():
    """HBM bytes of one step's mixed_linear calls from the committed rocprofv3 counter
    summary, or None when the GEMM source has changed since those counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "mixed_linear_hbm_traffic.md")
    src = os.path.join(ROOT, "paper_2609_33496_amd", "csrc", "cham_gemm.hip")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and line.split(":")[0].strip() in ("traffic_bytes_per_step", "gemm_source_sha256_16"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    if vals.get("gemm_source_sha256_16") != sha or "traffic_bytes_per_step" not in vals:
        return None
    return int(vals["traffic_bytes_per_step"])


def search_bytes(N: int, K: int, bits: int = 4) -> float:
    """Algorithmic bytes of the weight search of one layer: 4 B read per weight, the
    codes (bits / 8 B), the chosen format's block metadata for every channel (NF4 absmax 4 B /
    64, E8M0 1 B / 32 at W4; E8M0 at W8) and 13 B per channel (format, scale, zero, perm)."""
    meta = (4.0 / 64 + 1.0 / 32) if bits == 4 else 1.0 / 32
    return N * K * (4.0 + bits / 8.0 + meta) + 13.0 * N


def pack_bytes(N: int, K: int) -> float:
    """Algorithmic bytes of the packing pass: codes and block metadata read (once for the
    records, once for the column sums), 48 B of record per 32 weights written, 20 B per
    channel."""
    return N * K * (2 * (0.5 + 4.0 / 64 + 1.0 / 32) + 1.5) + 20.0 * N


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only (the library has no multi-GPU path); use --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    import __graft_entry__
    from paper_2609_33496_amd import cham, synth

    if not os.path.exists(cham.LIB_PATH):
        __graft_entry__.build()
    L = cham.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    S = ctypes.c_void_p(stream.cuda_stream)
    side = torch.cuda.Stream(device=dev)  # the weight search of each step (default priority)
    S_side = ctypes.c_void_p(side.cuda_stream)
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    if args.calib_copy_mib > 0:
        src = torch.ones(args.calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    layers = synth.sdxl_stack_layers()
    nl = len(layers)
    Ms = [ROWS[d] for (_, _, _, d) in layers]
    print(f"bench: building the {nl}-layer stack inputs on the GPU", file=sys.stderr, flush=True)
    # ---- inputs (synthetic, drawn on the GPU, resident in HBM before timing)
    Ws = [synth.hetero_weights_dev(1000 + li, N, K, dev) for li, (_, K, N, _) in enumerate(layers)]
    Xs = [synth.diffusion_acts_dev(0, li, args.t, M, K, dev) for li, ((_, K, _, _), M) in enumerate(zip(layers, Ms))]
    wqs = [cham.alloc_wq(N, K, cham.MASK_W4, dev, want_perm=True, want_packed=True) for (_, K, N, _) in layers]
    aqs = [cham.alloc_aq(M, K, dev) for (_, K, _, _), M in zip(layers, Ms)]
    Ys = [torch.empty((M, N), dtype=torch.float32, device=dev) for (_, _, N, _), M in zip(layers, Ms)]
    # one workspace per call kind, sized for the largest layer (the calls run in order)
    ws_lin = torch.empty(max(cham.workspace_bytes(cham.OP_LINEAR, M, N, K) for (_, K, N, _), M in zip(layers, Ms)),
                         dtype=torch.uint8, device=dev)
    ws_q = torch.empty(max(cham.workspace_bytes(cham.OP_QUANT_ACT, M, 0, K) for (_, K, _, _), M in zip(layers, Ms)),
                       dtype=torch.uint8, device=dev)
    # calibration pre-pass (setup, untimed): one batch of 256 rows per (layer, bucket) at the
    # bucket's middle timestep
    stats = cham.alloc_stats(nl, B_BUCKETS, dev)
    cham.act_stats_reset(stats)
    for b in range(B_BUCKETS):
        t = b * T_SCHED // B_BUCKETS + T_SCHED // (2 * B_BUCKETS)
        cal = [synth.diffusion_acts_dev(1, li, t, 256, K, dev) for li, (_, K, _, _) in enumerate(layers)]
        cham.act_stats_accumulate_batch(cal, list(range(nl)), [b] * nl, stats)
        del cal
    sched = cham.Schedule(T=T_SCHED)
    lut = cham.build_act_lut(stats, sched, want_kappa=True)
    # the host mirror of the LUT's formats, in pinned memory: each step refreshes it from
    # the LUT it builds, for the next step's lookups
    lut.F_host = torch.empty(lut.F.numel(), dtype=torch.uint8, pin_memory=True)
    lut.F_host.copy_(lut.F)
    bucket = cham.bucket(args.t, T_SCHED, B_BUCKETS)

    # prepared C structs (the step issues raw C-ABI calls)
    wq_s = [w.struct() for w in wqs]
    sbatch = cham.SearchBatch(Ws, wqs)
    # chunks of consecutive layers with about equal weight counts: the search of chunk c runs
    # on the side stream, the GEMMs of chunk c wait only for it, and the next step's search of
    # chunk c only for this step's GEMMs of chunk c
    nw = np.cumsum([N * K for (_, K, N, _) in layers])
    cuts = sorted({int(np.searchsorted(nw, nw[-1] * (c + 1) / args.search_chunks)) + 1
                   for c in range(max(args.search_chunks, 1) - 1)} - {0, nl})
    chunks = list(zip([0] + cuts, cuts + [nl]))
    sb_chunks = [cham.SearchBatch(Ws[a:b], wqs[a:b]) for a, b in chunks]
    tbatch = cham.StatsBatch(Xs, list(range(nl)), [bucket] * nl, stats)
    st_s, sc_s, lut_s = stats.struct(), sched.struct(), lut.struct()
    aq_s = [a.struct() for a in aqs]
    Fh = ctypes.c_void_p(lut.F_host.data_ptr())
    qsb = cham.QuantStatsBatch(Xs, list(range(nl)), aqs, lut, stats)
    ev = {k: [] for k in ("search", "gemm", "layer")}
    prev_done = [None] * len(chunks)
    f_copied = [None]

    def step(record=False, per_layer_events=False):
        searched = []
        for c, (a, b) in enumerate(chunks):
            if prev_done[c] is not None:
                side.wait_event(prev_done[c])
            if record and c == 0:
                e0 = torch.cuda.Event(enable_timing=True)
                e0.record(side)
            sbc = sb_chunks[c]
            rc = L.cham_select_weight_formats_batch(sbc.ptrs, sbc.structs, b - a, S_side)
            assert rc == 0, rc
            searched.append(torch.cuda.Event(enable_timing=record and c == len(chunks) - 1))
            searched[-1].record(side)
        if record:
            ev["search"].append((e0, searched[-1]))
        if f_copied[0] is not None:
            f_copied[0].synchronize()  # the formats of the LUT the previous step built
        rc = L.cham_quantize_act_lut_accumulate_batch(qsb.ptrs, qsb.layer, nl, args.t, ctypes.byref(qsb.l), Fh,
                                                      qsb.aq, ctypes.byref(qsb.s), P(qsb.ws), qsb.ws_bytes, S)
        assert rc == 0, rc
        rc = L.cham_build_act_lut(ctypes.byref(st_s), ctypes.byref(sc_s), None, ctypes.byref(lut_s), None, S)
        assert rc == 0, rc
        lut.F_host.copy_(lut.F, non_blocking=True)
        f_copied[0] = torch.cuda.Event()
        f_copied[0].record(stream)
        # the per-layer breakdown times the GEMMs alone: every chunk's search first
        for e in (searched if per_layer_events else searched[:1]):
            stream.wait_event(e)
        if record:
            e2 = torch.cuda.Event(enable_timing=True)
            e2.record(stream)
        marks = [e2] if record else []
        for c, (a, b) in enumerate(chunks):
            stream.wait_event(searched[c])
            for li in range(a, b):
                rc = L.cham_mixed_linear(ctypes.byref(qsb.aq[li]), ctypes.byref(wq_s[li]), P(Ys[li]), P(ws_lin),
                                         ws_lin.numel(), S)
                assert rc == 0, rc
                if per_layer_events and li + 1 < nl:
                    marks.append(torch.cuda.Event(enable_timing=True))
                    marks[-1].record(stream)
            prev_done[c] = torch.cuda.Event(enable_timing=record and c == len(chunks) - 1)
            prev_done[c].record(stream)
        end = prev_done[-1]
        if per_layer_events:
            marks.append(end)
            ev["layer"].append(list(zip(marks[:-1], marks[1:])))
        elif record:
            ev["gemm"].append((e2, end))

    print("bench: warmup", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    prev_done[:] = [t0] * len(chunks)
    for _ in range(args.steps):
        step(record=True)
    t1.record(stream)
    torch.cuda.synchronize()
    print("bench: timed steps done", file=sys.stderr, flush=True)
    ms_step = t0.elapsed_time(t1) / args.steps
    ms_search_step = float(np.mean([a.elapsed_time(b) for a, b in ev["search"]]))
    ms_gemm = float(np.mean([a.elapsed_time(b) for a, b in ev["gemm"]]))
    for _ in range(args.layer_steps):
        step(record=True, per_layer_events=True)
    torch.cuda.synchronize()

    flops = [2.0 * M * N * K for (_, K, N, _), M in zip(layers, Ms)]
    per_kind = {}
    if args.layer_steps > 0:
        us = np.mean([[a.elapsed_time(b) * 1e3 for a, b in st] for st in ev["layer"]], axis=0)
        for li, ((name, K, N, d), M) in enumerate(zip(layers, Ms)):
            kind = name.split(".")[0] + "." + name.split(".")[-1]
            by = M * K + N * K / 2 + 4.0 * M * N
            t_roof = max(flops[li] / (F16_PEAK_TFLOPS * 1e6), by / (HBM_PEAK_GBPS * 1e3))
            k = per_kind.setdefault(kind, {"calls": 0, "us": 0.0, "t_roof_us": 0.0, "fl": 0.0, "shape": f"{M}x{N}x{K}"})
            k["calls"] += 1
            k["us"] += float(us[li])
            k["t_roof_us"] += t_roof
            k["fl"] += flops[li]
        for k in per_kind.values():
            k["tflops"] = round(k.pop("fl") / (k["us"] * 1e-6) / 1e12, 1)
            k["frac_t_roof"] = round(k["t_roof_us"] / k["us"], 4)
            k["us_per_call"] = round(k["us"] / k["calls"], 2)
            k["us"] = round(k["us"], 1)
            k["t_roof_us"] = round(k["t_roof_us"], 1)

    total_flops = sum(flops)
    gemm_tflops = total_flops / (ms_gemm * 1e-3) / 1e12
    value = total_flops / (ms_step * 1e-3) / 1e12

    # ---- the weight search of the whole stack as its own call (no packing), then with packing
    print("bench: search timing", file=sys.stderr, flush=True)
    wq_np = [cham.alloc_wq(N, K, cham.MASK_W4, dev, want_perm=True) for (_, K, N, _) in layers]
    nb_search = cham.SearchBatch(Ws, wq_np)
    ms_search = time_calls(lambda: nb_search.run(stream), stream)
    ms_search_pack = time_calls(lambda: sbatch.run(stream), stream)
    sb = sum(search_bytes(N, K) for (_, K, N, _) in layers)
    pb = sum(pack_bytes(N, K) for (_, K, N, _) in layers)
    nweights = sum(N * K for (_, K, N, _) in layers)
    search_gbps = sb / (ms_search * 1e-3) / 1e9
    del wq_np, nb_search

    # ---- the step's 280 GEMMs alone (nothing beside them on the chip), for comparison with
    # their time inside the step, where the next chunk's search shares the chip with them
    def gemms():
        for li in range(nl):
            rc = L.cham_mixed_linear(ctypes.byref(qsb.aq[li]), ctypes.byref(wq_s[li]), P(Ys[li]), P(ws_lin),
                                     ws_lin.numel(), S)
            assert rc == 0, rc
    ms_gemm_alone = time_calls(gemms, stream)
    gemm_alone_tflops = total_flops / (ms_gemm_alone * 1e-3) / 1e12

    # ---- the activation side's parts, each timed alone on the launch stream: the step's
    # fused pass (4 B read + 1 B written per element, + 1/32 B of E8M0 for MX formats), the
    # LUT build, and for comparison the two passes it replaces: the batched moments (4 B read
    # per element) and the 280 quantize calls (5 B per element)
    print("bench: activation side", file=sys.stderr, flush=True)
    numel = sum(M * K for (_, K, _, _), M in zip(layers, Ms))

    def stats_call():
        rc = L.cham_act_stats_accumulate_batch(tbatch.ptrs, tbatch.numel, tbatch.layer, tbatch.bucket, nl,
                                               ctypes.byref(st_s), P(tbatch.ws), tbatch.ws_bytes, S)
        assert rc == 0, rc

    def lut_call():
        rc = L.cham_build_act_lut(ctypes.byref(st_s), ctypes.byref(sc_s), None, ctypes.byref(lut_s), None, S)
        assert rc == 0, rc

    def quant_calls():
        for li in range(nl):
            rc = L.cham_quantize_act_lut(P(Xs[li]), ctypes.byref(lut_s), Fh, li, args.t, 0, ctypes.byref(aq_s[li]),
                                         P(ws_q), ws_q.numel(), S)
            assert rc == 0, rc

    def fused_call():
        rc = L.cham_quantize_act_lut_accumulate_batch(qsb.ptrs, qsb.layer, nl, args.t, ctypes.byref(qsb.l), Fh,
                                                      qsb.aq, ctypes.byref(qsb.s), P(qsb.ws), qsb.ws_bytes, S)
        assert rc == 0, rc

    ms_fused = time_calls(fused_call, stream)
    ms_stats = time_calls(stats_call, stream)
    ms_lut = time_calls(lut_call, stream)
    ms_quant = time_calls(quant_calls, stream)
    qbytes = sum(M * K * (5.0 + (1.0 / 32 if int(lut.F_host[li * B_BUCKETS + bucket]) >= 3 else 0.0))
                 for li, ((_, K, _, _), M) in enumerate(zip(layers, Ms)))
    act_side = {
        "quantize_and_moments": {"ms": round(ms_fused, 4), "GBps": round(qbytes / (ms_fused * 1e-3) / 1e9, 1),
                                 "frac_hbm": round(qbytes / (ms_fused * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                                 "what": "the step's quantize_act_lut_accumulate_batch over the 280 layer inputs, "
                                         "5 B per element (+1/32 for MX)"},
        "stats": {"ms": round(ms_stats, 4), "GBps": round(4.0 * numel / (ms_stats * 1e-3) / 1e9, 1),
                  "frac_hbm": round(4.0 * numel / (ms_stats * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                  "what": "act_stats_accumulate_batch over the 280 layer inputs (binary64 power sums), 4 B per element"},
        "lut": {"ms": round(ms_lut, 4), "what": "build_act_lut, L = 280, B = 10"},
        "quantize": {"ms": round(ms_quant, 4), "GBps": round(qbytes / (ms_quant * 1e-3) / 1e9, 1),
                     "frac_hbm": round(qbytes / (ms_quant * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                     "what": "280 x quantize_act_lut (static LUT scales), 5 B per element (+1/32 for MX)"},
        "elements": int(numel),
    }

    fmts = [int(lut.F_host[li * B_BUCKETS + bucket]) for li in range(nl)]
    hist = np.bincount(torch.cat([w.fmt for w in wqs]).cpu().numpy(), minlength=9)
    afh = np.bincount(np.array(fmts), minlength=5)
    out = {
        "metric": "mixed_linear TFLOP/s + weight-search GB/s (frac of MI355X peak), 1 GPU",
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16-mfma(fp32 acc); w4 codes, a8 codes",
        "data": "synthetic (seeded hetero W4 rows; diffusion-mixture activations; drawn on the GPU)",
        "config": {"workload": "SDXL-like 70-block linear stack (10 blocks d=640 at M=8192, 60 blocks d=1280 at "
                               "M=2048; CFG batch 2), one sampler step of the 50-step sweep, W4 per-channel, A8 LUT "
                               "B=10 scaled-linear T=1000",
                   "linears": nl, "weights": nweights, "gemm_tflop_per_step": round(total_flops / 1e12, 3),
                   "timestep": args.t, "bucket": bucket, "search_chunks": len(chunks),
                   "act_format_hist": {cham.A_NAMES[i]: int(afh[i]) for i in range(5) if afh[i]},
                   "weight_format_hist": {cham.W_NAMES[i]: int(hist[i]) for i in range(9) if hist[i]}},
        "gemm_tflops": round(gemm_tflops, 3),
        "gemm_ms": round(ms_gemm, 4),
        "search": {"ms": round(ms_search, 4), "GBps": round(search_gbps, 1),
                   "frac_hbm": round(search_gbps / HBM_PEAK_GBPS, 4), "bytes": int(sb), "weights": nweights,
                   "what": "select_weight_formats_batch over the 280 layers without packing, HIP events over 3 "
                           "calls; algorithmic bytes: 4 B read + 0.5 B codes + block metadata per weight, 13 B per "
                           "channel"},
        "pack": {"ms": round(ms_search_pack - ms_search, 4),
                 "GBps": round(pb / max(ms_search_pack - ms_search, 1e-6) / 1e6, 1), "bytes": int(pb),
                 "what": "the same call writing each layer's packed GEMM layout, minus the search alone"},
        "search_span_in_step_ms": round(ms_search_step, 4),
        "activation_side": act_side,
        "roofline": {"bound": "mfma", "achieved": round(gemm_tflops, 3), "peak": F16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gemm_tflops / F16_PEAK_TFLOPS, 4),
                     "traffic": committed_traffic(),
                     "alone": {"ms": round(ms_gemm_alone, 4), "achieved": round(gemm_alone_tflops, 3),
                               "frac": round(gemm_alone_tflops / F16_PEAK_TFLOPS, 4),
                               "what": "the same 280 calls with nothing else on the chip (HIP events over 3 "
                                       "passes after the timed steps)"},
                     "per_layer": {"kinds": per_kind,
                                   "what": f"{args.layer_steps} untimed steps with an event between the GEMM calls "
                                           "(each adds a launch gap of about 2-3 us); t_roof = max(2MNK / f16 MFMA "
                                           "peak, (MK + NK/2 + 4MN) bytes / HBM peak), summed per kind"},
                     "kernel": "mixed_linear (gemm_kernel, k-split reduce_kernel; packed weights from the search); "
                               "achieved = 2MNK summed over the step's 280 calls / their HIP-event time on the launch "
                               "stream; traffic = HBM bytes of those 280 calls"},
    }
    if not args.no_extras:
        print("bench: single-step stack, PixArt-like search, dense comparison", file=sys.stderr, flush=True)
        out["single_step_stack"] = single_step_stack(cham, L, layers, Ms, Xs, wqs, stream, S)
        out["compact_weights"] = compact_weights(cham, L, layers, Ms, wqs, qsb.aq, Ys, ws_lin, stream, S,
                                                 ms_gemm_alone)
        out["pixart_search"] = pixart_search(cham, synth, stream, dev)
        out["dense_f16_reference"] = dense_reference(layers, Ms, stream)
    del Ys
    if not args.no_cpu_baseline:
        print("bench: CPU baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(layers, Ms, Ws, Xs, fmts, bucket, args.cpu_budget_s, total_flops)
    print(json.dumps(out), flush=True)


def time_calls(fn, stream, reps=3):
    """Mean HIP-event time (ms) of fn() over reps calls after one warm call."""
    import torch
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def compact_weights(cham, L, layers, Ms, wqs, aq_s, Ys, ws_lin, stream, S, ms_gemm_packed):
    """The step's 280 GEMMs on weights held only as the search's codes and metadata (no
    packed layout: each call derives the decode layout in its workspace first), beside the
    resident bytes per weight of that form and of the packed layout."""
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    lean = []
    for w in wqs:
        st = w.struct()  # a fresh descriptor: the packed layout dropped from it only
        st.packed = None
        lean.append(st)

    def run():
        for li in range(len(layers)):
            rc = L.cham_mixed_linear(ctypes.byref(aq_s[li]), ctypes.byref(lean[li]), P(Ys[li]), P(ws_lin),
                                     ws_lin.numel(), S)
            assert rc == 0, rc

    ms = time_calls(run, stream)
    nw = sum(N * K for (_, K, N, _) in layers)
    nch = sum(N for (_, K, N, _) in layers)
    compact = sum(N * K // 2 + N * (1 + 4 + 4) + 4 * (N * K // 64) + N * K // 32 for (_, K, N, _) in layers)
    packed = sum(int(cham.lib().cham_packed_bytes(N, K)) for (_, K, N, _) in layers)
    return {"gemm_ms": round(ms, 4), "gemm_ms_packed": round(ms_gemm_packed, 4),
            "resident_bytes_per_weight": round(compact / nw, 4),
            "packed_bytes_per_weight": round(packed / nw, 4), "channels": nch,
            "what": "280 x mixed_linear with wq.packed = NULL (the record pre-pass runs in each call's workspace); "
                    "resident = codes (4 bits) + NF4 absmax (4 B / 64) + E8M0 (1 B / 32) per weight + format, "
                    "scale and zero point per channel; gemm_ms_packed = the same calls on the packed layout, both "
                    "timed alone"}


def single_step_stack(cham, L, layers, Ms, Xs, wqs, stream, S):
    """The single-step (SDXL-Turbo-like) case on the same stack: batch 1 (M = 4096 / 1024
    rows: the first CFG half of each input), one fixed A8 format per layer from a B = 1 LUT
    routed by kurtosis alone (statistics at t = 999); quantize + GEMM over the 280 layers."""
    import torch
    from paper_2609_33496_amd import synth
    nl = len(layers)
    dev = Xs[0].device
    st = cham.alloc_stats(nl, 1, dev)
    cham.act_stats_reset(st)
    cal = [synth.diffusion_acts_dev(2, li, 999, 256, K, dev) for li, (_, K, _, _) in enumerate(layers)]
    cham.act_stats_accumulate_batch(cal, list(range(nl)), [0] * nl, st)
    del cal
    lut = cham.build_act_lut(st, cham.Schedule(snr_gate_on=0)).mirror()
    X1 = [X[: M // 2] for X, M in zip(Xs, Ms)]
    aqs = [cham.alloc_aq(M // 2, K, dev, with_e8m0=True) for (_, K, _, _), M in zip(layers, Ms)]
    Ys = [torch.empty((M // 2, N), dtype=torch.float32, device=dev) for (_, _, N, _), M in zip(layers, Ms)]
    ws_lin = torch.empty(max(cham.workspace_bytes(cham.OP_LINEAR, M // 2, N, K) for (_, K, N, _), M in zip(layers, Ms)),
                         dtype=torch.uint8, device=dev)
    ws_q = torch.empty(1 << 16, dtype=torch.uint8, device=dev)
    lut_s = lut.struct()
    Fh = ctypes.c_void_p(lut.F_host.data_ptr())
    aq_s = [a.struct() for a in aqs]
    wq_s = [w.struct() for w in wqs]
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
    marks = {}

    def run(record=False):
        for li in range(nl):
            assert L.cham_quantize_act_lut(P(X1[li]), ctypes.byref(lut_s), Fh, li, 999, 0, ctypes.byref(aq_s[li]),
                                           P(ws_q), ws_q.numel(), S) == 0
        if record:
            marks["g0"] = torch.cuda.Event(enable_timing=True)
            marks["g0"].record(stream)
        for li in range(nl):
            assert L.cham_mixed_linear(ctypes.byref(aq_s[li]), ctypes.byref(wq_s[li]), P(Ys[li]), P(ws_lin),
                                       ws_lin.numel(), S) == 0
        if record:
            marks["g1"] = torch.cuda.Event(enable_timing=True)
            marks["g1"].record(stream)

    run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    run(record=True)
    e1.record(stream)
    torch.cuda.synchronize()
    fl = sum(2.0 * (M // 2) * N * K for (_, K, N, _), M in zip(layers, Ms))
    ms = e0.elapsed_time(e1)
    ms_g = marks["g0"].elapsed_time(marks["g1"])
    fh = np.bincount(lut.F_host.numpy(), minlength=5)
    return {"ms": round(ms, 4), "tflops": round(fl / (ms * 1e-3) / 1e12, 1), "gemm_ms": round(ms_g, 4),
            "gemm_tflops": round(fl / (ms_g * 1e-3) / 1e12, 1),
            "act_format_hist": {cham.A_NAMES[i]: int(fh[i]) for i in range(5) if fh[i]},
            "what": "280 x (quantize_act_lut + mixed_linear) at batch 1 (M = 4096 / 1024), fixed per-layer A8 "
                    "formats (B = 1, kurtosis-only LUT at t = 999), weights packed by the step's search"}


def pixart_search(cham, synth, stream, dev):
    """The weight-format search over 28 PixArt-like DiT blocks (QKV, proj, fc1, fc2,
    cross-attention KV: 578 M weights) at W4 and at W8 {INT8-sym, INT8-asym, MXINT8}, one
    batched call each, no packing."""
    blocks = [(name, K, N) for _ in range(28) for (name, K, N, _) in synth.pixart_block_layers()]
    Ws = [synth.hetero_weights_dev(3000 + i, N, K, dev) for i, (_, K, N) in enumerate(blocks)]
    res = {}
    for mask, tag, bits in ((cham.MASK_W4, "w4", 4), (cham.MASK_W8, "w8", 8)):
        outs = [cham.alloc_wq(N, K, mask, dev, want_perm=True) for (_, K, N) in blocks]
        sb = cham.SearchBatch(Ws, outs)
        ms = time_calls(lambda: sb.run(stream), stream)
        by = sum(search_bytes(N, K, bits) for (_, K, N) in blocks)
        gbps = by / (ms * 1e-3) / 1e9
        hist = np.bincount(np.concatenate([o.fmt.cpu().numpy() for o in outs]), minlength=9)
        res[tag] = {"ms": round(ms, 4), "GBps": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4),
                    "format_hist": {cham.W_NAMES[i]: int(hist[i]) for i in range(9) if hist[i]}}
        del outs, sb
    res["weights"] = sum(N * K for (_, K, N) in blocks)
    res["what"] = "28 blocks x 5 linears in one batched call per palette, HIP events over 3 calls, the search's algorithmic bytes"
    return res


def dense_reference(layers, Ms, stream, reps=10):
    """For comparison only (not part of the path): the library's dense f16 GEMM (torch.matmul,
    f16 inputs and output, no per-channel decode) on the stack's eight distinct shapes,
    weighted by their count in the stack; TFLOP/s per shape and over the step."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(0)
    shapes = {}
    for (name, K, N, d), M in zip(layers, Ms):
        shapes.setdefault((M, N, K), 0)
        shapes[(M, N, K)] += 1
    res, tot_ms, tot_fl = {}, 0.0, 0.0
    for (M, N, K), cnt in shapes.items():
        a = torch.randn(M, K, dtype=torch.float16, device="cuda", generator=g)
        b = torch.randn(K, N, dtype=torch.float16, device="cuda", generator=g)
        for _ in range(3):
            torch.matmul(a, b)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            torch.matmul(a, b)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res[f"{M}x{N}x{K}"] = round(2.0 * M * N * K / (ms * 1e-3) / 1e12, 1)
        tot_ms += ms * cnt
        tot_fl += 2.0 * M * N * K * cnt
    return {"tflops": res, "step_tflops": round(tot_fl / (tot_ms * 1e-3) / 1e12, 1), "unit": "TFLOP/s",
            "what": "torch.matmul f16 x f16 -> f16 (library GEMM), same M, N, K; no decode, 2-byte output"}


# ---------------------------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample of the step
# ---------------------------------------------------------------------------------------------
def _oracle_chunk(job):
    """One unit of oracle work (run in a worker process or inline): returns seconds spent."""
    import oracle
    kind, arrs, p = job
    t = time.perf_counter()
    if kind == "search":
        oracle.select_weight_formats(arrs[0], oracle.MASK_W4, want_err=False, want_perm=False)
    elif kind == "stats":
        st = oracle.Stats(1, 1)
        st.accumulate(arrs[0], 0, 0)
    elif kind == "quant":
        oracle.quantize_act(arrs[0], p["fmt"], p["s"], p["z"], want_xhat=True)
    elif kind == "pairs":
        oracle.linear_pairs(arrs[0], arrs[1], p["mm"], p["nn"])
    return time.perf_counter() - t


def cpu_baseline(layers, Ms, Ws, Xs, act_fmts, bucket, budget_s, total_flops):
    """The CPU oracle (plain C, scalar, the same code the tests check against) on a bounded
    sample of the step, single-threaded and on all host cores (one process per core, each
    running the oracle on its own chunk): for one layer of each of the stack's eight kinds,
    output channels searched, activation rows accumulated into the moments and quantized,
    and single outputs computed; the LUT build over 280 x 10 in full.  Per-kind times are
    extrapolated to the kind's layers at full size and summed to a step time, reported as
    the step's GEMM-flop rate."""
    import multiprocessing as mp

    import oracle

    kinds = {}
    for li, ((name, K, N, d), M) in enumerate(zip(layers, Ms)):
        kinds.setdefault(name.split(".")[0] + "." + name.split(".")[-1], []).append(li)
    # the sample: per kind, chunks of work cut from the first layer of the kind
    jobs, scale = [], []
    for kind, lis in kinds.items():
        li = lis[0]
        _, K, N, _ = layers[li]
        M = Ms[li]
        W = Ws[li][:256].cpu().numpy()
        X = Xs[li][:256].cpu().numpy()
        lo, hi = oracle.minmax(X)
        s, z = oracle.scale_zp(act_fmts[li], lo, hi)
        wq = oracle.select_weight_formats(W[:64], oracle.MASK_W4, want_err=False, want_perm=False)
        Wh = oracle.dequant_weights(wq, K)
        xh = oracle.quantize_act(X[:64], act_fmts[li], s, z, want_xhat=True)[2]
        g = np.random.default_rng(li)
        n = len(lis)
        for c in range(4):
            jobs.append(("search", [W[64 * c:64 * c + 64]], {}))
            scale.append(n * N / 64.0)
            jobs.append(("stats", [X[64 * c:64 * c + 64]], {}))
            scale.append(n * M / 64.0)
            jobs.append(("quant", [X[64 * c:64 * c + 64]], {"fmt": act_fmts[li], "s": s, "z": z}))
            scale.append(n * M / 64.0)
            mm, nn = g.integers(0, 64, 2048), g.integers(0, 64, 2048)
            jobs.append(("pairs", [xh, Wh], {"mm": mm, "nn": nn}))
            scale.append(n * M * N / 2048.0)
    # the LUT over 280 x 10 from the accumulated moments (its cost in full, on one core)
    ost = oracle.Stats(len(layers), B_BUCKETS)
    t = time.perf_counter()
    oracle.build_lut(ost)
    t_lut = time.perf_counter() - t

    def run(pool):
        done, secs, t0 = np.zeros(len(jobs)), np.zeros(len(jobs)), time.perf_counter()
        rounds = 0
        while rounds == 0 or time.perf_counter() - t0 < budget_s:
            res = pool.map(_oracle_chunk, jobs) if pool else [_oracle_chunk(j) for j in jobs]
            secs += np.array(res)
            done += 1
            rounds += 1
        wall = time.perf_counter() - t0
        cpu = float(np.sum(secs))
        est = float(np.sum(secs / done * np.array(scale)))  # single-core seconds for the full step
        return est, wall, cpu, rounds

    est1, wall1, _, r1 = run(None)
    step1 = est1 + t_lut
    ncores = min(16, os.cpu_count() or 1)
    with mp.get_context("spawn").Pool(ncores) as pool:  # fresh interpreters: no GPU state
        estn, walln, cpun, rn = run(pool)
    # all cores: the same per-chunk costs spread over ncores workers, at the parallel efficiency
    # the pool achieved (CPU-seconds of work per wall second / cores)
    eff = min(1.0, cpun / (walln * ncores))
    stepn = estn / (ncores * eff) + t_lut
    cpu_model = platform.processor() or "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(total_flops / stepn / 1e12, 9), "unit": "TFLOP/s", "cores": ncores, "kind": "oracle",
            "value_1core": round(total_flops / step1 / 1e12, 9), "step_s_1core": round(step1, 1),
            "step_s_all_cores": round(stepn, 1), "parallel_efficiency": round(eff, 3),
            "nproc": os.cpu_count(), "cpu_model": cpu_model,
            "sample": f"one layer of each of the 8 kinds: 256 channels searched, 256 rows accumulated into the "
                      f"moments and quantized, 8192 single outputs per kind, repeated for {budget_s:.0f} s "
                      f"({r1} rounds on 1 core, {rn} on {ncores}); times extrapolated to the kind's layers at full "
                      f"size; LUT 280 x 10 in full"}


if __name__ == "__main__":
    main()
