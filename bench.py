"""Benchmark of the whole Chameleon quantized-linear hot path on one MI355X.

Workload: the SDXL-like 1280-wide transformer-block linear set at 1024 px with CFG batch 2 --
M = 2048 tokens through QKV 1280->3840, out-proj 1280->1280, GEGLU 1280->10240 and FF-out
5120->1280.  Weights are W4 with per-channel formats (heterogeneous synthetic rows);
activations are A8 in the format a lookup table built for B = 4 timestep buckets from
kurtosis and SNR (scaled-linear schedule 0.00085 -> 0.012, T = 1000) assigns.

One step = one pass of every step of the path over one batch, all inputs resident in HBM:
  select_weight_formats_batch (the 4 layers, one call, also writing each layer's packed GEMM
  layout) -> act_stats_accumulate_batch (the 4 layer inputs, one call) ->
  build_act_lut -> quantize_act_lut (4) -> mixed_linear (4).
The weight side and the activation side are independent until the GEMMs: the search runs on
a second stream (default priority) while the statistics, LUT and quantization run on the
launch stream, which waits for the search before the GEMMs; the next step's search waits
for this step's GEMMs (they read the packed weights it rewrites).

Printed: one JSON line.  `value` is mixed_linear TFLOP/s over the whole step time (GEMM
flops / step time; the search, statistics, LUT and quantization count against it).  The
`roofline` object is for the dominant kernel (the mixed-format GEMM), timed with HIP events
on the launch stream over the timed steps; the weight search's own HBM rate is reported
beside it.  `roofline.per_layer` breaks the GEMM time down by layer, from untimed steps run
after the timed ones with an event between the calls (--layer-steps; each such event adds a
launch gap, so the timed steps carry none).  `cpu_baseline` times the CPU oracle on a
bounded sample of the same step.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
F16_PEAK_TFLOPS = 2500.0   # dense f16/bf16 MFMA
T_SCHED = 1000
B_BUCKETS = 4
M_TOKENS = 2048
D = 1280


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--t", type=int, default=375, help="timestep of the benchmarked batch")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-dense-reference", action="store_true",
                   help="skip timing the library's dense f16 GEMM on the same shapes (a point of comparison)")
    p.add_argument("--cpu-budget-s", type=float, default=15.0)
    p.add_argument("--no-w8", action="store_true", help="skip the W8 x A8 GEMM timing after the benchmark")
    p.add_argument("--layer-steps", type=int, default=10,
                   help="untimed steps after the timed ones for the per-layer GEMM breakdown (0: none)")
    p.add_argument("--calib-copy-mib", type=int, default=0,
                   help="before timing, copy a buffer of this many MiB once (a kernel of known HBM traffic "
                        "for scaling hardware byte counters)")
    return p.parse_args()


def committed_traffic():
    """HBM bytes per mixed_linear call from the committed rocprofv3 counter summary, or None
    when the GEMM source has changed since those counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "mixed_linear_hbm_traffic.md")
    src = os.path.join(ROOT, "paper_2609_33496_amd", "csrc", "cham_gemm.hip")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if ":" in line and line.split(":")[0].strip() in ("traffic_bytes_per_call", "gemm_source_sha256_16"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    if vals.get("gemm_source_sha256_16") != sha or "traffic_bytes_per_call" not in vals:
        return None
    return int(vals["traffic_bytes_per_call"])


def search_bytes_per_weight(K: int) -> float:
    """Algorithmic bytes of the W4 search call per weight: 4 B read + 0.5 B codes + the
    block metadata written for every channel (NF4 absmax 4 B / 64, E8M0 1 B / 32) + 14 B per
    channel (format, scale, zero, perm, amortized over K); then the packed GEMM layout: the
    codes and block metadata read back (0.5 + 4/64 + 1/32 B), 48 B of record per 32 weights
    (1.5 B) and 16 B of channel parameters per channel."""
    search = 4.0 + 0.5 + 4.0 / 64 + 1.0 / 32 + 14.0 / K
    pack = 0.5 + 4.0 / 64 + 1.0 / 32 + 1.5 + 16.0 / K
    return search + pack


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

    layers = synth.sdxl_block_layers(D)
    # ---- inputs (synthetic, resident in HBM before timing)
    Ws, Xs = [], []
    for li, (name, K, N) in enumerate(layers):
        W, _ = synth.hetero_weights(100 + li, N, K)
        Ws.append(torch.from_numpy(W).to(dev))
        Xs.append(torch.from_numpy(synth.diffusion_acts(0, li, args.t, M_TOKENS, K)).to(dev))
    # the search also writes each layer's GEMM-ready layout (decode tables), which
    # mixed_linear then reads instead of deriving it again on every call
    wqs = [cham.alloc_wq(N, K, cham.MASK_W4, dev, want_perm=True, want_packed=True) for (_, K, N) in layers]
    aqs = [cham.alloc_aq(M_TOKENS, K, dev) for (_, K, N) in layers]
    Ys = [torch.empty((M_TOKENS, N), dtype=torch.float32, device=dev) for (_, K, N) in layers]
    stats = cham.alloc_stats(len(layers), B_BUCKETS, dev)
    cham.act_stats_reset(stats)
    # calibration pre-pass: two batches per bucket at the bucket's timesteps (setup, untimed)
    for b in range(B_BUCKETS):
        for i in range(2):
            t = b * T_SCHED // B_BUCKETS + (2 * i + 1) * T_SCHED // (4 * B_BUCKETS)
            for li, (_, K, _) in enumerate(layers):
                x = torch.from_numpy(synth.diffusion_acts(1, li, t, 512, K)).to(dev)
                cham.act_stats_accumulate(x, li, b, stats)
    sched = cham.Schedule(T=T_SCHED)
    lut = cham.build_act_lut(stats, sched, want_kappa=True)
    lut.mirror()
    bucket = cham.bucket(args.t, T_SCHED, B_BUCKETS)
    if args.calib_copy_mib > 0:
        src = torch.ones(args.calib_copy_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # prepared C structs and workspaces (the step issues raw C-ABI calls)
    ws_q = [torch.empty(max(cham.workspace_bytes(cham.OP_QUANT_ACT, M_TOKENS, 0, X.shape[1]), 256),
                        dtype=torch.uint8, device=dev) for X in Xs]
    ws_lin = [torch.empty(cham.workspace_bytes(cham.OP_LINEAR, M_TOKENS, N, K), dtype=torch.uint8, device=dev)
              for (_, K, N) in layers]
    wq_s = [w.struct() for w in wqs]
    sbatch = cham.SearchBatch(Ws, wqs)  # the block's four layers searched in one call
    # the four layer inputs' statistics in one call (as one calibration forward pass gives them)
    tbatch = cham.StatsBatch(Xs, list(range(len(layers))), [bucket] * len(layers), stats)
    st_s = stats.struct()
    sc_s = sched.struct()
    lut_s = lut.struct()
    aq_s = [a.struct() for a in aqs]
    Fh = ctypes.c_void_p(lut.F_host.data_ptr())
    P = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731

    ev = {k: [] for k in ("search", "gemm", "layer")}
    prev_end = [None]  # event: the previous step's GEMMs are done (or the timing start)

    def step(record=False, per_layer_events=False):
        e0 = e1 = None
        # weight side, on the second stream: after the previous step's GEMMs
        if prev_end[0] is not None:
            side.wait_event(prev_end[0])
        if record:
            e0 = torch.cuda.Event(enable_timing=True)
            e0.record(side)
        rc = L.cham_select_weight_formats_batch(sbatch.ptrs, sbatch.structs, len(layers), S_side)
        assert rc == 0, rc
        searched = torch.cuda.Event(enable_timing=record)
        searched.record(side)
        if record:
            ev["search"].append((e0, searched))
        # activation side, on the launch stream
        rc = L.cham_act_stats_accumulate_batch(tbatch.ptrs, tbatch.numel, tbatch.layer, tbatch.bucket, len(layers),
                                               ctypes.byref(st_s), P(tbatch.ws), tbatch.ws_bytes, S)
        assert rc == 0, rc
        rc = L.cham_build_act_lut(ctypes.byref(st_s), ctypes.byref(sc_s), None, ctypes.byref(lut_s), None, S)
        assert rc == 0, rc
        for li in range(len(layers)):
            rc = L.cham_quantize_act_lut(P(Xs[li]), ctypes.byref(lut_s), Fh, li, args.t, 0, ctypes.byref(aq_s[li]),
                                         P(ws_q[li]), ws_q[li].numel(), S)
            assert rc == 0, rc
        stream.wait_event(searched)
        if record:
            e2 = torch.cuda.Event(enable_timing=True)
            e2.record(stream)
        marks = [e2] if record else []
        for li in range(len(layers)):
            rc = L.cham_mixed_linear(ctypes.byref(aq_s[li]), ctypes.byref(wq_s[li]), P(Ys[li]), P(ws_lin[li]),
                                     ws_lin[li].numel(), S)
            assert rc == 0, rc
            if per_layer_events and li + 1 < len(layers):
                marks.append(torch.cuda.Event(enable_timing=True))
                marks[-1].record(stream)
        end = torch.cuda.Event(enable_timing=record)
        end.record(stream)
        prev_end[0] = end
        if per_layer_events:
            marks.append(end)
            ev["layer"].append(list(zip(marks[:-1], marks[1:])))
        elif record:
            ev["gemm"].append((e2, end))

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    prev_end[0] = t0  # the first timed search starts after the timing start
    for _ in range(args.steps):
        step(record=True)
    t1.record(stream)
    torch.cuda.synchronize()
    ms_total = t0.elapsed_time(t1)
    ms_step = ms_total / args.steps
    ms_search = float(np.mean([a.elapsed_time(b) for a, b in ev["search"]]))
    ms_gemm = float(np.mean([a.elapsed_time(b) for a, b in ev["gemm"]]))
    # per-layer breakdown from extra steps after the timed region: an event between calls
    # adds a launch gap (≈ 2–3 µs each), so the timed steps carry only the two around the GEMMs
    for _ in range(args.layer_steps):
        step(record=True, per_layer_events=True)
    torch.cuda.synchronize()
    # per layer: HIP-event time of its call (launch gap to the previous call included), and
    # its roofline time max(flops / f16 MFMA peak, algorithmic bytes / HBM peak), the bytes
    # being activation codes, 4-bit weight codes and the binary32 output
    per_layer = {}
    for li, (name, K, N) in enumerate(layers if args.layer_steps > 0 else []):
        us = float(np.mean([a.elapsed_time(b) for a, b in (st[li] for st in ev["layer"])])) * 1e3
        fl = 2.0 * M_TOKENS * N * K
        by = M_TOKENS * K + N * K / 2 + 4.0 * M_TOKENS * N
        t_roof = max(fl / (F16_PEAK_TFLOPS * 1e6), by / (HBM_PEAK_GBPS * 1e3))
        per_layer[name] = {"us": round(us, 2), "tflops": round(fl / us / 1e6, 1), "t_roof_us": round(t_roof, 2),
                           "frac_t_roof": round(t_roof / us, 4)}

    flops = sum(2.0 * M_TOKENS * N * K for (_, K, N) in layers)
    sbytes = sum(N * K * search_bytes_per_weight(K) for (_, K, N) in layers)
    gemm_tflops = flops / (ms_gemm * 1e-3) / 1e12
    value = flops / (ms_step * 1e-3) / 1e12
    search_gbps = sbytes / (ms_search * 1e-3) / 1e9

    fmts = [int(lut.F_host[li * B_BUCKETS + bucket]) for li in range(len(layers))]
    hist = np.bincount(torch.cat([w.fmt for w in wqs]).cpu().numpy(), minlength=9)
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
        "data": "synthetic (seeded hetero W4 rows; diffusion-mixture activations)",
        "config": {"workload": "SDXL-like 1280-wide block linears, M=2048 (1024 tokens x CFG 2), W4 per-channel, "
                               "A8 LUT B=4 scaled-linear T=1000",
                   "layers": [f"{n} {k}->{nn}" for (n, k, nn) in layers], "timestep": args.t, "bucket": bucket,
                   "act_formats": [cham.A_NAMES[f] for f in fmts],
                   "weight_format_hist": {cham.W_NAMES[i]: int(hist[i]) for i in range(9) if hist[i]}},
        "gemm_tflops": round(gemm_tflops, 3),
        "gemm_ms": round(ms_gemm, 4),
        "search_GBps": round(search_gbps, 2),
        "search_frac_hbm": round(search_gbps / HBM_PEAK_GBPS, 4),
        "search_ms": round(ms_search, 4),
        "roofline": {"bound": "mfma", "achieved": round(gemm_tflops, 3), "peak": F16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(gemm_tflops / F16_PEAK_TFLOPS, 4),
                     "traffic": committed_traffic(),
                     "per_layer": {"layers": per_layer,
                                   "what": f"{args.layer_steps} untimed steps after the timed ones with an event between "
                                           "the GEMM calls (each adds a launch gap of about 2-3 us); t_roof = max("
                                           "2MNK / f16 MFMA peak, (MK + NK/2 + 4MN) bytes / HBM peak)"},
                     "kernel": "mixed_linear (gemm_kernel, k-split reduce_kernel; the weights' decode layout comes packed from the search); achieved = 2MNK summed over the "
                               "4 calls / their HIP-event time; traffic = HBM bytes per call"},
    }
    if not args.no_dense_reference:
        out["dense_f16_reference"] = dense_reference(layers, stream)
    if not args.no_w8:
        for a, st_c in zip(aqs, aq_s):
            a.fmt = st_c.fmt  # the format the step's quantize calls wrote into the C structs
        out["w8a8_linear"] = w8_linear(cham, layers, Ws, aqs, stream)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(layers, Ws, Xs, fmts, args.cpu_budget_s)
    print(json.dumps(out), flush=True)


def dense_reference(layers, stream, reps=20):
    """For comparison only (not part of the path): the library's dense f16 GEMM (torch.matmul,
    f16 inputs and output, no per-channel decode) on the same shapes, timed after the
    benchmark with HIP events; TFLOP/s per layer."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(0)
    res = {}
    for (name, K, N) in layers:
        a = torch.randn(M_TOKENS, K, dtype=torch.float16, device="cuda", generator=g)
        b = torch.randn(K, N, dtype=torch.float16, device="cuda", generator=g)  # contiguous [K, N]
        for _ in range(3):
            torch.matmul(a, b)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            torch.matmul(a, b)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        res[name] = round(2.0 * M_TOKENS * N * K / (ms * 1e-3) / 1e12, 1)
    return {"tflops": res, "unit": "TFLOP/s",
            "what": "torch.matmul f16 x f16 -> f16 (library GEMM), same M, N, K; no decode, 2-byte output"}


def w8_linear(cham, layers, Ws, aqs, stream, reps=20):
    """The same four GEMMs with W8 weights (INT8-sym, INT8-asym, MXINT8 per channel: the
    8-bit palette) against the step's A8 activation codes, after the benchmark: each call
    timed with HIP events over `reps` calls; TFLOP/s per layer and over the four."""
    import torch
    res, tot_ms, tot_fl = {}, 0.0, 0.0
    for (name, K, N), W, aq in zip(layers, Ws, aqs):
        wq = cham.select_weight_formats(W, cham.MASK_W8, want_packed=True)
        Y = torch.empty((M_TOKENS, N), dtype=torch.float32, device=W.device)
        ws = torch.empty(cham.workspace_bytes(cham.OP_LINEAR, M_TOKENS, N, K), dtype=torch.uint8, device=W.device)
        for _ in range(3):
            cham.mixed_linear(aq, wq, Y=Y, ws=ws)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            cham.mixed_linear(aq, wq, Y=Y, ws=ws)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        fl = 2.0 * M_TOKENS * N * K
        res[name] = round(fl / (ms * 1e-3) / 1e12, 1)
        tot_ms += ms
        tot_fl += fl
    return {"tflops": res, "all_tflops": round(tot_fl / (tot_ms * 1e-3) / 1e12, 1), "unit": "TFLOP/s",
            "what": "mixed_linear with W8 per-channel weights (8-bit palette), the step's A8 codes; each call "
                    "timed alone after the benchmark"}


def cpu_baseline(layers, Ws, Xs, act_fmts, budget_s):
    """The CPU oracle (single-threaded C) on a bounded sample of the same step, scaled to
    the step's GEMM-flop throughput: per layer, output channels are searched, activation
    rows quantized and single outputs computed, each in chunks until its share of the
    budget is spent; the per-layer times are extrapolated to the full sizes."""
    import oracle

    def until(share, total, chunk, fn):  # run fn(first, count) in chunks for `share` seconds
        done, t0 = 0, time.perf_counter()
        while done < total and (done == 0 or time.perf_counter() - t0 < share):
            n = min(chunk, total - done)
            fn(done, n)
            done += n
        return done, time.perf_counter() - t0

    per_layer = budget_s / len(layers)
    total_s = 0.0
    flops = 0.0
    samples = []
    for li, (name, K, N) in enumerate(layers):
        W = Ws[li].cpu().numpy()
        X = Xs[li].cpu().numpy()
        M = X.shape[0]
        first = {}

        def search(a, n):
            wq = oracle.select_weight_formats(W[a:a + n], oracle.MASK_W4, want_err=False, want_perm=False)
            first.setdefault("wq", wq)
        nrows, ts = until(0.4 * per_layer, N, 32, search)
        t = time.perf_counter()
        lo, hi = oracle.minmax(X)
        s, z = oracle.scale_zp(act_fmts[li], lo, hi)
        t_mm = time.perf_counter() - t

        def quant(a, n):
            xh = oracle.quantize_act(X[a:a + n], act_fmts[li], s, z, want_xhat=True)[2]
            first.setdefault("xh", xh)
        mrows, tq = until(0.2 * per_layer, M, 64, quant)
        Wh = oracle.dequant_weights(first["wq"], K)
        xh = first["xh"]
        g = np.random.default_rng(li)

        def pairs(a, n):
            oracle.linear_pairs(xh, Wh, g.integers(0, xh.shape[0], n), g.integers(0, Wh.shape[0], n))
        npairs, tg = until(0.4 * per_layer, M * N, 4096, pairs)
        total_s += ts * N / nrows + t_mm + tq * M / mrows + tg * (M * N) / npairs
        flops += 2.0 * M * N * K
        samples.append(f"{name}: {nrows}/{N} channels searched, {mrows}/{M} rows quantized, {npairs} outputs")
    return {"value": round(flops / total_s / 1e12, 9), "unit": "TFLOP/s", "cores": 1, "kind": "oracle",
            "sample": "; ".join(samples) + f"; each part run for its share of {budget_s:.0f} s of CPU time, "
                      "per-layer times extrapolated to full size (stats/LUT omitted)"}


if __name__ == "__main__":
    main()
