#!/usr/bin/env python3
"""Benchmark of the W8A8 SmoothQuant hot path on one MI355X.

Step: one forward pass of Gemma-3-1B's FFN path over a batch of synthetic
tokens -- 26 FFN blocks (d = 1152, f = 6912) under a precision map, RMSNorm
glue, final RMSNorm and the lm_head (V = 262144) -- launched through the C ABI
(``w8a8_ffn_stack``) and replayed as a captured graph.  Default: the 26-layer
stack at M = 2048 prefill tokens, every FFN block INT8 (the paper's all26 map)
and the INT8 lm_head, so every product of the step runs on the INT8 path.

Printed (one JSON line): INT8 TOPS of the step, the roofline of its dominant
kernel (the INT8 gate/up GEMM with the fused GeGLU epilogue, bound by the
matrix cores at this size) against the published peak and a measured one,
the oracle timed on the host, and per layer group the INT8-vs-bf16 speedup,
decode GB/s and prefill TOPS.  Inputs are seeded synthetic tensors
(``paper_2608_28003_amd.synth``).  Times are medians of 15 repeats, each a
loop of at least 1 ms of work between two HIP events on the launch stream.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--m 2048] [--map all26]
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0       # MI355X HBM3E
INT8_PEAK_TOPS = 5000.0     # dense INT8 MFMA (published figure without sparsity)
BF16_PEAK_TFLOPS = 2500.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--m", type=int, default=2048)
    ap.add_argument("--map", default="all26")
    ap.add_argument("--no-extras", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain 256 MiB device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: this path has no multi-GPU mode "
              "(each GPU would run its own batch shard; the forward pass needs no collective)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_28003_amd import synth, w8a8

    if args.copy_probe:
        # A copy of known size: its FETCH_SIZE / WRITE_SIZE readings per
        # dispatch convert the counters of the other kernels into bytes.
        n = 256 << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(4):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "dispatches": 4}), flush=True)
        return

    w8a8.lib()  # fails loudly without the HIP library
    assert torch.cuda.is_available(), "bench.py needs the GPU"
    dev = torch.device("cuda:0")
    M, D, F, V, NL = args.m, synth.D_MODEL, synth.D_FF, synth.VOCAB, synth.N_LAYERS

    def dbf(u16):
        return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).to(dev)

    # ------------------------------------------------------------ inputs
    t0 = time.time()
    cfg = synth.stack_config(m=max(M, 64), n_layers=NL)
    log("synthetic weights drawn in %.1f s" % (time.time() - t0))
    x_all = dbf(cfg["x"])
    x = x_all[:M].contiguous()
    x_cal = dbf(cfg["x_cal"])
    w_layers = [{k: dbf(v) for k, v in L.items()} for L in cfg["layers"]]
    w_lm = dbf(cfg["w_lm"])
    del cfg

    # ------------------------------------------------------------ offline: a1 + a2 on the GPU
    t0 = time.time()
    bf16_layers = [w8a8.FfnBF16.from_weights(L["w_gate"], L["w_up"], L["w_down"]) for L in w_layers]
    int8_layers, fp8_layers = [], []
    a = torch.empty_like(x_cal)
    xc = x_cal.clone()
    ws_cal = torch.empty(w8a8.bf16_ffn_workspace_bytes(x_cal.shape[0], D, F), dtype=torch.uint8, device=dev)
    fo = torch.empty_like(x_cal)
    for l, L in enumerate(w_layers):
        w8a8.rmsnorm(xc, out=a)
        a_amax = w8a8.col_absmax(a)
        d_gu = w8a8.smooth_calibrate(a_amax, [L["w_gate"], L["w_up"]])
        h = w8a8.bf16_ffn_gate_up(bf16_layers[l], a)
        d_dn = w8a8.smooth_calibrate(w8a8.col_absmax(h), [L["w_down"]])
        int8_layers.append(w8a8.FfnW8A8.from_weights(L["w_gate"], L["w_up"], L["w_down"], d_gu, d_dn))
        if not args.no_extras:   # the FP8 (E4M3) variant, same smoothing factors
            fp8_layers.append(w8a8.fp8_ffn_layer(L["w_gate"], L["w_up"], L["w_down"], d_gu, d_dn))
        w8a8.bf16_ffn(bf16_layers[l], a, out=fo, ws=ws_cal)
        w8a8.rmsnorm_residual(xc, fo, out=xc)
    w8a8.rmsnorm(xc, out=a)
    d_lm = w8a8.smooth_calibrate(w8a8.col_absmax(a), [w_lm])
    lm_int8 = w8a8.LinearW8A8.from_weight(w_lm, d_lm)
    lm_fp8 = None if args.no_extras else w8a8.fp8_linear_layer(w_lm, d_lm)
    lm_bf16 = w8a8.pack_bf16(w_lm)
    torch.cuda.synchronize()
    # row-major (K x N) bf16 weights for the torch / hipBLASLt reference FFN
    torch_ffn = [] if args.no_extras else [
        (torch.cat([L["w_gate"], L["w_up"]], 0).t().contiguous(), L["w_down"].t().contiguous())
        for L in w_layers]
    del w_layers, ws_cal
    log("calibration + quantisation on the GPU in %.1f s" % (time.time() - t0))

    stack = w8a8.Stack(int8_layers, bf16_layers, lm_int8, lm_bf16, V)

    def ops_int8(prec, lm8, m):
        n8 = int(np.sum(prec))
        return n8 * 6.0 * m * D * F + (2.0 * m * D * V if lm8 else 0.0)

    def ops_all(m):
        return NL * 6.0 * m * D * F + 2.0 * m * D * V

    def make_graph(fn):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            fn()
            fn()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        torch.cuda.synchronize()
        return g

    def time_graph(g, reps=15, warm=3, min_ms=1.0):
        """Median over `reps` repeats of the seconds per replay; each repeat
        replays the graph for at least min_ms between two events recorded on
        the current stream (the one the graph and the library launch on)."""
        for _ in range(warm):
            g.replay()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        inner = max(1, int(np.ceil(min_ms / max(e0.elapsed_time(e1), 1e-3))))
        ts = []
        for _ in range(reps):
            e0.record()
            for _ in range(inner):
                g.replay()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / inner)
        return float(np.median(ts)) * 1e-3

    def time_eager(fn, reps, warm=3):
        for _ in range(warm):
            fn()
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t) / reps

    # ------------------------------------------------------------ the step
    prec = w8a8.precision_map(args.map)
    lm8 = True
    out = torch.empty((M, V), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(w8a8.stack_workspace_bytes(M, D, F, V), dtype=torch.uint8, device=dev)

    def step():
        stack.run(x, prec, lm8, out=out, ws=ws)

    g = make_graph(step)
    for _ in range(args.warmup):
        g.replay()
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(args.steps):
        g.replay()
    torch.cuda.synchronize()
    sec = (time.perf_counter() - t) / args.steps
    w8a8.Stack.status(ws)   # raises if a persistent decode launch gave up
    value = ops_int8(prec, lm8, M) / sec / 1e12
    eager_sec = time_eager(step, max(3, args.steps // 4), warm=1)
    log("step %.3f ms (graph), %.3f ms (eager launches): %.1f INT8 TOPS" % (sec * 1e3, eager_sec * 1e3, value))

    # ------------------------------------------------------------ dominant kernel roofline
    # INT8 gate/up GEMM with the fused GeGLU epilogue, the kernel with the
    # largest share of the step (26 launches), at the step's M and in its
    # launch configuration: a captured graph of its 26 per-layer launches
    # (16 MB of weights each, 415 MB in rotation, above the 256 MB memory-side
    # cache) is timed with HIP events on the launch stream; average launch
    # duration = median time per replay / 26.  At M = 2048 the kernel does
    # 2 M d (2 f) = 65.2 G integer ops on 16.3 MB of algorithmic bytes
    # (4000 op/B, far above the 629 op/B ridge): bound by the matrix cores.
    peaks = measured_peaks(torch)
    log("measured ceilings: INT8 MFMA loop %.0f TOPS, HBM read %.0f GB/s"
        % (peaks["mfma_i8_tops"], peaks["hbm_read_GBs"]))
    roofline = gate_up_roofline(torch, w8a8, int8_layers, x, M, D, F, NL, make_graph, time_graph,
                                peaks)
    log("gate/up kernel %.2f us: %.0f TOPS (%.1f %% of peak)"
        % (roofline["avg_launch_us"], roofline["achieved"], 100 * roofline["frac"]))

    result = {
        "metric": "W8A8 linear INT8 TOPS (% MFMA peak) + decode GB/s; INT8-vs-bf16 speedup",
        "value": round(value, 2), "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(sec * 1e3, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int8", "data": "synthetic",
        "config": {"workload": "26-layer FFN stack (Gemma-3-1B FFN shapes: 26 gated FFN blocks "
                               "1152 -> 6912 -> 1152) under the %s precision map + RMSNorm glue + "
                               "INT8 lm_head (1152 -> 262144), M=%d tokens, random-init"
                               % (args.map, M),
                   "m": M, "layers": NL, "map": args.map, "lm_head": "int8",
                   "launch": "captured graph", "int8_mfma_frac": round(value / INT8_PEAK_TOPS, 4),
                   "int8_mfma_frac_measured_peak": round(value / peaks["mfma_i8_tops"], 4),
                   "eager_ms_per_step": round(eager_sec * 1e3, 4)},
        "measured_peaks": peaks,
        "roofline": roofline,
    }

    # ------------------------------------------------------------ per layer group
    if not args.no_extras:
        result["groups"] = extras(torch, w8a8, stack, int8_layers, bf16_layers, lm_int8, lm_bf16,
                                  x_all, w_lm, M, D, F, V, NL, make_graph, time_graph, ops_int8,
                                  ops_all, sec, fp8_layers, lm_fp8, torch_ffn, peaks)

    if "groups" in result:  # decode: one token through the all26 map and the INT8 lm_head
        d1 = dict(result["groups"]["stack_maps_m1"]["FFN all26 + lm_head"])
        d1["hbm_frac"] = round(d1["weight_GBs"] / HBM_PEAK_GBS, 4)
        result["decode_m1"] = d1

    if "groups" in result:  # the M = 128 gate/up kernel against HBM (extra)
        result["gate_up_m128_hbm"] = result["groups"].pop("gate_up_m128_hbm")

    # ------------------------------------------------------------ oracle on the host
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(M)

    print(json.dumps(result), flush=True)


def measured_traffic(m):
    """HBM bytes per launch of the gate/up kernel at M = m from the committed
    counter summary, or None when there is none for this M or it was taken on
    other kernel or planner sources than the ones built here."""
    import hashlib
    import re
    path = os.path.join(ROOT, "profiles", "gate_up_geglu_m%d_hbm_traffic.md" % m)
    try:
        text = open(path).read()
        rec = json.loads(re.search(r"```json\n(.*?)\n```", text, re.S).group(1))
    except (OSError, AttributeError, ValueError):
        return None
    h = hashlib.sha256()
    for f in ("gemm.hip", "device.h", "kernels.h", "api.hip"):  # kernels and their plans
        with open(os.path.join(ROOT, "paper_2608_28003_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    if rec.get("m") != m or rec.get("source_sha256") != h.hexdigest():
        return None
    return rec["traffic_bytes"]


def measured_peaks(torch):
    """Ceilings measured on this device (libw8a8_peak.so): the INT8 matrix
    instruction in a register loop (2 workgroups of 4 waves per CU, 8
    independent chains a wave) and a streaming 16-byte read of 2 GiB (8x the
    memory-side cache) at the best of three grid sizes; medians of 15."""
    import ctypes
    from paper_2608_28003_amd import build as hip_build
    L = ctypes.CDLL(hip_build.PEAK_LIB_PATH)
    L.w8a8_peak_mfma_i8.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    L.w8a8_peak_mfma_i8_ops.argtypes = [ctypes.c_int, ctypes.c_int]
    L.w8a8_peak_mfma_i8_ops.restype = ctypes.c_double
    L.w8a8_peak_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p,
                                 ctypes.c_void_p]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    def med(launch):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for _ in range(3):
            launch()
        ts = []
        for _ in range(15):
            e0.record()
            launch()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3)
        return float(np.median(ts))

    blocks, iters = 2 * cus, 20000
    sink = torch.zeros(blocks, dtype=torch.int32, device="cuda:0")
    t = med(lambda: L.w8a8_peak_mfma_i8(blocks, iters, ctypes.c_void_p(sink.data_ptr()), st))
    tops = L.w8a8_peak_mfma_i8_ops(blocks, iters) / t / 1e12
    nbytes = 2 << 30
    buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0")
    best = 0.0
    for mult in (4, 8, 16):
        b = cus * mult
        t = med(lambda: L.w8a8_peak_read(ctypes.c_void_p(buf.data_ptr()), nbytes, b,
                                         ctypes.c_void_p(sink.data_ptr()), st))
        best = max(best, nbytes / t / 1e9)
    del buf
    return {"mfma_i8_tops": round(tops, 1), "hbm_read_GBs": round(best, 1),
            "note": "INT8 MFMA register loop and a 2 GiB streaming read on this device"}


def gate_up_roofline(torch, w8a8, int8_layers, x, M, D, F, NL, make_graph, time_graph, peaks):
    """Roofline entry of the INT8 gate/up GEMM with the GeGLU epilogue at M
    tokens: 26 per-layer launches in one captured graph, average launch
    duration from HIP events on the launch stream.  Algorithmic work per
    launch: 2 M d (2 f) integer ops; bytes 2 f d (both weights) + 8 f (their
    scales) + 4 d (smoothing) + 2 M d (the bf16 block input), the intermediate
    h excluded.  Below the ridge (5000 TOPS / 8 TB/s = 625 op/B) the bound is
    HBM, above it the matrix cores."""
    qx, sx = w8a8.quantize_act(x, int8_layers[0].gate.delta)
    h = torch.empty((M, F), dtype=torch.bfloat16, device=x.device)
    g = make_graph(lambda: [w8a8.ffn_gate_up(L, qx, sx, M, out=h) for L in int8_layers])
    t = time_graph(g) / NL
    del g
    ops = 2.0 * M * D * 2 * F
    nbytes = 2 * F * D + 8 * F + 4 * D + 2 * M * D
    common = {"kernel": "gemm_tile_kernel<int8, GeGLU epilogue> (FFN gate/up)",
              "avg_launch_us": round(t * 1e6, 3), "ops_per_launch": ops,
              "algorithmic_bytes_per_launch": nbytes, "m": M,
              "int8_tops": round(ops / t / 1e12, 1), "GBs": round(nbytes / t / 1e9, 1)}
    if ops / nbytes >= INT8_PEAK_TOPS * 1e12 / (HBM_PEAK_GBS * 1e9):
        achieved = ops / t / 1e12
        return dict({"bound": "mfma", "achieved": round(achieved, 1), "peak": INT8_PEAK_TOPS,
                     "unit": "TOP/s", "frac": round(achieved / INT8_PEAK_TOPS, 4),
                     "traffic": measured_traffic(M),
                     "measured_peak": peaks["mfma_i8_tops"],
                     "frac_of_measured_peak": round(achieved / peaks["mfma_i8_tops"], 4)}, **common)
    achieved = nbytes / t / 1e9
    return dict({"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                 "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                 "traffic": measured_traffic(M),
                 "measured_peak": peaks["hbm_read_GBs"],
                 "frac_of_measured_peak": round(achieved / peaks["hbm_read_GBs"], 4)}, **common)


def extras(torch, w8a8, stack, int8_layers, bf16_layers, lm_int8, lm_bf16, x_all, w_lm, M, D, F,
           V, NL, make_graph, time_graph, ops_int8, ops_all, step_sec, fp8_layers, lm_fp8,
           torch_ffn, peaks):
    dev = x_all.device
    groups = {}

    # --- the gate/up kernel at M = 128, where it is bound by HBM
    groups["gate_up_m128_hbm"] = gate_up_roofline(torch, w8a8, int8_layers,
                                                  x_all[:128].contiguous(), 128, D, F, NL,
                                                  make_graph, time_graph, peaks)

    # --- FFN block, decode and prefill, 26 distinct layers per timed pass
    for m in (1, 128, 2048):
        xm = (x_all[:m] if m <= x_all.shape[0] else
              x_all.repeat((m + x_all.shape[0] - 1) // x_all.shape[0], 1)[:m]).contiguous()
        y = torch.empty((m, D), dtype=torch.bfloat16, device=dev)
        ws8 = torch.empty(w8a8.ffn_workspace_bytes(m, D, F), dtype=torch.uint8, device=dev)
        wsb = torch.empty(w8a8.bf16_ffn_workspace_bytes(m, D, F), dtype=torch.uint8, device=dev)
        wsf = torch.empty(w8a8.fp8_ffn_workspace_bytes(m, D, F), dtype=torch.uint8, device=dev)
        g8 = make_graph(lambda: [w8a8.ffn(L, xm, out=y, ws=ws8) for L in int8_layers])
        gb = make_graph(lambda: [w8a8.bf16_ffn(L, xm, out=y, ws=wsb) for L in bf16_layers])
        gf = make_graph(lambda: [w8a8.fp8_ffn(L, xm, out=y, ws=wsf) for L in fp8_layers])

        def torch_block(wgu_t, wd_t):  # one GEMM for gate and up, GeGLU, down GEMM
            gu = torch.mm(xm, wgu_t)
            hh = torch.nn.functional.gelu(gu[:, :F], approximate="tanh") * gu[:, F:]
            torch.mm(hh, wd_t, out=y)
        gt = make_graph(lambda: [torch_block(a, b) for a, b in torch_ffn])
        t8 = time_graph(g8) / NL
        tb = time_graph(gb) / NL
        tf = time_graph(gf) / NL
        tt = time_graph(gt) / NL
        bytes8 = 3 * F * D + 2 * F * 4 + D * 4 + F * 4 + D * 4 + m * D * 2 * 2
        bytesb = 3 * F * D * 2 + m * D * 2 * 2
        ops = 6.0 * m * D * F
        groups["ffn_m%d" % m] = {
            "int8_us": round(t8 * 1e6, 2), "bf16_us": round(tb * 1e6, 2),
            "torch_bf16_us": round(tt * 1e6, 2),
            "speedup": round(tb / t8, 3), "speedup_vs_best_bf16": round(min(tb, tt) / t8, 3),
            "int8_GBs": round(bytes8 / t8 / 1e9, 1), "int8_hbm_frac": round(bytes8 / t8 / 1e9 / HBM_PEAK_GBS, 3),
            "bf16_GBs": round(bytesb / tb / 1e9, 1),
            "int8_tops": round(ops / t8 / 1e12, 1), "int8_mfma_frac": round(ops / t8 / 1e12 / INT8_PEAK_TOPS, 4),
            "fp8_us": round(tf * 1e6, 2), "fp8_speedup_vs_bf16": round(tb / tf, 3),
            "fp8_vs_int8": round(t8 / tf, 3),
            "note": "per FFN block incl. activation quant, GeGLU and requant; graph of 26 distinct layers"}
        del g8, gb, gf, gt
        log("ffn m=%d: int8 %.2f us, bf16 %.2f us, torch bf16 %.2f us, fp8 %.2f us"
            % (m, t8 * 1e6, tb * 1e6, tt * 1e6, tf * 1e6))

    # --- FFN GEMMs alone at M = 2048 (prefill), INT8 TOPS against the MFMA peak
    m = 2048
    xm = x_all.repeat((m + x_all.shape[0] - 1) // x_all.shape[0], 1)[:m].contiguous()
    qx, sx = w8a8.quantize_act(xm, int8_layers[0].gate.delta)
    h = torch.empty((m, F), dtype=torch.bfloat16, device=dev)
    qh, sh = w8a8.quantize_act(h.normal_(), int8_layers[0].down.delta)
    y = torch.empty((m, D), dtype=torch.bfloat16, device=dev)
    wsl = torch.empty(w8a8.linear_workspace_bytes(m, D, F), dtype=torch.uint8, device=dev)
    acc = torch.empty((m, D), dtype=torch.int32, device=dev)
    g_gu = make_graph(lambda: [w8a8.ffn_gate_up(L, qx, sx, m, out=h) for L in int8_layers])
    g_dn = make_graph(lambda: [w8a8.gemm_i8_i32(qh, m, L.down.wq, D, F, ws=wsl) for L in int8_layers])
    t_gu = time_graph(g_gu) / NL
    t_dn = time_graph(g_dn) / NL
    del g_gu, g_dn
    fqx, fsx = w8a8.fp8_quantize_act(xm, fp8_layers[0].gate.delta)
    fqh, _ = w8a8.fp8_quantize_act(h, fp8_layers[0].down.delta)
    wsf = torch.empty(w8a8.fp8_linear_workspace_bytes(m, D, F), dtype=torch.uint8, device=dev)
    f_gu = make_graph(lambda: [w8a8.fp8_ffn_gate_up(L, fqx, fsx, m, out=h) for L in fp8_layers])
    f_dn = make_graph(lambda: [w8a8.fp8_gemm_f32(fqh, m, L.down.wq, D, F, ws=wsf) for L in fp8_layers])
    tf_gu = time_graph(f_gu) / NL
    tf_dn = time_graph(f_dn) / NL
    del f_gu, f_dn
    groups["prefill_gemm_m2048"] = {
        "gate_up_us": round(t_gu * 1e6, 2), "gate_up_tops": round(4.0 * m * D * F / t_gu / 1e12, 1),
        "gate_up_mfma_frac": round(4.0 * m * D * F / t_gu / 1e12 / INT8_PEAK_TOPS, 4),
        "down_us": round(t_dn * 1e6, 2), "down_tops": round(2.0 * m * D * F / t_dn / 1e12, 1),
        "down_mfma_frac": round(2.0 * m * D * F / t_dn / 1e12 / INT8_PEAK_TOPS, 4),
        "fp8_gate_up_us": round(tf_gu * 1e6, 2), "fp8_down_us": round(tf_dn * 1e6, 2),
        "fp8_gate_up_tflops": round(4.0 * m * D * F / tf_gu / 1e12, 1),
        "fp8_down_tflops": round(2.0 * m * D * F / tf_dn / 1e12, 1)}
    log("prefill gemms m=2048: gate/up %.2f us, down %.2f us; fp8 %.2f / %.2f us"
        % (t_gu * 1e6, t_dn * 1e6, tf_gu * 1e6, tf_dn * 1e6))

    # --- attention projections (the same W8A8 linear on the attention shapes):
    # fused QKV 1152 -> 1536 (4 query heads + 1 key + 1 value head of 256, one
    # shared quantisation of x) and O 1024 -> 1152, 26 distinct layers per
    # timed pass, INT8 (quantisation included) vs our bf16 kernel vs torch.mm
    from paper_2608_28003_amd import synth
    NQ, NKV = 1024, 256
    NQKV = NQ + 2 * NKV
    att = []
    for l in range(NL):
        wqkv = torch.from_numpy(synth.to_bf16_bits(np.concatenate(
            [synth.normal(5100 + 4 * l + i, (n, D), synth.W_SIGMA) for i, n in enumerate((NQ, NKV, NKV))]))
            .view(np.int16)).view(torch.bfloat16).to(dev)
        wo = torch.from_numpy(synth.to_bf16_bits(synth.normal(5103 + 4 * l, (D, NQ), synth.W_SIGMA))
                              .view(np.int16)).view(torch.bfloat16).to(dev)
        att.append((wqkv, wo))
    xa_all = torch.from_numpy(synth.to_bf16_bits(synth.activations(
        5001, 256, D, synth.outlier_channels(5002, D, synth.n_outliers_1pct(D)), 30.0))
        .view(np.int16)).view(torch.bfloat16).to(dev)
    xo_all = torch.from_numpy(synth.to_bf16_bits(synth.activations(
        5007, 256, NQ, synth.outlier_channels(5009, NQ, synth.n_outliers_1pct(NQ)), 30.0))
        .view(np.int16)).view(torch.bfloat16).to(dev)
    qkv8 = [w8a8.LinearW8A8.from_weight(wq_, w8a8.smooth_calibrate(w8a8.col_absmax(xa_all), [wq_]))
            for wq_, _ in att]
    o8 = [w8a8.LinearW8A8.from_weight(wo_, w8a8.smooth_calibrate(w8a8.col_absmax(xo_all), [wo_]))
          for _, wo_ in att]
    qkv16 = [w8a8.pack_bf16(wq_) for wq_, _ in att]
    o16 = [w8a8.pack_bf16(wo_) for _, wo_ in att]
    qkv_t = [wq_.t().contiguous() for wq_, _ in att]
    o_t = [wo_.t().contiguous() for _, wo_ in att]
    for m in (1, 32, 256):
        entry = {}
        for name, xs_, L8, L16, Lt, n, k in (("qkv", xa_all, qkv8, qkv16, qkv_t, NQKV, D),
                                             ("o", xo_all, o8, o16, o_t, D, NQ)):
            xm = xs_[:m].contiguous()
            y = torch.empty((m, n), dtype=torch.bfloat16, device=dev)
            ws8 = torch.empty(max(1, w8a8.linear_workspace_bytes(m, n, k)), dtype=torch.uint8, device=dev)
            wsb_n = w8a8.bf16_linear_workspace_bytes(m, n, k)
            wsb = torch.empty(max(wsb_n, 1), dtype=torch.uint8, device=dev)
            g8 = make_graph(lambda: [w8a8.linear(L, xm, out=y, ws=ws8) for L in L8])
            gb = make_graph(lambda: [w8a8.bf16_linear(xm, wp, n, k, out=y, ws=wsb if wsb_n else None)
                                     for wp in L16])
            gt = make_graph(lambda: [torch.mm(xm, wt, out=y) for wt in Lt])
            t8, tb, tt = time_graph(g8) / NL, time_graph(gb) / NL, time_graph(gt) / NL
            del g8, gb, gt
            b8 = n * k + n * 4 + k * 4 + m * k * 2 + m * n * 2
            entry[name] = {"int8_us": round(t8 * 1e6, 2), "bf16_us": round(tb * 1e6, 2),
                           "torch_bf16_us": round(tt * 1e6, 2),
                           "speedup_vs_best_bf16": round(min(tb, tt) / t8, 3),
                           "int8_GBs": round(b8 / t8 / 1e9, 1),
                           "int8_tops": round(2.0 * m * n * k / t8 / 1e12, 2)}
        entry["note"] = ("per call incl. activation quantisation; 26 distinct layers per pass "
                         "(the INT8 weights, 46 MB, stay in the 256 MB memory-side cache)")
        groups["attn_proj_m%d" % m] = entry
    log("attention projections: " + ", ".join(
        "m=%d qkv %.2f/%.2f us o %.2f/%.2f us (int8/best bf16)" % (
            m, groups["attn_proj_m%d" % m]["qkv"]["int8_us"],
            min(groups["attn_proj_m%d" % m]["qkv"]["bf16_us"], groups["attn_proj_m%d" % m]["qkv"]["torch_bf16_us"]),
            groups["attn_proj_m%d" % m]["o"]["int8_us"],
            min(groups["attn_proj_m%d" % m]["o"]["bf16_us"], groups["attn_proj_m%d" % m]["o"]["torch_bf16_us"]))
        for m in (1, 32, 256)))

    # --- decode attention with a key/value cache (Sec. 2 layout: 4 query heads,
    # one key/value head of 256; Sec. 4: INT8 cache).  The kernel alone at a
    # few context lengths, INT8 cache vs bf16 cache, then 26 attention blocks
    # at one token (fused QKV projection, append-and-attend over the layer's
    # cache, O projection) under the attention layer sets Q_ATT, with the
    # global layers (0, 6, 12, 18) attending the whole context and the others
    # the last 1024 rows.
    HD = w8a8.HEAD_DIM
    attn_kernel = {}
    for T in (1024, 4096, 32768):
        kvd = synth.kv_decode_inputs(5800, T - 1)
        kt = torch.from_numpy(kvd["k"].view(np.int16)).view(torch.bfloat16).to(dev)
        vt = torch.from_numpy(kvd["v"].view(np.int16)).view(torch.bfloat16).to(dev)
        qkv1 = torch.from_numpy(kvd["qkv"].view(np.int16)).view(torch.bfloat16).to(dev)
        wsa = torch.empty(max(1, w8a8.attn_decode_workspace_bytes(T)), dtype=torch.uint8, device=dev)
        outa = torch.empty(NQ, dtype=torch.bfloat16, device=dev)
        ent = {}
        for kind in ("int8", "bf16"):
            cache = w8a8.KVCache(T, kind == "int8", dev)
            cache.fill(0, kt, vt)
            # 26 calls per replay (one per layer of a step), so the graph's own
            # launch is not charged to one call
            g = make_graph(lambda: [w8a8.attn_decode(qkv1, cache, T - 1, T, out=outa, ws=wsa)
                                    for _ in range(NL)])
            t = time_graph(g) / NL
            del g, cache
            row = 2 * HD + 8 if kind == "int8" else 4 * HD   # key + value codes and scales, or bf16
            ent[kind + "_us"] = round(t * 1e6, 2)
            ent[kind + "_GBs"] = round(T * row / t / 1e9, 1)
        ent["speedup_int8_cache"] = round(ent["bf16_us"] / ent["int8_us"], 3)
        attn_kernel["t%d" % T] = ent
        del kt, vt, wsa
    groups["attn_decode_kernel"] = attn_kernel
    log("attention decode kernel: " + ", ".join("T=%s int8 %.2f us (%.0f GB/s) bf16 %.2f us" % (
        k[1:], v["int8_us"], v["int8_GBs"], v["bf16_us"]) for k, v in attn_kernel.items()))

    CTX = 4096
    kvd = synth.kv_decode_inputs(5900, CTX - 1)
    kt = torch.from_numpy(kvd["k"].view(np.int16)).view(torch.bfloat16).to(dev)
    vt = torch.from_numpy(kvd["v"].view(np.int16)).view(torch.bfloat16).to(dev)
    caches = {}
    for kind in ("int8", "bf16"):
        caches[kind] = [w8a8.KVCache(CTX, kind == "int8", dev) for _ in range(NL)]
        for c in caches[kind]:
            c.fill(0, kt, vt)
    del kt, vt
    x1a = xa_all[:1].contiguous()
    qkv_b = torch.empty((1, NQKV), dtype=torch.bfloat16, device=dev)
    att_b = torch.empty((1, NQ), dtype=torch.bfloat16, device=dev)
    o_b = torch.empty((1, D), dtype=torch.bfloat16, device=dev)
    wsa = torch.empty(max(1, w8a8.attn_decode_workspace_bytes(CTX)), dtype=torch.uint8, device=dev)
    nb = max(w8a8.linear_workspace_bytes(1, NQKV, D), w8a8.linear_workspace_bytes(1, D, NQ),
             w8a8.bf16_linear_workspace_bytes(1, NQKV, D), w8a8.bf16_linear_workspace_bytes(1, D, NQ))
    wsl = torch.empty(max(1, nb), dtype=torch.uint8, device=dev)
    windows = [CTX if l in (0, 6, 12, 18) else 1024 for l in range(NL)]

    def blocks(prec, kind):
        for l in range(NL):
            if prec[l]:
                w8a8.linear(qkv8[l], x1a, out_dtype=torch.bfloat16, out=qkv_b, ws=wsl)
            else:
                w8a8.bf16_linear(x1a, qkv16[l], NQKV, D, out=qkv_b, ws=wsl)
            w8a8.attn_decode(qkv_b.view(-1), caches[kind][l], CTX - 1, windows[l], out=att_b.view(-1),
                             ws=wsa)
            if prec[l]:
                w8a8.linear(o8[l], att_b, out_dtype=torch.bfloat16, out=o_b, ws=wsl)
            else:
                w8a8.bf16_linear(att_b, o16[l], D, NQ, out=o_b, ws=wsl)

    att_maps = {}
    for name in ("none", "5+5", "10+10", "all26"):
        prec = w8a8.precision_map("bf16" if name == "none" else name)
        for kind in ("bf16", "int8"):
            g = make_graph(lambda: blocks(prec, kind))
            att_maps["Q_ATT %s, %s cache" % (name, kind)] = round(time_graph(g) * 1e6, 1)
            del g
    groups["attn_blocks_m1_ctx%d" % CTX] = {
        "us_per_step_26_blocks": att_maps,
        "note": "one token; per layer QKV projection + append-and-attend + O projection; "
                "global layers 0, 6, 12, 18 attend %d rows, the others 1024" % CTX}
    log("attention blocks at one token, context %d: " % CTX
        + ", ".join("%s %.1f us" % kv for kv in att_maps.items()))
    del caches, wsa, wsl
    del att, qkv8, o8, qkv16, o16, qkv_t, o_t

    # --- lm_head decode: INT8 vs our bf16 kernel vs torch.mm (hipBLASLt) bf16.
    # Each timed replay walks through copies of the weights (3 x 302 MB INT8,
    # 2 x 604 MB bf16; the memory-side cache holds 256 MB), so every call
    # reads its weights from HBM.
    n8, nb = 3, 2
    import ctypes
    from paper_2608_28003_amd import build as hip_build
    PL = ctypes.CDLL(hip_build.PEAK_LIB_PATH)
    PL.w8a8_peak_read_write.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                                        ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    sink = torch.zeros(1, dtype=torch.int32, device=dev)

    def rw_floor(wq, lg, m):
        rc = PL.w8a8_peak_read_write(ctypes.c_void_p(wq.data_ptr()), V, D, ctypes.c_void_p(lg.data_ptr()),
                                     m, 1024, ctypes.c_void_p(sink.data_ptr()),
                                     ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if rc != 0:
            raise RuntimeError("read/write probe failed: %d" % rc)

    lm8s = [lm_int8] + [w8a8.LinearW8A8(lm_int8.n, lm_int8.k, lm_int8.wq.clone(), lm_int8.s_w.clone(),
                                        lm_int8.delta) for _ in range(n8 - 1)]
    lmfs = [lm_fp8] + [w8a8.LinearW8A8(lm_fp8.n, lm_fp8.k, lm_fp8.wq.clone(), lm_fp8.s_w.clone(),
                                       lm_fp8.delta) for _ in range(n8 - 1)]
    lmbs = [lm_bf16] + [lm_bf16.clone() for _ in range(nb - 1)]
    w_lm_ts = [w_lm.t().contiguous() for _ in range(nb)]   # d x V, plain right operands
    for m in (1, 8, 64):
        xm = x_all[:m].contiguous()
        lg = torch.empty((m, V), dtype=torch.bfloat16, device=dev)
        ws8 = torch.empty(w8a8.lm_head_workspace_bytes(m, V, D), dtype=torch.uint8, device=dev)
        wsb_n = w8a8.bf16_linear_workspace_bytes(m, V, D)
        wsb = torch.empty(max(wsb_n, 1), dtype=torch.uint8, device=dev)
        wsf = torch.empty(w8a8.fp8_linear_workspace_bytes(m, V, D), dtype=torch.uint8, device=dev)
        g8 = make_graph(lambda: [w8a8.lm_head(L, xm, out=lg, ws=ws8) for L in lm8s])
        gb = make_graph(lambda: [w8a8.bf16_linear(xm, wp, V, D, out=lg, ws=wsb if wsb_n else None)
                                 for wp in lmbs])
        gt = make_graph(lambda: [torch.mm(xm, wt, out=lg) for wt in w_lm_ts])
        gf = make_graph(lambda: [w8a8.fp8_lm_head(L, xm, out=lg, ws=wsf) for L in lmfs])
        # the same weight bytes read and the same logits written by a kernel
        # that does no arithmetic: the practical floor of this call
        gp = make_graph(lambda: [rw_floor(L.wq, lg, m) for L in lm8s])
        tp = time_graph(gp) / n8
        t8 = time_graph(g8) / n8
        tb = time_graph(gb) / nb
        tt = time_graph(gt) / nb
        tf = time_graph(gf) / n8
        b8 = V * D + V * 4 + D * 4 + m * D * 2 + m * V * 2
        bb = V * D * 2 + m * D * 2 + m * V * 2
        groups["lm_head_m%d" % m] = {
            "int8_us": round(t8 * 1e6, 2), "bf16_ours_us": round(tb * 1e6, 2),
            "bf16_torch_us": round(tt * 1e6, 2), "speedup": round(min(tb, tt) / t8, 3),
            "int8_GBs": round(b8 / t8 / 1e9, 1), "int8_hbm_frac": round(b8 / t8 / 1e9 / HBM_PEAK_GBS, 3),
            "int8_frac_of_measured_read": round(b8 / t8 / 1e9 / peaks["hbm_read_GBs"], 3),
            "read_write_floor_us": round(tp * 1e6, 2),
            "int8_frac_of_read_write_floor": round(tp / t8, 3),
            "bf16_best_GBs": round(bb / min(tb, tt) / 1e9, 1),
            "fp8_us": round(tf * 1e6, 2), "fp8_GBs": round(b8 / tf / 1e9, 1),
            "note": "median of 15; each replay rotates over %d INT8 / %d bf16 weight copies" % (n8, nb)}
        del g8, gb, gt, gf, gp
        log("lm_head m=%d: int8 %.2f us, bf16 ours %.2f us, torch %.2f us, fp8 %.2f us, "
            "read+write floor %.2f us" % (m, t8 * 1e6, tb * 1e6, tt * 1e6, tf * 1e6, tp * 1e6))
    del w_lm_ts, lm8s, lmfs, lmbs

    # --- the paper's precision maps on the whole step: at the step's M and at
    # the 26-layer stack's prefill sizes M = 512 and 2048 (token rows repeat
    # the synthetic ones beyond the rows drawn; rows are independent)
    for mm in sorted({M, 512, 2048}):
        xm = (x_all[:mm] if mm <= x_all.shape[0] else
              x_all.repeat((mm + x_all.shape[0] - 1) // x_all.shape[0], 1)[:mm]).contiguous()
        out = torch.empty((mm, V), dtype=torch.bfloat16, device=dev)
        ws = torch.empty(w8a8.stack_workspace_bytes(mm, D, F, V), dtype=torch.uint8, device=dev)
        maps = {}
        base = None
        for name, mp, lm8 in [("bf16", "bf16", False), ("lm_head only", "bf16", True),
                              ("FFN 5+5", "5+5", False), ("FFN 5+5 + lm_head", "5+5", True),
                              ("FFN 10+10 + lm_head", "10+10", True), ("FFN all26", "all26", False),
                              ("FFN all26 + lm_head", "all26", True)]:
            prec = w8a8.precision_map(mp)
            gs = make_graph(lambda: stack.run(xm, prec, lm8, out=out, ws=ws))
            ts = time_graph(gs)
            del gs
            if base is None:
                base = ts
            maps[name] = {"ms": round(ts * 1e3, 4), "speedup_vs_bf16": round(base / ts, 3),
                          "effective_tops": round(ops_all(mm) / ts / 1e12, 1)}
        groups["stack_maps_m%d" % mm] = maps
        del out, ws
        log("stack at M=%d: " % mm + ", ".join("%s %.3f ms" % (k, v["ms"]) for k, v in maps.items()))
    # the same maps at decode (one token per step: the paper's batch-1 setting)
    x1 = x_all[:1].contiguous()
    out1 = torch.empty((1, V), dtype=torch.bfloat16, device=dev)
    ws1 = torch.empty(w8a8.stack_workspace_bytes(1, D, F, V), dtype=torch.uint8, device=dev)
    def weight_bytes(prec, lm8):
        # bytes of weights, scales and smoothing factors one decode step streams
        n8 = int(np.sum(prec))
        b = n8 * (3 * F * D + (2 * F + D) * 4 + (D + F) * 4) + (NL - n8) * 3 * F * D * 2
        return b + (V * D + 4 * V + 4 * D if lm8 else 2 * V * D)

    maps1, base1 = {}, None
    for name, mp, lm8 in [("bf16", "bf16", False), ("lm_head only", "bf16", True),
                          ("FFN 5+5 + lm_head", "5+5", True), ("FFN 10+10 + lm_head", "10+10", True),
                          ("FFN all26 + lm_head", "all26", True)]:
        prec = w8a8.precision_map(mp)
        gs = make_graph(lambda: stack.run(x1, prec, lm8, out=out1, ws=ws1))
        ts = time_graph(gs)
        del gs
        if base1 is None:
            base1 = ts
        wb = weight_bytes(prec, lm8)
        maps1[name] = {"us": round(ts * 1e6, 1), "speedup_vs_bf16": round(base1 / ts, 3),
                       "weight_GBs": round(wb / ts / 1e9, 1)}
    # the INT8 runs of layers take the persistent decode kernel; the same step
    # with one launch per GEMM, for reference
    prec = w8a8.precision_map("all26")
    w8a8.set_plan_override("NO_PERSISTENT", 1)
    gs = make_graph(lambda: stack.run(x1, prec, True, out=out1, ws=ws1))
    w8a8.clear_plan_overrides()
    ts = time_graph(gs)
    del gs
    maps1["FFN all26 + lm_head, one launch per GEMM"] = {
        "us": round(ts * 1e6, 1), "speedup_vs_bf16": round(base1 / ts, 3),
        "weight_GBs": round(weight_bytes(prec, True) / ts / 1e9, 1)}
    groups["stack_maps_m1"] = maps1
    # one decode step composed of separately timed parts: the FFN stack with
    # its lm_head (above) and the 26 attention blocks (projections + cache)
    att = groups["attn_blocks_m1_ctx4096"]["us_per_step_26_blocks"]
    composed = {}
    for name, ffn_key, att_key in [
            ("bf16", "bf16", "Q_ATT none, bf16 cache"),
            ("FFN 5+5 + lm_head", "FFN 5+5 + lm_head", "Q_ATT none, bf16 cache"),
            ("FFN all26 + lm_head", "FFN all26 + lm_head", "Q_ATT none, bf16 cache"),
            ("Attn+FFN 5+5 (Q_ATT all26) + lm_head", "FFN 5+5 + lm_head", "Q_ATT all26, bf16 cache"),
            ("Attn+FFN all26 + lm_head", "FFN all26 + lm_head", "Q_ATT all26, bf16 cache"),
            ("Attn+FFN all26 + lm_head + INT8 cache", "FFN all26 + lm_head", "Q_ATT all26, int8 cache"),
            ("Attn 5+5 + FFN 5+5 + lm_head + INT8 cache", "FFN 5+5 + lm_head", "Q_ATT 5+5, int8 cache")]:
        composed[name] = round(maps1[ffn_key]["us"] + att[att_key], 1)
    base_c = composed["bf16"]
    groups["decode_step_composed_ctx4096"] = {
        k: {"us": v, "speedup_vs_bf16": round(base_c / v, 3)} for k, v in composed.items()}
    log("composed decode step (context 4096): " + ", ".join("%s %.1f us" % kv for kv in composed.items()))
    # layer sensitivity (SQNR, dB) on 64 tokens and automatically chosen maps,
    # timed at the step's M against its all-bf16 step
    xm = x_all[:M].contiguous()
    out = torch.empty((M, V), dtype=torch.bfloat16, device=dev)
    ws = torch.empty(w8a8.stack_workspace_bytes(M, D, F, V), dtype=torch.uint8, device=dev)
    base = groups["stack_maps_m%d" % M]["bf16"]["ms"] * 1e-3
    xs = x_all[:64].contiguous()
    iso, prop = stack.sensitivity(xs, w8a8.precision_map("all26"))
    auto = {}
    for budget in (30.0, 40.0):
        prec, db = stack.select_map(xs, budget)
        gs = make_graph(lambda: stack.run(xm, prec, True, out=out, ws=ws))
        ts = time_graph(gs)
        del gs
        auto["budget_%g_db" % budget] = {
            "int8_layers": [int(i) for i in np.flatnonzero(prec)], "sqnr_db": round(db, 2),
            "ms_m%d" % M: round(ts * 1e3, 4), "speedup_vs_bf16": round(base / ts, 3)}
    groups["sensitivity_m64"] = {"isolated_db": [round(float(v), 2) for v in iso],
                                 "propagated_all26_db": [round(float(v), 2) for v in prop],
                                 "auto_maps": auto}
    log("auto maps: " + ", ".join("%s: %d INT8 layers, %.1f dB" % (k, len(v["int8_layers"]), v["sqnr_db"])
                                  for k, v in auto.items()))
    log("stack at M=1: " + ", ".join("%s %.1f us" % (k, v["us"]) for k, v in maps1.items()))
    groups["paper_context"] = {"note": "RTX 5090 + TensorRT-LLM, end-to-end decode tok/s at batch 1; not a target",
                               "FFN 5+5 + lm_head": 1.110, "FFN all26 + lm_head": 1.191}
    return groups


def cpu_baseline(M):
    """The oracle, untouched, on a bounded sample of the step: one INT8 FFN
    block (1152 -> 6912 -> 1152, smoothing factors calibrated by the oracle
    on 512 tokens) at the step's M, passes on all OpenMP threads until about
    8 s have been spent (at least 5, at most 30; the median is reported);
    and one pass on a single thread at M = 256."""
    import ctypes
    import oracle
    from paper_2608_28003_amd import synth
    oracle.build()
    cfg = synth.ffn_config(m=M)
    q = oracle.quantize_ffn(cfg["w_gate"], cfg["w_up"], cfg["w_down"], cfg["x_cal"])
    ops = 6.0 * M * synth.D_MODEL * synth.D_FF
    oracle.w8a8_ffn(cfg["x"][:16], q)   # thread pool up
    ts = []
    while len(ts) < 5 or (sum(ts) < 8.0 and len(ts) < 30):
        t0 = time.perf_counter()
        oracle.w8a8_ffn(cfg["x"], q)
        ts.append(time.perf_counter() - t0)
    t_med = float(np.median(ts))
    omp = ctypes.CDLL("libgomp.so.1")
    omp.omp_get_max_threads.restype = ctypes.c_int
    threads = omp.omp_get_max_threads()
    m1 = min(M, 256)
    omp.omp_set_num_threads(1)
    try:
        t0 = time.perf_counter()
        oracle.w8a8_ffn(cfg["x"][:m1], q)
        t1 = time.perf_counter() - t0
    finally:
        omp.omp_set_num_threads(threads)
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(ops / t_med / 1e12, 5), "unit": "TOPS", "cores": threads,
            "kind": "oracle", "cpu": model,
            "single_thread_tops": round(6.0 * m1 * synth.D_MODEL * synth.D_FF / t1 / 1e12, 6),
            "sample": "one INT8 FFN block (1152 -> 6912 -> 1152) of the 26 in the step, M=%d, "
                      "oracle C loops with OpenMP on %d threads: median of %d passes %.2f s "
                      "(%.1f s in all; the step runs 26 such blocks + the lm_head); single "
                      "thread at M=%d: %.2f s" % (M, threads, len(ts), t_med, sum(ts), m1, t1)}


if __name__ == "__main__":
    main()
