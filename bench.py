#!/usr/bin/env python3
"""Benchmark of the phase-specific quantized linear layer on one MI355X.

Workload: the 8B-scale MLP up-projection (Qwen3-8B shape: K = d_model = 4096,
N = d_ffn x 3 = 12288), prefill M = 2048 tokens with 0.5 % outlier channels
x30, decode batches 1 and 4; weights 0.02 N(0,1) with a log-normal row scale.
Inputs are seeded synthetic tensors already resident in HBM.

One step = the whole per-token hot path over one batch:
  1. NVFP4 activation quantization of X [2048, 4096] (static global scale),
  2. W4A4 NVFP4 GEMM -> bf16 Y [2048, 12288],
  3. LUT3 decode GEMV at batch 1 and at batch 4 (fp32 y).
Weight packing (NVFP4 and per-row LUT3) is offline and timed separately.

The decode weights of a step rotate over enough packed copies (>= 768 MiB)
that every GEMV streams its weights from HBM rather than from the 256 MiB
Infinity Cache; the activations X rotate over 16 copies for the same reason.

Besides the step, the run measures a decode sweep outside the timed steps:
one decode token through 64 stacked 27B-class blocks (q/k/v 7168x5120,
o 5120x5120, gate/up 34816x5120, down 5120x17408: 7.93 GB of LUT3 codes, all
distinct memory) at batch 1, 8 and 16, and the same in LUT2 at batch 1.

Prints one JSON line.  `ms_per_step` is the time of the timed steps (HIP
events on the launch stream around them, nothing else in between).  `value`
is the prefill linear throughput: 2*M*N*K over (quantization + GEMM) time,
each measured as back-to-back calls of that kernel alone between one pair of
events (the average includes the GPU-side gap between launches, no host or
event overhead); the GEMV rates are measured the same way.

`--calibrate-copy` instead runs a plain 256 MiB device copy five times: the
reference kernel whose FETCH_SIZE / WRITE_SIZE readings scale the GEMM's
counters into bytes (profiles/).
"""
import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "NVFP4 prefill GEMM TFLOPS (%FP4 peak); LUT3 decode GEMV GB/s (%HBM peak)"
PEAK_FP16_TFLOPS = 2500.0      # dense fp16/bf16 MFMA, MI355X
PEAK_FP4_TFLOPS = 10100.0      # dense fp4 MFMA, MI355X
PEAK_HBM_GBS = 8000.0
# sources that decide the GEMM's kernels and launches (tile geometry, column split)
GEMM_SOURCES = [os.path.join(ROOT, "paper_2609_26333_amd", "csrc", f) for f in ("gemm.hip", "dq_internal.hpp")]
GEMM_COUNTERS = os.path.join(ROOT, "profiles", "nvfp4_gemm_8b_up_proj_counters.md")
COPY_BYTES = 256 << 20


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-decode-sweep", action="store_true")
    p.add_argument("--sweep-blocks", type=int, default=64)
    p.add_argument("--decode-bytes", type=int, default=768 << 20,
                   help="total bytes of rotated decode weight copies")
    p.add_argument("--calibrate-copy", action="store_true")
    return p.parse_args()


def gemm_source_sha256():
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def gemm_traffic():
    """HBM bytes per GEMM call from the committed counter summary: the
    FETCH_SIZE and WRITE_SIZE readings of the call's kernel launches (a
    full-tile launch and, for a partial last round, a half-width-tile launch),
    each scaled by the bytes a plain copy of known size moves per KiB that the
    same counter reads.  None when the summary is missing or the GEMM sources
    have changed since."""
    try:
        text = open(GEMM_COUNTERS).read()
    except OSError:
        return None
    fields = dict(re.findall(r"^- `(\w+)`: `([^`]+)`", text, re.M))
    if fields.get("gemm_source_sha256") != gemm_source_sha256():
        return None
    try:
        fetch = float(fields["gemm_fetch_kib"]) * float(fields["fetch_bytes_per_kib"])
        write = float(fields["gemm_write_kib"]) * float(fields["write_bytes_per_kib"])
    except (KeyError, ValueError):
        return None
    return fetch + write


def calibrate_copy():
    import torch
    torch.cuda.set_device(0)
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read": COPY_BYTES, "bytes_written": COPY_BYTES,
                      "launches": 5}), flush=True)


def cpu_baseline(cfg, w, X, G_x, xds, min_seconds=10.0):
    """Time the CPU oracle on the same workload: the whole prefill layer
    (activation quantization + fp64 GEMM over the dequantized operands) and
    the batch-1 and batch-4 LUT3 GEMVs, repeated until min_seconds have
    passed.  Weight packing is offline and untimed."""
    from threadpoolctl import threadpool_info

    from oracle import linalg, lut, nvfp4
    qw, cw, Gw = nvfp4.quantize_dynamic(w)
    codes, table = lut.quantize_per_row(w, 3)
    w_hat = nvfp4.dequantize(qw, cw, Gw)
    M, K = X.shape
    N = w.shape[0]
    t_pre = t_dec = 0.0
    reps = 0
    start = time.perf_counter()
    while reps == 0 or time.perf_counter() - start < min_seconds:
        t0 = time.perf_counter()
        qa, ca, _ = nvfp4.quantize_bf16_activations(X, G_x)
        Y = linalg.gemm(nvfp4.dequantize(qa, ca, G_x), w_hat)
        t1 = time.perf_counter()
        for xd in xds.values():
            linalg.lut_gemv_per_row(xd, codes, table)
        t_pre += t1 - t0
        t_dec += time.perf_counter() - t1
        reps += 1
        del Y
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    dec_bytes = sum(N * K * 3 / 8 + N * 16 + xd.size * 2 + xd.shape[0] * N * 4 for xd in xds.values())
    return {
        "value": 2.0 * M * N * K * reps / t_pre / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
        "sample": (f"the whole layer {reps} times: NVFP4 quantization of X[{M},{K}] + fp64 GEMM against all "
                   f"{N} weight rows ({t_pre / reps:.2f} s each); decode: LUT3 dequantization + fp64 GEMV at "
                   f"batch {' and '.join(str(b) for b in xds)} ({t_dec / reps:.2f} s each, "
                   f"{dec_bytes * reps / t_dec / 1e9:.3f} GB/s); weight packing untimed"),
        "decode_gbps": dec_bytes * reps / t_dec / 1e9,
    }


def mxfp4_prefill(dq, torch, np, w, Xs, M, N, K, s, reps):
    """The MXFP4 W4A4 variant of the same prefill linear (OCP MX: E8M0 scale
    per 32, block scales applied inside the FP4 MFMA), timed apart from the
    NVFP4 steps: activation quantization and GEMM with HIP events around
    `reps` calls of each."""
    lib = dq.lib()
    sp = ctypes.c_void_p(s.cuda_stream)
    Wm = dq.dq_pack_mxfp4(torch.from_numpy(np.ascontiguousarray(w)).cuda())
    A = dq.MxFp4Tensor.empty(M, K)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    dA, dW = A.desc(), Wm.desc()
    n_x = len(Xs)

    def quant(i):
        return lib.dq_quantize_act_mxfp4(ctypes.c_void_p(Xs[i % n_x].data_ptr()), M, K, ctypes.byref(dA), sp)

    def gemm():
        return lib.dq_prefill_gemm_mxfp4(ctypes.byref(dA), ctypes.byref(dW), dq.OUT_BF16,
                                         ctypes.c_void_p(Y.data_ptr()), sp)
    for i in range(3):
        assert quant(i) == 0 and gemm() == 0
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ev[0].record(s)
    for i in range(reps):
        assert quant(i) == 0
    ev[1].record(s)
    for _ in range(reps):
        assert gemm() == 0
    ev[2].record(s)
    torch.cuda.synchronize()
    t_q = ev[0].elapsed_time(ev[1]) / reps * 1e-3
    t_g = ev[1].elapsed_time(ev[2]) / reps * 1e-3
    flops = 2.0 * M * N * K
    return {"quant_us": t_q * 1e6, "quant_GB/s": M * K * (2 + 0.5 + 1 / 32) / t_q / 1e9,
            "gemm_us": t_g * 1e6, "gemm_TFLOP/s": flops / t_g / 1e12,
            "frac_fp4_peak": flops / t_g / 1e12 / PEAK_FP4_TFLOPS,
            "linear_TFLOP/s_incl_quant": flops / (t_q + t_g) / 1e12,
            "note": "MXFP4 W4A4 (E2M1, E8M0 per 32 along K) on the scaled FP4 MFMA; same shapes and bf16 output"}


def nvfp4a16_decode(dq, torch, np, Wq, xd_dev, Bs, N, K, s, decode_bytes, reps):
    """Weight-only NVFP4 decode GEMV (format-disaggregated NVFP4) over the same
    packed NVFP4 weights the prefill GEMM uses, at the decode batches, with
    the weights rotated over enough copies to stream from HBM."""
    lib = dq.lib()
    sp = ctypes.c_void_p(s.cuda_stream)
    nbytes = Wq.codes.numel() + Wq.scales.numel()
    n_w = max(2, -(-decode_bytes // nbytes))
    Ws = [Wq] + [dq.NvFp4Tensor(Wq.codes.clone(), Wq.scales.clone(), Wq.G.clone(), N, K) for _ in range(n_w - 1)]
    ds = [x.desc() for x in Ws]
    out = {}
    for b in Bs:
        y = torch.empty((b, N), dtype=torch.float32, device="cuda")
        ws_n = dq.dq_decode_gemv_nvfp4_workspace_size(b, Wq)
        ws = torch.empty(max(ws_n, 16), dtype=torch.uint8, device="cuda")
        args_ = (ctypes.c_void_p(xd_dev[b].data_ptr()), b)
        call = lambda i: lib.dq_decode_gemv_nvfp4(*args_, ctypes.byref(ds[i % n_w]), dq.OUT_F32,  # noqa: E731
                                                 ctypes.c_void_p(y.data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                                                 ws_n, sp)
        for i in range(n_w):
            assert call(i) == 0
        torch.cuda.synchronize()
        ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ea.record(s)
        for i in range(reps):
            call(i)
        eb.record(s)
        torch.cuda.synchronize()
        t = ea.elapsed_time(eb) / reps * 1e-3
        alg = nbytes + b * K * 2 + b * N * 4
        out[f"b{b}"] = {"us": t * 1e6, "GB/s": alg / t / 1e9, "frac_hbm": alg / t / 1e9 / PEAK_HBM_GBS,
                        "bytes": alg}
    out["weight_copies"] = n_w
    out["note"] = "NVFP4 weights (4.5 bits), bf16 x, fp16 MFMA; back-to-back calls; one launch per call at these batches (K split inside each workgroup)"
    return out


def decode_sweep(dq, synth, torch, np, n_blocks, steps):
    """One decode token through n_blocks stacked 27B-class blocks (distinct
    copies of one packed block), LUT3 at batch 1, 8, 16 and LUT2 at batch 1."""
    cfg = synth.CONFIGS[4]
    lib = dq.lib()
    s = torch.cuda.current_stream()
    sp = ctypes.c_void_p(s.cuda_stream)
    out = {}
    Ws = [torch.from_numpy(synth.layer_weight(cfg, layer)).cuda() for layer in cfg.layers]
    for bits, batches in ((3, (1, 8, 16)), (2, (1,))):
        block = [dq.dq_pack_lut3(W, bits=bits, mode=dq.LUT_PER_ROW) for W in Ws]
        if bits == 2:
            del Ws
        stack = [block] + [[dq.LutWeight(l.codes.clone(), l.lut.clone(), None, None, l.rows, l.cols, bits,
                                         dq.LUT_PER_ROW) for l in block] for _ in range(n_blocks - 1)]
        descs = [[l.desc() for l in blk] for blk in stack]
        wbytes = sum(l.codes.numel() + l.lut.numel() * 2 for blk in stack for l in blk)
        for B in batches:
            xs = [torch.from_numpy(synth.decode_x(cfg, l.k, B).view(np.int16)).cuda() for l in cfg.layers]
            ys = [torch.empty((B, l.n), dtype=torch.float32, device="cuda") for l in cfg.layers]
            xp = [ctypes.c_void_p(t.data_ptr()) for t in xs]
            yp = [ctypes.c_void_p(t.data_ptr()) for t in ys]
            ws_n = max(dq.dq_decode_gemv_workspace_size(B, l) for l in block)
            ws = torch.empty(max(ws_n, 16), dtype=torch.uint8, device="cuda")
            wsp = ctypes.c_void_p(ws.data_ptr())

            def token():
                for d in descs:
                    for i in range(len(cfg.layers)):
                        assert lib.dq_decode_gemv(xp[i], B, ctypes.byref(d[i]), dq.OUT_F32, yp[i], wsp, ws_n,
                                                  sp) == 0
            token()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(steps):
                token()
            e1.record(s)
            torch.cuda.synchronize()
            t = e0.elapsed_time(e1) / steps * 1e-3
            io = n_blocks * sum(B * l.k * 2 + B * l.n * 4 for l in cfg.layers)
            gbs = (wbytes + io) / t / 1e9
            out[f"lut{bits}_b{B}"] = {"ms_per_token": t * 1e3, "GB/s": gbs, "frac_hbm": gbs / PEAK_HBM_GBS,
                                      "weight_bytes": wbytes, "gemv_launches": n_blocks * len(cfg.layers)}
        del stack, descs, block
        torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the kernels run on one GPU (one GPU's share of a sharded layer); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy()
        return
    import numpy as np
    import torch

    import paper_2609_26333_amd as dq
    import synth

    torch.cuda.set_device(0)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()   # noqa: E731
    cfg = synth.CONFIGS[1]
    layer = cfg.layers[0]
    M, N, K = cfg.m, layer.n, layer.k
    Bs = cfg.decode_batches

    w = synth.layer_weight(cfg, layer)
    X = synth.prefill_x(cfg, K)
    calib = synth.prefill_x(cfg, K, calib=True)
    xds = {b: synth.decode_x(cfg, K, b) for b in Bs}

    W_dev = dev(w)
    s = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    Wq = dq.dq_pack_nvfp4(W_dev)
    e1.record()
    torch.cuda.synchronize()
    t_pack_nvfp4 = e0.elapsed_time(e1)
    e0.record()
    Wl = dq.dq_pack_lut3(W_dev, bits=3, mode=dq.LUT_PER_ROW)
    e1.record()
    torch.cuda.synchronize()
    t_pack_lut = e0.elapsed_time(e1)
    del W_dev
    # LUT -> NVFP4 autocast of the packed LUT3 weight (the prefill view of a LUT model), once warm
    dq.dq_autocast_lut_to_nvfp4(Wl)
    torch.cuda.synchronize()
    e0.record()
    Wac = dq.dq_autocast_lut_to_nvfp4(Wl)
    e1.record()
    torch.cuda.synchronize()
    t_autocast = e0.elapsed_time(e1)
    del Wac

    # static activation scale from a calibration batch (running-max observer stand-in)
    A_cal = dq.dq_quantize_act_nvfp4(dev(calib.view(np.int16)))
    G_x = A_cal.G.clone()
    torch.cuda.synchronize()
    G_x_host = float(G_x.cpu()[0])

    # rotation buffers
    n_x = 16
    Xs = [dev(X.view(np.int16)) for _ in range(n_x)]
    lut_bytes = Wl.codes.numel() + Wl.lut.numel() * 2
    n_w = max(2, -(-args.decode_bytes // lut_bytes))
    Wls = [Wl] + [dq.LutWeight(Wl.codes.clone(), Wl.lut.clone(), None, None, N, K, 3, dq.LUT_PER_ROW)
                  for _ in range(n_w - 1)]
    xd_dev = {b: dev(xds[b].view(np.int16)) for b in Bs}
    A = dq.NvFp4Tensor.empty(M, K)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    ys = {b: torch.empty((b, N), dtype=torch.float32, device="cuda") for b in Bs}

    # prebuilt raw C-ABI calls (keeps host enqueue far ahead of the GPU)
    lib = dq.lib()
    sp = ctypes.c_void_p(s.cuda_stream)
    dA, dW = A.desc(), Wq.desc()
    dWls = [x.desc() for x in Wls]
    gx = ctypes.c_void_p(G_x.data_ptr())

    def quant(i):
        return lib.dq_quantize_act_nvfp4(ctypes.c_void_p(Xs[i % n_x].data_ptr()), M, K, gx, ctypes.byref(dA), sp)

    def gemm():
        return lib.dq_prefill_gemm(ctypes.byref(dA), None, None, ctypes.byref(dW), M, dq.OUT_BF16,
                                   ctypes.c_void_p(Y.data_ptr()), None, None, 0, sp)

    ws_n = max(dq.dq_decode_gemv_workspace_size(b, Wls[0]) for b in Bs)
    ws = torch.empty(max(ws_n, 16), dtype=torch.uint8, device="cuda")
    wsp = ctypes.c_void_p(ws.data_ptr())

    def gemv(i, b):
        return lib.dq_decode_gemv(ctypes.c_void_p(xd_dev[b].data_ptr()), b, ctypes.byref(dWls[i % n_w]),
                                  dq.OUT_F32, ctypes.c_void_p(ys[b].data_ptr()), wsp, ws_n, sp)

    def step(i):
        assert quant(i) == 0
        assert gemm() == 0
        for j, b in enumerate(Bs):
            assert gemv(i * len(Bs) + j, b) == 0

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    # the timed steps: nothing but the step's launches between the two events
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_start.record(s)
    for i in range(args.steps):
        step(args.warmup + i)
    t_end.record(s)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)

    # per-kernel rates: `reps` back-to-back calls of one kernel (rotating the
    # activation copies and decode weight copies) between one pair of events,
    # so the average includes the GPU-side gap between launches but no event
    # or host overhead
    reps = max(20, args.steps)

    def back_to_back(fn):
        for i in range(3):
            fn(i)
        torch.cuda.synchronize()
        ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ea.record(s)
        for i in range(reps):
            fn(i)
        eb.record(s)
        torch.cuda.synchronize()
        return ea.elapsed_time(eb) / reps

    per = {"quant": back_to_back(lambda i: quant(i)), "gemm": back_to_back(lambda i: gemm())}
    # the same quantizer fused with the RMSNorm that precedes the projection
    gamma = dev(synth.bf16_bits_from_f32((1.0 + 0.2 * synth.random_f32(7, (1, K))).astype(np.float32))[0]
                .view(np.int16))

    norm_ws = torch.empty(4 * M, dtype=torch.uint8, device="cuda")

    def norm_quant(i):
        return lib.dq_rmsnorm_quantize_act_nvfp4(ctypes.c_void_p(Xs[i % n_x].data_ptr()),
                                                 ctypes.c_void_p(gamma.data_ptr()), ctypes.c_float(1e-6), M, K, gx,
                                                 ctypes.byref(dA), ctypes.c_void_p(norm_ws.data_ptr()), 4 * M, sp)
    per["norm_quant"] = back_to_back(norm_quant)
    for b in Bs:
        per[f"gemv_b{b}"] = back_to_back(lambda i, b=b: gemv(i, b))

    flops = 2.0 * M * N * K
    quant_bytes = M * K * 2 + M * K / 2 + M * K / 16
    gemm_tflops = flops / (per["gemm"] * 1e-3) / 1e12
    prefill_tflops = flops / ((per["quant"] + per["gemm"]) * 1e-3) / 1e12
    decode = {}
    for b in Bs:
        nbytes = N * K * 3 / 8 + N * 8 * 2 + b * K * 2 + b * N * 4
        gbs = nbytes / (per[f"gemv_b{b}"] * 1e-3) / 1e9
        decode[f"b{b}"] = {"us": per[f"gemv_b{b}"] * 1e3, "GB/s": gbs, "frac_hbm": gbs / PEAK_HBM_GBS,
                           "bytes": nbytes}
    # algorithmic bytes of one GEMM call: the NVFP4 operands once, the bf16 output once
    gemm_alg_bytes = M * K * (0.5 + 1 / 16) + N * K * (0.5 + 1 / 16) + M * N * 2
    traffic = gemm_traffic()

    out = {
        "metric": METRIC, "value": prefill_tflops, "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": total_ms / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": "8B-scale MLP up-projection: K=4096, N=12288, prefill M=2048 (NVFP4 W4A4), "
                               "decode B=1,4 (LUT3 per-row fp16 tables)",
                   "M": M, "N": N, "K": K, "decode_batches": list(Bs), "static_G_x": G_x_host,
                   "decode_weight_copies": n_w, "x_copies": n_x},
        "prefill": {"quant_us": per["quant"] * 1e3, "quant_GB/s": quant_bytes / (per["quant"] * 1e-3) / 1e9,
                    "rmsnorm_quant_us": per["norm_quant"] * 1e3,
                    "gemm_us": per["gemm"] * 1e3, "gemm_TFLOP/s": gemm_tflops,
                    "frac_fp16_mfma_peak": gemm_tflops / PEAK_FP16_TFLOPS,
                    "frac_fp4_peak": gemm_tflops / PEAK_FP4_TFLOPS,
                    "linear_TFLOP/s_incl_quant": prefill_tflops},
        "decode": decode,
        "pack_ms": {"nvfp4": t_pack_nvfp4, "lut3_per_row": t_pack_lut, "lut3_to_nvfp4_autocast": t_autocast},
        "roofline": {"bound": "mfma", "kernel": "nvfp4_gemm_kernel (one launch per dq_prefill_gemm call)",
                     "achieved": gemm_tflops,
                     "peak": PEAK_FP16_TFLOPS, "unit": "TFLOP/s", "frac": gemm_tflops / PEAK_FP16_TFLOPS,
                     "traffic": traffic,
                     "traffic_note": (f"HBM bytes per GEMM call from FETCH_SIZE + WRITE_SIZE (copy-calibrated); "
                                      f"algorithmic bytes {gemm_alg_bytes:.4g}" if traffic is not None else
                                      "no counter summary for the current GEMM source"),
                     "note": "exact NVFP4 operands are dequantized to fp16 and multiplied on fp16 MFMA; "
                             "frac of the dense FP4 peak is prefill.frac_fp4_peak"},
    }
    out["mxfp4_prefill"] = mxfp4_prefill(dq, torch, np, w, Xs, M, N, K, s, args.steps)
    out["nvfp4a16_decode"] = nvfp4a16_decode(dq, torch, np, Wq, xd_dev, Bs, N, K, s, args.decode_bytes, reps)
    del Wls, dWls, Xs
    torch.cuda.empty_cache()
    if not args.no_decode_sweep:
        out["decode_sweep_27b_blocks"] = decode_sweep(dq, synth, torch, np, args.sweep_blocks, 5)
        out["decode_sweep_27b_blocks"]["blocks"] = args.sweep_blocks
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cfg, w, X, np.float32(G_x_host), xds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
