#!/usr/bin/env python3
"""Benchmark of the phase-specific quantized linear layer on one MI355X.

Workload (the largest single-GPU one): the decode-heavy sweep over 64
stacked 27B-class blocks plus an NVFP4 prefill at M = 32768 tokens.

* Prefill: NVFP4 activation quantization (static global scale from a
  calibration batch) of X [32768, 17408] bf16, then the W4A4 NVFP4 GEMM with
  the 27B MLP down-projection W [5120, 17408] -> bf16 Y [32768, 5120].
* Decode: one token through 64 stacked 27B blocks (q/k/v 7168x5120, o
  5120x5120, gate/up 34816x5120, down 5120x17408; one packed block copied to
  64 distinct buffers: 7.98 GB in LUT3, 5.31 GB in LUT2, far beyond the 256 MB
  Infinity Cache) at batch 1, 8 and 16, in LUT3 and in LUT2 (per-row fp16
  tables).  Each (format, batch) token is one captured HIP graph of 256
  GEMV launches, replayed.
Weights 0.02 N(0,1) times a log-normal row scale; activations N(0,1) with
0.5 % outlier channels x30 (seeded synthetic tensors, resident in HBM).

One step = prefill quantization + GEMM + the six decode tokens.  The run
does `warmup` steps (phases interleaved), then times `steps` steps between
two HIP events on the launch stream (`ms_per_step`), the steps' prefill
passes first and then their decode tokens, so that each phase runs under its
own sustained load; HIP events around every phase of every timed step give
each phase's average duration.  `value` is the prefill linear's
throughput 2*M*N*K / (quantization + GEMM); `roofline` is the GEMM kernel
against the dense FP4 peak (its fp16-MFMA fraction alongside), and
`roofline_decode` the LUT3 batch-1 token against HBM.  Outside the timed
steps the run also measures the 27B down-projection at M = 8192 with fused
activation quantization, the 27B block chained at M = 4096 with NVFP4
epilogues, the MXFP4 variant of the prefill GEMM, the NVFP4A16 decode GEMV,
the engine clock under GEMM and GEMV load, and the CPU oracle on a bounded
sample of the same workload.

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
import subprocess
import sys
import tempfile
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "NVFP4 prefill GEMM TFLOPS (%FP4 peak); LUT3 decode GEMV GB/s (%HBM peak)"
PEAK_FP16_TFLOPS = 2500.0      # dense fp16/bf16 MFMA, MI355X
PEAK_FP4_TFLOPS = 10100.0      # dense fp4 MFMA, MI355X
PEAK_HBM_GBS = 8000.0
# sources that decide the GEMM's kernels and launches
GEMM_SOURCES = [os.path.join(ROOT, "paper_2609_26333_amd", "csrc", f) for f in ("gemm.hip", "dq_internal.hpp", "dq_device.hpp")]
GEMM_COUNTERS = os.path.join(ROOT, "profiles", "nvfp4_gemm_27b_down_m32768_counters.md")
COPY_BYTES = 256 << 20
# The paper's end-to-end figure for this method, quoted as context only: a
# whole-model time to first token on other hardware, not a kernel rate and
# not comparable with the numbers measured here (paper Sec. 1 and Sec. 3.2,
# hardware as stated in Sec. 3.1).
PAPER_CONTEXT = {
    "what": "time to first token, Qwen3.8-27B at an 8K-token prompt, llama.cpp",
    "weight_only_iq1s_s": 12.27, "odp_nvfp4_prefiller_s": 6.90, "speedup": 1.78,
    "speedup_range_4k_to_32k": [1.38, 1.78],
    "hardware": "one NVIDIA GB10 (DGX Spark)",
    "note": "context only; no absolute TFLOP/s or GB/s is published for this path",
}
SWEEP = ((3, 1), (3, 8), (3, 16), (2, 1), (2, 8), (2, 16))

# Clock sampler: a separate process, started before this one touches the GPU,
# that appends amd-smi's per-XCD graphics clocks with a timestamp to a file.
SAMPLER = r"""
import json, subprocess, sys, time
out = sys.argv[1]
while True:
    t = time.time()
    try:
        r = subprocess.run(["amd-smi", "metric", "-c", "--json"], capture_output=True, text=True, timeout=20)
        d = json.loads(r.stdout)
        clk = d["gpu_data"][0]["clock"] if "gpu_data" in d else d[0]["clock"]
        v = [c["clk"]["value"] for k, c in clk.items() if k.startswith("gfx_") and isinstance(c.get("clk"), dict)]
        rec = {"t0": t, "t1": time.time(), "gfx_mhz": v}
    except Exception as e:
        rec = {"t0": t, "t1": time.time(), "error": str(e)[:200]}
    with open(out, "a") as f:
        f.write(json.dumps(rec) + "\n")
    time.sleep(0.05)
"""


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extras", action="store_true", help="skip the measurements outside the timed steps")
    p.add_argument("--no-sclk", action="store_true")
    p.add_argument("--sweep-blocks", type=int, default=64)
    p.add_argument("--calibrate-copy", action="store_true")
    p.add_argument("--summarize-trace", metavar="CSV", help="print a rocprofv3 kernel trace grouped by kernel and grid")
    p.add_argument("--summarize-counters", metavar="CSV", help="print rocprofv3 counters grouped by kernel and grid")
    return p.parse_args()


def short_kernel_name(name):
    """Kernel name without namespaces, return type and argument list."""
    n = name.strip('"')
    n = re.sub(r"^void ", "", n)
    n = n.replace("dq::(anonymous namespace)::", "").replace("dq::", "")
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):        # the argument list: the first "(" outside template brackets
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            cut = i
            break
    return n[:cut].replace("(anonymous namespace)::", "")


def summarize_trace(path, top=40):
    """Markdown table of a rocprofv3 kernel trace: dispatches grouped by kernel,
    grid and workgroup size, with calls and average / min / max duration."""
    import csv
    groups = {}
    for r in csv.DictReader(open(path)):
        key = (short_kernel_name(r["Kernel_Name"]), int(r["Grid_Size_X"]), int(r["Workgroup_Size_X"]))
        groups.setdefault(key, []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    rows = sorted(groups.items(), key=lambda kv: -sum(kv[1]))[:top]
    print("| kernel | grid (work-items) | workgroup | calls | average (us) | min (us) | max (us) | total (us) |")
    print("|---|---:|---:|---:|---:|---:|---:|---:|")
    for (k, g, w), d in rows:
        print(f"| `{k}` | {g} | {w} | {len(d)} | {sum(d) / len(d):.3f} | {min(d):.3f} | {max(d):.3f} | {sum(d):.1f} |")


def summarize_counters(path):
    """Markdown table of a rocprofv3 counter collection: the average value per
    dispatch of each counter, grouped by kernel and grid size."""
    import csv
    groups = {}
    for r in csv.DictReader(open(path)):
        key = (short_kernel_name(r["Kernel_Name"]), int(r["Grid_Size"]), r["Counter_Name"])
        groups.setdefault(key, {}).setdefault(int(r["Dispatch_Id"]), 0.0)
        groups[key][int(r["Dispatch_Id"])] += float(r["Counter_Value"])
    print("| kernel | grid (work-items) | counter | dispatches | average per dispatch |")
    print("|---|---:|---|---:|---:|")
    for (k, g, c), d in sorted(groups.items()):
        v = list(d.values())
        print(f"| `{k}` | {g} | {c} | {len(v)} | {sum(v) / len(v):.6g} |")


def gemm_source_sha256():
    h = hashlib.sha256()
    for f in GEMM_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def gemm_traffic():
    """HBM bytes per GEMM call from the committed counter summary: FETCH_SIZE
    and WRITE_SIZE of the GEMM kernel, each scaled by the bytes a plain copy
    of known size moves per KiB that the same counter reads.  None when the
    summary is missing or the GEMM sources have changed since."""
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


def clock_window(path, t0, t1):
    """Median per-XCD graphics clock (MHz) of the samples taken inside [t0, t1]."""
    if path is None or not os.path.exists(path):
        return None
    vals = []
    for line in open(path):
        try:
            r = json.loads(line)
        except ValueError:
            continue
        if "gfx_mhz" in r and r["t0"] >= t0 and r["t1"] <= t1:
            vals += r["gfx_mhz"]
    if not vals:
        return None
    vals.sort()
    return {"median_mhz": vals[len(vals) // 2], "min_mhz": vals[0], "max_mhz": vals[-1], "readings": len(vals)}


def cpu_baseline(w_down, X, G_x, min_seconds=10.0):
    """The CPU oracle on a bounded sample of the same workload, repeated until
    min_seconds have passed: the prefill linear for 32 of the 32768 token rows
    (NVFP4 quantization + fp64 GEMM against all 5120 weight rows) and the
    batch-1 LUT3 GEMV of one block's down-projection (dequantization + fp64
    GEMV).  Weight packing is offline and untimed."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import linalg, lut, nvfp4
    cfg = synth.STACK_27B_M32768
    qw, cw, Gw = nvfp4.quantize_dynamic(w_down)
    w_hat = nvfp4.dequantize(qw, cw, Gw)
    codes, table = lut.quantize_per_row(w_down, 3)
    xd = synth.decode_x(cfg, w_down.shape[1], 1)
    rows = 32
    Xs = X[:rows]
    N, K = w_down.shape
    t_pre = t_dec = 0.0
    reps = 0
    start = time.perf_counter()
    while reps == 0 or time.perf_counter() - start < min_seconds:
        t0 = time.perf_counter()
        qa, ca, _ = nvfp4.quantize_bf16_activations(Xs, G_x)
        linalg.gemm(nvfp4.dequantize(qa, ca, G_x), w_hat)
        t1 = time.perf_counter()
        linalg.lut_gemv_per_row(xd, codes, table)
        t_pre += t1 - t0
        t_dec += time.perf_counter() - t1
        reps += 1
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    dec_bytes = N * K * 3 / 8 + N * 16 + K * 2 + N * 4
    return {
        "value": 2.0 * rows * N * K * reps / t_pre / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
        "sample": (f"prefill linear for {rows} of the 32768 token rows (NVFP4 quantization of X[{rows},{K}] + fp64 "
                   f"GEMM against all {N} weight rows), {reps} times, {t_pre / reps:.2f} s each; decode: LUT3 "
                   f"dequantization + fp64 GEMV of one 27B down-projection ({N}x{K}) at batch 1, "
                   f"{t_dec / reps:.2f} s each = {dec_bytes * reps / t_dec / 1e9:.3f} GB/s; packing untimed"),
        "decode_gbps": dec_bytes * reps / t_dec / 1e9,
        "host": host_info(threadpool_info()),
    }


def host_info(pools):
    """The host the oracle ran on: logical CPUs, the CPU model, and the BLAS /
    OpenMP thread pools numpy uses."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_count": os.cpu_count(), "model": model,
            "thread_pools": [{"api": i.get("user_api"), "library": i.get("internal_api"),
                              "threads": i.get("num_threads")} for i in pools]}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the kernels run on one GPU (one GPU's share of a sharded layer); "
              f"--gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.summarize_trace or args.summarize_counters:
        if args.summarize_trace:
            summarize_trace(args.summarize_trace)
        if args.summarize_counters:
            summarize_counters(args.summarize_counters)
        return
    sampler = clk_path = None
    if not args.no_sclk:
        clk_path = os.path.join(tempfile.mkdtemp(prefix="dq_clk_"), "clk.jsonl")
        try:
            sampler = subprocess.Popen([sys.executable, "-c", SAMPLER, clk_path], stdout=subprocess.DEVNULL,
                                       stderr=subprocess.DEVNULL)
        except OSError:
            sampler = clk_path = None
    try:
        out = run(args, clk_path)
    finally:
        if sampler is not None:
            sampler.kill()
            sampler.wait()
    print(json.dumps(out), flush=True)


def run(args, clk_path):
    import numpy as np
    import torch

    import paper_2609_26333_amd as dq
    import synth

    torch.cuda.set_device(0)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()   # noqa: E731
    lib = dq.lib()
    s = torch.cuda.current_stream()
    sp = ctypes.c_void_p(s.cuda_stream)
    ev = lambda: torch.cuda.Event(enable_timing=True)   # noqa: E731

    # ---------------------------------------------------------------- prefill inputs
    cfg = synth.STACK_27B_M32768
    layers = {l.name: l for l in cfg.layers}
    down = layers["down"]
    M, N, K = cfg.m, down.n, down.k
    w_down = synth.layer_weight(cfg, down)
    Wq = dq.dq_pack_nvfp4(dev(w_down))
    X_host = synth.prefill_x(cfg, K)
    X = dev(X_host.view(np.int16))
    calib = dev(synth.prefill_x(cfg, K, m=2048, calib=True).view(np.int16))
    G_x = dq.dq_quantize_act_nvfp4(calib).G.clone()   # static scale: the dynamic rule on the calibration batch
    del calib
    A = dq.NvFp4Tensor.empty(M, K)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    dA, dW = A.desc(), Wq.desc()
    gx = ctypes.c_void_p(G_x.data_ptr())

    def quant():
        assert lib.dq_quantize_act_nvfp4(ctypes.c_void_p(X.data_ptr()), M, K, gx, ctypes.byref(dA), sp) == 0

    def gemm():
        assert lib.dq_prefill_gemm(ctypes.byref(dA), None, None, ctypes.byref(dW), M, dq.OUT_BF16,
                                   ctypes.c_void_p(Y.data_ptr()), None, None, 0, None, 0, sp) == 0

    # ---------------------------------------------------------------- decode sweep
    Ws = {l.name: dev(synth.layer_weight(cfg, l)) for l in cfg.layers}
    stacks, wbytes = {}, {}
    for bits in (3, 2):
        block = [dq.dq_pack_lut3(Ws[l.name], bits=bits, mode=dq.LUT_PER_ROW) for l in cfg.layers]
        stacks[bits] = [block] + [[dq.LutWeight(w.codes.clone(), w.lut.clone(), None, None, w.rows, w.cols, bits,
                                                dq.LUT_PER_ROW) for w in block] for _ in range(args.sweep_blocks - 1)]
        wbytes[bits] = sum(w.codes.numel() + w.lut.numel() * 2 for blk in stacks[bits] for w in blk)
    del Ws
    torch.cuda.empty_cache()
    xs = {B: [dev(synth.decode_x(cfg, l.k, B).view(np.int16)) for l in cfg.layers] for B in (1, 8, 16)}
    ys = {B: [torch.empty((B, l.n), dtype=torch.float32, device="cuda") for l in cfg.layers] for B in (1, 8, 16)}
    graphs, keep = {}, []
    cap = torch.cuda.Stream()
    for bits, B in SWEEP:
        descs = [[w.desc() for w in blk] for blk in stacks[bits]]
        ws_n = max(dq.dq_decode_gemv_workspace_size(B, w) for w in stacks[bits][0])
        ws = torch.empty(max(ws_n, 16), dtype=torch.uint8, device="cuda")
        keep += [descs, ws]

        def token(stream, descs=descs, B=B, ws=ws, ws_n=ws_n):
            p = ctypes.c_void_p(stream.cuda_stream)
            for d in descs:
                for i in range(len(cfg.layers)):
                    assert lib.dq_decode_gemv(ctypes.c_void_p(xs[B][i].data_ptr()), B, ctypes.byref(d[i]), dq.OUT_F32,
                                              ctypes.c_void_p(ys[B][i].data_ptr()), ctypes.c_void_p(ws.data_ptr()),
                                              ws_n, p) == 0
        token(s)            # warm: kernel attributes and plans are set up outside the capture
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            token(torch.cuda.current_stream())
        graphs[(bits, B)] = g
    torch.cuda.synchronize()

    # ---------------------------------------------------------------- timed steps
    # The timed region runs the K steps' prefill passes (quantization + GEMM)
    # back to back, then their decode tokens: each phase at the clock the
    # chip holds under that phase's own sustained load, as on a prefill
    # engine and a decode engine of disaggregated serving.  The warm-up steps
    # interleave the phases (quantization, GEMM, then the six tokens); their
    # GEMM durations are reported separately (after ~25 ms of HBM-bound
    # decode kernels the power management holds a lower clock for the next
    # several milliseconds).
    def prefill_pass(pm):
        pm[0].record(s)
        quant()
        pm[1].record(s)
        gemm()
        pm[2].record(s)

    def decode_pass(dm):
        dm[0].record(s)
        for j, key in enumerate(SWEEP):
            graphs[key].replay()
            dm[1 + j].record(s)

    warm_pm = [[ev() for _ in range(3)] for _ in range(args.warmup)]
    for w in range(args.warmup):
        prefill_pass(warm_pm[w])
        decode_pass([ev() for _ in range(len(SWEEP) + 1)])
    torch.cuda.synchronize()
    gemm_interleaved_ms = [m[1].elapsed_time(m[2]) for m in warm_pm[1:]]   # the first warm-up step is cold
    pms = [[ev() for _ in range(3)] for _ in range(args.steps)]
    dms = [[ev() for _ in range(len(SWEEP) + 1)] for _ in range(args.steps)]
    t_start, t_end = ev(), ev()
    t_start.record(s)
    for i in range(args.steps):
        prefill_pass(pms[i])
    for i in range(args.steps):
        decode_pass(dms[i])
    t_end.record(s)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    spans = [[m[0].elapsed_time(m[1]), m[1].elapsed_time(m[2])] + [d[j].elapsed_time(d[j + 1]) for j in range(len(SWEEP))]
             for m, d in zip(pms, dms)]   # ms, per step: quantization, GEMM, the six tokens
    n_ph = 2 + len(SWEEP)
    ph = [sum(sp_[j] for sp_ in spans) / args.steps for j in range(n_ph)]
    ph_med = [float(np.median([sp_[j] for sp_ in spans])) for j in range(n_ph)]
    t_quant, t_gemm = ph[0] * 1e-3, ph[1] * 1e-3

    flops = 2.0 * M * N * K
    gemm_tflops = flops / t_gemm / 1e12
    prefill_tflops = flops / (t_quant + t_gemm) / 1e12
    quant_bytes = M * K * 2 + M * K / 2 + M * K / 16
    decode = {}
    io = {B: args.sweep_blocks * sum(B * l.k * 2 + B * l.n * 4 for l in cfg.layers) for B in (1, 8, 16)}
    for j, (bits, B) in enumerate(SWEEP):
        t = ph[2 + j] * 1e-3
        gbs = (wbytes[bits] + io[B]) / t / 1e9
        decode[f"lut{bits}_b{B}"] = {"ms_per_token": t * 1e3, "ms_per_token_median": ph_med[2 + j],
                                     "GB/s": gbs, "frac_hbm": gbs / PEAK_HBM_GBS,
                                     "bytes": wbytes[bits] + io[B],
                                     "gemv_launches": args.sweep_blocks * len(cfg.layers)}
    gemm_alg_bytes = M * K * (0.5 + 1 / 16) + N * K * (0.5 + 1 / 16) + M * N * 2
    traffic = gemm_traffic()
    out = {
        "metric": METRIC, "value": prefill_tflops, "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": total_ms / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic",
        "config": {"workload": ("decode-heavy sweep over 64 stacked 27B-class blocks (LUT3 and LUT2 per-row "
                                "tables, batch 1/8/16) plus NVFP4 prefill at M=32768 on the 27B down-projection "
                                "(K=17408, N=5120)"),
                   "M": M, "N": N, "K": K, "decode_batches": [1, 8, 16], "sweep_blocks": args.sweep_blocks,
                   "static_G_x": float(G_x.cpu()[0]), "decode_tokens": "captured HIP graphs, 256 GEMVs each"},
        "prefill": {"quant_us": t_quant * 1e6, "quant_us_median": ph_med[0] * 1e3,
                    "gemm_us_median": ph_med[1] * 1e3, "quant_GB/s": quant_bytes / t_quant / 1e9,
                    "quant_frac_hbm": quant_bytes / t_quant / 1e9 / PEAK_HBM_GBS,
                    "gemm_us": t_gemm * 1e6, "gemm_TFLOP/s": gemm_tflops,
                    "frac_fp4_peak": gemm_tflops / PEAK_FP4_TFLOPS,
                    "frac_fp16_mfma_peak": gemm_tflops / PEAK_FP16_TFLOPS,
                    "linear_TFLOP/s_incl_quant": prefill_tflops,
                    "gemm_us_interleaved": (float(np.median(gemm_interleaved_ms)) * 1e3 if gemm_interleaved_ms
                                            else None),
                    "order": ("timed: the steps' prefill passes back to back, then their decode tokens; "
                              "gemm_us_interleaved: median GEMM of the warm-up steps after the first, each "
                              "right after the previous step's six decode tokens")},
        "decode": decode,
        "roofline": {"bound": "mfma", "kernel": "nvfp4_gemm_kernel (one launch per dq_prefill_gemm call)",
                     "achieved": gemm_tflops, "peak": PEAK_FP4_TFLOPS, "unit": "TFLOP/s",
                     "frac": gemm_tflops / PEAK_FP4_TFLOPS,
                     "frac_fp16_mfma": gemm_tflops / PEAK_FP16_TFLOPS,
                     "traffic": traffic,
                     "traffic_note": (f"HBM bytes per GEMM call from FETCH_SIZE + WRITE_SIZE (copy-calibrated); "
                                      f"algorithmic bytes {gemm_alg_bytes:.4g}" if traffic is not None else
                                      f"no counter summary for the current GEMM source; algorithmic bytes "
                                      f"{gemm_alg_bytes:.4g}"),
                     "note": "exact NVFP4 (E4M3 scale per 16) runs on the fp16 MFMA after exact dequantization, "
                             "whose dense peak is a quarter of the FP4 peak"},
        "roofline_decode": {"bound": "hbm", "kernel": "LUT3 batch-1 token: 256 dq_decode_gemv launches",
                            "achieved": decode["lut3_b1"]["GB/s"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                            "frac": decode["lut3_b1"]["frac_hbm"]},
        "paper_context": PAPER_CONTEXT,
    }
    if not args.no_extras:
        out["decode_differencing"] = decode_differencing(dq, torch, lib, s, stacks[3], xs[1], ys[1], cfg,
                                                         graphs[(3, 1)])
        del graphs, keep
        torch.cuda.synchronize()
        out["sclk"] = measure_clocks(dq, torch, lib, s, sp, gemm, stacks, xs, ys, cfg, clk_path)
        del stacks
        torch.cuda.empty_cache()
        out["mxfp4_prefill_m32768"] = mxfp4_prefill(dq, torch, lib, s, sp, w_down, X, M, N, K)
        up8b = synth.UP_8B_M2048
        up = up8b.layers[0]
        out["mxfp4_prefill_8b_up_m2048"] = mxfp4_prefill(dq, torch, lib, s, sp, synth.layer_weight(up8b, up),
                                                         dev(synth.prefill_x(up8b, up.k).view(np.int16)), up8b.m,
                                                         up.n, up.k, reps=100)
        del A, Y, X
        torch.cuda.empty_cache()
        out["fused_down_27b_m8192"] = fused_down_m8192(dq, synth, torch, np, lib, s, sp)
        out["block_chain_27b_m4096"] = block_chain_m4096(dq, synth, torch, np, lib, s, sp)
        out["nvfp4a16_decode_27b_down"] = nvfp4a16_decode(dq, torch, lib, s, sp, Wq, N, K)
        out["rmsnorm_quant_27b_hidden"] = rmsnorm_quant(dq, synth, torch, np, lib, s, sp)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w_down, X_host, np.float32(out["config"]["static_G_x"]))
    return out


def decode_differencing(dq, torch, lib, s, stack, xs, ys, cfg, g_full):
    """N-vs-2N differencing of the LUT3 batch-1 token: replays of a captured
    graph over the first half of the blocks and of the full token's graph
    (median of 7 timings of 5 replays each); the difference over the blocks
    it adds is the per-block cost without the graph launch."""
    half = len(stack) // 2
    descs = [[w.desc() for w in blk] for blk in stack[:half]]
    cap = torch.cuda.Stream()
    g_half = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_half, stream=cap):
        p = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        for d in descs:
            for i in range(len(cfg.layers)):
                assert lib.dq_decode_gemv(ctypes.c_void_p(xs[i].data_ptr()), 1, ctypes.byref(d[i]), dq.OUT_F32,
                                          ctypes.c_void_p(ys[i].data_ptr()), None, 0, p) == 0
    torch.cuda.synchronize()

    def med(g):
        g.replay()
        torch.cuda.synchronize()
        ts = []
        for _ in range(7):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            for _ in range(5):
                g.replay()
            e1.record(s)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / 5)
        return sorted(ts)[len(ts) // 2]

    t_half, t_full = med(g_half), med(g_full)
    n_full = len(stack)
    return {"blocks": [half, n_full], "ms_per_replay_median": [t_half, t_full],
            "us_per_block_differenced": (t_full - t_half) / (n_full - half) * 1e3,
            "us_per_block_full_replay": t_full / n_full * 1e3,
            "note": "LUT3 batch 1; graph over the first half of the blocks vs the whole token"}


def timed(torch, s, fn, reps, warm_s=0.3):
    """Mean time of `reps` back-to-back calls, after at least warm_s seconds of
    back-to-back calls: the engine clock ramps up over tens of milliseconds
    of sustained load (a few calls right after an idle gap run up to 20 %
    slower), and the timed steps of the workload run in that sustained state."""
    fn()
    torch.cuda.synchronize()
    t0 = time.time()
    while time.time() - t0 < warm_s:
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for _ in range(reps):
        fn()
    e1.record(s)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps * 1e-3


def measure_clocks(dq, torch, lib, s, sp, gemm, stacks, xs, ys, cfg, clk_path):
    """Engine clock while the GPU runs back-to-back prefill GEMMs (about 2 s)
    and back-to-back LUT3 batch-1 GEMVs over the 64 blocks (about 2 s)."""
    if clk_path is None:
        return None
    res = {}
    gemm()
    torch.cuda.synchronize()
    t0 = time.time()
    for _ in range(450):
        gemm()
    torch.cuda.synchronize()
    res["prefill_gemm"] = clock_window(clk_path, t0, time.time())
    descs = [[w.desc() for w in blk] for blk in stacks[3]]
    t0 = time.time()
    for _ in range(700):
        for d in descs:
            for i in range(len(cfg.layers)):
                lib.dq_decode_gemv(ctypes.c_void_p(xs[1][i].data_ptr()), 1, ctypes.byref(d[i]), dq.OUT_F32,
                                   ctypes.c_void_p(ys[1][i].data_ptr()), None, 0, sp)
        if time.time() - t0 > 2.0:
            break
    torch.cuda.synchronize()
    res["decode_gemv_lut3_b1"] = clock_window(clk_path, t0, time.time())
    res["source"] = "amd-smi metric -c (per-XCD graphics clock), sampled by a helper process"
    return res


def mxfp4_prefill(dq, torch, lib, s, sp, w, X, M, N, K, reps=5):
    """The MXFP4 W4A4 variant of the same prefill linear (OCP MX: E8M0 scale
    per 32, block scales applied inside the FP4 MFMA)."""
    Wm = dq.dq_pack_mxfp4(torch.from_numpy(w).cuda())
    A = dq.MxFp4Tensor.empty(M, K)
    Y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    dA, dW = A.desc(), Wm.desc()
    t_q = timed(torch, s, lambda: lib.dq_quantize_act_mxfp4(ctypes.c_void_p(X.data_ptr()), M, K, ctypes.byref(dA),
                                                            sp), reps)
    t_g = timed(torch, s, lambda: lib.dq_prefill_gemm_mxfp4(ctypes.byref(dA), ctypes.byref(dW), dq.OUT_BF16,
                                                            ctypes.c_void_p(Y.data_ptr()), sp), reps)
    flops = 2.0 * M * N * K
    return {"quant_us": t_q * 1e6, "quant_GB/s": M * K * (2 + 0.5 + 1 / 32) / t_q / 1e9,
            "gemm_us": t_g * 1e6, "gemm_TFLOP/s": flops / t_g / 1e12,
            "frac_fp4_peak": flops / t_g / 1e12 / PEAK_FP4_TFLOPS,
            "linear_TFLOP/s_incl_quant": flops / (t_q + t_g) / 1e12,
            "note": "MXFP4 W4A4 (E2M1, E8M0 per 32 along K) on the scaled FP4 MFMA; same shapes, bf16 output"}


def fused_down_m8192(dq, synth, torch, np, lib, s, sp):
    """27B MLP down-projection at an 8K prompt: M = 8192, K = 17408, N = 5120,
    activation quantization fused into the prefill call (static scale, the
    NVFP4 copy of X in a caller workspace)."""
    cfg = synth.DOWN_27B_M8192
    layer = cfg.layers[0]
    M, N, K = cfg.m, layer.n, layer.k
    W = dq.dq_pack_nvfp4(torch.from_numpy(synth.layer_weight(cfg, layer)).cuda())
    X = torch.from_numpy(synth.prefill_x(cfg, K).view(np.int16)).cuda()
    G = dq.dq_quantize_act_nvfp4(torch.from_numpy(synth.prefill_x(cfg, K, m=2048, calib=True).view(np.int16))
                                 .cuda()).G.clone()
    Y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    ws_n = dq.dq_prefill_gemm_workspace_size(M, K)
    ws = torch.empty(ws_n, dtype=torch.uint8, device="cuda")
    dW = W.desc()
    t = timed(torch, s, lambda: lib.dq_prefill_gemm(None, ctypes.c_void_p(X.data_ptr()), ctypes.c_void_p(G.data_ptr()),
                                                    ctypes.byref(dW), M, dq.OUT_BF16, ctypes.c_void_p(Y.data_ptr()),
                                                    None, None, 0, ctypes.c_void_p(ws.data_ptr()), ws_n, sp), 10)
    # the two halves of the fused call, each timed alone: the quantization
    # pass bounds what folding it into the GEMM could save
    A = dq.NvFp4Tensor.empty(M, K)
    dA = A.desc()
    t_q = timed(torch, s, lambda: lib.dq_quantize_act_nvfp4(ctypes.c_void_p(X.data_ptr()), M, K,
                                                            ctypes.c_void_p(G.data_ptr()), ctypes.byref(dA), sp), 10)
    t_g = timed(torch, s, lambda: lib.dq_prefill_gemm(ctypes.byref(dA), None, None, ctypes.byref(dW), M, dq.OUT_BF16,
                                                      ctypes.c_void_p(Y.data_ptr()), None, None, 0, None, 0, sp), 10)
    flops = 2.0 * M * N * K
    return {"us": t * 1e6, "TFLOP/s": flops / t / 1e12, "frac_fp4_peak": flops / t / 1e12 / PEAK_FP4_TFLOPS,
            "frac_fp16_mfma_peak": flops / t / 1e12 / PEAK_FP16_TFLOPS,
            "quant_pass_us": t_q * 1e6, "gemm_alone_us": t_g * 1e6,
            "note": "one dq_prefill_gemm call with X: quantization pass into the workspace, then the GEMM; "
                    "quant_pass_us and gemm_alone_us time the two halves alone"}


def block_chain_m4096(dq, synth, torch, np, lib, s, sp):
    """The 27B block's linears chained on one stream at M = 4096: activation
    quantization and q/k/v (bf16 out); quantization of the attention-output
    stand-in and o with an NVFP4 epilogue (static scale) feeding gate/up with
    SwiGLU and an NVFP4 epilogue feeding down (bf16 out)."""
    cfg = synth.BLOCK_27B_M4096
    L = {l.name: l for l in cfg.layers}
    M = cfg.m
    W = {n: dq.dq_pack_nvfp4(torch.from_numpy(synth.layer_weight(cfg, L[n])).cuda()) for n in L}
    X = torch.from_numpy(synth.prefill_x(cfg, 5120).view(np.int16)).cuda()
    At = torch.from_numpy(synth.attn_out_standin(cfg, M, 5120).view(np.int16)).cuda()
    g = lambda v: torch.tensor([v], dtype=torch.float32, device="cuda")   # noqa: E731
    Gx = dq.dq_quantize_act_nvfp4(X[:2048]).G.clone()
    Ga = dq.dq_quantize_act_nvfp4(At[:2048]).G.clone()
    Go, Gh = g(0.02), g(0.05)
    A1, A2 = dq.NvFp4Tensor.empty(M, 5120), dq.NvFp4Tensor.empty(M, 5120)
    Ho = dq.NvFp4Tensor.empty(M, 5120)
    Hg = dq.NvFp4Tensor.empty(M, 17408)
    Yqkv = torch.empty((M, 7168), dtype=torch.bfloat16, device="cuda")
    Yd = torch.empty((M, 5120), dtype=torch.bfloat16, device="cuda")
    d = {k: v.desc() for k, v in W.items()}
    dA1, dA2, dHo, dHg = A1.desc(), A2.desc(), Ho.desc(), Hg.desc()
    P = ctypes.c_void_p
    by = ctypes.byref

    def chain():
        assert lib.dq_quantize_act_nvfp4(P(X.data_ptr()), M, 5120, P(Gx.data_ptr()), by(dA1), sp) == 0
        assert lib.dq_prefill_gemm(by(dA1), None, None, by(d["qkv"]), M, dq.OUT_BF16, P(Yqkv.data_ptr()), None, None,
                                   0, None, 0, sp) == 0
        assert lib.dq_quantize_act_nvfp4(P(At.data_ptr()), M, 5120, P(Ga.data_ptr()), by(dA2), sp) == 0
        assert lib.dq_prefill_gemm(by(dA2), None, None, by(d["o"]), M, dq.OUT_NVFP4, None, P(Go.data_ptr()), by(dHo),
                                   0, None, 0, sp) == 0
        assert lib.dq_prefill_gemm(by(dHo), None, None, by(d["gate_up"]), M, dq.OUT_NVFP4, None, P(Gh.data_ptr()),
                                   by(dHg), dq.EPI_SWIGLU, None, 0, sp) == 0
        assert lib.dq_prefill_gemm(by(dHg), None, None, by(d["down"]), M, dq.OUT_BF16, P(Yd.data_ptr()), None, None,
                                   0, None, 0, sp) == 0
    t = timed(torch, s, chain, 10)
    flops = 2.0 * M * sum(l.n * l.k for l in cfg.layers)
    return {"us": t * 1e6, "TFLOP/s": flops / t / 1e12, "frac_fp4_peak": flops / t / 1e12 / PEAK_FP4_TFLOPS,
            "frac_fp16_mfma_peak": flops / t / 1e12 / PEAK_FP16_TFLOPS, "TFLOP": flops / 1e12,
            "note": "2 activation quantizations + 4 GEMMs (q/k/v bf16, o -> NVFP4, gate/up + SwiGLU -> NVFP4, "
                    "down bf16), back-to-back on one stream"}


def rmsnorm_quant(dq, synth, torch, np, lib, s, sp):
    """RMSNorm fused with the NVFP4 activation quantizer (static scale) on the
    27B hidden state at M = 4096 and M = 32768, K = 5120, next to the plain
    activation quantizer of the same tensor."""
    cfg = synth.BLOCK_27B_M4096
    K = 5120
    out = {}
    X0 = torch.from_numpy(synth.prefill_x(cfg, K).view(np.int16)).cuda()
    gamma = torch.from_numpy(synth.bf16_bits_from_f32((1.0 + 0.2 * synth.random_f32(7, (1, K))).astype(np.float32))[0]
                             .view(np.int16)).cuda()
    G = dq.dq_quantize_act_nvfp4(X0[:2048]).G.clone()
    for M in (4096, 32768):
        X = X0.repeat(M // X0.shape[0], 1)
        A = dq.NvFp4Tensor.empty(M, K)
        dA = A.desc()
        P = ctypes.c_void_p
        t_n = timed(torch, s, lambda: lib.dq_rmsnorm_quantize_act_nvfp4(P(X.data_ptr()), P(gamma.data_ptr()),
                                                                         ctypes.c_float(1e-6), M, K, P(G.data_ptr()),
                                                                         ctypes.byref(dA), None, 0, sp), 20)
        t_q = timed(torch, s, lambda: lib.dq_quantize_act_nvfp4(P(X.data_ptr()), M, K, P(G.data_ptr()),
                                                                ctypes.byref(dA), sp), 20)
        nbytes = M * K * (2 + 0.5 + 1 / 16)
        out[f"m{M}"] = {"rmsnorm_quant_us": t_n * 1e6, "rmsnorm_quant_GB/s": nbytes / t_n / 1e9,
                        "quant_us": t_q * 1e6, "quant_GB/s": nbytes / t_q / 1e9}
    out["note"] = "one pass over X (static scale, K <= 8192); algorithmic bytes: X read once, NVFP4 written"
    return out


def nvfp4a16_decode(dq, torch, lib, s, sp, Wq, N, K):
    """Weight-only NVFP4 decode GEMV (format-disaggregated NVFP4) on the 27B
    down-projection's NVFP4 weights, rotated over 16 copies (800 MB) so that
    they stream from HBM."""
    copies = [Wq] + [dq.NvFp4Tensor(Wq.codes.clone(), Wq.scales.clone(), Wq.G.clone(), N, K) for _ in range(15)]
    ds = [c.desc() for c in copies]
    nbytes = Wq.codes.numel() + Wq.scales.numel()
    out = {}
    for B in (1, 16):
        x = torch.randn(B, K, device="cuda").to(torch.bfloat16)
        y = torch.empty((B, N), dtype=torch.float32, device="cuda")
        ws_n = dq.dq_decode_gemv_nvfp4_workspace_size(B, Wq)
        ws = torch.empty(max(ws_n, 16), dtype=torch.uint8, device="cuda")
        it = iter(range(1 << 30))
        t = timed(torch, s, lambda: lib.dq_decode_gemv_nvfp4(ctypes.c_void_p(x.data_ptr()), B,
                                                             ctypes.byref(ds[next(it) % len(ds)]), dq.OUT_F32,
                                                             ctypes.c_void_p(y.data_ptr()),
                                                             ctypes.c_void_p(ws.data_ptr()), ws_n, sp), 32)
        alg = nbytes + B * K * 2 + B * N * 4
        out[f"b{B}"] = {"us": t * 1e6, "GB/s": alg / t / 1e9, "frac_hbm": alg / t / 1e9 / PEAK_HBM_GBS}
    out["note"] = "NVFP4 weights (4.5 bits/weight), bf16 x; back-to-back calls over 16 weight copies"
    return out


if __name__ == "__main__":
    main()
