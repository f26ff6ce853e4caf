#!/usr/bin/env python3
"""Benchmark of the NVFP4 ScaleSweep hot path on one MI355X.

One step quantizes every weight of a Llama-3-8B-shaped decoder layer (bfloat16, block 16,
dynamic global scale with D = 256) with ScaleSweep under both objectives, MSE and WMSE: one
batched call per objective over the layer's 7 tensors (each tensor's |x| reduction spread over
the workgroups of the previous tensor's quantization grid).  `value` is the bfloat16 input consumed
per second (both objectives read the layer).  The line also carries:
  * per-method GB/s of the same GPU's AbsMax (D = 448), 4/6 and each ScaleSweep objective,
    batched over the layer and as 7 single-tensor calls, and the time relative to AbsMax;
  * `roofline` for the dominant kernel (the WMSE sweep kernel), from HIP events around its
    launches on the stream it runs on;
  * `cpu_baseline`: the oracle on the host, single-threaded, on a bounded sample;
  * `rows`: the window variants, the reference scales (optimal real scale, FP8-quantized
    optimum, gap report) and the online quantizer (static S, swizzled scales, importance
    vectors), each timed on its own workload (skipped with --no-rows).
Inputs are synthetic (workloads.py) and resident in HBM before timing starts.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

# MI355X figures used for the rooflines.
HBM_PEAK_GBS = 8000.0
# binary32 vector: 157.3 TFLOP/s published = 256 CU x 4 SIMD x 32 lanes x 2.4 GHz lane-ops
VALU_PEAK_TOPS = 256 * 4 * 32 * 2.4e9 / 1e12    # 78.64 T lane-ops/s (an FMA is one lane-op)
# Algorithmic VALU lane-operations per element-candidate evaluation: scale, round,
# reconstruct-and-subtract, square-and-accumulate (+ one weight multiply for WMSE).
OPS_PER_EVAL = {"scalesweep_mse": 4, "scalesweep_wmse": 5}
CANDIDATES_16 = {"scalesweep_mse": 11, "scalesweep_wmse": 16}
DOMINANT = "scalesweep_wmse"
DOMINANT_SYMBOL = "quant_kernel<3, unsigned short, 16, false>"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target length of the oracle's CPU-baseline sample")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU baseline")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain device copy of known size (for counter scaling)")
    ap.add_argument("--no-rows", action="store_true",
                    help="skip the window / reference-scale / online / GPTQ measurements")
    ap.add_argument("--profile-config", choices=("c0", "c2", "c3", "c3w", "c4", "f3", "f4"), default=None,
                    help="run only one other configuration's launches (a few of each, for "
                         "rocprofv3 counter runs) and exit: c0 the FP32 1024x1024 matrix, c2 the "
                         "8192x8192 block-size sweep, c3 the online tensors, c4 one "
                         "Llama-3-70B-shaped layer, f3 the fused SwiGLU quantizer and its "
                         "unfused pair, f4 GPTQ on q_proj")
    ap.add_argument("--c4-layers", type=int, default=80,
                    help="Llama-3-70B-shaped layers to stream through the WMSE quantizer "
                         "(80, the default, is the whole model)")
    return ap.parse_args()


def kernel_source_hash() -> str:
    src = (ROOT / "paper_2606_07618_amd" / "csrc" / "nvfp4ss.hip").read_bytes()
    return hashlib.sha256(src).hexdigest()[:16]


def read_traffic():
    """HBM bytes per launch of the dominant kernel from the committed counter summary (two
    rocprofv3 --pmc runs, FETCH_SIZE and WRITE_SIZE, scaled by a plain copy's readings), or
    None if the counters were taken on another version of the kernel source."""
    f = ROOT / "profiles" / "traffic_scalesweep_wmse_llama8b_layer.txt"
    if not f.exists():
        return None
    d = dict(line.split(None, 1) for line in f.read_text().splitlines() if line.strip())
    if d.get("kernel_source_sha256_16", "").strip() != kernel_source_hash():
        return None
    return int(d["hbm_bytes_per_launch"])


def read_valu():
    """Executed VALU lane-instructions per launch of the dominant kernel (rocprofv3
    SQ_INSTS_VALU x 64, mean over the layer's 7 tensors) from the committed counter summary, or
    None if the counters were taken on another version of the kernel source."""
    f = ROOT / "profiles" / "valu_scalesweep_wmse_llama8b_layer.txt"
    if not f.exists():
        return None
    d = dict(line.split(None, 1) for line in f.read_text().splitlines() if line.strip())
    if d.get("kernel_source_sha256_16", "").strip() != kernel_source_hash():
        return None
    return float(d["valu_lane_instructions_per_launch"])


def host_cpu():
    """The host CPU's model name and the cores this process may run on."""
    model = None
    try:
        for line in Path("/proc/cpuinfo").read_text().splitlines():
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def _timed(torch, fn, reps):
    """Mean milliseconds of fn over reps calls, HIP events on the current stream (which the
    library launches on)."""
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def _median_call(torch, fn, reps):
    """Median milliseconds of single calls of fn (HIP events around each call on the current
    stream), after one untimed call."""
    fn()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for e0, e1 in ev:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    ts = sorted(e0.elapsed_time(e1) for e0, e1 in ev)
    return ts[reps // 2]


def measure_c0(nv, workloads, torch, dev):
    """The FP32 [1024, 1024] N(0, 1) matrix (seed 0), ScaleSweep-MSE with D = 448 and a
    dynamic S (its amax pass, scale fold and sweep), per-call latency: median of 50 calls, each
    timed with HIP events.  At 4 MiB the call is launch-bound, so no roofline fraction."""
    x = torch.from_numpy(workloads.c0_matrix()).to(dev)
    ws = nv.workspace(dev)
    out = {"workload": "fp32 [1024, 1024] N(0, 1) seed 0, block 16, D = 448, dynamic S",
           "timing": "median of 50 single calls (HIP events)"}
    for m in ("absmax", "scalesweep_mse"):
        o = nv.quantize(x, m, 16, fp8_range=448.0, ws=ws)
        us = 1e3 * _median_call(torch, lambda: nv.quantize(x, m, 16, fp8_range=448.0, ws=ws,
                                                             out=o), 50)
        out[m] = {"us_per_call": round(us, 2), "input_GBps": round(4 * x.numel() / us / 1e3, 1)}
    return out


def swiglu_inputs(workloads, torch, dev, tokens=8192, inter=14336):
    """The MLP of a Llama-3-8B-shaped layer for `tokens` tokens: gate and up activations
    [tokens, 14336] bf16 (gate ~ 3 N(0, 1), up ~ N(0, 1) with 4 outlier channels x20) and the
    down projection's input-channel importance (one vector)."""
    g = workloads.generator(dev, 81, 1)
    gate = (torch.randn((tokens, inter), generator=g, device=dev) * 3.0).to(torch.bfloat16)
    up = torch.randn((tokens, inter), generator=g, device=dev)
    up[:, torch.randperm(inter, generator=g, device=dev)[:4]] *= 20.0
    up = up.to(torch.bfloat16)
    imp = workloads.column_importance(inter, g, dev, tokens=256)[None].contiguous()
    return gate, up, imp


def measure_fused_swiglu(nv, workloads, torch, dev):
    """The online quantizer fused into its producer (the SwiGLU product feeding down_proj)
    against the producer kernel followed by the online quantizer, static S, swizzled scales:
    median of 50 single calls each (HIP events), per method, with the algorithmic HBM bytes
    (fused: 4 B read + 0.5625 B written per element; unfused: 4 + 2 for the producer, then
    2 + 0.5625 for the quantizer)."""
    gate, up, imp = swiglu_inputs(workloads, torch, dev)
    n = gate.numel()
    h = nv.swiglu(gate, up)
    S = 0.004
    out = {"workload": "Llama-3-8B MLP activation of 8192 tokens: gate, up [8192, 14336] bf16 -> "
                       "NVFP4 of bf16(silu(gate) * up), static S, swizzled scales, block 16",
           "timing": "median of 50 single calls (HIP events)",
           "bytes_per_element": {"fused": 4.5625, "unfused": 8.5625}}
    ms_prod = _median_call(torch, lambda: nv.swiglu(gate, up, out=h), 50)
    out["producer_alone_ms"] = round(ms_prod, 4)
    for m in ("absmax", "scalesweep_mse", "scalesweep_wmse"):
        wt = imp if m == "scalesweep_wmse" else None
        o1 = nv.quantize_online_swiglu(gate, up, m, S, wt, layout="swizzled")
        o2 = nv.quantize_online(h, m, S, 16, wt, layout="swizzled")
        fused = _median_call(torch, lambda: nv.quantize_online_swiglu(gate, up, m, S, wt, layout="swizzled",
                                                                      out=o1), 50)

        def unfused():
            nv.swiglu(gate, up, out=h)
            nv.quantize_online(h, m, S, 16, wt, layout="swizzled", out=o2)

        unf = _median_call(torch, unfused, 50)
        out[m] = {"fused_ms": round(fused, 4), "unfused_ms": round(unf, 4),
                  "time_saved": round(1.0 - fused / unf, 3),
                  "fused_hbm_GBps_algorithmic": round(4.5625 * n / fused / 1e6, 1),
                  "unfused_hbm_GBps_algorithmic": round(8.5625 * n / unf / 1e6, 1)}
    del gate, up, h
    return out


def measure_rows(nv, workloads, torch, dev, layer):
    """Window variants, reference scales and the online quantizer, each on its own
    workload, as milliseconds per call and GB/s of bf16 input."""
    out = {}
    x, w = layer["gate_proj"]
    n = x.numel()
    S = 1.0e-4
    win = {}
    for name, wt, mode, lo, hi in (("tight_mse", None, "tight", 0, 0),
                                   ("offsets_-3_7_mse", None, "offsets", -3, 7),
                                   ("tight_wmse", w, "tight", 0, 0),
                                   ("offsets_-8_7_wmse", w, "offsets", -8, 7),
                                   ("exhaustive_mse", None, "offsets", -126, 126)):
        ms = _timed(torch, lambda: nv.quantize_window(x, 16, wt, mode, lo, hi, 256.0, S),
                    3 if name.startswith("exhaustive") else 10)
        win[name] = {"ms": round(ms, 4), "input_GBps": round(2 * n / ms / 1e6, 1)}
    out["f2_windows"] = {"workload": "gate_proj [14336, 4096] bf16, block 16, static S", **win}

    # dequantization of the same tensor: 0.5 B of nibbles + 1/16 B of scale per element in,
    # 4 B of binary32 out
    q, sc, Sg = nv.quantize(x, "scalesweep_wmse", 16, weight=w)
    xh = torch.empty(x.shape, dtype=torch.float32, device=dev)
    ms = _timed(torch, lambda: nv.dequant(q, sc, Sg, 16, out=xh), 10)
    out["a10_dequant"] = {"workload": "gate_proj [14336, 4096], block 16, binary32 out",
                          "ms": round(ms, 4),
                          "hbm_GBps_algorithmic": round(n * (0.5 + 1 / 16 + 4) / ms / 1e6, 1)}
    del xh

    xq, wq = layer["q_proj"]
    _, _, Sq = nv.quantize(xq, "scalesweep_mse", 16)
    ref = {}
    for blk in (16, 128):
        ms = _timed(torch, lambda: nv.block_optimum(xq, Sq, blk, wq), 2)
        ref[f"block_optimum_n{blk}"] = {"ms": round(ms, 3),
                                        "Gelem_per_s": round(xq.numel() / ms / 1e6, 3)}
    gaps = nv.gap_report(xq, 16, wq)
    out["f1_reference_scales"] = {"workload": "q_proj [4096, 4096] bf16, WMSE weights", **ref,
                                  "gaps_wmse": {k: round(v, 5) for k, v in gaps.items()}}

    # block-size sweep on one 8192 x 8192 weight: time per call (dynamic S) and the objective
    # gap of every rule to the optimal real block scale, for both objectives
    x2, w2 = workloads.square8192(dev)
    n2 = x2.numel()
    sweep = {}
    for blk in (16, 32, 64, 128):
        per = {}
        for m in ("absmax", "four_over_six", "scalesweep_mse", "scalesweep_wmse"):
            wt = w2 if m in ("scalesweep_wmse",) else None
            ms = _timed(torch, lambda: nv.quantize(x2, m, blk, weight=wt), 10)
            per[m] = {"ms": round(ms, 4), "input_GBps": round(2 * n2 / ms / 1e6, 1)}
        gaps_mse = nv.gap_report(x2, blk, None)
        gaps_wmse = nv.gap_report(x2, blk, w2)
        sweep[f"n{blk}"] = {**per, "gap_to_optimum_mse": {k: round(v, 5) for k, v in gaps_mse.items()},
                            "gap_to_optimum_wmse": {k: round(v, 5) for k, v in gaps_wmse.items()}}
    out["c2_block_sizes"] = {"workload": "one [8192, 8192] bf16 weight, dynamic S, WMSE weights of "
                                         "8192 columns", **sweep}
    del x2, w2

    t = workloads.online_tensors(dev)
    onl = {"timing": "median of 50 single calls (HIP events)"}
    for name in ("act", "k", "v", "q"):
        xo = t[name].reshape(-1, t[name].shape[-1])
        for m in ("absmax", "scalesweep_mse"):
            o = nv.quantize_online(xo, m, 0.002, 16, layout="swizzled")
            ms = _median_call(torch, lambda: nv.quantize_online(xo, m, 0.002, 16, layout="swizzled",
                                                                out=o), 50)
            onl[f"{name}_{m}"] = {"shape": list(t[name].shape), "ms": round(ms, 4),
                                  "input_GBps": round(2 * xo.numel() / ms / 1e6, 1)}
            o = nv.quantize(xo, m, 16)
            ms = _median_call(torch, lambda: nv.quantize(xo, m, 16, out=o), 50)
            onl[f"{name}_{m}_dynamic_S"] = {"ms": round(ms, 4),
                                            "input_GBps": round(2 * xo.numel() / ms / 1e6, 1)}
    g = workloads.generator(dev, 77)
    imp = workloads.column_importance(8192, g, dev, tokens=256)[None].contiguous()
    table8 = {}
    for B in (128, 1024, 8192, 32768):
        xb = torch.randn((B, 8192), generator=g, device=dev).to(torch.bfloat16)
        table8[str(B)] = {m: round(1e3 * _timed(torch, lambda: nv.quantize_online(
            xb, m, 0.002, 16, imp, layout="swizzled"), 20), 1)
            for m in ("absmax", "scalesweep_mse", "scalesweep_wmse")}
    del t
    t = workloads.online_tensors(dev)
    k2 = t["k"].reshape(-1, 128)
    ms_imp = _timed(torch, lambda: nv.channel_sq_norms(k2, t["k"].shape[2], 8, 1, 4), 5)
    out["f3_online"] = {"workload": "online tensors (activations [8192, 4096]; K, V "
                                    "[16, 8, 4096, 128]; Q [16, 32, 4096, 128]), static S, "
                                    "swizzled scales", **onl,
                        "hidden8192_us_per_call": table8,
                        "importance_q_from_k_ms": round(ms_imp, 4)}
    del t

    out["f3_fused_swiglu"] = measure_fused_swiglu(nv, workloads, torch, dev)

    # GPTQ (LDLQ) with ScaleSweep-WMSE scales fixed beforehand, q_proj and a synthetic Hessian
    H, scg, Sg = gptq_inputs(nv, workloads, torch, dev, xq)
    ms_gptq = _timed(torch, lambda: nv.ldlq(xq, H, scg, Sg, 16, 0.01, check=False), 3)
    out["f4_gptq"] = {"workload": "q_proj [4096, 4096] bf16, Hessian X^T X of 1024 synthetic "
                                  "tokens, ScaleSweep-WMSE scales, damping 0.01",
                      "ms_per_call": round(ms_gptq, 2)}
    return out


def gptq_inputs(nv, workloads, torch, dev, xq):
    """A synthetic Hessian X^T X of 1024 tokens (columns of log-normal scale) for the weight xq,
    and xq's ScaleSweep-WMSE scales with the Hessian diagonal as importance."""
    g = workloads.generator(dev, 61, 99)
    X = torch.randn((1024, xq.shape[1]), generator=g, device=dev, dtype=torch.float64) * \
        torch.exp(0.7 * torch.randn(xq.shape[1], generator=g, device=dev, dtype=torch.float64))
    H = (X.T @ X).contiguous()
    del X
    imp = torch.diagonal(H).float().contiguous()
    _, scg, Sg = nv.quantize(xq, "scalesweep_wmse", 16, weight=imp)
    return H, scg, Sg


def measure_llama70b(nv, workloads, torch, dev, layers):
    """The Llama-3-70B-shaped model streamed layer by layer: each layer's weights are generated
    on the device (timed on the wall clock, separately), then quantized with ScaleSweep-WMSE in
    one batched call (dynamic S per tensor), timed with HIP events around the call.  That first
    call per layer is the streamed pass: its times summed over all layers are the model's
    kernel time.  Two more calls per layer give a median per layer as well, so that a one-off
    stall of the box can be told from the kernels' cost; the slowest single call is reported."""
    stream_ms, median_ms, elems, worst = 0.0, 0.0, 0, 0.0
    gen_s, quant_wall_s = 0.0, 0.0
    t_all = time.perf_counter()
    for li in range(layers):
        torch.cuda.synchronize()
        t_g = time.perf_counter()
        lay = workloads.llama70b_layer(li, dev)
        xs = [lay[n][0] for n in lay]
        ws_ = [lay[n][1] for n in lay]
        outs = [(torch.empty((x.shape[0], x.shape[1] // 2), dtype=torch.uint8, device=dev),
                 torch.empty((x.shape[0], x.shape[1] // 16), dtype=torch.uint8, device=dev),
                 torch.empty(1, dtype=torch.float32, device=dev)) for x in xs]
        bws = torch.empty(nv.nvfp4_batched_workspace_bytes(len(xs)) // 4, dtype=torch.int32,
                          device=dev)
        torch.cuda.synchronize()
        gen_s += time.perf_counter() - t_g
        call = lambda: nv.quantize_batched(xs, "scalesweep_wmse", 16, weights=ws_, ws=bws,
                                           outs=outs)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t_q = time.perf_counter()
        e0.record()
        call()
        e1.record()
        torch.cuda.synchronize()
        quant_wall_s += time.perf_counter() - t_q
        first = e0.elapsed_time(e1)
        ts = sorted([first] + [_timed(torch, call, 1) for _ in range(2)])
        stream_ms += first
        median_ms += ts[1]
        worst = max(worst, ts[2])
        elems += sum(x.numel() for x in xs)
        del lay, xs, ws_, outs, bws
        print(f"llama70b layer {li + 1}/{layers}: {stream_ms:.1f} ms of kernel time so far",
              file=sys.stderr, flush=True)
    wall_s = time.perf_counter() - t_all
    return {"workload": "Llama-3-70B-shaped decoder layers (q/o 8192^2, k/v 1024x8192, "
                        "gate/up 28672x8192, down 8192x28672), bf16, ScaleSweep-WMSE, block 16, "
                        "dynamic S per tensor, weights generated per layer on the device",
            "layers": layers, "elements": elems,
            "kernel_ms_total": round(stream_ms, 2),
            "input_GBps": round(2 * elems / stream_ms / 1e6, 1),
            "ms_per_layer": round(stream_ms / layers, 3),
            "quant_wall_s": round(quant_wall_s, 3),
            "generation_wall_s": round(gen_s, 3),
            "wall_s_total": round(wall_s, 3),
            "timing": "kernel time: HIP events around the one streamed call per layer; "
                      "quant_wall_s: host clock around those calls (launch to completion); "
                      "wall_s_total also holds generation and the two repeat calls",
            "median_of_3_kernel_ms_total": round(median_ms, 2),
            "median_of_3_input_GBps": round(2 * elems / median_ms / 1e6, 1),
            "slowest_call_ms": round(worst, 3)}


def profile_config(name, nv, workloads, torch, dev, copy_calibration):
    """The launches of one configuration, three of each, for counter runs (rocprofv3 groups
    its dispatches by kernel and grid).  Inputs as in the timed measurements."""
    reps = 3
    ran = []

    def run(label, fn):
        for _ in range(reps):
            fn()
        torch.cuda.synchronize()
        ran.append(label)

    if name == "c0":
        x = torch.from_numpy(workloads.c0_matrix()).to(dev)
        run("c0 fp32 [1024, 1024] scalesweep_mse D=448 dynamic",
            lambda: nv.quantize(x, "scalesweep_mse", 16, fp8_range=448.0))
    elif name == "c2":
        x, w = workloads.square8192(dev)
        for blk in (16, 32, 64, 128):
            for m in ("absmax", "four_over_six", "scalesweep_mse", "scalesweep_wmse"):
                wt = w if m == "scalesweep_wmse" else None
                run(f"c2 [8192, 8192] n={blk} {m} dynamic",
                    lambda: nv.quantize(x, m, blk, weight=wt))
    elif name == "c3":
        t = workloads.online_tensors(dev)
        for nm in ("act", "k", "v", "q"):
            xo = t[nm].reshape(-1, t[nm].shape[-1])
            for m in ("absmax", "scalesweep_mse"):
                run(f"c3 {nm} {list(t[nm].shape)} {m} static S swizzled",
                    lambda: nv.quantize_online(xo, m, 0.002, 16, layout="swizzled"))
    elif name == "c3w":
        g = workloads.generator(dev, 77)
        xb = torch.randn((32768, 8192), generator=g, device=dev).to(torch.bfloat16)
        for m in ("absmax", "scalesweep_mse"):
            run(f"c3w hidden-8192 activations [32768, 8192] {m} static S swizzled",
                lambda: nv.quantize_online(xb, m, 0.002, 16, layout="swizzled"))
    elif name == "f3":
        gate, up, imp = swiglu_inputs(workloads, torch, dev)
        h = nv.swiglu(gate, up)
        run("f3 swiglu producer [8192, 14336]", lambda: nv.swiglu(gate, up, out=h))
        for m in ("absmax", "scalesweep_mse", "scalesweep_wmse"):
            wt = imp if m == "scalesweep_wmse" else None
            run(f"f3 fused {m}", lambda: nv.quantize_online_swiglu(gate, up, m, 0.004, wt, layout="swizzled"))
            run(f"f3 unfused quantizer {m}", lambda: nv.quantize_online(h, m, 0.004, 16, wt, layout="swizzled"))
    elif name == "f4":
        xq = workloads.llama8b_layer(dev)["q_proj"][0]
        H, scg, Sg = gptq_inputs(nv, workloads, torch, dev, xq)
        run("f4 GPTQ q_proj [4096, 4096] bf16, ScaleSweep-WMSE scales, damping 0.01",
            lambda: nv.ldlq(xq, H, scg, Sg, 16, 0.01, check=False))
    else:
        lay = workloads.llama70b_layer(0, dev)
        xs = [lay[n][0] for n in lay]
        ws_ = [lay[n][1] for n in lay]
        outs = [nv.quantize(x, "scalesweep_wmse", 16, weight=w) for x, w in zip(xs, ws_)]
        run("c4 Llama-3-70B-shaped layer 0, scalesweep_wmse batched, dynamic S",
            lambda: nv.quantize_batched(xs, "scalesweep_wmse", 16, weights=ws_, outs=outs))
    if copy_calibration:     # a plain 436 MB device copy, for scaling FETCH/WRITE_SIZE
        src = torch.empty(436207616 // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        ran.append("copy of 436207616 bytes")
    print(json.dumps({"profile_config": name, "launches_each": reps, "ran": ran}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the path is built and "
              "measured on a single MI355X", file=sys.stderr)
        sys.exit(2)

    import torch

    import workloads
    import paper_2606_07618_amd as nv

    dev = torch.device("cuda:0")
    if args.profile_config:
        profile_config(args.profile_config, nv, workloads, torch, dev, args.copy_calibration)
        return
    layer = workloads.llama8b_layer(dev)
    names = list(layer)
    xs = [layer[n][0] for n in names]
    ws_col = [layer[n][1] for n in names]
    n_elem = sum(x.numel() for x in xs)
    in_bytes = 2 * n_elem
    ws = nv.workspace(dev)

    def alloc(x, block=16):
        r, c = x.shape
        return (torch.empty((r, c // 2), dtype=torch.uint8, device=dev),
                torch.empty((r, c // block), dtype=torch.uint8, device=dev),
                torch.empty(1, dtype=torch.float32, device=dev))

    outs = {m: [alloc(x) for x in xs] for m in
            ("absmax", "four_over_six", "scalesweep_mse", "scalesweep_wmse")}

    bws = torch.empty(nv.nvfp4_batched_workspace_bytes(len(xs)) // 4, dtype=torch.int32,
                      device=dev)

    def run(method, static=None):
        for i, x in enumerate(xs):
            w = ws_col[i] if method in ("scalesweep_wmse",) else None
            nv.quantize(x, method, 16, weight=w, ws=ws, out=outs[method][i],
                        static_scale=0.0 if static is None else static[i])

    def run_batched(method):
        nv.quantize_batched(xs, method, 16, weights=ws_col if method == "scalesweep_wmse" else None,
                            ws=bws, outs=outs[method])

    def step():
        run_batched("scalesweep_mse")
        run_batched("scalesweep_wmse")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = 1e3 * elapsed / args.steps
    value = 2 * in_bytes * args.steps / elapsed / 1e9

    # ---- per-method throughput (events on the current stream, which the library uses) ----
    reps = max(4, args.steps // 5)
    per_method, per_method_single = {}, {}
    for m in ("absmax", "four_over_six", "scalesweep_mse", "scalesweep_wmse"):
        for table, fn in ((per_method, run_batched), (per_method_single, run)):
            fn(m)
            torch.cuda.synchronize()
            groups = []                  # median of 5 timed groups: robust to a stray stall
            for _ in range(5):
                t_a = time.perf_counter()
                for _ in range(reps):
                    fn(m)
                torch.cuda.synchronize()
                groups.append((time.perf_counter() - t_a) * 1e3 / reps)
            ms = sorted(groups)[2]
            table[m] = {"ms_per_layer": round(ms, 4),
                        "input_GBps": round(in_bytes / ms / 1e6, 1),
                        "Gelem_per_s": round(n_elem / ms / 1e6, 2)}
    overhead = {m: round(per_method[m]["ms_per_layer"] / per_method["absmax"]["ms_per_layer"], 3)
                for m in ("four_over_six", "scalesweep_mse", "scalesweep_wmse")}

    # ---- dominant kernel alone: static-scale calls launch only the sweep kernel ----------
    scales_dyn = [float(o[2].item()) for o in outs[DOMINANT]]
    stream = torch.cuda.current_stream(dev)
    launch_ms = []
    for i, x in enumerate(xs):
        nv.quantize(x, DOMINANT, 16, weight=ws_col[i], out=outs[DOMINANT][i],
                    static_scale=scales_dyn[i])
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            nv.quantize(x, DOMINANT, 16, weight=ws_col[i], out=outs[DOMINANT][i],
                        static_scale=scales_dyn[i])
        e1.record(stream)
        torch.cuda.synchronize()
        launch_ms.append(e0.elapsed_time(e1) / reps)
    avg_launch_s = sum(launch_ms) / len(launch_ms) / 1e3
    # the same launches with L2 and MALL flushed before each (a 512 MiB fill between launches)
    flush = torch.empty(128 * 1024 * 1024, dtype=torch.float32, device=dev)
    cold_ms = []
    for i, x in enumerate(xs):
        per = []
        for r in range(reps):
            flush.fill_(float(r))
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            nv.quantize(x, DOMINANT, 16, weight=ws_col[i], out=outs[DOMINANT][i],
                        static_scale=scales_dyn[i])
            e1.record(stream)
            torch.cuda.synchronize()
            per.append(e0.elapsed_time(e1))
        cold_ms.append(sorted(per)[len(per) // 2])
    del flush
    evals_per_launch = n_elem / len(xs) * CANDIDATES_16[DOMINANT]
    ops_per_launch = evals_per_launch * OPS_PER_EVAL[DOMINANT]
    achieved = ops_per_launch / avg_launch_s / 1e12
    alg_bytes = (2 + 0.5 + 1 / 16) * n_elem / len(xs)          # read bf16, write q + scales
    roofline = {
        "bound": "alu", "achieved": round(achieved, 2), "peak": round(VALU_PEAK_TOPS, 2),
        "unit": "TOP/s", "frac": round(achieved / VALU_PEAK_TOPS, 3),
        "traffic": read_traffic(),
        "kernel": DOMINANT_SYMBOL, "avg_launch_us": round(avg_launch_s * 1e6, 2),
        "avg_launch_us_cold": round(sum(cold_ms) / len(cold_ms) * 1e3, 2),
        "algorithmic_ops_per_launch": int(ops_per_launch),
        "hbm_GBps_algorithmic": round(alg_bytes / avg_launch_s / 1e9, 1),
        "hbm_frac": round(alg_bytes / avg_launch_s / 1e9 / HBM_PEAK_GBS, 3),
    }
    # executed VALU lane-instructions (counters) per launch over the same launch time: the
    # kernel skips candidates that provably lose, so this can sit below `frac`
    valu = read_valu()
    roofline["executed_frac"] = (None if valu is None else
                                 round(valu / avg_launch_s / 1e12 / VALU_PEAK_TOPS, 3))
    roofline["executed_valu_lane_instr_per_launch"] = None if valu is None else int(valu)

    rows = None if args.no_rows else measure_rows(nv, workloads, torch, dev, layer)
    if rows is not None:
        rows["c0_fp32_1024"] = measure_c0(nv, workloads, torch, dev)
    if rows is not None and args.c4_layers > 0:
        rows["c4_llama70b_streamed"] = measure_llama70b(nv, workloads, torch, dev, args.c4_layers)

    if args.copy_calibration:
        src = torch.empty(in_bytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    # ---- CPU baseline: the oracle, one thread, on a bounded sample of the same layer -----
    cpu = None
    if not args.no_cpu:
        import oracle

        host = [(workloads.host_array(x), w.cpu().numpy()) for x, w in zip(xs, ws_col)]
        rows_per = 8
        done_elems, t_cpu = 0, 0.0
        while t_cpu < args.cpu_seconds and rows_per <= 4096:
            done_elems, t_start = 0, time.perf_counter()
            for xh, wh in host:
                sub = xh[:rows_per]
                oracle.quantize("scalesweep_mse", sub, 16, 256.0)
                oracle.quantize("scalesweep_wmse", sub, 16, 256.0, 0.0, wh)
                done_elems += sub.size
            t_cpu = time.perf_counter() - t_start
            if t_cpu < args.cpu_seconds / 4:
                rows_per *= 4
            elif t_cpu < args.cpu_seconds:
                rows_per *= 2
            else:
                break
        cpu = {"value": round(2 * 2 * done_elems / t_cpu / 1e9, 4), "unit": "GB/s", "cores": 1,
               "kind": "oracle",
               "sample": f"first {rows_per} rows of each of the 7 layer tensors "
                         f"({done_elems} bf16 elements), ScaleSweep MSE and WMSE, "
                         f"dynamic S of the sample; {t_cpu:.1f} s on one host thread"}
        # the same sample on the host's cores: the oracle's C calls release the GIL, so row
        # chunks run in parallel threads (S of each tensor's sample first, as above)
        from concurrent.futures import ThreadPoolExecutor
        model, avail = host_cpu()
        cpu["cpu_model"] = model
        cpu["cores_available"] = avail
        threads = max(1, min(16, avail))
        t_start = time.perf_counter()
        subs = [(xh[:rows_per], wh) for xh, wh in host]
        scales = [oracle.tensor_scale(sub, 256.0) for sub, _ in subs]
        tasks = []
        for (sub, wh), S_t in zip(subs, scales):
            step = max(1, -(-sub.shape[0] // threads))
            for r0 in range(0, sub.shape[0], step):
                tasks.append((sub[r0:r0 + step], wh, S_t))

        def work(task):
            part, wh, S_t = task
            oracle.quantize("scalesweep_mse", part, 16, 256.0, S_t)
            oracle.quantize("scalesweep_wmse", part, 16, 256.0, S_t, wh)

        with ThreadPoolExecutor(threads) as pool:
            list(pool.map(work, tasks))
        t_par = time.perf_counter() - t_start
        cpu["all_cores"] = {"value": round(2 * 2 * done_elems / t_par / 1e9, 4), "unit": "GB/s",
                            "cores": threads, "seconds": round(t_par, 2),
                            "note": "same sample, row chunks on a thread pool"}

    line = {
        "metric": "ScaleSweep NVFP4 quant GB/s (BF16 in) + % HBM/VALU roofline; overhead vs AbsMax",
        "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "llama3_8b_decoder_layer_weights_bf16", "tensors": {
            n: list(x.shape) for n, x in zip(names, xs)}, "elements": n_elem, "block": 16,
            "objectives": ["scalesweep_mse", "scalesweep_wmse"],
            "global_scale": "dynamic, S = amax / (6 * 256)", "value_counts": "bf16 input bytes of both objectives",
            "calls": "nvfp4_quant_batched over the 7 tensors, one call per objective"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "per_method": per_method,
        "per_method_single_calls": per_method_single,
        "rows": rows,
        "time_vs_absmax": overhead,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
