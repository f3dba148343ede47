"""Benchmark: one worker's VGG-16 CIFAR conv stack step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]

A step is the full forward and backward of the 13-layer VGG-16 conv stack on
a batch of 128 synthetic 3x32x32 images in fp32 (conv fwd with fused ReLU,
fused ReLU + 2x2 maxpool fwd/bwd, data and weight gradients of every layer,
including the first layer's data gradient), with every input resident in
HBM.  The step is ~60 short kernel launches, so it is captured once in a HIP
graph (through torch.cuda.graph: libsb enqueues on the current stream) and
the timed region is one replay of a graph of K steps, bracketed by HIP events.

Prints one JSON line: `value` is images/s; the line also carries the
achieved TFLOP/s (nominal 2*N*K*C*9*H*W per pass, and the valid-tap count
that leaves out padded taps), a per-call duration table, the roofline of the
dominant kernel and the fp64 CPU oracle's rate on a small sample of the same
workload.  Per-call durations come from a second timed region: each call of
the step captured K times back to back in its own graph, replayed between
two HIP events on the stream the kernels run on.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_MFMA_TFLOPS = 157.3      # MI355X dense fp32 matrix peak (256 CU x 2.4 GHz x 256 FLOP/clk)
PEAK_HBM_GBS = 8000.0


def layer_flops(L, n):
    """(valid-tap, nominal) FLOPs of one conv pass of layer L at batch n."""
    from paper_2112_15317_amd.configs import _valid_taps
    nominal = 2 * n * L.k * L.c * 9 * L.h * L.w
    valid = 2 * n * L.k * L.c * _valid_taps(L.h) * _valid_taps(L.w)
    return valid, nominal


def pool_bytes(L, n, esize=4):
    """Algorithmic HBM bytes of one fused ReLU + maxpool pass: per 2x2 window
    4 inputs + 1 output + 1 code byte (fwd), or 1 input + 1 code + 4 outputs
    (bwd) -- 5 elements + 1 byte either way."""
    windows = n * L.k * (L.h // 2) * (L.w // 2)
    return windows * (5 * esize + 1)


def cpu_baseline(sample_n):
    """Time the fp64 oracle on `sample_n` images of the same VGG-16 step."""
    import numpy as np
    import oracle
    from oracle import stack as OS
    from paper_2112_15317_amd import configs, synth
    layers = configs.conv_layers(configs.VGG16, 3, 32)
    x = synth.normal((sample_n, 3, 32, 32), 0, synth.TID.IMAGES)
    ws = [synth.he_normal_conv3x3(L.k, L.c, 0, synth.TID.CONV_W + L.index) for L in layers]
    bs = [np.zeros(L.k, np.float32) for L in layers]
    dy = synth.normal((sample_n, 512, 1, 1), 0, synth.TID.DY_TOP)
    pools = [L.pool_after for L in layers]
    t0 = time.perf_counter()
    OS.vgg_step(x, ws, bs, pools, dy)
    dt = time.perf_counter() - t0
    return {"value": round(sample_n / dt, 3), "unit": "images/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": "%d images of the same VGG-16 CIFAR fwd+bwd step (fp64 oracle), %.1f s"
                      % (sample_n, dt)}


def kernel_name(key, call_args):
    """Name of the main kernel a step call launches (as a profiler shows it)."""
    from paper_2112_15317_amd import sb
    kind, _ = key
    if kind in ("fwd", "dgrad", "wgrad"):
        p = {"fwd": sb.SB_PASS_FWD, "dgrad": sb.SB_PASS_BWD_DATA,
             "wgrad": sb.SB_PASS_BWD_WEIGHT}[kind]
        return sb.sb_conv3x3_plan_string(call_args[0], p)
    return "sb::relu_maxpool_%s_kernel<float, 2>" % kind.split("_")[1]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--batch", type=int, default=128)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=16)
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this library has no multi-GPU path "
              "(collectives are outside its scope); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2112_15317_amd import configs, synth
    from paper_2112_15317_amd.stack import ConvStack, capture_graph

    torch.cuda.set_device(0)
    n, K = args.batch, args.steps
    layers = configs.conv_layers(configs.VGG16, 3, 32)
    st = ConvStack(configs.VGG16, n, 3, 32, "f32")
    x = synth.normal((n, 3, 32, 32), 0, synth.TID.IMAGES)
    ws = [synth.he_normal_conv3x3(L.k, L.c, 0, synth.TID.CONV_W + L.index) for L in layers]
    dy = synth.normal((n, 512, 1, 1), 0, synth.TID.DY_TOP)
    st.load_inputs(x, ws, None, dy)
    calls = st.step_calls()

    def run_step():
        for _, fn, a in calls:
            fn(*a)

    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)

    # Timed region 1 (headline): one replay of a graph of K steps.
    g = capture_graph(run_step, K)
    g.replay()
    torch.cuda.synchronize()
    ev0.record()
    g.replay()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / K

    # Timed region 2: every call of the step, K launches back to back in a
    # graph of its own, between two events -> average duration per launch.
    per_call = {}
    for key, fn, a in calls:
        gc = capture_graph(lambda: fn(*a), K)
        gc.replay()
        torch.cuda.synchronize()
        ev0.record()
        gc.replay()
        ev1.record()
        torch.cuda.synchronize()
        per_call[key] = ev0.elapsed_time(ev1) / K
        del gc

    fl = configs.stack_flops(layers, n)
    tf_nom = fl["nominal"] / (ms * 1e-3) / 1e12
    tf_valid = fl["valid"] / (ms * 1e-3) / 1e12

    # Group the calls by kernel; the dominant kernel has the largest time per step.
    groups = {}
    for key, fn, a in calls:
        name = kernel_name(key, a)
        base = name.split(" grid=")[0]
        kind, i = key
        L = layers[i]
        work = layer_flops(L, n)[0] if kind in ("fwd", "dgrad", "wgrad") else pool_bytes(L, n)
        gr = groups.setdefault(base, {"ms": 0.0, "work": 0, "calls": [], "split": False})
        gr["ms"] += per_call[key]
        gr["work"] += work
        gr["calls"].append("%s%d" % (kind, i + 1))
        gr["split"] |= "+" in name
    dom = max(groups, key=lambda k: groups[k]["ms"])
    G = groups[dom]
    avg_us = G["ms"] * 1e3 / len(G["calls"])
    if "relu_maxpool" in dom:
        achieved = G["work"] / (G["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    else:
        achieved = G["work"] / (G["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_FP32_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_MFMA_TFLOPS, 4)}
    roof.update({"traffic": None, "kernel": dom, "calls": G["calls"],
                 "avg_us": round(avg_us, 2), "work_per_step": G["work"],
                 "includes_split_reduce": G["split"]})

    out = {
        "metric": "images/sec/GPU VGG-CIFAR conv fwd+bwd; achieved TFLOP/s vs MFMA peak",
        "value": round(n / (ms * 1e-3), 1),
        "unit": "images/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "VGG-16 CIFAR conv stack fwd+bwd (13 conv, 5 relu+maxpool), "
                               "batch 128, 3x32x32, fp32, NCHW",
                   "global_batch": n, "seq_len": None, "parallelism": "none (1 GPU)"},
        "launch": "HIP graph of %d steps" % K,
        "tflops_nominal": round(tf_nom, 2), "tflops_valid_tap": round(tf_valid, 2),
        "frac_fp32_mfma_peak_nominal": round(tf_nom / PEAK_FP32_MFMA_TFLOPS, 4),
        "roofline": roof,
        "sum_of_calls_ms": round(sum(per_call.values()), 4),
        "per_call_us": {"%s%d" % (k[0], k[1] + 1): round(v * 1e3, 1) for k, v in per_call.items()},
        "per_kernel_us_per_step": {k: round(v["ms"] * 1e3, 1) for k, v in
                                   sorted(groups.items(), key=lambda kv: -kv[1]["ms"])},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_sample)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
