"""Benchmark: one worker's VGG-16 CIFAR conv stack step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]

A step is the full forward and backward of the 13-layer VGG-16 conv stack on
a batch of 128 synthetic 3x32x32 images in fp32 (conv fwd with fused ReLU,
fused ReLU + 2x2 maxpool fwd/bwd, data and weight gradients of every layer,
including the first layer's data gradient), inputs resident in HBM.  Prints
one JSON line.  `value` is images/s; the line also carries the achieved
TFLOP/s (nominal 2*N*K*C*9*H*W per pass, and the valid-tap count that leaves
out padded taps), the roofline of the dominant kernel measured with HIP
events inside the timed region, and the fp64 CPU oracle's rate on a small
sample of the same workload.
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

PEAK_FP32_MFMA_TFLOPS = 157.3      # MI355X dense fp32 matrix peak (256 CU x 2.4 GHz x 256)
PEAK_HBM_GBS = 8000.0


def layer_flops(L, n, kind):
    """Algorithmic (valid-tap) FLOPs of one pass of one layer, and nominal."""
    from paper_2112_15317_amd.configs import _valid_taps
    nominal = 2 * n * L.k * L.c * 9 * L.h * L.w
    valid = 2 * n * L.k * L.c * _valid_taps(L.h) * _valid_taps(L.w)
    return valid, nominal


def pool_bytes(L, n, kind, esize=4):
    """Algorithmic HBM bytes of a fused ReLU + maxpool pass: per 2x2 window
    4 inputs + 1 output + 1 code byte (fwd), 1 input + 1 code + 4 outputs (bwd)."""
    windows = n * L.k * (L.h // 2) * (L.w // 2)
    return windows * (5 * esize + 1)


def cpu_baseline(sample_n=2):
    """Time the fp64 oracle on `sample_n` images of the same VGG-16 stack."""
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
    return {"value": sample_n / dt, "unit": "images/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": "%d images of the same VGG-16 CIFAR fwd+bwd step, fp64, %.1f s" % (sample_n, dt)}


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
              "(collectives are out of scope); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2112_15317_amd import configs, synth
    from paper_2112_15317_amd.stack import ConvStack, EventTimer

    torch.cuda.set_device(0)
    n = args.batch
    layers = configs.conv_layers(configs.VGG16, 3, 32)
    st = ConvStack(configs.VGG16, n, 3, 32, "f32")
    x = synth.normal((n, 3, 32, 32), 0, synth.TID.IMAGES)
    ws = [synth.he_normal_conv3x3(L.k, L.c, 0, synth.TID.CONV_W + L.index) for L in layers]
    dy = synth.normal((n, 512, 1, 1), 0, synth.TID.DY_TOP)
    st.load_inputs(x, ws, None, dy)
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        st.step()
    torch.cuda.synchronize()

    # Timed region: K steps, every libsb call bracketed by HIP events on the
    # stream it is launched on (torch's current stream).
    timer = EventTimer()
    st.call = timer
    t_start = torch.cuda.Event(enable_timing=True)
    t_stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for _ in range(args.steps):
        st.step()
    t_stop.record()
    torch.cuda.synchronize()
    st.call = lambda key, fn, *a: fn(*a)
    ms = t_start.elapsed_time(t_stop) / args.steps

    fl = configs.stack_flops(layers, n)
    tf_nom = fl["nominal"] / (ms * 1e-3) / 1e12
    tf_valid = fl["valid"] / (ms * 1e-3) / 1e12

    # Dominant call: the (pass, layer) with the largest total time.
    tot = timer.total_ms()
    mean = timer.mean_ms()
    key = max(tot, key=tot.get)
    kind, li = key
    L = layers[li]
    if kind in ("fwd", "dgrad", "wgrad"):
        alg, _ = layer_flops(L, n, kind)
        achieved = alg / (mean[key] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_FP32_MFMA_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_MFMA_TFLOPS, 4),
                "traffic": None, "kernel": "%s conv%d (%dx%d, %dx%d)" % (kind, li + 1, L.c, L.k, L.h, L.w),
                "avg_us": round(mean[key] * 1e3, 2), "flops_per_launch": alg}
    else:
        b = pool_bytes(L, n, kind)
        achieved = b / (mean[key] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None,
                "kernel": "%s pool%d" % (kind, li + 1), "avg_us": round(mean[key] * 1e3, 2)}

    per_call = {"%s%d" % (k[0], k[1] + 1): round(v * 1e3, 1) for k, v in sorted(mean.items())}
    out = {
        "metric": "images/sec/GPU VGG-CIFAR conv fwd+bwd; achieved TFLOP/s vs MFMA peak",
        "value": round(n / (ms * 1e-3), 1),
        "unit": "images/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": "VGG-16 CIFAR conv stack fwd+bwd (13 conv, 5 relu+maxpool), "
                               "batch 128, 3x32x32, fp32, NCHW",
                   "global_batch": n, "seq_len": None, "parallelism": "none (1 GPU)"},
        "tflops_nominal": round(tf_nom, 2), "tflops_valid_tap": round(tf_valid, 2),
        "frac_fp32_mfma_peak_nominal": round(tf_nom / PEAK_FP32_MFMA_TFLOPS, 4),
        "roofline": roof,
        "per_call_us": per_call,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.cpu_sample)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
