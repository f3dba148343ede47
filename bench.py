"""Benchmark: one SplitBrain worker's compute share on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline] [--only]
                    [--workload vgg16-cifar-f32 | vgg16-imagenet-bf16 |
                                fc-shard-f32 | hybrid-f32 | paper-variant-f32 |
                                exchange-f32]
                    [--profile-pass]

Default workload (the headline): one step of the 13-layer VGG-16 conv stack,
forward and backward (conv fwd with fused ReLU, fused ReLU + 2x2 maxpool
fwd/bwd, data and weight gradients of every layer, including the first
layer's data gradient), on a batch of 128 synthetic 3x32x32 images in fp32,
every input resident in HBM.  Other workloads:

  vgg16-imagenet-bf16  the same stack on 32 images of 3x224x224, bf16
                       activations and filters, fp32 accumulation;
  fc-shard-f32         one FC column shard, forward and backward, on a
                       gathered batch of 512 rows: X 512x4096, the shard's
                       1024 of 4096 output columns;
  hybrid-f32           the worker step: the VGG-16 CIFAR stack on 128 local
                       images, FC0 (512 -> 1024 of 4096, ReLU) and FC1 (4096
                       -> 1024 of 4096) shards on the gathered batch of 512,
                       then backward through both;
  paper-variant-f32    the same worker step for the paper's own VGG variant
                       (seven convs, FC 4096 -> 1024 -> 1024 -> 10) in an MP
                       group of 2: 128 local images, 256 gathered rows;
  exchange-f32         the modulo- and shard-layer data movement of one MP
                       group of 4 workers held on this device, at the hybrid
                       step's shapes, over the 4 modulo iterations: gather
                       128 x 512 rows, assemble 128 x 4096 from 1024-column
                       shards, sum and split the partial gradients back.

A step is one or several dozen kernel launches, so it is captured once in a
HIP graph (through torch.cuda.graph: libsb enqueues on the current stream)
and the timed region is one replay of a graph of K steps, bracketed by HIP
events on that stream.

Prints one JSON line: `value` is images/s (TFLOP/s for the FC shard alone,
GB/s for the exchange data movement);
the line carries the achieved TFLOP/s (nominal 2*N*K*C*9*H*W per conv pass;
the valid-tap count leaves out padded taps), a per-call duration table, the
roofline of the dominant kernel and the fp64 CPU oracle's rate on a sample
of the same workload.  Per-call durations come from a second timed region:
each call of the step captured K times back to back in a graph of its own,
replayed between two HIP events on the stream the kernels run on.

The default run (the headline workload, no --only) then times every other
workload the same way in the same process and adds their rate, step time
and dominant-kernel roofline to the line under `other_workloads`; the
headline's fields and timed regions are unaffected.

--profile-pass runs W + K plain (eager, ungraphed) steps and then three
copies of a 256 MiB buffer, and prints a one-line summary: the program that
hardware-counter runs of the profiler measure (the copy is the reference of
known size that scales the HBM byte counters).
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published dense peaks (no sparsity) and HBM bandwidth.
PEAK_MFMA_TFLOPS = {"f32": 157.3, "bf16": 2500.0}
PEAK_HBM_GBS = 8000.0
COPY_MIB = 256
TRAIN_LR = 0.01                                # SGD rate of the training-step workload

CIFAR_METRIC = "images/sec/GPU VGG-CIFAR conv fwd+bwd; achieved TFLOP/s vs MFMA peak"
FC_SHAPE = (512, 4096, 1024, 4096)            # gathered rows, k_in, shard columns, full columns
HYBRID_FC = [(512, 4096), (4096, 4096)]       # (in, out) of FC0, FC1; 4 replicas, 4 shards


def layer_flops(L, n):
    """(valid-tap, nominal) FLOPs of one conv pass of layer L at batch n."""
    from paper_2112_15317_amd.configs import _valid_taps
    nominal = 2 * n * L.k * L.c * 9 * L.h * L.w
    valid = 2 * n * L.k * L.c * _valid_taps(L.h) * _valid_taps(L.w)
    return valid, nominal


def pool_bytes(L, n, esize):
    """Algorithmic HBM bytes of one fused ReLU + maxpool pass: per 2x2 window
    4 inputs + 1 output + 1 code byte (fwd), or 1 input + 1 code + 4 outputs
    (bwd) -- 5 elements + 1 byte either way."""
    windows = n * L.k * (L.h // 2) * (L.w // 2)
    return windows * (5 * esize + 1)


def fc_flops(desc, kind, has_dx=True):
    """FLOPs of an FC shard call: 2*m*k_in*n_shard per product."""
    one = 2 * desc.m * desc.k_in * desc.n_shard
    return one if kind == "fc_fwd" else one * (2 if has_dx else 1)


def csrc_digest():
    """sha256 over the HIP sources: a stored counter reading is only valid
    for the kernels it was taken on."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2112_15317_amd", "csrc", "*"))):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def stored_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed counter summaries
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known size), or None
    when there is no reading or the kernels changed since it was taken."""
    digest = csrc_digest()
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*hbm_traffic*.md"))):
        with open(path) as fh:
            text = fh.read()
        m = re.search(r"^csrc_sha256: *([0-9a-f]+)", text, re.M)
        w = re.search(r"^workload: *(\S+)", text, re.M)
        if not m or m.group(1) != digest or not w or w.group(1) != workload:
            continue
        col = None
        for line in text.splitlines():
            if not line.startswith("|"):
                continue
            cells = [c.strip().strip("`") for c in line.strip().strip("|").split("|")]
            if "traffic_bytes_per_launch" in cells:
                col = cells.index("traffic_bytes_per_launch")
            elif col is not None and len(cells) > col and cells[0] == kernel:
                return int(cells[col])
    return None


# ----------------------------------------------------------------- inputs --
def vgg_inputs(n, hw, top):
    import numpy as np
    from paper_2112_15317_amd import configs, synth
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x = synth.normal((n, 3, hw, hw), 0, synth.TID.IMAGES)
    ws = [synth.he_normal_conv3x3(L.k, L.c, 0, synth.TID.CONV_W + L.index) for L in layers]
    bs = [np.zeros(L.k, np.float32) for L in layers]
    dy = synth.normal((n, 512, top, top), 0, synth.TID.DY_TOP)
    return layers, x, ws, bs, dy


def fc_inputs(rows=None):
    import numpy as np
    from paper_2112_15317_amd import synth
    m, kin, ns, nfull = FC_SHAPE
    m = rows or m
    x = synth.relu_normal((m, kin), 0, synth.TID.FC_X)
    w = np.ascontiguousarray(synth.xavier_uniform(kin, nfull, 0, synth.TID.FC_W)[:, :ns])
    b = np.zeros(ns, np.float32)
    dy = synth.normal((m, ns), 0, synth.TID.FC_DY)
    return x, w, b, dy


def hybrid_inputs(n, schedule, fc_shapes, group):
    """Inputs of a worker step: conv stack on n local images, FC shards on the
    rows gathered from `group` replicas, each FC split in `group` shards."""
    import numpy as np
    from paper_2112_15317_amd import configs, synth
    layers = configs.conv_layers(schedule, 3, 32)
    x = synth.normal((n, 3, 32, 32), 0, synth.TID.IMAGES)
    ws = [synth.he_normal_conv3x3(L.k, L.c, 0, synth.TID.CONV_W + L.index) for L in layers]
    bs = [np.zeros(L.k, np.float32) for L in layers]
    m = n * group
    ns = [fo // group for _, fo in fc_shapes]
    fw = [np.ascontiguousarray(synth.xavier_uniform(fi, fo, 0, synth.TID.FC_W + j)[:, :ns[j]])
          for j, (fi, fo) in enumerate(fc_shapes)]
    fb = [np.zeros(k, np.float32) for k in ns]
    rows = synth.relu_normal((m - n, fc_shapes[0][0]), 0, synth.TID.X0_REMOTE)
    cols = [synth.relu_normal((m, fc_shapes[j][0] - ns[j - 1]), 0,
                              synth.TID.X1_REMOTE if j == 1 else synth.TID.COLS_REMOTE + j)
            for j in range(1, len(fc_shapes))]
    dy = synth.normal((m, ns[-1]), 0, synth.TID.FC_DY)
    return layers, x, ws, bs, fw, fb, rows, cols, dy


# --------------------------------------------------------------- workloads --
class Workload:
    """What a benchmark run needs: the step's calls, its work, its baseline."""
    name = text = metric = dtype = None
    images = 0            # images per step (0: not an image workload)
    layers = ()

    def build(self):      # -> list of (key, libsb fn, args)
        raise NotImplementedError

    def flops(self):      # -> {"nominal": F, "valid": F}
        raise NotImplementedError

    def cpu_baseline(self, sample):
        raise NotImplementedError


class VggWorkload(Workload):
    def __init__(self, name, batch, hw, dtype, metric, text, layout="nchw"):
        self.name, self.n, self.hw, self.dtype = name, batch, hw, dtype
        self.metric, self.text, self.images = metric, text, batch
        self.top = hw // 32
        self.layout = layout

    def build(self):
        from paper_2112_15317_amd import configs
        from paper_2112_15317_amd.stack import ConvStack
        self.layers, x, ws, _, dy = vgg_inputs(self.n, self.hw, self.top)
        self.st = ConvStack(configs.VGG16, self.n, 3, self.hw, self.dtype, layout=self.layout)
        self.st.load_inputs(x, ws, None, dy)
        return self.st.step_calls()

    def flops(self):
        from paper_2112_15317_amd import configs
        return configs.stack_flops(self.layers, self.n)

    def cpu_baseline(self, sample):
        import oracle
        from oracle import stack as OS
        sample = sample or (self.n if self.hw <= 32 else 8)
        layers, x, ws, bs, dy = vgg_inputs(sample, self.hw, self.top)
        bf16 = self.dtype == "bf16"
        if bf16:
            x = oracle.round_bf16(x)
            ws = [oracle.round_bf16(w) for w in ws]
            dy = oracle.round_bf16(dy)
        pools = [L.pool_after for L in layers]
        reps = 3 if self.hw <= 32 else 1
        t0 = time.perf_counter()
        for _ in range(reps):
            OS.vgg_step(x, ws, bs, pools, dy, bf16=bf16)
        dt = time.perf_counter() - t0
        return {"value": round(reps * sample / dt, 3), "unit": "images/s",
                "cores": oracle.num_threads(), "kind": "oracle",
                "sample": "%d x the fwd+bwd step on %d images (fp64 oracle%s), %.1f s"
                          % (reps, sample, ", bf16 rounding at storage points" if bf16 else "",
                             dt)}


class FcWorkload(Workload):
    name = "fc-shard-f32"
    dtype = "f32"
    metric = "TFLOP/s FC column shard fwd+bwd on the gathered batch (fp32)"
    text = ("FC column shard fwd+bwd: X 512x4096 gathered rows, W_shard 4096x1024 "
            "(1024 of 4096 output columns), partial dX 512x4096, dW 4096x1024, fp32")

    def build(self):
        import torch
        from paper_2112_15317_amd.stack import FCShard
        m, kin, ns, _ = FC_SHAPE
        x, w, b, dy = fc_inputs()
        self.fc = FCShard(m, kin, ns)
        t = lambda a: torch.from_numpy(a).cuda()
        self.x, self.dy = t(x), t(dy)
        self.fc.W.copy_(t(w))
        self.fc.b.copy_(t(b))
        self.y = torch.empty((m, ns), device="cuda")
        self.dx = torch.empty((m, kin), device="cuda")
        return [(("fc_fwd", 0),) + self.fc.fwd_call(self.x, self.y),
                (("fc_bwd", 0),) + self.fc.bwd_call(self.x, self.dy, None, self.dx)]

    def flops(self):
        f = fc_flops(self.fc.desc_f, "fc_fwd") + fc_flops(self.fc.desc_b, "fc_bwd")
        return {"nominal": f, "valid": f}

    def cpu_baseline(self, sample):
        import oracle
        sample = sample or FC_SHAPE[0]
        x, w, b, dy = fc_inputs(sample)
        reps = 3
        t0 = time.perf_counter()
        for _ in range(reps):
            oracle.fc_fwd(x, w, b)
            oracle.fc_bwd(x, w, dy)
        dt = time.perf_counter() - t0
        f = reps * 6 * sample * FC_SHAPE[1] * FC_SHAPE[2]
        return {"value": round(f / dt / 1e12, 5), "unit": "TFLOP/s",
                "cores": oracle.num_threads(), "kind": "oracle",
                "sample": "%d x fwd+bwd of the shard on %d gathered rows (fp64 oracle), %.1f s"
                          % (reps, sample, dt)}


class HybridWorkload(Workload):
    dtype = "f32"
    images = 128

    def __init__(self, name, schedule, fc_shapes, group, metric, text):
        self.name, self.schedule, self.fc_shapes, self.group = name, schedule, fc_shapes, group
        self.metric, self.text = metric, text

    def build(self):
        from paper_2112_15317_amd.stack import HybridStep
        inp = hybrid_inputs(self.images, self.schedule, self.fc_shapes, self.group)
        self.layers = inp[0]
        self.hs = HybridStep(self.schedule, self.images, 3, 32, self.group, self.fc_shapes,
                             self.group)
        self.hs.load_inputs(*inp[1:])
        return self.hs.step_calls()

    def flops(self):
        from paper_2112_15317_amd import configs
        f = configs.stack_flops(self.layers, self.images)
        extra = sum(fc_flops(s.desc_f, "fc_fwd") + fc_flops(s.desc_b, "fc_bwd")
                    for s in self.hs.fc)
        return {"nominal": f["nominal"] + extra, "valid": f["valid"] + extra}

    def cpu_baseline(self, sample):
        import oracle
        from oracle import stack as OS
        n = self.images
        layers, x, ws, bs, fw, fb, rows, cols, dy = hybrid_inputs(
            n, self.schedule, self.fc_shapes, self.group)
        pools = [L.pool_after for L in layers]
        t0 = time.perf_counter()
        OS.hybrid_step(x, ws, bs, pools, fw, fb, rows, cols, dy)
        dt = time.perf_counter() - t0
        return {"value": round(n / dt, 3), "unit": "images/s",
                "cores": oracle.num_threads(), "kind": "oracle",
                "sample": "1 x the whole hybrid step, %d local images (fp64 oracle), %.1f s"
                          % (n, dt)}


def group_inputs(n, schedule, fc_shapes, K):
    """Inputs of an MP group's training step: worker 0's conv stack on n
    local images, the other workers' conv outputs, the full dense layers
    (worker r's shard = its 1/K of the columns) and the labels of every
    iteration's gathered rows."""
    import numpy as np
    from paper_2112_15317_amd import configs, synth
    layers = configs.conv_layers(schedule, 3, 32)
    x = synth.normal((n, 3, 32, 32), 0, synth.TID.IMAGES)
    ws = [synth.he_normal_conv3x3(L.k, L.c, 0, synth.TID.CONV_W + L.index) for L in layers]
    bs = [np.zeros(L.k, np.float32) for L in layers]
    fw = [synth.xavier_uniform(fi, fo, 0, synth.TID.FC_W + j)
          for j, (fi, fo) in enumerate(fc_shapes)]
    fb = [np.zeros(fo, np.float32) for _, fo in fc_shapes]
    remote = synth.relu_normal((K - 1, n, fc_shapes[0][0]), 0, synth.TID.X0_REMOTE)
    labels = synth.labels(K * n, fc_shapes[-1][1], 0, synth.TID.LABELS).reshape(K, n)
    return layers, x, ws, bs, fw, fb, remote, labels


class GroupWorkload(Workload):
    """Training step of an MP group of K (sec. 3.1): worker 0's conv stack,
    K modulo iterations of every worker's FC shards with an SGD step after
    each, the conv backward and update."""
    dtype = "f32"
    images = 128

    def __init__(self, name, schedule, fc_shapes, K, metric, text):
        self.name, self.schedule, self.fc_shapes, self.K = name, schedule, fc_shapes, K
        self.metric, self.text = metric, text

    def build(self):
        from paper_2112_15317_amd import partition as P
        from paper_2112_15317_amd.stack import GroupTrainStep
        inp = group_inputs(self.images, self.schedule, self.fc_shapes, self.K)
        self.layers = inp[0]
        plan = P.fc_plan(P.partition(P.vgg_net(self.schedule, 3, 32, self.fc_shapes), self.K))
        self.gs = GroupTrainStep(self.schedule, self.images, 3, 32, plan, lr=TRAIN_LR)
        self.gs.load_inputs(*inp[1:])
        return self.gs.step_calls()

    def call_bytes(self, key, args):
        gs, (kind, j) = self.gs, key
        K, B = gs.K, gs.B
        if kind == "loss":           # logits read, gradient written, labels and losses
            return 2 * B * gs.classes * 4 + 2 * B * 4
        if kind in ("mfwd", "mbwd"):
            return 4 * (2 * B * gs.F if kind == "mfwd" else (K + 1) * B * gs.F)
        if kind in ("sfwd", "sbwd"):
            ns = gs.ns[j] if kind == "sfwd" else gs.ns[j - 1]
            return 4 * (2 * K * B * ns if kind == "sfwd" else (K + 1) * K * B * ns)
        # sgd: each parameter read and written, its gradient read
        if kind == "sgd_fc":
            n = sum(w.numel() + b.numel() for w, b in zip(gs.W, gs.b))
        else:
            n = sum(w.numel() + b.numel() for w, b in zip(gs.conv.W, gs.conv.b))
        return 12 * n

    def flops(self):
        from paper_2112_15317_amd import configs
        f = configs.stack_flops(self.layers, self.images)
        gs = self.gs
        # K iterations x K workers' shards, forward and backward (both products).
        extra = sum(gs.K * gs.K * 6 * gs.B * gs.ins[j] * gs.ns[j] for j in range(gs.L))
        return {"nominal": f["nominal"] + extra, "valid": f["valid"] + extra}

    def cpu_baseline(self, sample):
        import oracle
        from oracle import stack as OS
        layers, x, ws, bs, fw, fb, remote, labels = group_inputs(
            self.images, self.schedule, self.fc_shapes, self.K)
        pools = [L.pool_after for L in layers]
        t0 = time.perf_counter()
        OS.group_train_step(x, ws, bs, pools, fw, fb, remote, labels, TRAIN_LR)
        dt = time.perf_counter() - t0
        return {"value": round(self.images / dt, 3), "unit": "images/s",
                "cores": oracle.num_threads(), "kind": "oracle",
                "sample": "1 x the whole training step of the group, %d local images on "
                          "worker 0 (fp64 oracle), %.1f s" % (self.images, dt)}


class ExchangeWorkload(Workload):
    """Modulo / shard layers of one MP group (sec. 3.1, 3.2) on one device."""
    name = "exchange-f32"
    dtype = "f32"
    metric = "GB/s modulo + shard layer data movement of one MP group on one GPU (fp32)"
    text = ("modulo and shard layers of an MP group of 4 workers held on one GPU, all 4 "
            "modulo iterations: gather 128x512 (of 4 local batches of 128x512), assemble "
            "128x4096 from 4 shards of 128x1024, sum 4 partial 128x4096 gradients into the "
            "shards' slices and 4 partial 128x512 into the local rows, fp32")
    K, B, F, NS = 4, 128, 512, 1024

    def inputs(self):
        from paper_2112_15317_amd import synth
        K, B, F, NS = self.K, self.B, self.F, self.NS
        T = synth.TID.MISC
        return (synth.normal((K, B, F), 0, T + 11), synth.normal((K, B, K * NS), 0, T + 12),
                synth.normal((K, B, NS), 0, T + 13), synth.normal((K, B, F), 0, T + 14))

    def build(self):
        import numpy as np
        import torch
        from paper_2112_15317_amd import sb
        K, B, F, NS = self.K, self.B, self.F, self.NS
        local, dfull, parts, dg = (torch.from_numpy(a.astype(np.float32)).cuda()
                                   for a in self.inputs())
        self.t = dict(local=local, dfull=dfull, parts=parts, dg=dg,
                      gathered=torch.empty((B, F), device="cuda"),
                      full=torch.empty((B, K * NS), device="cuda"),
                      dparts=torch.empty((K, B, NS), device="cuda"),
                      dlocal=torch.empty((K, B, F), device="cuda"))
        md, sd = sb.modulo_desc(K, K, B, F), sb.shard_desc(K, K, B, NS)
        t = self.t
        calls = []
        for k in range(K):
            calls += [(("mfwd", k), sb.sb_modulo_fwd, (md, 0, k, t["local"], t["gathered"])),
                      (("sfwd", k), sb.sb_shard_fwd, (sd, 0, t["parts"], t["full"])),
                      (("sbwd", k), sb.sb_shard_bwd, (sd, 0, t["dfull"], t["dparts"])),
                      (("mbwd", k), sb.sb_modulo_bwd, (md, 0, k, t["dg"], t["dlocal"]))]
        return calls

    def call_bytes(self, key, args=None):
        K, B, F, NS = self.K, self.B, self.F, self.NS
        kind = key[0]
        return 4 * {"mfwd": 2 * B * F, "sfwd": 2 * K * B * NS,
                    "sbwd": K * B * K * NS + K * B * NS, "mbwd": K * B * F + B * F}[kind]

    def bytes_per_step(self):
        return self.K * sum(self.call_bytes((k, 0)) for k in ("mfwd", "sfwd", "sbwd", "mbwd"))

    def flops(self):
        return {"nominal": 0, "valid": 0}

    def cpu_baseline(self, sample):
        from oracle import modulo as OM
        import numpy as np
        local, dfull, parts, dg = self.inputs()
        K = self.K
        reps = 0
        t0 = time.perf_counter()
        while reps == 0 or time.perf_counter() - t0 < 10.0:   # about 10 s of CPU work
            dl = np.zeros_like(dg)
            for k in range(K):
                OM.modulo_fwd(local, 0, k, K)
                OM.shard_fwd(parts, 0, K)
                OM.shard_bwd(dfull, 0, K, np.zeros_like(parts))
                dl = OM.modulo_bwd(dg, 0, k, K, dl)
            reps += 1
        dt = time.perf_counter() - t0
        return {"value": round(reps * self.bytes_per_step() / dt / 1e9, 3), "unit": "GB/s",
                "cores": 1, "kind": "oracle",
                "sample": "%d x the whole step (4 modulo iterations; fp64 numpy oracle, one "
                          "thread), %.1f s" % (reps, dt)}



class AverageWorkload(Workload):
    """Model averaging of DP replicas (sec. 2, sec. 4) on one device."""
    name = "average-f32"
    dtype = "f32"
    metric = "GB/s model averaging of data-parallel replicas on one GPU (fp32)"
    text = ("model averaging of 4 data-parallel replicas held on one GPU: every replica's "
            "VGG-16 conv parameters (14,714,688 fp32 weights and biases) replaced by the "
            "mean of the 4, in place")
    W = 4

    def n(self):
        from paper_2112_15317_amd import configs
        return sum(L.k * L.c * 9 + L.k for L in configs.conv_layers(configs.VGG16, 3, 32))

    def build(self):
        import torch
        from paper_2112_15317_amd import sb, synth
        self.p = torch.from_numpy(synth.normal((self.W, self.n()), 0, synth.TID.MISC + 15)).cuda()
        return [(("avg", 0), sb.sb_model_average, (self.W, 1, self.p))]

    def call_bytes(self, key=None, args=None):
        return 2 * self.W * self.n() * 4          # every slot read once and written once

    def bytes_per_step(self):
        return self.call_bytes()

    def flops(self):
        return {"nominal": 0, "valid": 0}

    def cpu_baseline(self, sample):
        from oracle import average as OA
        from paper_2112_15317_amd import synth
        rows = sample or 1 << 20                   # parameters per replica in the sample
        p = synth.normal((self.W, rows), 0, synth.TID.MISC + 15)
        reps = 0
        t0 = time.perf_counter()
        while reps == 0 or time.perf_counter() - t0 < 10.0:   # about 10 s of CPU work
            OA.model_average(p, 1)
            reps += 1
        dt = time.perf_counter() - t0
        return {"value": round(reps * 2 * self.W * rows * 4 / dt / 1e9, 3), "unit": "GB/s",
                "cores": 1, "kind": "oracle",
                "sample": "%d x averaging 4 replicas of %d parameters (fp64 numpy oracle, one "
                          "thread), %.1f s" % (reps, rows, dt)}

def workloads():
    from paper_2112_15317_amd import configs
    return {
        "vgg16-cifar-f32": VggWorkload(
            "vgg16-cifar-f32", 128, 32, "f32", CIFAR_METRIC,
            "VGG-16 CIFAR conv stack fwd+bwd (13 conv, 5 relu+maxpool), batch 128, 3x32x32, "
            "fp32"),
        "vgg16-imagenet-bf16": VggWorkload(
            "vgg16-imagenet-bf16", 32, 224, "bf16",
            "images/sec/GPU VGG-16 ImageNet-shaped conv fwd+bwd (bf16); achieved TFLOP/s vs "
            "MFMA peak",
            "VGG-16 ImageNet-shaped conv stack fwd+bwd (13 conv, 5 relu+maxpool), batch 32, "
            "3x224x224, bf16 activations and filters, fp32 accumulation", layout="c8"),
        "fc-shard-f32": FcWorkload(),
        "hybrid-f32": HybridWorkload(
            "hybrid-f32", configs.VGG16, HYBRID_FC, 4,
            "images/sec/GPU hybrid worker step (VGG-16 CIFAR conv DP + FC shards MP), fp32",
            "hybrid worker step: VGG-16 CIFAR conv stack on 128 local images, then FC0 "
            "512->1024 (of 4096, ReLU) and FC1 4096->1024 (of 4096) shards on the gathered 512 "
            "rows, fwd+bwd, fp32"),
        "paper-variant-f32": GroupWorkload(
            "paper-variant-f32", configs.PAPER_VARIANT_CONV, configs.PAPER_VARIANT_FC, 2,
            "images/sec/GPU training step of the paper's VGG variant (Table 1) in an MP group "
            "of 2, fp32",
            "training step of the paper's VGG variant in an MP group of 2 on one GPU: seven "
            "3x3 convs (64,64,M,128,128,M,256,256,256,M) on worker 0's 128 local 3x32x32 "
            "images; 2 modulo iterations, each gathering 128 rows (64 per worker) and running "
            "both workers' column shards of FC 4096->1024->1024->10 with shard layers "
            "between them, log-softmax + NLL of the full 10-class logits, the backward and an "
            "FC SGD step at lr/2; then the conv backward and SGD at lr; fp32"),
        "exchange-f32": ExchangeWorkload(),
        "average-f32": AverageWorkload(),
    }


def kernel_name(key, call_args, dtype):
    """Name of the main kernel a step call launches (as a profiler shows it);
    FC calls launch several GEMMs and are grouped by call."""
    from paper_2112_15317_amd import sb
    kind, j = key
    if kind in ("fwd", "dgrad", "wgrad", "fwd_pool"):
        p = {"fwd": sb.SB_PASS_FWD, "dgrad": sb.SB_PASS_BWD_DATA,
             "wgrad": sb.SB_PASS_BWD_WEIGHT, "fwd_pool": sb.SB_PASS_FWD_POOL}[kind]
        return sb.sb_conv3x3_plan_string(call_args[0], p)
    if kind == "wgrad_many":       # one launch of the batched kernel for the group
        wl = call_args[0]
        name = sb.sb_conv3x3_plan_string(wl.descs[0], sb.SB_PASS_BWD_WEIGHT).split(" grid=")[0]
        return name.replace("conv3x3_wgrad_f32<", "conv3x3_wgrad_f32_many<") + \
            " grid=%dx1x2" % wl.count
    if kind.startswith("fc_"):
        d = call_args[0]
        return "sb_fc_shard_%s m=%d k_in=%d n_shard=%d" % (kind[3:], d.m, d.k_in, d.n_shard)
    if kind == "pack":
        return "sb::filter_pack_many"
    if kind in ("mfwd", "mbwd", "sfwd", "sbwd"):
        return "sb::%s_%s_kernel<4>" % ("modulo" if kind[0] == "m" else "shard",
                                        "fwd" if kind[1:] == "fwd" else "bwd")
    if kind == "loss":
        return "sb::log_softmax_nll_kernel"
    if kind in ("sgd_fc", "sgd_conv"):
        return "sb::sgd_update_kernel"
    if kind == "avg":
        return "sb::model_average_kernel<4>"
    if call_args[5] == sb.SB_NCHW8C:
        return "sb::relu_maxpool_%s_c8" % kind.split("_")[1]
    return "sb::relu_maxpool_%s_kernel<%s, 2>" % (
        kind.split("_")[1], "float" if dtype == "f32" else "unsigned short")


def call_work(wl, key, args):
    """Algorithmic work of one call: (amount, 'flop' | 'bytes')."""
    kind, i = key
    if kind in ("fwd", "dgrad", "wgrad", "fwd_pool"):
        return layer_flops(wl.layers[i], args[0].n)[0], "flop"
    if kind == "wgrad_many":       # the group's layers, from their descriptors
        from paper_2112_15317_amd.configs import _valid_taps
        return sum(2 * d.n * d.k * d.c * _valid_taps(d.h) * _valid_taps(d.w)
                   for d in args[0].descs), "flop"
    if kind.startswith("fc_"):
        return fc_flops(args[0], kind, kind == "fc_fwd" or args[5] is not None), "flop"
    if kind in ("mfwd", "mbwd", "sfwd", "sbwd", "loss", "sgd_fc", "sgd_conv", "avg"):
        return wl.call_bytes(key, args), "bytes"
    esize = 4 if wl.dtype == "f32" else 2
    if kind == "pack":             # every layer's filters read, twice packed written
        return sum(3 * L.k * L.c * 9 * esize for L in wl.layers), "bytes"
    return pool_bytes(wl.layers[i], args[0], esize), "bytes"


def measure(wl, K, warmup):
    """Time workload `wl` (already chosen and configured) on the current
    GPU: warm-up steps, timed region 1 (a graph of K steps), timed region 2
    (each call K times in a graph of its own).  Returns the JSON fields."""
    import torch
    from paper_2112_15317_amd.stack import capture_graph
    dtype = wl.dtype
    calls = wl.build()

    def run_step():
        for _, fn, a in calls:
            fn(*a)

    for _ in range(warmup):
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
    del g

    # Timed region 2: every call of the step, K launches back to back in a
    # graph of its own, between two events -> average duration per launch.
    per_call = []                 # ms per launch, in the order of `calls`
    for key, fn, a in calls:
        gc = capture_graph(lambda: fn(*a), K)
        gc.replay()
        torch.cuda.synchronize()
        ev0.record()
        gc.replay()
        ev1.record()
        torch.cuda.synchronize()
        per_call.append(ev0.elapsed_time(ev1) / K)
        del gc
    # Call names: kind + 1-based index, "#n" for a repeated key (a group
    # step runs the same layer's call once per worker and iteration).
    names, seen = [], {}
    for key, _, _ in calls:
        base = "%s%d" % (key[0], key[1] + 1)
        seen[base] = seen.get(base, 0) + 1
        names.append(base if seen[base] == 1 else "%s#%d" % (base, seen[base]))

    fl = wl.flops()
    peak = PEAK_MFMA_TFLOPS[dtype]
    tf_nom = fl["nominal"] / (ms * 1e-3) / 1e12
    tf_valid = fl["valid"] / (ms * 1e-3) / 1e12
    moved = getattr(wl, "bytes_per_step", None)

    # Group the calls by kernel; the dominant kernel has the largest time per step.
    groups = {}
    for (key, fn, a), t, cname in zip(calls, per_call, names):
        name = kernel_name(key, a, dtype)
        base = name.split(" grid=")[0]
        work, unit = call_work(wl, key, a)
        gr = groups.setdefault(base, {"ms": 0.0, "work": 0, "unit": unit, "calls": [],
                                      "split": False})
        gr["ms"] += t
        gr["work"] += work
        gr["calls"].append(cname)
        gr["split"] |= bool(re.search(r"grid=\d+x\d+x([2-9]|\d\d)", name))
    dom = max(groups, key=lambda k: groups[k]["ms"])
    G = groups[dom]
    launches = len(G["calls"])
    avg_us = G["ms"] * 1e3 / launches
    if G["unit"] == "bytes":
        achieved = G["work"] / (G["ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    else:
        achieved = G["work"] / (G["ms"] * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4)}
    roof.update({"traffic": stored_traffic(dom, wl.name), "kernel": dom,
                 "calls": G["calls"], "avg_us": round(avg_us, 2),
                 "work_per_launch": G["work"] // launches,
                 "work_unit": "bytes" if G["unit"] == "bytes" else "valid-tap FLOP",
                 "includes_split_reduce": G["split"]})

    if wl.images:
        value, unit = round(wl.images / (ms * 1e-3), 1), "images/s"
    elif moved:
        value, unit = round(moved() / (ms * 1e-3) / 1e9, 1), "GB/s"
    else:
        value, unit = round(tf_nom, 2), "TFLOP/s"
    out = {
        "metric": wl.metric,
        "value": value,
        "unit": unit,
        "n_gpus": 1, "steps": K, "warmup": warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dtype, "data": "synthetic",
        "config": dict({"workload": wl.text, "global_batch": wl.images or FC_SHAPE[0],
                        "parallelism": "none (1 GPU)"},
                       **({"layout": wl.layout} if isinstance(wl, VggWorkload) else {})),
        "launch": "HIP graph of %d steps" % K,
        "tflops_nominal": None if moved else round(tf_nom, 2),
        "tflops_valid_tap": None if moved else round(tf_valid, 2),
        "frac_mfma_peak_nominal": None if moved else round(tf_nom / peak, 4),
        "roofline": roof,
        "sum_of_calls_ms": round(sum(per_call), 4),
        "per_call_us": {n: round(v * 1e3, 1) for n, v in zip(names, per_call)},
        "per_kernel_us_per_step": {k: round(v["ms"] * 1e3, 1) for k, v in
                                   sorted(groups.items(), key=lambda kv: -kv[1]["ms"])},
    }
    return out


def main():
    W = workloads()
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", choices=sorted(W), default="vgg16-cifar-f32")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="images (rows for the FC shard) the oracle times")
    ap.add_argument("--profile-pass", action="store_true")
    ap.add_argument("--layout", choices=["nchw", "c8"], default=None,
                    help="activation layout of a VGG stack (default: the workload's)")
    ap.add_argument("--only", action="store_true",
                    help="time the chosen workload alone (by default the headline run "
                         "also times every other workload, reported under "
                         "other_workloads)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: this library has no multi-GPU path "
              "(collectives are outside its scope); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    wl = W[args.workload]
    if args.layout is not None:
        if not isinstance(wl, VggWorkload):
            ap.error("--layout applies to the VGG stack workloads")
        wl.layout = args.layout
    torch.cuda.set_device(0)
    K = args.steps

    if args.profile_pass:
        calls = wl.build()
        for _ in range(args.warmup + K):
            for _, fn, a in calls:
                fn(*a)
        torch.cuda.synchronize()
        a = torch.empty(COPY_MIB << 18, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        a.fill_(1.0)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"profile_pass": args.workload, "steps": args.warmup + K,
                          "copy_bytes": COPY_MIB << 20, "csrc_sha256": csrc_digest()}),
              flush=True)
        return

    out = measure(wl, K, args.warmup)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = wl.cpu_baseline(args.cpu_sample)
    if not args.only and args.workload == "vgg16-cifar-f32" and args.layout is None:
        # The other workloads at their own configurations, same process and
        # GPU, after the headline's timed regions (their rate, step time and
        # dominant kernel's roofline; no CPU baselines).
        others = {}
        for name, other in W.items():
            if name == args.workload:
                continue
            try:
                o = measure(other, K, args.warmup)
                others[name] = {k: o[k] for k in ("metric", "value", "unit", "ms_per_step",
                                                  "dtype", "config")}
                others[name]["roofline"] = {k: o["roofline"][k] for k in
                                            ("kernel", "bound", "achieved", "unit", "frac")}
            except Exception as e:          # reported, never hides the headline
                others[name] = {"error": "%s: %s" % (type(e).__name__, e)}
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
        out["other_workloads"] = others
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
