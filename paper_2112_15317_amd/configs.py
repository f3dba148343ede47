"""Workload shapes: the VGG conv stacks, the FC shards and the paper's variant.

Shapes only, no arithmetic.  ``M`` in a channel schedule is a 2x2/2 max
pool (which the library fuses with the ReLU of the conv before it).
"""
from __future__ import annotations

from dataclasses import dataclass

POOL = "M"

# VGG-16 convolutional schedule (13 conv layers, five pools).
VGG16 = [64, 64, POOL, 128, 128, POOL, 256, 256, 256, POOL,
         512, 512, 512, POOL, 512, 512, 512, POOL]

# The paper's VGG variant (Table 1): seven convs 3->64->64->128->128->256->
# 256->256; three pools bring 32x32 down to 4x4 so that the flattened
# 256x4x4 output feeds FC0 with 4096 inputs; FC 4096->1024->1024->10.
PAPER_VARIANT_CONV = [64, 64, POOL, 128, 128, POOL, 256, 256, 256, POOL]
PAPER_VARIANT_FC = [(4096, 1024), (1024, 1024), (1024, 10)]


@dataclass(frozen=True)
class ConvLayer:
    index: int        # 0-based position in the stack
    c: int            # input channels
    k: int            # output channels
    h: int            # input (= output) height
    w: int            # input (= output) width
    pool_after: bool  # a fused ReLU + 2x2 max pool follows


def conv_layers(schedule, in_ch: int, hw: int):
    """Expand a channel schedule into per-layer shapes."""
    layers = []
    c, h = in_ch, hw
    i = 0
    for j, item in enumerate(schedule):
        if item == POOL:
            continue
        pool = j + 1 < len(schedule) and schedule[j + 1] == POOL
        layers.append(ConvLayer(i, c, item, h, h, pool))
        c = item
        if pool:
            h //= 2
        i += 1
    return layers


def stack_flops(layers, n: int, with_layer1_dgrad: bool = True) -> dict:
    """Nominal multiply-add FLOPs (2 per MAC, padded taps counted) of one
    fwd + dgrad + wgrad pass, and the valid-tap count (padding excluded)."""
    nominal = 0
    valid = 0
    for L in layers:
        per_pass = 2 * n * L.k * L.c * 9 * L.h * L.w
        taps = _valid_taps(L.h) * _valid_taps(L.w)
        per_valid = 2 * n * L.k * L.c * taps
        passes = 3 if (L.index > 0 or with_layer1_dgrad) else 2
        nominal += passes * per_pass
        valid += passes * per_valid
    return {"nominal": nominal, "valid": valid}


def _valid_taps(n: int) -> int:
    # Sum over output positions of the number of in-range taps along one axis.
    return sum(sum(1 for d in (-1, 0, 1) if 0 <= p + d < n) for p in range(n))


# The five benchmark / parity workloads.
CONFIGS = {
    1: dict(kind="conv", n=8, c=3, hw=32, k=64, dtype="f32", seed=0),
    2: dict(kind="stack", schedule=VGG16, n=128, in_ch=3, hw=32, dtype="f32", seed=0),
    3: dict(kind="fc", m=512, k_in=4096, n_full=4096, shards=4, dtype="f32", seed=0),
    4: dict(kind="hybrid", schedule=VGG16, n=128, in_ch=3, hw=32, replicas=4,
            fc=[(512, 4096), (4096, 4096)], shards=4, dtype="f32", seed=0),
    5: dict(kind="stack", schedule=VGG16, n=32, in_ch=3, hw=224, dtype="bf16", seed=0),
}
