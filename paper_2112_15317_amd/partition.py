"""Host-side model partitioning (sec. 3.1, Layer Partitioning).

The paper's procedure walks a sequential CNN and builds its hybrid
counterpart: layers that reshape, pad, convolve or pool are never split and
need an unpartitioned input; element-wise functional layers (ReLU, dropout)
follow whatever width their input has; a fully connected (LINEAR) layer is
split to 1/K of its outputs when model parallelism is on and its
computation-to-communication ratio (CCR) is large enough.  A modulo layer is
inserted before the first split FC layer (its input is still whole), a shard
layer before every later FC layer whose input is partitioned, and a shard
layer before LOG_SOFTMAX when the output is partitioned, so the loss sees
the complete output.

Two dimensions travel along the walk: ``dim``, the width of the current
activation on this worker, and ``dim_full``, its width in the unsplit
model.  They differ exactly while the activation is partitioned.

The paper leaves the CCR and its threshold unstated.  Here the CCR of a
LINEAR layer of ``i`` inputs and ``o`` outputs is its forward plus backward
arithmetic per example, ``3 * 2 * i * o`` FLOP, over the bytes its model
parallelism exchanges per example, its fp32 input and output gradient-sized
activations, ``4 * (i + o)``; the default threshold, 1 FLOP/byte, splits
every FC layer of the paper's VGG variant (whose three FC layers it splits
for their memory, sec. 5).

Host code: this module computes nothing on the GPU.  ``fc_plan`` turns the
partitioned list into the call sequence of the training step
(``stack.GroupTrainStep``): its modulo, shard, split dense and loss layers,
in order.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional


# Layer kinds of the paper's sequential CNNs, plus the two it inserts.
SEQ, RESHAPE, PAD, CONV, POOLING, DROPOUT, RELU, LINEAR, LOG_SOFTMAX = (
    "SEQ", "RESHAPE", "PAD", "CONV", "POOLING", "DROPOUT", "RELU", "LINEAR", "LOG_SOFTMAX")
MODULO, SHARD = "MODULO", "SHARD"
_UNSPLIT = (RESHAPE, PAD, CONV, POOLING)
_ELEMENTWISE = (DROPOUT, RELU)


@dataclass
class Layer:
    """A layer with flattened input and output widths (features per example).

    ``out_dim`` of a split LINEAR layer is its own share of the outputs;
    ``full_out`` is the unsplit layer's.  MODULO carries the width it
    gathers (``in_dim``); SHARD the partition width (``in_dim``) and the full
    width it assembles (``out_dim``).
    """
    kind: str
    in_dim: int = 0
    out_dim: int = 0
    children: List["Layer"] = field(default_factory=list)
    shards: int = 1                  # LINEAR: 1 / shards of the outputs live here
    full_out: Optional[int] = None   # LINEAR: outputs of the unsplit layer

    def resize(self, dim: int) -> int:
        """Output width for an input of width ``dim``."""
        if self.kind in _ELEMENTWISE or self.kind == LOG_SOFTMAX:
            return dim
        if dim != self.in_dim:
            raise ValueError("%s expects %d inputs, gets %d" % (self.kind, self.in_dim, dim))
        return self.out_dim


def seq(*layers: Layer) -> Layer:
    return Layer(SEQ, children=list(layers))


def linear(i: int, o: int) -> Layer:
    return Layer(LINEAR, i, o, full_out=o)


def ccr(layer: Layer) -> float:
    """FLOP of forward + backward per byte exchanged, per example."""
    i, o = layer.in_dim, layer.full_out or layer.out_dim
    return 6.0 * i * o / (4.0 * (i + o))


# How each layer kind treats the width of its input (sec. 3.1, Layer
# Partitioning): layers that reshape, pad, convolve or pool see whole
# examples only; element-wise layers keep whatever width they are given; a
# dense layer may be split over its outputs; the loss needs the whole output.
_ROLE = {RESHAPE: "whole", PAD: "whole", CONV: "whole", POOLING: "whole",
         DROPOUT: "pointwise", RELU: "pointwise", LINEAR: "dense", LOG_SOFTMAX: "loss"}


def flatten(net: Layer) -> List[Layer]:
    """The leaves of nested SEQ containers, in order."""
    if net.kind != SEQ:
        return [net]
    return [leaf for child in net.children for leaf in flatten(child)]


def partition(net: Layer, workers: int, threshold: float = 1.0) -> List[Layer]:
    """The hybrid layer list of ``net`` for MP groups of ``workers`` (the
    paper's K; 1 = no model parallelism).

    A fold over the flattened layers that carries two widths per example:
    the activation as this worker holds it (``local``) and as the unsplit
    model has it (``whole``); they differ exactly while the activation is
    partitioned.  Before a dense layer with a partitioned input a SHARD
    layer restores the whole width; a dense layer with a whole input that is
    split becomes the first split layer, so a MODULO layer goes in front of
    it (the input is still per-worker data, gathered by rows); before the
    loss a partitioned output is made whole by a SHARD layer."""
    if workers < 1:
        raise ValueError("workers must be >= 1")
    leaves = flatten(net)
    if not leaves:
        return []
    out: List[Layer] = []
    local = whole = leaves[0].in_dim

    for layer in leaves:
        role = _ROLE.get(layer.kind)
        if role is None:
            raise ValueError("no partitioning rule for layer kind %r" % layer.kind)
        if role == "whole":
            if local != whole:
                raise ValueError("%s cannot take a column-split input (%d of %d features)"
                                 % (layer.kind, local, whole))
            local = whole = layer.resize(whole)
            out.append(layer)
        elif role == "pointwise":
            local = layer.resize(local)
            out.append(layer)
        elif role == "dense":
            if layer.in_dim != whole:
                raise ValueError("dense layer of %d inputs after %d features"
                                 % (layer.in_dim, whole))
            split = workers > 1 and ccr(layer) > threshold
            if local != whole:
                out.append(Layer(SHARD, local, whole))
            elif split:
                out.append(Layer(MODULO, whole, whole))
            full_out = layer.full_out or layer.out_dim
            if split:
                if full_out % workers:
                    raise ValueError("%d outputs cannot be split evenly over %d workers"
                                     % (full_out, workers))
                layer = Layer(LINEAR, layer.in_dim, full_out // workers, shards=workers,
                              full_out=full_out)
            out.append(layer)
            local, whole = layer.out_dim, full_out
        else:                                   # the loss
            if local != whole:
                out.append(Layer(SHARD, local, whole))
                local = whole
            out.append(layer)
    return out


def fc_plan(layers: List[Layer]):
    """The model-parallel tail of a partitioned layer list as the training
    step runs it: from the MODULO layer on, a list of
    ``("modulo", features)``, ``("linear", in, shard_out, full_out, relu)``
    (relu: a ReLU follows the layer), ``("shard", part, full)`` and
    ``("loss", classes)`` entries.  Dropout is not part of any workload and
    is refused, as is a tail that does not start with a MODULO layer."""
    kinds = [l.kind for l in layers]
    if MODULO not in kinds:
        raise ValueError("no model-parallel part: the list has no MODULO layer")
    tail = layers[kinds.index(MODULO):]
    plan = []
    for i, l in enumerate(tail):
        if l.kind == MODULO:
            plan.append(("modulo", l.in_dim))
        elif l.kind == LINEAR:
            relu = i + 1 < len(tail) and tail[i + 1].kind == RELU
            plan.append(("linear", l.in_dim, l.out_dim, l.full_out or l.out_dim, relu))
        elif l.kind == SHARD:
            plan.append(("shard", l.in_dim, l.out_dim))
        elif l.kind == LOG_SOFTMAX:
            width = plan[-1][2] if plan[-1][0] == "shard" else plan[-1][3]
            plan.append(("loss", width))
        elif l.kind == RELU:
            continue                              # fused into the layer before
        else:
            raise ValueError("%s in the model-parallel part is not supported" % l.kind)
    return plan


def fc_shards(layers: List[Layer]):
    """(input width, shard outputs, full outputs) of every split LINEAR layer."""
    return [(l.in_dim, l.out_dim, l.full_out) for l in layers
            if l.kind == LINEAR and l.shards > 1]


def parameters(layers: List[Layer], conv_params: int = 0) -> int:
    """Parameters one worker holds: the given conv parameters plus its FC
    weight (and bias) columns."""
    return conv_params + sum(l.in_dim * l.out_dim + l.out_dim for l in layers
                             if l.kind == LINEAR)


def vgg_net(schedule, in_ch: int, hw: int, fc) -> Layer:
    """A sequential VGG-style CNN as a layer list: 3x3 convs (each followed
    by a ReLU) and 2x2 pools per the channel schedule, a flatten, the dense
    layers ``fc`` [(in, out)] with a ReLU between them, then LOG_SOFTMAX."""
    from .configs import POOL
    layers, c = [], in_ch
    for v in schedule:
        if v == POOL:
            layers.append(Layer(POOLING, c * hw * hw, c * (hw // 2) ** 2))
            hw //= 2
        else:
            layers += [Layer(CONV, c * hw * hw, v * hw * hw), Layer(RELU)]
            c = v
    layers.append(Layer(RESHAPE, c * hw * hw, c * hw * hw))
    for j, (i, o) in enumerate(fc):
        layers.append(linear(i, o))
        if j < len(fc) - 1:
            layers.append(Layer(RELU))
    layers.append(Layer(LOG_SOFTMAX))
    return seq(*layers)
