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

Host code: this module computes nothing on the GPU and feeds the driver
(``stack.HybridStep``) its shard shapes.
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


def partition(net: Layer, workers: int, threshold: float = 1.0) -> List[Layer]:
    """The hybrid layer list of ``net`` for MP groups of ``workers`` (the
    paper's K; 1 = no model parallelism)."""
    if workers < 1:
        raise ValueError("workers must be >= 1")
    use_mp = workers > 1
    out: List[Layer] = []
    first = net.children[0] if net.kind == SEQ and net.children else net
    start = _first_dim(first)
    state = {"dim": start, "dim_full": start}

    def split(layer: Layer) -> Layer:
        o = layer.full_out or layer.out_dim
        if o % workers:
            raise ValueError("%d outputs do not split in %d shards" % (o, workers))
        return Layer(LINEAR, layer.in_dim, o // workers, shards=workers, full_out=o)

    def walk(layer: Layer) -> None:
        dim, full = state["dim"], state["dim_full"]
        k = layer.kind
        if k == SEQ:
            for child in layer.children:
                walk(child)
            return
        if k in _UNSPLIT:
            if dim != full:
                raise ValueError("partitioned input unsupported by %s" % k)
            state["dim"] = state["dim_full"] = layer.resize(dim)
        elif k in _ELEMENTWISE:
            state["dim"] = layer.resize(dim)        # follows the partitioned width
        elif k == LINEAR:
            if layer.in_dim != full:
                raise ValueError("LINEAR expects %d inputs, the model gives %d"
                                 % (layer.in_dim, full))
            if dim == full:
                # Whole input: the first FC layer to split gets the modulo layer.
                if use_mp and ccr(layer) > threshold:
                    out.append(Layer(MODULO, full, full))
                    layer = split(layer)
            else:
                # Partitioned input: assemble the full input first.
                out.append(Layer(SHARD, dim, full))
                if use_mp and ccr(layer) > threshold:
                    layer = split(layer)
            state["dim"] = layer.out_dim
            state["dim_full"] = layer.full_out or layer.out_dim
        elif k == LOG_SOFTMAX:
            if dim != full:
                out.append(Layer(SHARD, dim, full))
                state["dim"] = full
        else:
            raise ValueError("unknown layer kind %s" % k)
        out.append(layer)

    walk(net)
    return out


def _first_dim(layer: Layer) -> int:
    while layer.kind == SEQ:
        layer = layer.children[0]
    return layer.in_dim


def fc_shards(layers: List[Layer]):
    """(input width, shard outputs, full outputs) of every split LINEAR layer."""
    return [(l.in_dim, l.out_dim, l.full_out) for l in layers
            if l.kind == LINEAR and l.shards > 1]


def parameters(layers: List[Layer], conv_params: int = 0) -> int:
    """Parameters one worker holds: the given conv parameters plus its FC
    weight (and bias) columns."""
    return conv_params + sum(l.in_dim * l.out_dim + l.out_dim for l in layers
                             if l.kind == LINEAR)
