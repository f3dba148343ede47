"""Oracle composition of the worker share: the conv stack and the hybrid step.

TEST INFRASTRUCTURE (see the package docstring): composes the pinned fp64
layer functions of this package in the order the paper's worker runs them
(sec. 3.1 and sec. 4: the convolutional layers run data-parallel on the
local batch; the FC layers, split to 1/K of their outputs, run on the batch
gathered by the modulo layer; backward runs the same path in reverse).

The stack's layer list is an input: ``weights[l]`` (KCRS), ``biases[l]`` and
``pool_after[l]`` (a ReLU + 2x2 max pool follows conv l; otherwise a ReLU
follows it).  The stack must end with a pool.

With ``bf16=True`` every tensor the bf16 GPU path stores in bfloat16 is
rounded to bfloat16 at the same point: conv outputs (before the pool, or
after the fused ReLU), the pooled outputs (already bf16 values), and the
activation gradients produced by the data-gradient convolution.  Weight and
bias gradients stay in full precision.
"""
from __future__ import annotations

import numpy as np

from . import (_f64, conv3x3_bwd_data, conv3x3_bwd_weight, conv3x3_fwd,
               fc_bwd, fc_fwd, relu_maxpool_bwd, relu_maxpool_fwd, round_bf16)
from .train import log_softmax_nll, sgd_update


def _identity(a):
    return a


def vgg_forward(x, weights, biases, pool_after, bf16=False):
    """Forward of the conv stack.  Returns a dict with
    ``A``: list of layer inputs A[0] = x ... A[L] = stack output,
    ``Z``: {l: pre-pool conv output} for pooled layers,
    ``idx``: {l: pool window codes} for pooled layers."""
    rnd = round_bf16 if bf16 else _identity
    if not pool_after[-1]:
        raise ValueError("the stack must end with a pooled layer")
    A = [_f64(x)]
    Z, idx = {}, {}
    for l, w in enumerate(weights):
        if pool_after[l]:
            z = rnd(conv3x3_fwd(A[l], w, biases[l], relu=False))
            y, code = relu_maxpool_fwd(z)
            Z[l], idx[l] = z, code
            A.append(y)
        else:
            A.append(rnd(conv3x3_fwd(A[l], w, biases[l], relu=True)))
    return {"A": A, "Z": Z, "idx": idx}


def vgg_backward(fwd, weights, pool_after, dy_top, bf16=False, want_dx=True):
    """Backward of the conv stack from the gradient of its output.
    Returns ``dZ`` (gradient at each conv output, after the ReLU/pool),
    ``dA`` (gradient arriving at each pooled output), ``dW``, ``db`` and
    ``dX`` (gradient of the stack input; None unless want_dx)."""
    rnd = round_bf16 if bf16 else _identity
    A, idx = fwd["A"], fwd["idx"]
    L = len(weights)
    dZ, dA, dW, db = {}, {}, {}, {}
    g = dy_top                      # gradient at the output of layer L-1
    dX = None
    for l in reversed(range(L)):
        if pool_after[l]:
            dA[l] = g
            g = relu_maxpool_bwd(g, idx[l])
        dZ[l] = g
        dW[l], db[l] = conv3x3_bwd_weight(A[l], g)
        if l > 0:
            mask = None if pool_after[l - 1] else A[l]
            g = rnd(conv3x3_bwd_data(g, weights[l], mask_src=mask))
        elif want_dx:
            dX = rnd(conv3x3_bwd_data(g, weights[0]))
    return {"dZ": dZ, "dA": dA, "dW": dW, "db": db, "dX": dX}


def vgg_step(x, weights, biases, pool_after, dy_top, bf16=False, want_dx=True):
    f = vgg_forward(x, weights, biases, pool_after, bf16=bf16)
    b = vgg_backward(f, weights, pool_after, dy_top, bf16=bf16, want_dx=want_dx)
    return f, b


def hybrid_step(x, weights, biases, pool_after, fc_w, fc_b, rows_remote, cols_remote, dy,
                train=None):
    """One worker's step of the hybrid scheme on one device, with L FC shards.

    ``train`` (a dict with ``labels``, ``logits_remote``, ``lr``, ``shards``)
    makes it a whole training step: the last shard's output and the other
    shards' columns ``logits_remote`` form the full logits (the shard layer
    before the LOG_SOFTMAX layer, sec. 3.1), whose log-softmax + NLL over the
    gathered rows (batch mean) gives the last shard's output gradient in
    place of ``dy``; after the backward, SGD at rate ``lr`` updates the conv
    parameters and, with the gradient divided by ``shards`` (the paper's K,
    sec. 3.1 Modulo Layer), the FC shards.

    The local conv stack output (flattened, one row per image, NCHW order)
    fills the first rows of the gathered FC0 input; ``rows_remote`` supplies
    the rows of the other replicas.  The shard output of FC j-1 (ReLU) fills
    the first feature columns of FC j's input; ``cols_remote[j-1]`` supplies
    the other shards' columns.  The last shard's output has no ReLU and
    receives the gradient ``dy``.  Backward: FC j's partial input gradient
    restricted to this shard's own columns of the layer below, masked by that
    layer's ReLU, is its output gradient; FC0's partial input gradient
    restricted to this replica's rows is the gradient of the conv stack
    output.  (The cross-worker sums of the partial gradients are collectives
    and are not part of one worker's compute.)
    """
    L = len(fc_w)
    f = vgg_forward(x, weights, biases, pool_after)
    top = f["A"][-1]
    n = top.shape[0]
    feat = int(np.prod(top.shape[1:]))
    xs = [np.concatenate([top.reshape(n, feat), np.asarray(rows_remote, np.float64)], axis=0)]
    ys = []
    for j in range(L):
        y = fc_fwd(xs[j], fc_w[j], fc_b[j], relu=j < L - 1)
        ys.append(y)
        if j < L - 1:
            xs.append(np.concatenate([y, np.asarray(cols_remote[j], np.float64)], axis=1))
    dxp, dw, db, dys = [None] * L, [None] * L, [None] * L, [None] * L
    loss = dz = None
    if train is not None:
        z = np.concatenate([ys[-1], np.asarray(train["logits_remote"], np.float64)], axis=1)
        _, loss, dz = log_softmax_nll(z, train["labels"], 1.0 / z.shape[0])
        g = np.ascontiguousarray(dz[:, :ys[-1].shape[1]])
    else:
        g = np.asarray(dy, np.float64)
    for j in reversed(range(L)):
        dys[j] = g
        dxp[j], dw[j], db[j] = fc_bwd(xs[j], fc_w[j], g,
                                      mask_src=ys[j] if j < L - 1 else None)
        if j > 0:
            g = np.ascontiguousarray(dxp[j][:, :ys[j - 1].shape[1]])
    dtop = np.ascontiguousarray(dxp[0][:n]).reshape(top.shape)
    b = vgg_backward(f, weights, pool_after, dtop)
    out = {"fwd": f, "bwd": b, "xs": xs, "ys": ys, "dys": dys, "dxp": dxp, "dw": dw, "db": db}
    if train is not None:
        lr, k = train["lr"], 1.0 / train["shards"]
        out.update(loss=loss, dz=dz,
                   conv_w_new=[sgd_update(w, b["dW"][i], lr, 1.0) for i, w in enumerate(weights)],
                   conv_b_new=[sgd_update(bb, b["db"][i], lr, 1.0) for i, bb in enumerate(biases)],
                   fc_w_new=[sgd_update(w, dw[j], lr, k) for j, w in enumerate(fc_w)],
                   fc_b_new=[sgd_update(bb, db[j], lr, k) for j, bb in enumerate(fc_b)])
    return out
