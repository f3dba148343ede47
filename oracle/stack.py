"""Oracle composition of the worker share: the conv stack and the hybrid step.

TEST INFRASTRUCTURE (see the package docstring): composes the pinned fp64
layer functions of this package in the order the paper's worker runs them
(sec. 3.1 and sec. 4: the convolutional layers run data-parallel on the
local batch; the FC layers, split to 1/K of their outputs, run on the batch
gathered by the modulo layer; backward runs the same path in reverse).

The stack's layer list is an input: ``weights[l]`` (KCRS), ``biases[l]`` and
``pool_after[l]`` (a ReLU + 2x2 max pool follows conv l; otherwise a ReLU
follows it).  The stack must end with a pool.

``store`` names the element type the GPU path keeps its activations and
activation gradients in: with ``"bf16"`` (or ``bf16=True``) / ``"f32"``
every such tensor is rounded to bfloat16 / float32 (nearest, ties to even)
at the point where the GPU stores it: conv outputs (before the pool, or
after the fused ReLU), the pooled outputs (already representable), the
activation gradients the data-gradient convolution produces and, in the
hybrid step, the FC shard outputs and partial input gradients.  Weight and
bias gradients stay in full precision.  The rounded chain is what the
per-call parity tests feed the GPU: every call's inputs are the oracle's own
tensors, held exactly in the GPU's storage type.  ``store=None`` keeps
everything in float64.
"""
from __future__ import annotations

import numpy as np

from . import (_f64, conv3x3_bwd_data, conv3x3_bwd_weight, conv3x3_fwd,
               fc_bwd, fc_fwd, relu_maxpool_bwd, relu_maxpool_fwd, round_bf16, round_f32)
from .average import model_average
from .modulo import modulo_bwd, modulo_fwd, shard_bwd, shard_fwd
from .train import log_softmax_nll, sgd_update


def _identity(a):
    return a


def _rounder(store, bf16=False):
    if bf16 or store == "bf16":
        return round_bf16
    if store == "f32":
        return round_f32
    if store is None:
        return _identity
    raise ValueError("store must be None, 'f32' or 'bf16'")


def vgg_forward(x, weights, biases, pool_after, bf16=False, store=None):
    """Forward of the conv stack.  Returns a dict with
    ``A``: list of layer inputs A[0] = x ... A[L] = stack output,
    ``Z``: {l: pre-pool conv output} for pooled layers,
    ``idx``: {l: pool window codes} for pooled layers."""
    rnd = _rounder(store, bf16)
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


def vgg_backward(fwd, weights, pool_after, dy_top, bf16=False, want_dx=True, store=None):
    """Backward of the conv stack from the gradient of its output.
    Returns ``dZ`` (gradient at each conv output, after the ReLU/pool),
    ``dA`` (gradient arriving at each pooled output), ``dW``, ``db`` and
    ``dX`` (gradient of the stack input; None unless want_dx)."""
    rnd = _rounder(store, bf16)
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


def vgg_step(x, weights, biases, pool_after, dy_top, bf16=False, want_dx=True, store=None):
    f = vgg_forward(x, weights, biases, pool_after, bf16=bf16, store=store)
    b = vgg_backward(f, weights, pool_after, dy_top, bf16=bf16, want_dx=want_dx, store=store)
    return f, b


def hybrid_step(x, weights, biases, pool_after, fc_w, fc_b, rows_remote, cols_remote, dy,
                store=None):
    """One worker's forward and backward of the hybrid scheme on one device,
    with L FC shards and no update (so the gathered rows of all K modulo
    iterations can go through the FC shards in one batch: with no update in
    between, the iterations' results are the same rows in another order and
    their weight gradients add up to the same sums).

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
    rnd = _rounder(store)
    f = vgg_forward(x, weights, biases, pool_after, store=store)
    top = f["A"][-1]
    n = top.shape[0]
    feat = int(np.prod(top.shape[1:]))
    xs = [np.concatenate([top.reshape(n, feat), np.asarray(rows_remote, np.float64)], axis=0)]
    ys = []
    for j in range(L):
        y = rnd(fc_fwd(xs[j], fc_w[j], fc_b[j], relu=j < L - 1))
        ys.append(y)
        if j < L - 1:
            xs.append(np.concatenate([y, np.asarray(cols_remote[j], np.float64)], axis=1))
    dxp, dw, db, dys = [None] * L, [None] * L, [None] * L, [None] * L
    g = np.asarray(dy, np.float64)
    for j in reversed(range(L)):
        dys[j] = g
        dxp[j], dw[j], db[j] = fc_bwd(xs[j], fc_w[j], g,
                                      mask_src=ys[j] if j < L - 1 else None)
        dxp[j] = rnd(dxp[j])
        if j > 0:
            g = np.ascontiguousarray(dxp[j][:, :ys[j - 1].shape[1]])
    dtop = np.ascontiguousarray(dxp[0][:n]).reshape(top.shape)
    b = vgg_backward(f, weights, pool_after, dtop, store=store)
    return {"fwd": f, "bwd": b, "xs": xs, "ys": ys, "dys": dys, "dxp": dxp, "dw": dw, "db": db}


def group_train_step(x, weights, biases, pool_after, fc_w, fc_b, local_remote, labels, lr):
    """One training step of an MP group of K workers, as sec. 3.1 (Modulo
    Layer, Shard Layer) runs it, with the FC side of every worker of the
    group and the conv stack of worker 0.

    * Worker 0 runs its conv stack forward once on its local batch of B
      images (``x``); ``local_remote`` [K-1][B][F] holds the flattened conv
      outputs of workers 1 .. K-1 (their own data-parallel stacks, not
      computed here).  K = ``len(local_remote) + 1`` and B must divide by K.
    * Then K modulo iterations k = 0 .. K-1.  Each gathers a batch of B rows,
      B/K from every worker of the group (block k of its local batch), with
      the modulo layer's index map; runs every FC layer as K column shards
      (worker r holds columns r*Ns .. (r+1)*Ns - 1 of ``fc_w[j]`` and
      ``fc_b[j]``, the full layers), a shard layer assembling the full input
      of the next layer from the K partitions (and the full logits before
      LOG_SOFTMAX); evaluates log-softmax + NLL of the full logits against
      ``labels[k]`` [B] (the labels of iteration k's gathered rows), averaged
      over the B rows; backpropagates: the last shards take their columns of
      the full logits' gradient (every worker evaluates the same loss), each
      later shard layer sums the group's partial input gradients over each
      worker's slice, and the modulo layer sums them back into the local
      rows of the workers that supplied them.  After the backward of
      iteration k every FC shard takes an SGD step with its gradient divided
      by K, so iteration k + 1 runs on the updated FC weights.
    * After the K iterations, worker 0's local rows hold the gradient of its
      conv output for the whole local batch; the conv stack runs backward
      and its parameters take one SGD step at rate ``lr``.

    Everything is float64.  Returns a dict with the conv forward and
    backward (``fwd``, ``bwd``), the per-iteration records ``iters``, the
    updated parameters (``fc_w_new``, ``fc_b_new`` as full layers,
    ``conv_w_new``, ``conv_b_new``) and ``dlocal`` [K][B][F], every worker's
    conv-output gradient as the modulo layer delivers it.
    """
    K = len(local_remote) + 1
    L = len(fc_w)
    f = vgg_forward(x, weights, biases, pool_after)
    top = f["A"][-1]
    B = top.shape[0]
    feat = int(np.prod(top.shape[1:]))
    if B % K:
        raise ValueError("the local batch must divide into K blocks")
    local = np.concatenate([top.reshape(1, B, feat), np.asarray(local_remote, np.float64)])
    W = [np.array(w, np.float64) for w in fc_w]
    bvec = [np.array(b, np.float64) for b in fc_b]
    ns = []
    for w in W:
        if w.shape[1] % K:
            raise ValueError("FC outputs must split in K shards")
        ns.append(w.shape[1] // K)
    cols = [[slice(r * n, (r + 1) * n) for r in range(K)] for n in ns]
    dlocal = np.zeros_like(local)
    iters = []
    for k in range(K):
        gathered = modulo_fwd(local, 0, k, K)
        xs, parts = [gathered], []
        for j in range(L):
            pj = [fc_fwd(xs[j], W[j][:, cols[j][r]], bvec[j][cols[j][r]], relu=j < L - 1)
                  for r in range(K)]
            parts.append(pj)
            xs.append(shard_fwd(np.stack(pj), 0, K))
        logits = xs[-1]
        _, loss, dz = log_softmax_nll(logits, labels[k], 1.0 / B)
        dws, dbs = [None] * L, [None] * L
        dfull = [None] * L
        dpart = None
        for j in reversed(range(L)):
            gw, gb, gx = [], [], []
            for r in range(K):
                dy = dz[:, cols[j][r]] if j == L - 1 else dpart[r]
                dx, dw, db = fc_bwd(xs[j], W[j][:, cols[j][r]], np.ascontiguousarray(dy),
                                    mask_src=parts[j][r] if j < L - 1 else None)
                gx.append(dx)
                gw.append(dw)
                gb.append(db)
            dws[j], dbs[j], dfull[j] = gw, gb, np.stack(gx)
            if j > 0:
                dpart = shard_bwd(dfull[j], 0, K, np.zeros((K, B, ns[j - 1])))
            else:
                dlocal = modulo_bwd(dfull[0], 0, k, K, dlocal)
        iters.append({"gathered": gathered, "xs": xs, "parts": parts, "logits": logits,
                      "loss": loss, "dz": dz, "dfull": dfull, "dw": dws, "db": dbs,
                      "w_before": [w.copy() for w in W], "b_before": [b.copy() for b in bvec]})
        for j in range(L):
            for r in range(K):
                W[j][:, cols[j][r]] = sgd_update(W[j][:, cols[j][r]], dws[j][r], lr, 1.0 / K)
                bvec[j][cols[j][r]] = sgd_update(bvec[j][cols[j][r]], dbs[j][r], lr, 1.0 / K)
    dtop = np.ascontiguousarray(dlocal[0]).reshape(top.shape)
    b = vgg_backward(f, weights, pool_after, dtop)
    return {"fwd": f, "bwd": b, "iters": iters, "dlocal": dlocal,
            "fc_w_new": W, "fc_b_new": bvec,
            "conv_w_new": [sgd_update(w, b["dW"][i], lr, 1.0) for i, w in enumerate(weights)],
            "conv_b_new": [sgd_update(bb, b["db"][i], lr, 1.0) for i, bb in enumerate(biases)]}


def averaged_group_training(groups, weights, biases, pool_after, fc_w, fc_b, steps, period,
                            lr):
    """Training of G MP groups that start from the same model and average it
    every ``period`` steps (sec. 4: the workers exchange the parameters up to
    the modulo layer every few batches, and the FC shards are averaged
    across the MP groups; sec. 2: the reduce is the mean of the replicas).

    ``groups[g]`` = (x, local_remote, labels): group g's inputs, the same at
    every step (one fixed synthetic batch per group).  Each step runs
    ``group_train_step`` in every group on that group's parameters; after
    steps period, 2 period, ... every parameter tensor (each conv layer's
    filters and bias, each FC layer as the full matrix: its shard r in every
    group is averaged with shard r of the others) is replaced in every group
    by the mean over the groups, in increasing group index.  Returns the
    per-group parameters after ``steps`` steps: a list of dicts with
    ``conv_w``, ``conv_b``, ``fc_w``, ``fc_b``.
    """
    G = len(groups)
    state = [{"conv_w": [np.array(w, np.float64) for w in weights],
              "conv_b": [np.array(b, np.float64) for b in biases],
              "fc_w": [np.array(w, np.float64) for w in fc_w],
              "fc_b": [np.array(b, np.float64) for b in fc_b]} for _ in range(G)]
    for s in range(steps):
        for g, (x, remote, labels) in enumerate(groups):
            p = state[g]
            r = group_train_step(x, p["conv_w"], p["conv_b"], pool_after, p["fc_w"], p["fc_b"],
                                 remote, labels, lr)
            state[g] = {"conv_w": r["conv_w_new"], "conv_b": r["conv_b_new"],
                        "fc_w": r["fc_w_new"], "fc_b": r["fc_b_new"]}
        if (s + 1) % period == 0:
            for key in ("conv_w", "conv_b", "fc_w", "fc_b"):
                for i in range(len(state[0][key])):
                    mean = model_average(np.stack([state[g][key][i] for g in range(G)]), 1)
                    for g in range(G):
                        state[g][key][i] = mean[g]
    return state
