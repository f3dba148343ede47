"""fp64 CPU oracle for the loss on the complete model output and the SGD
update that closes a training step.

TEST INFRASTRUCTURE.  Only the test suite (``tests/``), the smoke check in
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` use this
module.  It shares no code with the HIP library and never loads it.

* Loss (sec. 3.1, Layer Partitioning): when the last FC layer is
  partitioned, a shard layer before the LOG_SOFTMAX layer gives every
  worker the full output, so the output error is that of a complete local
  model.  The criterion on log-probabilities is the negative log-likelihood
  of the true class.  With logits z (one row per example), the
  log-softmax is z minus the log of the row's sum of exponentials, the loss
  of a row is minus the log-probability at its label, and the gradient of
  ``scale * sum(loss)`` with respect to z is
  ``scale * (softmax(z) - onehot(label))``.  The row maximum is subtracted
  before exponentiating (the log-sum-exp is unchanged by any shift).  A
  label outside the class range has no loss: NaN, with a NaN gradient row.
* Update (sec. 4: SGD on mini-batches; sec. 3.1, Modulo Layer: the FC
  layers, updated K times as often as the convolutional layers, divide
  their gradients by K): a parameter moves against its gradient by the
  learning rate times a per-tensor scale (1 for the conv layers, 1/K for
  the FC shards).
"""
from __future__ import annotations

import numpy as np


def log_softmax_nll(z, labels, scale):
    """Returns (logp, loss, dz) in float64 for logits z [m][classes] and
    integer labels [m]."""
    z = np.asarray(z, np.float64)
    labels = np.asarray(labels, np.int64)
    m, classes = z.shape
    mx = z.max(axis=1, keepdims=True)
    lse = mx + np.log(np.exp(z - mx).sum(axis=1, keepdims=True))
    logp = z - lse
    valid = (labels >= 0) & (labels < classes)
    rows = np.arange(m)
    safe = np.where(valid, labels, 0)
    loss = np.where(valid, -logp[rows, safe], np.nan)
    onehot = np.zeros_like(z)
    onehot[rows[valid], labels[valid]] = 1.0
    dz = scale * (np.exp(logp) - onehot)
    dz[~valid] = np.nan
    return logp, loss, dz


def sgd_update(w, g, lr, scale):
    """The parameter after one SGD step: w - lr * scale * g (float64)."""
    return np.asarray(w, np.float64) - lr * scale * np.asarray(g, np.float64)
