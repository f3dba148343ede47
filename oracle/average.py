"""fp64 CPU oracle for model averaging across the emulated workers of one
device: the reduce step of data parallelism (sec. 2: replicas are brought to
a global model by averaging them; sec. 4: every worker exchanges the
parameters up to the modulo layer every few batches, and the FC model
shards are averaged across the MP groups).

TEST INFRASTRUCTURE.  Only the test suite (``tests/``), the smoke check in
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` use this
module.  It shares no code with the HIP library and never loads it.

``params`` holds one slot per worker (axis 0, worker id w = 0 .. N-1).
Workers form MP groups of ``mp`` consecutive ids (sec. 3.2); worker
``g * mp + r`` holds shard ``r`` of its group.  Averaging replaces every slot
by the mean over the workers that hold the same parameters: with ``mp = 1``
all N workers (conv layers, pure DP); with ``mp > 1`` the N / mp workers with
the same offset r, one per group (the inter-group averaging of FC shards).
The sum runs in increasing worker id, in float64, then is divided by the
number of workers in the set.
"""
from __future__ import annotations

import numpy as np


def model_average(params, mp: int):
    p = np.asarray(params, np.float64)
    n = p.shape[0]
    if mp < 1 or n % mp:
        raise ValueError("workers must be a multiple of mp")
    out = np.empty_like(p)
    groups = n // mp
    for r in range(mp):
        members = [g * mp + r for g in range(groups)]
        acc = np.zeros_like(p[0])
        for w in members:
            acc = acc + p[w]
        mean = acc / len(members)
        for w in members:
            out[w] = mean
    return out
