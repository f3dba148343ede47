"""fp64 CPU oracle for the data movement around the FC shards on one device:
the modulo layer and the shard layer (sec. 3.1, Modulo Layer and Shard
Layer) with the group-MP worker numbering (sec. 3.2, Group MP Extension).

TEST INFRASTRUCTURE.  Only the test suite (``tests/``), the smoke check in
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` use this
module.  It shares no code with the HIP library and never loads it.

One device holds the buffers of every emulated worker: axis 0 of each array
below is the worker id w = 0 .. N-1.  Workers form MP groups of ``mp``
consecutive ids (sec. 3.2: group id = worker id // mp; ``mp = 1`` is pure
data parallelism, ``mp = N`` a single group).  Within a group the paper's K
is ``mp``.

Modulo layer, iteration k (the counter modulo K) of worker ``iproc``:
  * forward: gathered example b of the group comes from worker
    ``remote(b) = group_first + b // (B/K)`` (the paper's b / size, offset by
    the group's first worker id), and from that worker's local row
    ``k * B/K + b % (B/K)`` (each iteration takes the next block of B/K local
    examples; a worker's own block is the "starred" local copy).
  * backward: every worker of the group holds a gradient with respect to the
    whole gathered batch (partial: its FC shard sees only its own output
    columns); the owner of gathered example b receives, in its local row,
    the sum of the group's gradients at b.
Shard layer of worker ``iproc``'s group:
  * forward: the full input of the next layer is the group's partitions side
    by side, worker (group_first + r) supplying columns r*Ns .. (r+1)*Ns - 1
    (the output-column split of the FC shard);
  * backward: each worker holds a gradient with respect to the full input
    (partial); worker (group_first + r) receives the sum of the group's
    gradients over its column slice.
Sums run over the group's workers in increasing id, in float64.
"""
from __future__ import annotations

import numpy as np


def group_first(iproc: int, mp: int) -> int:
    """First worker id of iproc's MP group (sec. 3.2: groups of mp workers)."""
    return (iproc // mp) * mp


def remote(b: int, batch: int, mp: int, iproc: int) -> int:
    """Worker whose local batch supplies gathered example b (sec. 3.1, Modulo
    Layer: b divided by the block size B/K; sec. 3.2: within iproc's group)."""
    size = batch // mp
    return group_first(iproc, mp) + b // size


def local_row(b: int, k: int, batch: int, mp: int) -> int:
    """Row of the supplying worker's local batch that is gathered example b in
    iteration k: block k of B/K rows, same position within the block."""
    size = batch // mp
    return k * size + b % size


def _check_modulo(shape, iproc, k, mp):
    n, batch, _ = shape
    if mp < 1 or n % mp or batch % mp or not 0 <= iproc < n or not 0 <= k < mp:
        raise ValueError("bad modulo arguments")


def modulo_fwd(local: np.ndarray, iproc: int, k: int, mp: int) -> np.ndarray:
    """local [N][B][F] -> gathered batch [B][F] of iproc's group, iteration k."""
    local = np.asarray(local, dtype=np.float64)
    _check_modulo(local.shape, iproc, k, mp)
    n, batch, feat = local.shape
    out = np.empty((batch, feat))
    for b in range(batch):
        out[b] = local[remote(b, batch, mp, iproc), local_row(b, k, batch, mp)]
    return out


def modulo_bwd(dgathered: np.ndarray, iproc: int, k: int, mp: int,
               dlocal: np.ndarray) -> np.ndarray:
    """dgathered [N][B][F]: each worker's gradient w.r.t. its gathered batch.
    Writes, for every worker r of iproc's group, rows k*B/K .. (k+1)*B/K - 1
    of dlocal[r] (the sums over the group); other rows are left as they are.
    Returns dlocal (a float64 copy of the argument)."""
    dgathered = np.asarray(dgathered, dtype=np.float64)
    _check_modulo(dgathered.shape, iproc, k, mp)
    n, batch, feat = dgathered.shape
    dlocal = np.array(dlocal, dtype=np.float64)
    g0 = group_first(iproc, mp)
    for b in range(batch):
        acc = np.zeros(feat)
        for w in range(g0, g0 + mp):
            acc = acc + dgathered[w, b]
        dlocal[remote(b, batch, mp, iproc), local_row(b, k, batch, mp)] = acc
    return dlocal


def _check_shard(n, iproc, mp):
    if mp < 1 or n % mp or not 0 <= iproc < n:
        raise ValueError("bad shard arguments")


def shard_fwd(parts: np.ndarray, iproc: int, mp: int) -> np.ndarray:
    """parts [N][M][Ns]: each worker's partitioned output -> the full input
    [M][mp*Ns] of the next layer in iproc's group (sec. 3.1, Shard Layer)."""
    parts = np.asarray(parts, dtype=np.float64)
    n, rows, ns = parts.shape
    _check_shard(n, iproc, mp)
    g0 = group_first(iproc, mp)
    out = np.empty((rows, mp * ns))
    for r in range(mp):
        for m in range(rows):
            out[m, r * ns:(r + 1) * ns] = parts[g0 + r, m]
    return out


def shard_bwd(dfull: np.ndarray, iproc: int, mp: int, dparts: np.ndarray) -> np.ndarray:
    """dfull [N][M][mp*Ns]: each worker's gradient w.r.t. the full input.
    Writes dparts[g0 + r] = sum over the group of columns r*Ns .. (r+1)*Ns - 1,
    for every worker of iproc's group; returns dparts (a float64 copy)."""
    dfull = np.asarray(dfull, dtype=np.float64)
    n, rows, width = dfull.shape
    _check_shard(n, iproc, mp)
    if width % mp:
        raise ValueError("bad shard arguments")
    ns = width // mp
    dparts = np.array(dparts, dtype=np.float64)
    g0 = group_first(iproc, mp)
    for r in range(mp):
        for m in range(rows):
            acc = np.zeros(ns)
            for w in range(g0, g0 + mp):
                acc = acc + dfull[w, m, r * ns:(r + 1) * ns]
            dparts[g0 + r, m] = acc
    return dparts
