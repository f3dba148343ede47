"""Pins of the modulo / shard-layer oracle (oracle/modulo.py) against things
other than itself: the paper's B = 2, K = 2 walk-through
(tests/golden/modulo_b2_k2.txt), the special cases of sec. 3.2 (mp = 1 is
plain data parallelism; the four-worker, two-group example), the
each-example-once property of the K iterations, adjoint identities between
the forward gathers and the backward sums, and the column-shard product
against an unsharded numpy matmul.  A wrong block index, a wrong source
worker, a dropped or duplicated worker in a sum, or a transposed shard
order fails at least one of them.
"""
import os

import numpy as np
import pytest

from oracle import modulo as M

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "modulo_b2_k2.txt")
rng = np.random.default_rng(2112)


def _walkthrough():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if line and not line.startswith("#"):
            rows.append(tuple(int(v) for v in line.split()))
    return rows


def _tagged(n, batch, feat):
    """local[w][b][f] = 1000 w + 10 b + f: every value names its source."""
    w, b, f = np.meshgrid(np.arange(n), np.arange(batch), np.arange(feat), indexing="ij")
    return (1000 * w + 10 * b + f).astype(np.float64)


def test_walkthrough_forward():
    rows = _walkthrough()
    assert len(rows) == 8
    local = _tagged(2, 2, 3)
    for k, worker, slot, src_w, src_row, starred in rows:
        got = M.modulo_fwd(local, worker, k, mp=2)
        np.testing.assert_array_equal(got[slot], local[src_w, src_row])
        assert M.remote(slot, 2, 2, worker) == src_w
        assert M.local_row(slot, k, 2, 2) == src_row
        assert bool(starred) == (src_w == worker)


def test_walkthrough_backward():
    """The starred slot of each worker receives the sum of both workers'
    gradients; the other slot's sum goes to the other worker."""
    rows = _walkthrough()
    dg = rng.standard_normal((2, 2, 3))
    for k, worker, slot, src_w, src_row, _ in rows:
        out = M.modulo_bwd(dg, worker, k, 2, np.full((2, 2, 3), np.nan))
        np.testing.assert_array_equal(out[src_w, src_row], dg[0, slot] + dg[1, slot])
        # Rows of other iterations stay untouched.
        assert np.isnan(out[:, 1 - k]).all()


def test_pure_data_parallel_is_transparent():
    """mp = 1 (sec. 3.2): every worker is its own group and the layer hands
    its local batch through unchanged."""
    local = rng.standard_normal((3, 5, 4))
    for i in range(3):
        np.testing.assert_array_equal(M.modulo_fwd(local, i, 0, 1), local[i])
        out = M.modulo_bwd(local, i, 0, 1, np.zeros_like(local))
        np.testing.assert_array_equal(out[i], local[i])


def test_four_workers_two_groups():
    """Four workers, mp = 2 (sec. 3.2's example): workers 0,1 and 2,3 form
    the groups; worker 3 gathers only from workers 2 and 3."""
    local = _tagged(4, 4, 2)
    for k in range(2):
        got = M.modulo_fwd(local, 3, k, 2)
        src = got[:, 0] // 1000
        np.testing.assert_array_equal(src, [2, 2, 3, 3])
        np.testing.assert_array_equal(M.modulo_fwd(local, 2, k, 2), got)
        np.testing.assert_array_equal((got[:, 0] % 1000) // 10, [2 * k, 2 * k + 1] * 2)
    assert [M.group_first(i, 2) for i in range(4)] == [0, 0, 2, 2]


@pytest.mark.parametrize("n,mp,batch", [(4, 4, 8), (6, 3, 9), (4, 2, 6), (2, 2, 2)])
def test_each_example_once_per_k_iterations(n, mp, batch):
    """Over the K iterations a group gathers each local example of each of
    its workers exactly once."""
    local = _tagged(n, batch, 1)
    for i in range(0, n, mp):
        seen = np.concatenate([M.modulo_fwd(local, i, k, mp)[:, 0] for k in range(mp)])
        expect = local[i:i + mp, :, 0].ravel()
        np.testing.assert_array_equal(np.sort(seen), np.sort(expect))


@pytest.mark.parametrize("n,mp,batch,feat", [(4, 4, 8, 3), (6, 3, 9, 2), (4, 2, 6, 5)])
def test_modulo_adjoint(n, mp, batch, feat):
    """<fwd(L), D> = <L, bwd(D)> with D placed on one worker of the group
    (the others zero): the backward writes exactly the rows the forward
    read, with nothing dropped or doubled."""
    local = rng.standard_normal((n, batch, feat))
    for i in range(n):
        for k in range(mp):
            d = rng.standard_normal((batch, feat))
            dg = np.zeros((n, batch, feat))
            dg[i] = d
            lhs = np.sum(M.modulo_fwd(local, i, k, mp) * d)
            back = M.modulo_bwd(dg, i, k, mp, np.zeros((n, batch, feat)))
            rhs = np.sum(local * back)
            assert abs(lhs - rhs) <= 1e-12 * (1 + abs(lhs))


def test_modulo_bwd_sums_every_group_worker():
    n, mp, batch, feat = 6, 3, 6, 2
    dg = rng.standard_normal((n, batch, feat))
    out = M.modulo_bwd(dg, 4, 1, mp, np.zeros((n, batch, feat)))
    # Group {3, 4, 5}; block 1 is local rows 2..3; worker 3 + r owns slots 2r, 2r+1.
    for r in range(3):
        for j in range(2):
            np.testing.assert_allclose(out[3 + r, 2 + j], dg[3:6, 2 * r + j].sum(axis=0),
                                       rtol=1e-15, atol=0)
    assert not out[:3].any() and not out[3:, :2].any() and not out[3:, 4:].any()


@pytest.mark.parametrize("mp,rows,k_in,ns", [(4, 5, 6, 3), (2, 3, 4, 5), (1, 2, 3, 4)])
def test_shard_fwd_is_the_unsharded_layer(mp, rows, k_in, ns):
    """Column shards of X*W side by side equal the unsharded product
    (numpy matmul), i.e. worker r of the group supplies columns r*Ns..."""
    x = rng.standard_normal((rows, k_in))
    w = rng.standard_normal((k_in, mp * ns))
    n = 2 * mp
    parts = np.zeros((n, rows, ns))
    for r in range(mp):
        parts[mp + r] = x @ w[:, r * ns:(r + 1) * ns]
    got = M.shard_fwd(parts, mp + mp - 1, mp)
    np.testing.assert_allclose(got, x @ w, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("mp,rows,k_in,ns", [(4, 5, 6, 3), (2, 3, 4, 5)])
def test_shard_bwd_reduces_partial_input_gradients(mp, rows, k_in, ns):
    """Each worker's upper-layer shard W_r yields the partial gradient
    dY_r W_r^T over the full input; worker r's slice of their sum equals the
    same slice of the unsharded dY W^T (numpy matmul)."""
    # Upper layer: input width mp*ns (the shard layer's full output), output
    # columns split over the group.
    w_up = rng.standard_normal((mp * ns, mp * k_in))
    dy = rng.standard_normal((rows, mp * k_in))
    dpart = np.stack([dy[:, r * k_in:(r + 1) * k_in] @ w_up[:, r * k_in:(r + 1) * k_in].T
                      for r in range(mp)])
    full = dy @ w_up.T
    got = M.shard_bwd(dpart, 0, mp, np.zeros((mp, rows, ns)))
    for r in range(mp):
        np.testing.assert_allclose(got[r], full[:, r * ns:(r + 1) * ns], rtol=1e-12, atol=1e-12)


def test_shard_adjoint():
    n, mp, rows, ns = 4, 2, 3, 5
    parts = rng.standard_normal((n, rows, ns))
    for i in range(n):
        d = rng.standard_normal((rows, mp * ns))
        dfull = np.zeros((n, rows, mp * ns))
        dfull[i] = d
        lhs = np.sum(M.shard_fwd(parts, i, mp) * d)
        rhs = np.sum(parts * M.shard_bwd(dfull, i, mp, np.zeros_like(parts)))
        assert abs(lhs - rhs) <= 1e-12 * (1 + abs(lhs))


@pytest.mark.parametrize("args", [dict(iproc=4), dict(k=2), dict(mp=3)])
def test_modulo_rejects_bad_arguments(args):
    a = dict(iproc=0, k=0, mp=2)
    a.update(args)
    with pytest.raises(ValueError):
        M.modulo_fwd(np.zeros((4, 4, 1)), a["iproc"], a["k"], a["mp"])
