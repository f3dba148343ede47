"""Pins of the model-averaging oracle (oracle/average.py) against numpy's own
mean and invariants of averaging.  No GPU."""
import numpy as np
import pytest

from oracle import average as A
from paper_2112_15317_amd import synth


def _slots(n, size, seed):
    return synth.normal((n, size), seed, synth.TID.MISC).astype(np.float64)


def test_pure_data_parallel_is_numpy_mean():
    p = _slots(5, 37, 1)
    out = A.model_average(p, 1)
    np.testing.assert_allclose(out, np.broadcast_to(p.mean(axis=0), p.shape), rtol=1e-15)


def test_group_mp_averages_each_shard_across_groups():
    # 6 workers in 3 groups of 2: shard 0 lives on workers 0, 2, 4 and
    # shard 1 on 1, 3, 5 (sec. 3.2 worker numbering).
    p = _slots(6, 11, 2)
    out = A.model_average(p, 2)
    for r in range(2):
        np.testing.assert_allclose(out[r::2], np.broadcast_to(p[r::2].mean(axis=0), (3, 11)),
                                   rtol=1e-15)


@pytest.mark.parametrize("n,mp", [(4, 1), (6, 2), (8, 4), (4, 4)])
def test_invariants(n, mp):
    p = _slots(n, 23, 3)
    out = A.model_average(p, mp)
    # Idempotent; each averaging set keeps its sum; a single group is untouched.
    np.testing.assert_allclose(A.model_average(out, mp), out, rtol=1e-15, atol=1e-15)
    for r in range(mp):
        np.testing.assert_allclose(out[r::mp].sum(axis=0), p[r::mp].sum(axis=0), rtol=1e-13,
                                   atol=1e-13)
    if mp == n:
        np.testing.assert_array_equal(out, p)
    # Identical replicas stay as they are.
    same = np.broadcast_to(p[0], p.shape)
    np.testing.assert_allclose(A.model_average(same, mp), same, rtol=1e-15)


def test_rejects_a_partial_group():
    with pytest.raises(ValueError):
        A.model_average(_slots(6, 3, 4), 4)
