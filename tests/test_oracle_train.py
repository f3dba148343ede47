"""Pins of the loss and update oracle (oracle/train.py) against things other
than itself: an independent library (scipy's log_softmax, torch's
cross-entropy and autograd in float64), closed forms (uniform logits, two
classes, a quadratic's minimum), central finite differences and invariants.
No GPU."""
import numpy as np
import pytest
import scipy.special
import torch

from oracle import train as T
from paper_2112_15317_amd import synth


def _logits(m, c, seed, spread=3.0):
    return synth.normal((m, c), seed, synth.TID.MISC).astype(np.float64) * spread


def _labels(m, c, seed):
    return np.random.Generator(np.random.PCG64(seed)).integers(0, c, size=m)


@pytest.mark.parametrize("m,c", [(7, 10), (3, 1000), (5, 1), (4, 2)])
def test_log_softmax_matches_scipy(m, c):
    z = _logits(m, c, m + c)
    logp, loss, _ = T.log_softmax_nll(z, _labels(m, c, 1), 1.0)
    np.testing.assert_allclose(logp, scipy.special.log_softmax(z, axis=1), rtol=0, atol=1e-13)
    # Large logits: the shift by the row maximum keeps it finite and exact.
    zl = z * 1000.0
    logp_l, _, _ = T.log_softmax_nll(zl, _labels(m, c, 1), 1.0)
    np.testing.assert_allclose(logp_l, scipy.special.log_softmax(zl, axis=1), rtol=1e-12, atol=1e-9)


def test_mean_loss_and_gradient_match_torch_cross_entropy():
    m, c = 16, 10
    z = _logits(m, c, 3)
    lab = _labels(m, c, 4)
    zt = torch.tensor(z, dtype=torch.float64, requires_grad=True)
    ref = torch.nn.functional.cross_entropy(zt, torch.tensor(lab), reduction="mean")
    ref.backward()
    _, loss, dz = T.log_softmax_nll(z, lab, 1.0 / m)
    assert abs(loss.mean() - ref.item()) < 1e-13
    np.testing.assert_allclose(dz, zt.grad.numpy(), rtol=0, atol=1e-15)


def test_uniform_logits_give_log_classes():
    for c in (1, 2, 10, 1000):
        z = np.full((3, c), 0.75)
        lab = np.array([0, c - 1, c // 2])
        logp, loss, dz = T.log_softmax_nll(z, lab, 0.5)
        np.testing.assert_allclose(loss, np.log(c), rtol=1e-15)
        np.testing.assert_allclose(logp, -np.log(c), rtol=1e-15)
        expect = np.full((3, c), 0.5 / c)
        expect[np.arange(3), lab] -= 0.5
        np.testing.assert_allclose(dz, expect, rtol=1e-14, atol=1e-17)


def test_two_classes_is_softplus_of_the_margin():
    z = _logits(9, 2, 5)
    lab = _labels(9, 2, 6)
    _, loss, _ = T.log_softmax_nll(z, lab, 1.0)
    margin = z[np.arange(9), 1 - lab] - z[np.arange(9), lab]
    np.testing.assert_allclose(loss, np.logaddexp(0.0, margin), rtol=1e-14)


def test_gradient_matches_central_differences():
    m, c, scale = 3, 5, 0.37
    z = _logits(m, c, 7)
    lab = _labels(m, c, 8)
    _, _, dz = T.log_softmax_nll(z, lab, scale)
    h = 1e-6
    fd = np.zeros_like(z)
    for i in range(m):
        for j in range(c):
            zp, zm = z.copy(), z.copy()
            zp[i, j] += h
            zm[i, j] -= h
            fd[i, j] = scale * (T.log_softmax_nll(zp, lab, 1.0)[1].sum() -
                                T.log_softmax_nll(zm, lab, 1.0)[1].sum()) / (2 * h)
    np.testing.assert_allclose(dz, fd, rtol=0, atol=1e-8)


def test_invariants_and_shift():
    z = _logits(6, 12, 9)
    lab = _labels(6, 12, 10)
    logp, loss, dz = T.log_softmax_nll(z, lab, 1.0)
    np.testing.assert_allclose(np.exp(logp).sum(axis=1), 1.0, rtol=1e-14)
    np.testing.assert_allclose(dz.sum(axis=1), 0.0, atol=1e-15)
    assert np.all(loss > 0)
    logp2, loss2, dz2 = T.log_softmax_nll(z + 123.25, lab, 1.0)
    np.testing.assert_allclose(logp2, logp, atol=1e-12)
    np.testing.assert_allclose(dz2, dz, atol=1e-15)


def test_label_out_of_range_gives_nan_row_only():
    z = _logits(4, 5, 11)
    lab = np.array([0, 5, -1, 4])
    _, loss, dz = T.log_softmax_nll(z, lab, 1.0)
    assert np.isnan(loss[1]) and np.isnan(loss[2]) and np.all(np.isnan(dz[[1, 2]]))
    _, ref_loss, ref_dz = T.log_softmax_nll(z[[0, 3]], lab[[0, 3]], 1.0)
    np.testing.assert_array_equal(loss[[0, 3]], ref_loss)
    np.testing.assert_array_equal(dz[[0, 3]], ref_dz)


def test_sgd_reaches_a_quadratics_minimum_and_divides_by_k():
    # f(w) = |w - a|^2 / 2 has gradient w - a: one step of lr * scale = 1
    # lands on a; with scale 1/K it covers 1/K of the way (sec. 3.1: the FC
    # gradients divided by K).
    w = synth.normal((40,), 12, synth.TID.MISC).astype(np.float64)
    a = synth.normal((40,), 13, synth.TID.MISC).astype(np.float64)
    np.testing.assert_allclose(T.sgd_update(w, w - a, 1.0, 1.0), a, rtol=0, atol=1e-15)
    for K in (2, 4):
        np.testing.assert_allclose(T.sgd_update(w, w - a, 1.0, 1.0 / K) - a,
                                   (1.0 - 1.0 / K) * (w - a), rtol=1e-14, atol=1e-15)
