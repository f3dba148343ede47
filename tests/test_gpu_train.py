"""GPU parity of the loss and update entry points (sb_log_softmax_nll,
sb_sgd_update) against the fp64 oracle (oracle/train.py), on seeded inputs:
ragged class counts, row strides wider than the rows, one-class and
thousand-class rows, out-of-range labels, empty and many-tensor updates."""
import numpy as np
import pytest
import torch

from oracle import train as T
from paper_2112_15317_amd import sb, synth
from tests.helpers import TOL, print_case, rel_l2

pytestmark = pytest.mark.gpu


def _labels(m, c, seed):
    return np.random.Generator(np.random.PCG64(seed)).integers(0, c, size=m).astype(np.int32)


@pytest.mark.parametrize("m,c,ldz", [(256, 10, 10), (33, 1000, 1000), (7, 65, 72), (5, 1, 1),
                                     (130, 3, 4), (1, 64, 64), (4, 129, 129)])
def test_log_softmax_nll(m, c, ldz):
    print_case("log_softmax_nll", m=m, c=c, ldz=ldz)
    z = (synth.normal((m, ldz), 21, synth.TID.MISC) * 3.0).astype(np.float32)
    lab = _labels(m, c, 22)
    scale = 1.0 / m
    zd = torch.from_numpy(z).cuda()
    ld = torch.from_numpy(lab).cuda()
    logp = torch.full((m, ldz), -7.0, device="cuda")
    dz = torch.full((m, ldz), -7.0, device="cuda")
    loss = torch.full((m,), float("nan"), device="cuda")
    sb.sb_log_softmax_nll(m, c, zd, ld, scale, logp, loss, dz, ldz=ldz)
    torch.cuda.synchronize()
    rl, rloss, rdz = T.log_softmax_nll(z[:, :c], lab, scale)
    assert rel_l2(logp.cpu().numpy()[:, :c], rl) <= TOL["f32"]
    assert rel_l2(loss.cpu().numpy(), rloss) <= TOL["f32"]
    assert rel_l2(dz.cpu().numpy()[:, :c], rdz) <= TOL["f32"]
    # Columns between the row width and the row stride are left alone.
    assert torch.all(logp[:, c:] == -7.0) and torch.all(dz[:, c:] == -7.0)
    # Fixed reduction order: a second call is bitwise identical.
    dz2 = torch.empty_like(dz)
    dz2.copy_(dz)
    loss2 = torch.empty_like(loss)
    sb.sb_log_softmax_nll(m, c, zd, ld, scale, None, loss2, dz2, ldz=ldz)
    torch.cuda.synchronize()
    assert torch.equal(loss, loss2) and torch.equal(dz, dz2)


def test_log_softmax_nll_large_logits_and_bad_labels():
    m, c = 6, 40
    print_case("log_softmax_nll_edge", m=m, c=c)
    z = (synth.normal((m, c), 23, synth.TID.MISC) * 500.0).astype(np.float32)
    lab = _labels(m, c, 24)
    lab[1], lab[4] = c, -3
    dz = torch.empty((m, c), device="cuda")
    loss = torch.empty((m,), device="cuda")
    sb.sb_log_softmax_nll(m, c, torch.from_numpy(z).cuda(), torch.from_numpy(lab).cuda(), 1.0,
                          None, loss, dz)
    torch.cuda.synchronize()
    _, rloss, rdz = T.log_softmax_nll(z, lab, 1.0)
    got_loss, got_dz = loss.cpu().numpy(), dz.cpu().numpy()
    bad = [1, 4]
    good = [0, 2, 3, 5]
    assert np.all(np.isnan(got_loss[bad])) and np.all(np.isnan(got_dz[bad]))
    assert np.all(np.isfinite(got_loss[good])) and np.all(np.isfinite(got_dz[good]))
    assert rel_l2(got_loss[good], rloss[good]) <= TOL["f32"]
    assert rel_l2(got_dz[good], rdz[good]) <= TOL["f32"]


@pytest.mark.parametrize("sizes", [[1], [5, 1024, 4099, 0, 17], [64] * 64, [3 * 64 * 9, 64, 1 << 20]])
def test_sgd_update(sizes):
    print_case("sgd_update", sizes=sizes[:6], count=len(sizes))
    lr = 0.05
    ws, items, ref = [], [], []
    for t, n in enumerate(sizes):
        w = synth.normal((n,), 30 + t, synth.TID.MISC).astype(np.float32)
        g = synth.normal((n,), 130 + t, synth.TID.MISC).astype(np.float32)
        scale = 1.0 if t % 2 == 0 else 0.25
        wd, gd = torch.from_numpy(w).cuda(), torch.from_numpy(g).cuda()
        ws.append(wd)
        items.append((wd, gd, scale))
        # Bound of one fp32 fused multiply-add with the step lr * scale
        # rounded to fp32: about an ulp of each term.
        ref.append((T.sgd_update(w, g, lr, scale),
                    2.5e-7 * (np.abs(w) + lr * scale * np.abs(g).astype(np.float64))))
    sb.sb_sgd_update(sb.SgdList(items), lr)
    torch.cuda.synchronize()
    for wd, (r, bound) in zip(ws, ref):
        if r.size:
            got = wd.cpu().numpy().astype(np.float64)
            assert rel_l2(got, r) <= TOL["f32"]
            assert np.all(np.abs(got - r) <= bound)


def test_sgd_update_unaligned_views():
    # Tensors that start 4 bytes past a 16-byte boundary take the element path.
    base_w = torch.from_numpy(synth.normal((1031,), 40, synth.TID.MISC).astype(np.float32)).cuda()
    base_g = torch.from_numpy(synth.normal((1031,), 41, synth.TID.MISC).astype(np.float32)).cuda()
    before = base_w.cpu().numpy().copy()
    w, g = base_w[1:1028], base_g[3:1030]
    wh, gh = w.cpu().numpy().astype(np.float64), g.cpu().numpy().astype(np.float64)
    ref = T.sgd_update(wh, gh, 0.5, 1.0 / 3)
    sb.sb_sgd_update(sb.SgdList([(w, g, 1.0 / 3)]), 0.5)
    torch.cuda.synchronize()
    got = w.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - ref) <= 2.5e-7 * (np.abs(wh) + np.abs(gh) / 6))
    after = base_w.cpu().numpy()
    assert after[0] == before[0] and np.array_equal(after[1028:], before[1028:])
