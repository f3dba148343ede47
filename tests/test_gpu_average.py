"""GPU parity of sb_model_average and sb_model_average_replicas against the
fp64 oracle (oracle/average.py): pure data-parallel replicas, group-MP shard
averaging, replicas in separate buffers, unaligned and odd sizes, padding
between slots left alone, single-group no-op; and two MP groups of the
paper's VGG variant trained one step each and averaged (stack.AveragedGroups)
against the oracle's averaged training."""
import numpy as np
import pytest
import torch

from oracle import average as A
from paper_2112_15317_amd import sb, synth
from tests.helpers import print_case

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("workers,mp,n,stride", [(4, 1, 1000, 1000), (6, 2, 1001, 1003),
                                                 (8, 4, 4096, 4100), (4, 4, 10, 10),
                                                 (3, 1, 5, 8), (16, 2, 1 << 16, 1 << 16)])
def test_model_average(workers, mp, n, stride):
    print_case("model_average", workers=workers, mp=mp, n=n, stride=stride)
    buf = synth.normal((workers * stride,), 50, synth.TID.MISC)
    t = torch.from_numpy(buf).cuda()
    sb.sb_model_average(workers, mp, t, n=n, stride=stride)
    torch.cuda.synchronize()
    got = t.cpu().numpy().reshape(workers, stride)
    src = buf.reshape(workers, stride)
    ref = A.model_average(src[:, :n], mp)
    # fp32 sums of at most 8 terms in the oracle's order, one division.
    np.testing.assert_allclose(got[:, :n], ref, rtol=2e-6, atol=1e-6)
    np.testing.assert_array_equal(got[:, n:], src[:, n:])          # padding untouched
    # Averaging again changes nothing beyond rounding.
    sb.sb_model_average(workers, mp, t, n=n, stride=stride)
    torch.cuda.synchronize()
    np.testing.assert_allclose(t.cpu().numpy().reshape(workers, stride)[:, :n], got[:, :n],
                               rtol=2e-6, atol=1e-6)


@pytest.mark.parametrize("replicas,n,offset", [(2, 1000, 0), (3, 1001, 0), (5, 4096, 1),
                                               (8, 1 << 16, 0), (1, 100, 0)])
def test_model_average_replicas(replicas, n, offset):
    """Replicas in separate buffers (offset: elements past a 16-byte boundary,
    the element-wise path); every buffer gets the mean, the bytes around
    each range stay as they were."""
    print_case("model_average_replicas", replicas=replicas, n=n, offset=offset)
    src = [synth.normal((n + offset + 3,), 60 + r, synth.TID.MISC) for r in range(replicas)]
    bufs = [torch.from_numpy(a).cuda() for a in src]
    views = [b[offset:offset + n] for b in bufs]
    sb.sb_model_average_replicas(views)
    torch.cuda.synchronize()
    ref = A.model_average(np.stack([a[offset:offset + n] for a in src]), 1)
    for r in range(replicas):
        got = bufs[r].cpu().numpy()
        np.testing.assert_allclose(got[offset:offset + n], ref[r], rtol=2e-6, atol=1e-6)
        np.testing.assert_array_equal(got[:offset], src[r][:offset])
        np.testing.assert_array_equal(got[offset + n:], src[r][offset + n:])
    for r in range(1, replicas):
        assert torch.equal(views[r], views[0])


def test_averaged_groups_training_step():
    """Two MP groups of the paper's VGG variant (K = 2) on different data,
    each through one training step, then the model average (period 1):
    every parameter tensor against the oracle's averaged training, and the
    two groups' models identical bit for bit."""
    from oracle import stack as OS
    from paper_2112_15317_amd import configs
    from paper_2112_15317_amd import partition as P
    from paper_2112_15317_amd.stack import AveragedGroups
    from tests.helpers import TOL, rel_l2, to_host
    from tests.test_gpu_stack import _group_inputs
    K, n, G, lr = 2, 4, 2, 0.05
    fc = configs.PAPER_VARIANT_FC
    print_case("averaged_groups", K=K, n=n, groups=G)
    plan = P.fc_plan(P.partition(P.vgg_net(configs.PAPER_VARIANT_CONV, 3, 32, fc), K))
    per = [_group_inputs(n, K, fc, 31 + g) for g in range(G)]
    layers, _, wts, bs, fw, fb, _, _ = per[0]
    groups = [(x, remote, labels) for _, x, _, _, _, _, remote, labels in per]
    ag = AveragedGroups(configs.PAPER_VARIANT_CONV, n, 3, 32, plan, G, 1, lr=lr)
    ag.load_inputs(groups, wts, bs, fw, fb)
    ag.step()
    torch.cuda.synchronize()
    pools = [L.pool_after for L in layers]
    ref = OS.averaged_group_training(groups, wts, bs, pools, fw, fb, 1, 1, lr)
    tol = TOL["f32"]
    g0 = ag.groups[0]
    for j in range(g0.L):
        assert rel_l2(g0.full_weights(j) - fw[j], ref[0]["fc_w"][j] - fw[j]) <= tol, "W_fc%d" % j
        assert rel_l2(g0.full_bias(j) - fb[j], ref[0]["fc_b"][j] - fb[j]) <= tol, "b_fc%d" % j
    for L in layers:
        i = L.index
        assert rel_l2(to_host(g0.conv.W[i]) - wts[i], ref[0]["conv_w"][i] - wts[i]) <= tol
        assert rel_l2(to_host(g0.conv.b[i]) - bs[i], ref[0]["conv_b"][i] - bs[i]) <= tol
    for ts in ag.sets:
        for t in ts[1:]:
            assert torch.equal(t, ts[0])
