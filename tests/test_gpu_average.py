"""GPU parity of sb_model_average against the fp64 oracle (oracle/average.py):
pure data-parallel replicas, group-MP shard averaging, unaligned and odd
sizes, padding between slots left alone, single-group no-op."""
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
