"""GPU test of the no-allocation weight gradient (sb_conv3x3_bwd_weight_noalloc).

It must equal sb_conv3x3_bwd_weight (caller workspace) bit for bit: the same
kernels and the same split plan, only the partials' home differs.  Two calls
in a row share the library's scratch array, the second on a smaller input,
so stale partials of the first would show in the second.  Both are also held
to the oracle's tolerance.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2112_15317_amd import sb, synth
from tests.helpers import TOL, print_case, rel_l2, to_dev, to_host

pytestmark = pytest.mark.gpu

# (n, c, h, k, dtype): every case splits its reduction (uses the scratch).
CASES = [(32, 64, 16, 128, "f32"), (4, 32, 8, 64, "f32"),
         (8, 64, 28, 128, "bf16"), (2, 16, 14, 64, "bf16")]


def _run_pair(n, c, h, k, dtype, seed):
    code = sb.SB_F32 if dtype == "f32" else sb.SB_BF16
    d = sb.conv_desc(n, c, h, h, k, code)
    need = sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_WEIGHT)
    assert 0 < need <= sb.SB_NOALLOC_SCRATCH_BYTES
    x = np.maximum(synth.normal((n, c, h, h), seed, synth.TID.IMAGES), 0)
    dy = synth.normal((n, k, h, h), seed, synth.TID.DY_TOP)
    xd, dyd = to_dev(x, dtype), to_dev(dy, dtype)
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")
    dw_ref = torch.full((k, c, 3, 3), float("nan"), device="cuda")
    db_ref = torch.full((k,), float("nan"), device="cuda")
    dw = torch.full((k, c, 3, 3), float("nan"), device="cuda")
    db = torch.full((k,), float("nan"), device="cuda")
    sb.sb_conv3x3_bwd_weight(d, xd, dyd, dw_ref, db_ref, ws)
    sb.sb_conv3x3_bwd_weight_noalloc(d, xd, dyd, dw, db)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw_ref) and torch.equal(db, db_ref)
    xh, dyh = to_host(xd), to_host(dyd)          # the values the kernels read
    rdw, rdb = O.conv3x3_bwd_weight(xh, dyh)
    assert rel_l2(to_host(dw), rdw) <= TOL["f32"]
    assert rel_l2(to_host(db), rdb) <= TOL["f32"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_weight_gradient_matches_workspace_call(dtype):
    big, small = [c for c in CASES if c[4] == dtype]
    print_case("noalloc_wgrad", big=big, small=small)
    _run_pair(*big, seed=61)
    _run_pair(*small, seed=62)           # smaller input, same scratch array
