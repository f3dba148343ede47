"""GPU parity of the ImageNet-shaped VGG-16 step in bf16 (batch 32 at
224x224, bf16 activations and filters, fp32 accumulation, channel-blocked
activations with the input's 3 channels zero-padded to 8), every call in
full, with the benchmark's seeded inputs (see tests/test_gpu_full_size.py
for the method).  Oracle arrays are laid out (and padded) like the stack's
buffers before they are uploaded or compared, so the padding is checked
too: the padded channels' data and filter gradients must be zero.

Per call, on the oracle's chain rounded to bf16 at the GPU's storage points:
pool codes and routed gradients bit for bit, bf16 outputs within relative L2
2e-2, fp32 weight and bias gradients (sums of exact bf16 products) within
1e-4.

End to end, each side takes its own decisions.  In bf16 the two sides round
sums that differ in their last fp32 bits, so windows whose two largest
values are a bf16 step or two apart can pick differently: every differing
code must be such a near-tie of the oracle's values (within 2^-6 of the
tensor's largest magnitude) and their number is printed.  Forward tensors
meet the bf16 bound.  Gradients of layers above every differing window meet
their bounds; below one they are printed and must be finite (each such
window sends one gradient element elsewhere; the per-call checks carry the
parity claim for those calls).
"""
import numpy as np
import pytest
import torch

import oracle as O
from oracle import stack as OS
from paper_2112_15317_amd import configs
from paper_2112_15317_amd.stack import ConvStack
from tests.chain import conv_io, host_nchw, near_tie_flips, run_and_check
from tests.helpers import TOL, print_case, rel_l2
from tests.test_gpu_full_size import _id, bench_vgg_inputs, stack_keys

pytestmark = pytest.mark.gpu

N, HW = 32, 224
LAYERS = configs.conv_layers(configs.VGG16, 3, HW)


def _fused():
    """The layers whose forward pools in the kernel (host-side queries; no
    library, no such calls)."""
    try:
        return ConvStack.fused_layers(configs.VGG16, N, 3, HW, "bf16", "c8")
    except Exception:
        return set()


FUSED = _fused()


@pytest.fixture(scope="module")
def cfg5():
    print_case("cfg5_chain", n=N, hw=HW)
    x, ws, bs, dy = bench_vgg_inputs(N, HW)
    xb, wsb, dyb = O.round_bf16(x), [O.round_bf16(w) for w in ws], O.round_bf16(dy)
    pools = [L.pool_after for L in LAYERS]
    f, b = OS.vgg_step(xb, wsb, bs, pools, dyb, store="bf16")
    st = ConvStack(configs.VGG16, N, 3, HW, "bf16", layout="c8")
    assert st.fused == FUSED
    st.load_inputs(x, ws, bs, dy)            # rounded to bf16 on the way in
    calls = {c[0]: c for c in st.step_calls()}
    run_and_check(calls[("pack", 0)], [], [])
    yield {"st": st, "f": f, "b": b, "calls": calls, "inputs": (x, ws, bs, dy)}


@pytest.mark.parametrize("key", stack_keys(LAYERS, FUSED)[1:], ids=_id)
def test_vgg16_imagenet_bf16_call_on_oracle_chain(cfg5, key):
    print_case("cfg5_call", call=_id(key), n=N, hw=HW)
    ups, checks = conv_io(cfg5["st"], cfg5["f"], cfg5["b"], key)
    worst = run_and_check(cfg5["calls"][key], ups, checks)
    print("relative L2:", worst)


def test_vgg16_imagenet_bf16_step_end_to_end(cfg5):
    print_case("cfg5_end_to_end", n=N, hw=HW)
    st, f, b = cfg5["st"], cfg5["f"], cfg5["b"]
    st.load_inputs(*cfg5["inputs"])
    st.step()
    torch.cuda.synchronize()
    tol = TOL["bf16"]
    flips = {}
    for L in st.layers:
        i = L.index
        if L.pool_after:
            z = f["Z"][i]
            if i not in st.fused:                # a fused layer stores no Z
                assert rel_l2(host_nchw(st, st.Z[i], z.shape), z) <= tol, "Z%d" % i
            flips[i] = near_tie_flips(z, f["idx"][i], host_nchw(st, st.idx[i], z.shape),
                                      2.0 ** -6 * np.max(np.abs(z)))
        a = f["A"][i + 1]
        assert rel_l2(host_nchw(st, st.A[i + 1], a.shape), a) <= tol, "A%d" % (i + 1)
    deepest = max([i for i, c in flips.items() if c] or [-1])
    report = {"near_tie_windows": flips}
    for L in st.layers:
        i = L.index
        for name, buf, ref, t in [("dZ%d" % i, st.grad_at_conv_output(i), b["dZ"][i], tol),
                                  ("dW%d" % i, st.dW[i], b["dW"][i], tol),
                                  ("db%d" % i, st.db[i], b["db"][i], tol)]:
            got = host_nchw(st, buf, ref.shape)
            e = rel_l2(got, ref)
            report[name] = round(e, 5)
            assert np.all(np.isfinite(got)), name
            if i > deepest:
                assert e <= t, "%s: %.3g" % (name, e)
    report["dX"] = round(rel_l2(host_nchw(st, st.gA[0], b["dX"].shape), b["dX"]), 5)
    print(report)
