"""GPU parity of the channel-blocked layout (SB_NCHW8C, bf16): conv forward,
data gradient (with and without the ReLU mask), weight and bias gradient,
fused ReLU + max pooling forward and backward, against the fp64 oracle.

The oracle works on NCHW arrays; the tests lay the seeded inputs out as
[n][c/8][h][w][8] on the device and bring the outputs back to NCHW on the
host.  Inputs are bf16 values (the oracle sees exactly what the kernels
read); bf16 outputs are held to relative L2 2e-2, fp32 weight and bias
gradients (sums of exact bf16 products) to 1e-4, pool codes and routed
gradients bit for bit.  Shapes: the padded first layer (8 channels, one
real-data block), a 32-channel output tile, ragged heights and widths,
short and long channel loops, grids small enough to split the reduction."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2112_15317_amd import sb, synth
from tests.helpers import TOL, print_case, rel_l2

pytestmark = pytest.mark.gpu

# (n, c, h, w, k)
SHAPES = [(2, 8, 32, 32, 64), (2, 16, 16, 16, 32), (3, 64, 33, 40, 24), (2, 64, 14, 14, 64),
          (4, 24, 9, 12, 16), (2, 128, 28, 28, 128), (1, 512, 14, 14, 512),
          (2, 64, 56, 56, 64), (1, 256, 32, 64, 256), (3, 8, 30, 36, 72)]


def c8(a):
    """NCHW host array -> channel-blocked bf16 device tensor."""
    n, c, h, w = a.shape
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)
    return t.reshape(n, c // 8, 8, h, w).permute(0, 1, 3, 4, 2).contiguous().cuda()


def nchw(t):
    """Channel-blocked device tensor -> NCHW float64 host array."""
    n, cb, h, w, e = t.shape
    u = t.permute(0, 1, 4, 2, 3).reshape(n, cb * e, h, w).cpu()
    return u.to(torch.float64).numpy() if u.dtype != torch.uint8 else u.numpy()


def bf(a):
    return O.round_bf16(a)


def _ws(nbytes):
    return torch.full((max(int(nbytes), 256),), 0xFF, dtype=torch.uint8, device="cuda")


def _inputs(n, c, h, w, k, seed):
    x = bf(np.maximum(synth.normal((n, c, h, w), seed, synth.TID.IMAGES), 0))
    wt = bf(synth.he_normal_conv3x3(k, c, seed, synth.TID.CONV_W))
    b = synth.normal((k,), seed, synth.TID.CONV_B, std=0.1)
    dy = bf(synth.normal((n, k, h, w), seed, synth.TID.DY_TOP))
    mask = bf(synth.normal((n, c, h, w), seed, synth.TID.MISC))
    return x, wt, b, dy, mask


def _desc(shape, relu=False):
    n, c, h, w, k = shape
    return sb.conv_desc(n, c, h, w, k, sb.SB_BF16, relu=relu, layout=sb.SB_NCHW8C)


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("relu", [False, True])
def test_c8_conv_fwd(shape, relu):
    n, c, h, w, k = shape
    print_case("c8_conv_fwd", shape=shape, relu=relu)
    x, wt, b, _, _ = _inputs(n, c, h, w, k, 41)
    d = _desc(shape, relu)
    ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD))
    y = torch.full((n, k // 8, h, w, 8), float("nan"), dtype=torch.bfloat16, device="cuda")
    wd = torch.from_numpy(wt.astype(np.float32)).to(torch.bfloat16).cuda()
    sb.sb_conv3x3_fwd(d, c8(x), wd, torch.from_numpy(b).cuda(), y, ws)
    torch.cuda.synchronize()
    ref = bf(O.conv3x3_fwd(x, wt, b, relu=relu))
    assert rel_l2(nchw(y), ref) <= TOL["bf16"]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("masked", [False, True])
def test_c8_conv_bwd_data(shape, masked):
    n, c, h, w, k = shape
    print_case("c8_conv_bwd_data", shape=shape, masked=masked)
    _, wt, _, dy, mask = _inputs(n, c, h, w, k, 42)
    d = _desc(shape)
    ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_DATA))
    dx = torch.full((n, c // 8, h, w, 8), float("nan"), dtype=torch.bfloat16, device="cuda")
    wd = torch.from_numpy(wt.astype(np.float32)).to(torch.bfloat16).cuda()
    sb.sb_conv3x3_bwd_data(d, c8(dy), wd, c8(mask) if masked else None, dx, ws)
    torch.cuda.synchronize()
    ref = bf(O.conv3x3_bwd_data(dy, wt, mask_src=mask if masked else None))
    assert rel_l2(nchw(dx), ref) <= TOL["bf16"]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_c8_conv_bwd_weight(shape):
    n, c, h, w, k = shape
    print_case("c8_conv_bwd_weight", shape=shape)
    x, _, _, dy, _ = _inputs(n, c, h, w, k, 43)
    d = _desc(shape)
    ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_WEIGHT))
    dw = torch.full((k, c, 3, 3), float("nan"), device="cuda")
    db = torch.full((k,), float("nan"), device="cuda")
    sb.sb_conv3x3_bwd_weight(d, c8(x), c8(dy), dw, db, ws)
    torch.cuda.synchronize()
    rdw, rdb = O.conv3x3_bwd_weight(x, dy)
    assert rel_l2(dw.cpu().numpy(), rdw) <= TOL["f32"]
    assert rel_l2(db.cpu().numpy(), rdb) <= TOL["f32"]
    # Fixed summation order: a second call is bitwise identical.
    dw2 = torch.empty_like(dw)
    sb.sb_conv3x3_bwd_weight(d, c8(x), c8(dy), dw2, None, ws)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw2)


def test_c8_packed_filters_match_unpacked():
    """The channel-blocked passes take the same packed filters as the NCHW
    bf16 kernels (SB_PACKED_FILTERS) and give the same bits."""
    shape = (2, 64, 28, 28, 64)
    n, c, h, w, k = shape
    print_case("c8_packed", shape=shape)
    x, wt, b, dy, mask = _inputs(n, c, h, w, k, 44)
    wd = torch.from_numpy(wt.astype(np.float32)).to(torch.bfloat16).cuda()
    outs = []
    for packed in (False, True):
        d = sb.conv_desc(n, c, h, w, k, sb.SB_BF16, relu=True, packed=packed,
                         layout=sb.SB_NCHW8C)
        db_ = sb.conv_desc(n, c, h, w, k, sb.SB_BF16, packed=packed, layout=sb.SB_NCHW8C)
        ws = _ws(max(sb.sb_conv3x3_workspace_bytes(d, 0), sb.sb_conv3x3_workspace_bytes(db_, 1)))
        wf, wb = wd, wd
        if packed:
            wf = torch.empty(sb.sb_conv3x3_packed_bytes(d, 0), dtype=torch.uint8, device="cuda")
            wb = torch.empty(sb.sb_conv3x3_packed_bytes(d, 1), dtype=torch.uint8, device="cuda")
            sb.sb_conv3x3_pack_filters(d, 0, wd, wf)
            sb.sb_conv3x3_pack_filters(d, 1, wd, wb)
        y = torch.empty((n, k // 8, h, w, 8), dtype=torch.bfloat16, device="cuda")
        dx = torch.empty((n, c // 8, h, w, 8), dtype=torch.bfloat16, device="cuda")
        sb.sb_conv3x3_fwd(d, c8(x), wf, torch.from_numpy(b).cuda(), y, ws)
        sb.sb_conv3x3_bwd_data(db_, c8(dy), wb, c8(mask), dx, ws)
        torch.cuda.synchronize()
        outs.append((y, dx))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


POOL_SHAPES = [(2, 8, 4, 6), (3, 64, 28, 28), (2, 128, 14, 10), (1, 16, 224, 224)]


@pytest.mark.parametrize("shape", POOL_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_c8_relu_maxpool(shape, dtype):
    n, c, h, w = shape
    print_case("c8_relu_maxpool", shape=shape, dtype=dtype)
    x = synth.normal((n, c, h, w), 51, synth.TID.IMAGES)
    # Constructed ties and all-negative windows in the first image.
    x[0, :, 0, 0] = x[0, :, 0, 1] = 2.5
    x[0, :, 2:4, 2:4] = -1.0
    dy = synth.normal((n, c, h // 2, w // 2), 51, synth.TID.DY_TOP)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    code = sb.SB_F32 if dtype == "f32" else sb.SB_BF16

    def dev(a):
        t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(tdt)
        nn_, cc, hh, ww = a.shape
        return t.reshape(nn_, cc // 8, 8, hh, ww).permute(0, 1, 3, 4, 2).contiguous().cuda()
    xd, dyd = dev(x), dev(dy)
    y = torch.full((n, c // 8, h // 2, w // 2, 8), float("nan"), dtype=tdt, device="cuda")
    idx = torch.full((n, c // 8, h // 2, w // 2, 8), 0x55, dtype=torch.uint8, device="cuda")
    dx = torch.full((n, c // 8, h, w, 8), float("nan"), dtype=tdt, device="cuda")
    sb.sb_relu_maxpool_fwd(n, c, h, w, code, sb.SB_NCHW8C, xd, y, idx)
    sb.sb_relu_maxpool_bwd(n, c, h, w, code, sb.SB_NCHW8C, dyd, idx, dx)
    torch.cuda.synchronize()
    xv, dyv = nchw(xd), nchw(dyd)                       # the values the kernels read
    ry, ridx = O.relu_maxpool_fwd(xv)
    np.testing.assert_array_equal(nchw(idx), ridx)
    np.testing.assert_array_equal(nchw(y), ry)
    np.testing.assert_array_equal(nchw(dx), O.relu_maxpool_bwd(dyv, ridx))


# Forward with fused ReLU + 2x2 pooling (sb_conv3x3_fwd_pool): shapes whose
# plan is one split (8x32 tiles with 64 and 32 output channels, a ragged
# last tile row, 16x16 tiles).
FUSED_SHAPES = [(32, 32, 64, 64, 64), (32, 16, 64, 64, 32), (40, 32, 50, 64, 64),
                (32, 64, 28, 28, 512)]


@pytest.mark.parametrize("shape", FUSED_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_c8_conv_fwd_pool(shape):
    """The fused call equals, bit for bit, the forward then the pool kernel
    (the same sums, rounded at the same point, pooled by the same rule), and
    against the oracle (pooling of the bf16-rounded fp64 forward) the pooled
    values meet 2e-2 and every differing code is a certified near-tie of the
    oracle's window values (the two sides round sums that differ in their
    last fp32 bits)."""
    from tests.chain import near_tie_flips
    n, c, h, w, k = shape
    print_case("c8_conv_fwd_pool", shape=shape)
    x, wt, b, _, _ = _inputs(n, c, h, w, k, 61)
    d = _desc(shape)
    need = sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD_POOL)
    assert need != sb.SIZE_MAX, "planned as one split"
    ws = _ws(need)
    wd = torch.from_numpy(wt.astype(np.float32)).to(torch.bfloat16).cuda()
    bd = torch.from_numpy(b).cuda()
    xd = c8(x)
    pooled = (n, k // 8, h // 2, w // 2, 8)
    y = torch.full(pooled, float("nan"), dtype=torch.bfloat16, device="cuda")
    idx = torch.full(pooled, 0x55, dtype=torch.uint8, device="cuda")
    sb.sb_conv3x3_fwd_pool(d, xd, wd, bd, y, idx, ws)
    z = torch.full((n, k // 8, h, w, 8), float("nan"), dtype=torch.bfloat16, device="cuda")
    y2 = torch.full(pooled, float("nan"), dtype=torch.bfloat16, device="cuda")
    idx2 = torch.full(pooled, 0x55, dtype=torch.uint8, device="cuda")
    sb.sb_conv3x3_fwd(d, xd, wd, bd, z, ws)
    sb.sb_relu_maxpool_fwd(n, k, h, w, sb.SB_BF16, sb.SB_NCHW8C, z, y2, idx2)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2), "codes differ from the unfused forward and pool"
    assert torch.equal(y.view(torch.int16), y2.view(torch.int16)), "pooled values differ"
    zr = bf(O.conv3x3_fwd(x, wt, b))
    ry, ridx = O.relu_maxpool_fwd(zr)
    assert rel_l2(nchw(y), ry) <= TOL["bf16"]
    flips = near_tie_flips(zr, ridx, nchw(idx), 2.0 ** -6 * np.max(np.abs(zr)))
    print("near-tie windows:", flips)
