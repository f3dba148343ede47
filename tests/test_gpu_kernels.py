"""GPU parity of every libsb entry point against the fp64 oracle, at sizes the
oracle finishes in seconds: several tiles, ragged tails, degenerate shapes.

All inputs come from the seeded generators; both sides get identical values.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2112_15317_amd import sb, synth
from tests.helpers import TOL, print_case, rel_l2, to_dev, to_host

pytestmark = pytest.mark.gpu


def _ws(nbytes):
    # The workspace needs no initialisation: hand it over full of NaN bytes.
    return torch.full((max(int(nbytes), 256),), 0xFF, dtype=torch.uint8, device="cuda")


# ------------------------------------------------------------------ pool --
POOL_SHAPES = [(2, 3, 4, 4), (3, 5, 6, 10), (1, 1, 2, 2), (4, 7, 8, 6), (2, 64, 32, 32),
               (2, 5, 6, 16), (1, 3, 4, 24),    # 4-window vector form
               (1, 3, 2, 30), (128, 512, 2, 2)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", POOL_SHAPES)
def test_relu_maxpool_fwd_bwd(shape, dtype):
    n, c, h, w = shape
    print_case("relu_maxpool", shape=shape, dtype=dtype)
    x = synth.normal(shape, 7, synth.TID.MISC + 1)
    dy = synth.normal((n, c, h // 2, w // 2), 7, synth.TID.MISC + 2)
    xd, dyd = to_dev(x, dtype), to_dev(dy, dtype)
    tdt = xd.dtype
    y = torch.empty((n, c, h // 2, w // 2), dtype=tdt, device="cuda")
    idx = torch.empty((n, c, h // 2, w // 2), dtype=torch.uint8, device="cuda")
    dx = torch.full(shape, 7.0, dtype=tdt, device="cuda")          # must be overwritten
    code = sb.SB_F32 if dtype == "f32" else sb.SB_BF16
    sb.sb_relu_maxpool_fwd(n, c, h, w, code, sb.SB_NCHW, xd, y, idx)
    sb.sb_relu_maxpool_bwd(n, c, h, w, code, sb.SB_NCHW, dyd, idx, dx)
    torch.cuda.synchronize()
    y_ref, idx_ref = O.relu_maxpool_fwd(xd.cpu())
    np.testing.assert_array_equal(idx.cpu().numpy(), idx_ref)
    np.testing.assert_array_equal(to_host(y), y_ref)               # a selection: exact
    dx_ref = O.relu_maxpool_bwd(dyd.cpu(), idx_ref)
    np.testing.assert_array_equal(to_host(dx), dx_ref)


def test_relu_maxpool_constructed_ties():
    x = np.array([[1.0, 1.0, 0.2, 0.7, -1.0, -0.5, 0.0, -1.0, -3.0, -2.0],
                  [0.5, 1.0, 0.7, 0.7, -2.0, -0.5, -1.0, -1.0, 5.0, 5.0]], np.float32)
    x = x.reshape(1, 1, 2, 10)
    xd = to_dev(x)
    y = torch.empty((1, 1, 1, 5), device="cuda")
    idx = torch.empty((1, 1, 1, 5), dtype=torch.uint8, device="cuda")
    sb.sb_relu_maxpool_fwd(1, 1, 2, 10, sb.SB_F32, sb.SB_NCHW, xd, y, idx)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(idx.cpu().numpy().ravel(), [0, 1, 0x81, 0x80, 2])
    np.testing.assert_array_equal(y.cpu().numpy().ravel(), np.float32([1.0, 0.7, 0.0, 0.0, 5.0]))


# ------------------------------------------------------------------ conv --
CONV_SHAPES = [
    # n, c, h, w, k
    (8, 3, 32, 32, 64),      # the single-layer workload (3 -> 64, 32x32, batch 8)
    (2, 5, 7, 9, 70),        # ragged everywhere: channels, rows, cols, out-channel tile
    (3, 16, 16, 16, 32),
    (5, 24, 8, 8, 96),
    (9, 40, 4, 4, 72),
    (33, 20, 2, 2, 130),     # more images than one tile holds, ragged
    (5, 40, 2, 2, 36),       # 2x2 in one image stage: unsplit, two ragged row and column tiles
    (2, 12, 5, 37, 17),
    (3, 40, 8, 8, 70),       # 8x8 two-group blocks, odd chunk count (groups uneven)
    (2, 33, 9, 12, 20),      # the same with ragged rows and columns
    (2, 64, 6, 40, 80),      # 32-wide tiles, 32-channel blocks, ragged columns and k
    (2, 36, 20, 20, 64),     # 16-wide tiles, ragged channel block
    (2, 48, 14, 14, 64),     # 8x8 tiles over 14x14 (rows not a multiple of 4)
    (2, 3, 6, 36, 40),       # RGB-like input (output staged through LDS, 4-pixel pieces,
                             # ragged column tile); 3-channel data gradient in two groups
                             # over an odd number of chunks
    (3, 2, 5, 38, 12),       # the same with an odd width (element-wise stores)
    (2, 12, 5, 38, 3),       # at most 4 output channels (vector-ALU kernel): forward
    (3, 20, 9, 33, 1),       # with bias and ReLU, ragged row and column tiles, a
    (2, 16, 8, 40, 4),       # partial last channel chunk; 1, 2, 3 and 4 channels
    (1, 9, 3, 64, 2),
    (1, 1, 1, 1, 1),         # degenerate: every tap but the centre is padding
    (1, 9, 3, 1, 5),
]


def _conv_inputs(n, c, h, w, k, seed):
    x = synth.normal((n, c, h, w), seed, synth.TID.IMAGES)
    wt = synth.he_normal_conv3x3(k, c, seed, synth.TID.CONV_W)
    b = synth.normal((k,), seed, synth.TID.CONV_B)
    dy = synth.normal((n, k, h, w), seed, synth.TID.DY_TOP)
    mask = synth.normal((n, c, h, w), seed, synth.TID.MISC)
    return x, wt, b, dy, mask


DTYPES = ["f32", "bf16"]


def _code(dtype):
    return sb.SB_F32 if dtype == "f32" else sb.SB_BF16


def _tdt(dtype):
    return torch.float32 if dtype == "f32" else torch.bfloat16


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", CONV_SHAPES)
@pytest.mark.parametrize("relu", [False, True])
def test_conv_fwd(shape, relu, dtype):
    n, c, h, w, k = shape
    print_case("conv_fwd", shape=shape, relu=relu, dtype=dtype)
    x, wt, b, _, _ = _conv_inputs(n, c, h, w, k, 11)
    d = sb.conv_desc(n, c, h, w, k, _code(dtype), relu=relu)
    ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD))
    y = torch.full((n, k, h, w), float("nan"), dtype=_tdt(dtype), device="cuda")
    xd, wd = to_dev(x, dtype), to_dev(wt, dtype)
    sb.sb_conv3x3_fwd(d, xd, wd, to_dev(b), y, ws)
    torch.cuda.synchronize()
    # The oracle gets exactly the values the kernel read (bf16-rounded).
    ref = O.conv3x3_fwd(to_host(xd), to_host(wd), b, relu=relu)
    assert rel_l2(to_host(y), ref) <= TOL[dtype]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", CONV_SHAPES)
@pytest.mark.parametrize("masked", [False, True])
def test_conv_bwd_data(shape, masked, dtype):
    n, c, h, w, k = shape
    print_case("conv_bwd_data", shape=shape, masked=masked, dtype=dtype)
    _, wt, _, dy, mask = _conv_inputs(n, c, h, w, k, 12)
    d = sb.conv_desc(n, c, h, w, k, _code(dtype))
    ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_DATA))
    dx = torch.full((n, c, h, w), float("nan"), dtype=_tdt(dtype), device="cuda")
    dyd, wd, md = to_dev(dy, dtype), to_dev(wt, dtype), to_dev(mask, dtype)
    sb.sb_conv3x3_bwd_data(d, dyd, wd, md if masked else None, dx, ws)
    torch.cuda.synchronize()
    ref = O.conv3x3_bwd_data(to_host(dyd), to_host(wd), mask_src=to_host(md) if masked else None)
    assert rel_l2(to_host(dx), ref) <= TOL[dtype]


# bf16 outputs are rounded from the fp32 accumulator to nearest, ties to
# even.  One live product per output (centre tap 1.5 on channel 0, every
# other filter value zero) makes the accumulator exactly 1.5 * input, which
# often lies halfway between two bf16 values; the expected bits come from
# torch's CPU rounding.  The shapes reach the bf16 MFMA epilogue (unsplit and
# through the split reduction) and the fp32-MFMA kernels' bf16 stores.
ROUNDING_SHAPES = [(2, 16, 32, 32, 64), (2, 64, 16, 16, 64), (2, 64, 4, 4, 64), (3, 5, 5, 7, 8),
                   (4, 64, 2, 2, 96)]


@pytest.mark.parametrize("shape", ROUNDING_SHAPES)
@pytest.mark.parametrize("pass_", ["fwd", "bwd_data"])
def test_bf16_store_rounds_ties_to_even(shape, pass_):
    n, c, h, w, k = shape
    print_case("bf16_rounding", shape=shape, pass_=pass_)
    # Forward: inputs x [n, c], filters [k, c]; data gradient: the same
    # layer transposed (dy [n, k] in, dx [n, c] out), the live filter value
    # on k = 0.
    cin, cout = (c, k) if pass_ == "fwd" else (k, c)
    src = synth.normal((n, cin, h, w), 3, synth.TID.IMAGES).astype(np.float32)
    src_d = torch.from_numpy(src).to(torch.bfloat16).cuda()
    wt = np.zeros((k, c, 3, 3), np.float32)
    if pass_ == "fwd":
        wt[:, 0, 1, 1] = 1.5
    else:
        wt[0, :, 1, 1] = 1.5
    wd = torch.from_numpy(wt).to(torch.bfloat16).cuda()
    d = sb.conv_desc(n, c, h, w, k, sb.SB_BF16)
    out = torch.full((n, cout, h, w), float("nan"), dtype=torch.bfloat16, device="cuda")
    if pass_ == "fwd":
        ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD))
        sb.sb_conv3x3_fwd(d, src_d, wd, None, out, ws)
    else:
        ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_DATA))
        sb.sb_conv3x3_bwd_data(d, src_d, wd, None, out, ws)
    torch.cuda.synchronize()
    exact = src_d.float().cpu()[:, :1] * 1.5                  # fp32-exact products
    expect = exact.to(torch.bfloat16).expand(n, cout, h, w)
    got = out.cpu()
    assert torch.equal(got.view(torch.int16), expect.contiguous().view(torch.int16))
    # The case really has ties (rounding up and down both occur).
    halfway = (exact.view(torch.int32) & 0xFFFF) == 0x8000
    assert int(halfway.sum()) > 0


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", CONV_SHAPES)
def test_conv_bwd_weight(shape, dtype):
    n, c, h, w, k = shape
    print_case("conv_bwd_weight", shape=shape, dtype=dtype)
    x, _, _, dy, _ = _conv_inputs(n, c, h, w, k, 13)
    d = sb.conv_desc(n, c, h, w, k, _code(dtype))
    ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_WEIGHT))
    dw = torch.full((k, c, 3, 3), float("nan"), device="cuda")
    db = torch.full((k,), float("nan"), device="cuda")
    xd, dyd = to_dev(x, dtype), to_dev(dy, dtype)
    sb.sb_conv3x3_bwd_weight(d, xd, dyd, dw, db, ws)
    torch.cuda.synchronize()
    dw_ref, db_ref = O.conv3x3_bwd_weight(to_host(xd), to_host(dyd))
    # dw and db are fp32 sums of exact bf16 x bf16 products: the fp32 bound.
    assert rel_l2(to_host(dw), dw_ref) <= TOL["f32"]
    assert rel_l2(to_host(db), db_ref) <= TOL["f32"]
    # Fixed summation order: a second call is bitwise identical.
    dw2 = torch.empty_like(dw)
    db2 = torch.empty_like(db)
    sb.sb_conv3x3_bwd_weight(d, xd, dyd, dw2, db2, ws)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw2) and torch.equal(db, db2)


# bf16 shapes that reach each staging width of the bf16 MFMA kernels (8, 4,
# 2 or 1 columns per load, from the image width) on each tile shape (32, 16
# and 8 columns wide), with ragged channel and k blocks.
WGRAD_BF16_SHAPES = [
    (2, 40, 5, 36, 64),      # 32-wide tiles, 4 columns per load
    (1, 32, 4, 34, 70),      # 32-wide tiles, 2 columns per load
    (2, 32, 6, 18, 64),      # 16-wide tiles, 2 columns per load
    (2, 20, 7, 19, 33),      # 16-wide tiles, 1 column per load, 16-channel blocks
    (2, 40, 9, 24, 70),      # 16-wide tiles, 8 columns per load, two column tiles
    (2, 48, 9, 11, 64),      # 8-wide tiles, 1 column per load
    (1, 64, 3, 64, 128),     # 32-wide tiles, two full column tiles
    # 64 or more input channels, ragged in c and k
    (2, 70, 5, 40, 140),     # 32-wide tiles, 8 columns per load, three c and three k tiles
    (2, 64, 6, 20, 96),      # 16-wide tiles, 4 columns per load
    (2, 100, 9, 10, 130),    # 8-wide tiles, 2 columns per load
    (1, 72, 3, 37, 200),     # 32-wide tiles, 1 column per load
]


def _dev_at(a, offset):
    """a as a bf16 device tensor starting `offset` elements into a buffer."""
    buf = torch.empty(a.size + offset, dtype=torch.bfloat16, device="cuda")
    t = buf[offset:].view(a.shape)
    t.copy_(to_dev(a, "bf16"))
    return t


@pytest.mark.parametrize("shape", WGRAD_BF16_SHAPES)
@pytest.mark.parametrize("offset", [0, 1])
def test_conv_fwd_bwd_data_bf16_staging(shape, offset):
    """The bf16 forward and data-gradient kernels over the same staging
    widths; offset = 1 element takes the one-column halo loads."""
    n, c, h, w, k = shape
    print_case("conv_fwd_bwd_data_bf16", shape=shape, offset=offset)
    x, wt, b, dy, mask = _conv_inputs(n, c, h, w, k, 16)
    df = sb.conv_desc(n, c, h, w, k, sb.SB_BF16, relu=True)
    dd = sb.conv_desc(n, c, h, w, k, sb.SB_BF16)
    ws = _ws(max(sb.sb_conv3x3_workspace_bytes(df, sb.SB_PASS_FWD),
                 sb.sb_conv3x3_workspace_bytes(dd, sb.SB_PASS_BWD_DATA)))
    xd, dyd, md = _dev_at(x, offset), _dev_at(dy, offset), _dev_at(mask, offset)
    wd = to_dev(wt, "bf16")
    y = torch.full((n, k, h, w), float("nan"), dtype=torch.bfloat16, device="cuda")
    sb.sb_conv3x3_fwd(df, xd, wd, to_dev(b), y, ws)
    dx = torch.full((n, c, h, w), float("nan"), dtype=torch.bfloat16, device="cuda")
    sb.sb_conv3x3_bwd_data(dd, dyd, wd, md, dx, ws)
    torch.cuda.synchronize()
    ref = O.conv3x3_fwd(to_host(xd), to_host(wd), b, relu=True)
    assert rel_l2(to_host(y), ref) <= TOL["bf16"]
    ref = O.conv3x3_bwd_data(to_host(dyd), to_host(wd), mask_src=to_host(md))
    assert rel_l2(to_host(dx), ref) <= TOL["bf16"]


@pytest.mark.parametrize("shape", WGRAD_BF16_SHAPES)
@pytest.mark.parametrize("offset", [0, 1])
def test_conv_bwd_weight_bf16_staging(shape, offset):
    """offset = 1 element shifts both tensors off their 16-byte alignment,
    which takes the one-column staging whatever the width."""
    n, c, h, w, k = shape
    print_case("conv_bwd_weight_bf16", shape=shape, offset=offset)
    x, _, _, dy, _ = _conv_inputs(n, c, h, w, k, 15)
    d = sb.conv_desc(n, c, h, w, k, sb.SB_BF16)
    ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_WEIGHT))
    xd, dyd = _dev_at(x, offset), _dev_at(dy, offset)
    dw = torch.full((k, c, 3, 3), float("nan"), device="cuda")
    db = torch.full((k,), float("nan"), device="cuda")
    sb.sb_conv3x3_bwd_weight(d, xd, dyd, dw, db, ws)
    torch.cuda.synchronize()
    dw_ref, db_ref = O.conv3x3_bwd_weight(to_host(xd), to_host(dyd))
    assert rel_l2(to_host(dw), dw_ref) <= TOL["f32"]
    assert rel_l2(to_host(db), db_ref) <= TOL["f32"]


PACKED_SHAPES = [(8, 3, 32, 32, 64), (2, 5, 7, 9, 70), (9, 40, 4, 4, 72), (33, 20, 2, 2, 130),
                 (2, 64, 6, 40, 80), (2, 36, 20, 20, 64), (2, 48, 14, 14, 64), (2, 12, 5, 37, 17),
                 (2, 12, 5, 38, 3)]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", PACKED_SHAPES)
def test_conv_packed_filters_match(shape, dtype):
    """Filters packed once (sb_conv3x3_pack_filters) and passed with
    SB_PACKED_FILTERS give bit-identical results to calls that pack them
    themselves, forward and data gradient."""
    n, c, h, w, k = shape
    print_case("conv_packed_filters", shape=shape, dtype=dtype)
    x, wt, b, dy, mask = _conv_inputs(n, c, h, w, k, 17)
    code = _code(dtype)
    xd, wd, dyd, md = to_dev(x, dtype), to_dev(wt, dtype), to_dev(dy, dtype), to_dev(mask, dtype)
    bd = to_dev(b)
    for pass_ in (sb.SB_PASS_FWD, sb.SB_PASS_BWD_DATA):
        d = sb.conv_desc(n, c, h, w, k, code, relu=pass_ == sb.SB_PASS_FWD)
        dp = sb.conv_desc(n, c, h, w, k, code, relu=pass_ == sb.SB_PASS_FWD, packed=True)
        ws = _ws(sb.sb_conv3x3_workspace_bytes(d, pass_))
        wsp = _ws(sb.sb_conv3x3_workspace_bytes(dp, pass_))
        packed = torch.full((max(sb.sb_conv3x3_packed_bytes(d, pass_), 256),), 0xFF,
                            dtype=torch.uint8, device="cuda")
        sb.sb_conv3x3_pack_filters(d, pass_, wd, packed)
        if pass_ == sb.SB_PASS_FWD:
            shape_out = (n, k, h, w)
            ref = torch.full(shape_out, float("nan"), dtype=_tdt(dtype), device="cuda")
            got = torch.full_like(ref, float("nan"))
            sb.sb_conv3x3_fwd(d, xd, wd, bd, ref, ws)
            sb.sb_conv3x3_fwd(dp, xd, packed, bd, got, wsp)
        else:
            shape_out = (n, c, h, w)
            ref = torch.full(shape_out, float("nan"), dtype=_tdt(dtype), device="cuda")
            got = torch.full_like(ref, float("nan"))
            sb.sb_conv3x3_bwd_data(d, dyd, wd, md, ref, ws)
            sb.sb_conv3x3_bwd_data(dp, dyd, packed, md, got, wsp)
        torch.cuda.synchronize()
        assert torch.equal(ref, got)
    # And against the oracle once (forward).
    y = torch.empty((n, k, h, w), dtype=_tdt(dtype), device="cuda")
    dp = sb.conv_desc(n, c, h, w, k, code, relu=True, packed=True)
    d = sb.conv_desc(n, c, h, w, k, code, relu=True)
    packed = torch.empty((max(sb.sb_conv3x3_packed_bytes(d, 0), 256),), dtype=torch.uint8,
                         device="cuda")
    sb.sb_conv3x3_pack_filters(d, 0, wd, packed)
    sb.sb_conv3x3_fwd(dp, xd, packed, bd, y, _ws(sb.sb_conv3x3_workspace_bytes(dp, 0)))
    torch.cuda.synchronize()
    assert rel_l2(to_host(y), O.conv3x3_fwd(to_host(xd), to_host(wd), b, relu=True)) <= TOL[dtype]


@pytest.mark.parametrize("dtype", DTYPES)
def test_conv_pack_filters_many_matches_single(dtype):
    """One batched packing of several layers and passes writes exactly what
    the per-layer packings write."""
    code = _code(dtype)
    items = []
    for j, (n, c, h, w, k) in enumerate(PACKED_SHAPES):
        wt = to_dev(synth.he_normal_conv3x3(k, c, 18 + j, synth.TID.CONV_W), dtype)
        d = sb.conv_desc(n, c, h, w, k, code)
        for pass_ in (sb.SB_PASS_FWD, sb.SB_PASS_BWD_DATA):
            nb = max(sb.sb_conv3x3_packed_bytes(d, pass_), 256)
            one = torch.full((nb,), 0xAB, dtype=torch.uint8, device="cuda")
            many = torch.full((nb,), 0xAB, dtype=torch.uint8, device="cuda")
            sb.sb_conv3x3_pack_filters(d, pass_, wt, one)
            items.append((d, pass_, wt, many, one))
    print_case("pack_filters_many", dtype=dtype, tasks=len(items))
    sb.sb_conv3x3_pack_filters_many(sb.PackList([(d, p_, w_, m) for d, p_, w_, m, _ in items]))
    torch.cuda.synchronize()
    for d, p_, _, many, one in items:
        assert torch.equal(many, one), (d.n, d.c, d.h, d.w, d.k, p_)


# Forward with fused ReLU + 2x2 pooling on NCHW fp32 (sb_conv3x3_fwd_pool):
# unsplit plans pooling in the epilogue (4x32 tiles, 8x16 tiles with two
# channel tiles, the two-group 8x8 tiles on whole 8x8 images, the same tiles
# over 14x14 images: ragged tiles and pooled edge) and split plans pooling in
# the split reduction (a small batch, the whole-image 4x4 and 2x2 tiles, a
# ragged output-channel tile).
FUSED_F32_SHAPES = [(64, 64, 32, 32, 64), (128, 64, 16, 16, 128), (128, 128, 8, 8, 256),
                    (128, 64, 14, 14, 64), (2, 64, 32, 32, 64), (128, 512, 4, 4, 512),
                    (128, 512, 2, 2, 512), (33, 64, 2, 2, 130), (33, 40, 4, 4, 70)]


@pytest.mark.parametrize("shape", FUSED_F32_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_conv_fwd_pool_f32(shape):
    """The fused call equals, bit for bit, the forward then the pool kernel
    (the same sums, pooled by the same rule), and against the oracle the
    pooled values meet 1e-4 and every differing code is a certified near-tie
    of the oracle's window values (the two sides' sums differ in their last
    bits)."""
    from tests.chain import NEAR_TIE_REL, near_tie_flips
    n, c, h, w, k = shape
    print_case("conv_fwd_pool_f32", shape=shape)
    x, wt, b, _, _ = _conv_inputs(n, c, h, w, k, 62)
    d = sb.conv_desc(n, c, h, w, k, sb.SB_F32)
    need = sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD_POOL)
    assert need != sb.SIZE_MAX, "pooled in the call"
    ws = _ws(need)
    xd, wd, bd = to_dev(x), to_dev(wt), to_dev(b)
    pooled = (n, k, h // 2, w // 2)
    y = torch.full(pooled, float("nan"), device="cuda")
    idx = torch.full(pooled, 0x55, dtype=torch.uint8, device="cuda")
    sb.sb_conv3x3_fwd_pool(d, xd, wd, bd, y, idx, ws)
    z = torch.full((n, k, h, w), float("nan"), device="cuda")
    y2 = torch.full(pooled, float("nan"), device="cuda")
    idx2 = torch.full(pooled, 0x55, dtype=torch.uint8, device="cuda")
    sb.sb_conv3x3_fwd(d, xd, wd, bd, z, _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD)))
    sb.sb_relu_maxpool_fwd(n, k, h, w, sb.SB_F32, sb.SB_NCHW, z, y2, idx2)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2), "codes differ from the unfused forward and pool"
    assert torch.equal(y.view(torch.int32), y2.view(torch.int32)), "pooled values differ"
    zr = O.conv3x3_fwd(x, wt, b)
    ry, ridx = O.relu_maxpool_fwd(zr)
    assert rel_l2(to_host(y), ry) <= TOL["f32"]
    flips = near_tie_flips(zr, ridx, idx.cpu().numpy(), NEAR_TIE_REL["f32"] * np.max(np.abs(zr)))
    print("near-tie windows:", flips)


def test_conv_bwd_weight_without_bias_grad():
    n, c, h, w, k = 2, 8, 6, 6, 20
    x, _, _, dy, _ = _conv_inputs(n, c, h, w, k, 14)
    d = sb.conv_desc(n, c, h, w, k, sb.SB_F32)
    ws = _ws(sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_WEIGHT))
    dw = torch.empty((k, c, 3, 3), device="cuda")
    sb.sb_conv3x3_bwd_weight(d, to_dev(x), to_dev(dy), dw, None, ws)
    torch.cuda.synchronize()
    assert rel_l2(to_host(dw), O.conv3x3_bwd_weight(x, dy)[0]) <= TOL["f32"]


def test_workspace_too_small_is_reported():
    d = sb.conv_desc(128, 512, 2, 2, 512, sb.SB_F32)
    need = sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD)
    assert need > 0
    x = torch.zeros((128, 512, 2, 2), device="cuda")
    wt = torch.zeros((512, 512, 3, 3), device="cuda")
    y = torch.zeros((128, 512, 2, 2), device="cuda")
    with pytest.raises(sb.SBError) as e:
        sb.sb_conv3x3_fwd(d, x, wt, None, y, _ws(need // 2))
    assert e.value.status == sb.SB_ERR_WORKSPACE


# -------------------------------------------------------------- FC shard --
# The FC workloads' shapes (hybrid step: 512 gathered rows; group training
# step: 128 rows, FC 4096 -> 512 and 1024 -> 5 shards), ragged shapes, and a
# tall reduction whose weight gradient is split (bias gradient summed apart).
# (64, 4128, 256): the forward's reduction splits into ranges of an odd
# number of k tiles (the GEMM's two-set operand pipeline ends on either set).
FC_SHAPES = [(512, 4096, 1024), (512, 512, 1024), (128, 4096, 512), (128, 1024, 5),
             (37, 70, 50), (130, 200, 257), (1, 1, 1), (64, 33, 129), (4096, 64, 64),
             (64, 4128, 256)]


def _fc_inputs(m, kin, ns, seed):
    x = synth.relu_normal((m, kin), seed, synth.TID.FC_X)
    wfull = synth.xavier_uniform(kin, ns * 2, seed, synth.TID.FC_W)
    w = np.ascontiguousarray(wfull[:, :ns])
    b = synth.normal((ns,), seed, synth.TID.FC_B)
    dy = synth.normal((m, ns), seed, synth.TID.FC_DY)
    mask = synth.normal((m, ns), seed, synth.TID.MISC)
    return x, w, b, dy, mask


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", FC_SHAPES)
@pytest.mark.parametrize("relu", [False, True])
def test_fc_fwd(shape, relu, dtype):
    m, kin, ns = shape
    print_case("fc_fwd", shape=shape, relu=relu, dtype=dtype)
    x, w, b, _, _ = _fc_inputs(m, kin, ns, 21)
    d = sb.fc_desc(m, kin, ns, _code(dtype), relu=relu)
    ws = _ws(sb.sb_fc_workspace_bytes(d, sb.SB_FC_FWD))
    y = torch.full((m, ns), float("nan"), dtype=_tdt(dtype), device="cuda")
    xd, wd = to_dev(x, dtype), to_dev(w, dtype)
    sb.sb_fc_shard_fwd(d, xd, wd, to_dev(b), y, ws)
    torch.cuda.synchronize()
    # The oracle gets the values the kernel read; bf16 outputs are rounded.
    ref = O.fc_fwd(to_host(xd), to_host(wd), b, relu=relu)
    if dtype == "bf16":
        ref = O.round_bf16(ref)
    assert rel_l2(to_host(y), ref) <= TOL[dtype]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", FC_SHAPES)
@pytest.mark.parametrize("masked", [False, True])
def test_fc_bwd(shape, masked, dtype):
    m, kin, ns = shape
    print_case("fc_bwd", shape=shape, masked=masked, dtype=dtype)
    x, w, _, dy, mask = _fc_inputs(m, kin, ns, 22)
    d = sb.fc_desc(m, kin, ns, _code(dtype))
    ws = _ws(sb.sb_fc_workspace_bytes(d, sb.SB_FC_BWD))
    dxp = torch.full((m, kin), float("nan"), dtype=_tdt(dtype), device="cuda")
    dw = torch.full((kin, ns), float("nan"), device="cuda")
    db = torch.full((ns,), float("nan"), device="cuda")
    xd, wd, dyd, md = (to_dev(a, dtype) for a in (x, w, dy, mask))
    sb.sb_fc_shard_bwd(d, xd, wd, dyd, md if masked else None, dxp, dw, db, False, ws)
    torch.cuda.synchronize()
    rdx, rdw, rdb = O.fc_bwd(to_host(xd), to_host(wd), to_host(dyd),
                             mask_src=to_host(md) if masked else None)
    if dtype == "bf16":
        rdx = O.round_bf16(rdx)
    assert rel_l2(to_host(dxp), rdx) <= TOL[dtype]
    # dW and db are fp32 sums of exact products of the bf16 values.
    assert rel_l2(to_host(dw), rdw) <= TOL["f32"]
    assert rel_l2(to_host(db), rdb) <= TOL["f32"]


@pytest.mark.parametrize("m,kin,ns,K", [(512, 300, 96, 4), (16384, 64, 64, 4)])
def test_fc_bwd_accumulates_over_modulo_iterations(m, kin, ns, K):
    """K calls with accumulate=1 on the K row blocks equal one call on all
    rows (the FC shard's gradient summed over the modulo iterations); the
    second shape splits the weight-gradient product."""
    x, w, _, dy, _ = _fc_inputs(m, kin, ns, 23)
    blk = m // K
    d = sb.fc_desc(blk, kin, ns)
    ws = _ws(sb.sb_fc_workspace_bytes(d, sb.SB_FC_BWD))
    dw = torch.empty((kin, ns), device="cuda")
    db = torch.empty((ns,), device="cuda")
    xd, wd, dyd = to_dev(x), to_dev(w), to_dev(dy)
    for q in range(K):
        sb.sb_fc_shard_bwd(d, xd[q * blk:(q + 1) * blk], wd, dyd[q * blk:(q + 1) * blk], None,
                           None, dw, db, q > 0, ws)
    torch.cuda.synchronize()
    _, rdw, rdb = O.fc_bwd(x, w, dy)
    assert rel_l2(to_host(dw), rdw) <= TOL["f32"]
    assert rel_l2(to_host(db), rdb) <= TOL["f32"]


def test_fc_strided_rows():
    """x, y, dy and the mask read with row strides larger than their width."""
    m, kin, ns, ldx, ldy = 70, 48, 40, 64, 100
    x, w, b, dy, mask = _fc_inputs(m, kin, ns, 24)
    xbig = np.zeros((m, ldx), np.float32); xbig[:, :kin] = x
    ybig = torch.zeros((m, ldy), device="cuda")
    dybig = np.zeros((m, ldy), np.float32); dybig[:, :ns] = dy
    mbig = np.zeros((m, ldy), np.float32); mbig[:, :ns] = mask
    df = sb.fc_desc(m, kin, ns, ldx=ldx, ldy=ldy, relu=True)
    db_ = sb.fc_desc(m, kin, ns, ldx=ldx, ldy=ldy)
    ws = _ws(max(sb.sb_fc_workspace_bytes(df, 0), sb.sb_fc_workspace_bytes(db_, 1)))
    xd = to_dev(xbig)
    sb.sb_fc_shard_fwd(df, xd, to_dev(w), to_dev(b), ybig, ws)
    dxp = torch.full((m, ldx), 5.0, device="cuda")
    dw = torch.empty((kin, ns), device="cuda")
    sb.sb_fc_shard_bwd(db_, xd, to_dev(w), to_dev(dybig), to_dev(mbig), dxp, dw, None, False, ws)
    torch.cuda.synchronize()
    assert rel_l2(to_host(ybig)[:, :ns], O.fc_fwd(x, w, b, relu=True)) <= TOL["f32"]
    assert np.all(to_host(ybig)[:, ns:] == 0.0)                     # untouched
    rdx, rdw, _ = O.fc_bwd(x, w, dy, mask_src=mask)
    assert rel_l2(to_host(dxp)[:, :kin], rdx) <= TOL["f32"]
    assert np.all(to_host(dxp)[:, kin:] == 5.0)
    assert rel_l2(to_host(dw), rdw) <= TOL["f32"]


def test_fc_unaligned_operands():
    """Operands that start off a 16-byte boundary take the element-wise
    staging path; results are the same."""
    m, kin, ns = 96, 128, 64
    x, w, b, dy, mask = _fc_inputs(m, kin, ns, 25)
    base = torch.zeros(m * kin + 1, device="cuda")
    xd = base[1:].view(m, kin)
    xd.copy_(to_dev(x))
    df = sb.fc_desc(m, kin, ns, relu=True)
    db_ = sb.fc_desc(m, kin, ns)
    ws = _ws(max(sb.sb_fc_workspace_bytes(df, 0), sb.sb_fc_workspace_bytes(db_, 1)))
    y = torch.empty((m, ns), device="cuda")
    sb.sb_fc_shard_fwd(df, xd, to_dev(w), to_dev(b), y, ws)
    dx = torch.empty((m, kin), device="cuda")
    dw = torch.empty((kin, ns), device="cuda")
    dbias = torch.empty((ns,), device="cuda")
    sb.sb_fc_shard_bwd(db_, xd, to_dev(w), to_dev(dy), to_dev(mask), dx, dw, dbias, False, ws)
    torch.cuda.synchronize()
    assert rel_l2(to_host(y), O.fc_fwd(x, w, b, relu=True)) <= TOL["f32"]
    rdx, rdw, rdb = O.fc_bwd(x, w, dy, mask_src=mask)
    assert rel_l2(to_host(dx), rdx) <= TOL["f32"]
    assert rel_l2(to_host(dw), rdw) <= TOL["f32"]
    assert rel_l2(to_host(dbias), rdb) <= TOL["f32"]
