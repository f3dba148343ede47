"""Pins of the fp64 oracle against things other than itself.

Each test checks one oracle function against an independent library routine
(torch CPU float64: conv2d, max_pool2d, autograd), a closed form (1x1 conv =
matmul, delta kernels = identity / shift), an invariant (adjoint identities,
shard concatenation, conservation in the pool backward) or brute-force finite
differences on tiny inputs.  Together they are chosen so that a dropped term,
a wrong sign, a wrong index, a flipped kernel or a transposed operand in the
oracle fails at least one of them.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O
from oracle import stack as OS

rng = np.random.default_rng(1234)


def _t(a, grad=False):
    t = torch.tensor(np.asarray(a, dtype=np.float64))
    if grad:
        t.requires_grad_(True)
    return t


# ------------------------------------------------------------------ conv --
@pytest.mark.parametrize("n,c,h,w,k", [(1, 1, 1, 1, 1), (2, 3, 5, 4, 3), (1, 4, 2, 2, 5),
                                       (3, 2, 7, 6, 2), (1, 3, 1, 5, 2)])
def test_conv_fwd_matches_torch_conv2d(n, c, h, w, k):
    x = rng.standard_normal((n, c, h, w))
    wt = rng.standard_normal((k, c, 3, 3))
    b = rng.standard_normal(k)
    ref = F.conv2d(_t(x), _t(wt), _t(b), stride=1, padding=1).numpy()
    got = O.conv3x3_fwd(x, wt, b)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    got_relu = O.conv3x3_fwd(x, wt, b, relu=True)
    np.testing.assert_allclose(got_relu, np.maximum(ref, 0), rtol=1e-12, atol=1e-12)


def test_conv_centre_tap_is_channel_matmul():
    x = rng.standard_normal((2, 5, 4, 3))
    m = rng.standard_normal((6, 5))
    wt = np.zeros((6, 5, 3, 3))
    wt[:, :, 1, 1] = m
    ref = np.einsum("kc,nchw->nkhw", m, x)
    np.testing.assert_allclose(O.conv3x3_fwd(x, wt), ref, rtol=1e-13, atol=1e-13)


def test_conv_delta_kernels_identity_and_shift():
    x = rng.standard_normal((2, 3, 5, 6))
    eye = np.zeros((3, 3, 3, 3))
    for c in range(3):
        eye[c, c, 1, 1] = 1.0
    np.testing.assert_array_equal(O.conv3x3_fwd(x, eye), x)
    # Tap (0,0) reads the input at (h-1, w-1): cross-correlation, zero fill.
    shift = np.zeros((3, 3, 3, 3))
    for c in range(3):
        shift[c, c, 0, 0] = 1.0
    want = np.zeros_like(x)
    want[:, :, 1:, 1:] = x[:, :, :-1, :-1]
    np.testing.assert_array_equal(O.conv3x3_fwd(x, shift), want)
    # Tap (2,1) reads (h+1, w).
    shift2 = np.zeros((3, 3, 3, 3))
    for c in range(3):
        shift2[c, c, 2, 1] = 1.0
    want2 = np.zeros_like(x)
    want2[:, :, :-1, :] = x[:, :, 1:, :]
    np.testing.assert_array_equal(O.conv3x3_fwd(x, shift2), want2)


def test_conv_fwd_at_matches_full():
    x = rng.standard_normal((2, 3, 6, 5))
    wt = rng.standard_normal((4, 3, 3, 3))
    b = rng.standard_normal(4)
    full = O.conv3x3_fwd(x, wt, b, relu=True)
    flat = rng.choice(full.size, 37, replace=False)
    np.testing.assert_array_equal(O.conv3x3_fwd_at(x, wt, flat, b, relu=True), full.ravel()[flat])


@pytest.mark.parametrize("n,c,h,w,k", [(2, 3, 5, 4, 3), (1, 6, 2, 2, 4), (2, 2, 3, 7, 5)])
def test_conv_adjoint_identities(n, c, h, w, k):
    """<conv(X;W), dZ> = <X, bwd_data(dZ;W)> = <W, bwd_weight(X,dZ)>."""
    x = rng.standard_normal((n, c, h, w))
    wt = rng.standard_normal((k, c, 3, 3))
    dz = rng.standard_normal((n, k, h, w))
    lhs = np.sum(O.conv3x3_fwd(x, wt) * dz)
    dx = O.conv3x3_bwd_data(dz, wt)
    dw, db = O.conv3x3_bwd_weight(x, dz)
    assert abs(lhs - np.sum(x * dx)) <= 1e-12 * (1 + abs(lhs))
    assert abs(lhs - np.sum(wt * dw)) <= 1e-12 * (1 + abs(lhs))
    np.testing.assert_allclose(db, dz.sum(axis=(0, 2, 3)), rtol=1e-13)


@pytest.mark.parametrize("n,c,h,w,k", [(2, 3, 5, 4, 3), (1, 4, 2, 2, 2), (2, 5, 4, 4, 6)])
def test_conv_bwd_matches_torch_autograd(n, c, h, w, k):
    x = _t(rng.standard_normal((n, c, h, w)), True)
    wt = _t(rng.standard_normal((k, c, 3, 3)), True)
    b = _t(rng.standard_normal(k), True)
    dz = rng.standard_normal((n, k, h, w))
    F.conv2d(x, wt, b, padding=1).backward(_t(dz))
    dx = O.conv3x3_bwd_data(dz, wt.detach().numpy())
    dw, db = O.conv3x3_bwd_weight(x.detach().numpy(), dz)
    np.testing.assert_allclose(dx, x.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(db, b.grad.numpy(), rtol=1e-11, atol=1e-11)


def test_conv_bwd_data_mask_is_relu_derivative():
    """bwd_data with mask source A = relu(Zp) is the gradient w.r.t. Zp of
    <conv(relu(Zp)), dZ> (torch autograd, ReLU'(0) = 0)."""
    zp = rng.standard_normal((2, 3, 4, 5))
    zp[0, 0, 0, :2] = 0.0                       # exact zeros: no gradient
    wt = rng.standard_normal((4, 3, 3, 3))
    dz = rng.standard_normal((2, 4, 4, 5))
    zt = _t(zp, True)
    F.conv2d(torch.relu(zt), _t(wt), padding=1).backward(_t(dz))
    got = O.conv3x3_bwd_data(dz, wt, mask_src=np.maximum(zp, 0))
    np.testing.assert_allclose(got, zt.grad.numpy(), rtol=1e-11, atol=1e-11)
    assert np.all(got[0, 0, 0, :2] == 0.0)


def test_conv_bwd_finite_differences():
    x = rng.standard_normal((1, 2, 3, 3))
    wt = rng.standard_normal((2, 2, 3, 3))
    dz = rng.standard_normal((1, 2, 3, 3))
    loss = lambda xx, ww: float(np.sum(O.conv3x3_fwd(xx, ww) * dz))
    dx = O.conv3x3_bwd_data(dz, wt)
    dw, _ = O.conv3x3_bwd_weight(x, dz)
    eps = 1e-6
    for idx in np.ndindex(x.shape):
        e = np.zeros_like(x); e[idx] = eps
        assert abs((loss(x + e, wt) - loss(x - e, wt)) / (2 * eps) - dx[idx]) < 1e-7
    for idx in np.ndindex(wt.shape):
        e = np.zeros_like(wt); e[idx] = eps
        assert abs((loss(x, wt + e) - loss(x, wt - e)) / (2 * eps) - dw[idx]) < 1e-7


def test_conv_bwd_at_matches_full():
    x = rng.standard_normal((2, 3, 5, 4))
    wt = rng.standard_normal((4, 3, 3, 3))
    dz = rng.standard_normal((2, 4, 5, 4))
    mask = np.maximum(rng.standard_normal(x.shape), 0)
    dx = O.conv3x3_bwd_data(dz, wt, mask_src=mask)
    f = rng.choice(dx.size, 29, replace=False)
    np.testing.assert_array_equal(O.conv3x3_bwd_data_at(dz, wt, f, mask_src=mask), dx.ravel()[f])
    dw, _ = O.conv3x3_bwd_weight(x, dz)
    f = rng.choice(dw.size, 31, replace=False)
    np.testing.assert_array_equal(O.conv3x3_bwd_weight_at(x, dz, f), dw.ravel()[f])


# ------------------------------------------------------- relu + maxpool --
def test_relu_maxpool_fwd_matches_torch():
    x = rng.standard_normal((3, 4, 6, 8))
    y, idx = O.relu_maxpool_fwd(x)
    ref, ridx = F.max_pool2d(_t(x), 2, 2, return_indices=True)
    np.testing.assert_array_equal(y, np.maximum(ref.numpy(), 0.0))
    # torch's flat index inside the plane -> window position (row-major).
    ri = ridx.numpy()
    pos = (ri // 8 % 2) * 2 + (ri % 8 % 2)
    np.testing.assert_array_equal(idx & 3, pos)
    np.testing.assert_array_equal((idx & 0x80) != 0, ref.numpy() <= 0)
    assert np.all((idx & 0x7C) == 0)


def test_relu_maxpool_constructed_ties_and_signs():
    x = np.array([[[[1.0, 1.0], [0.5, 1.0]],        # tie: first max (pos 0)
                   [[0.2, 0.7], [0.7, 0.7]],        # tie among 1,2,3 -> pos 1
                   [[-1.0, -0.5], [-2.0, -0.5]],    # all negative -> flag, pos 1
                   [[0.0, -1.0], [-1.0, -1.0]],     # max exactly 0 -> flag
                   [[-3.0, -2.0], [5.0, 5.0]]]])    # tie at 2,3 -> pos 2
    x = x.reshape(1, 5, 2, 2)
    y, idx = O.relu_maxpool_fwd(x)
    np.testing.assert_array_equal(y.ravel(), [1.0, 0.7, 0.0, 0.0, 5.0])
    np.testing.assert_array_equal(idx.ravel(), [0, 1, 0x80 | 1, 0x80 | 0, 2])
    assert not np.signbit(y.ravel()[3])           # +0, not -0


def test_relu_maxpool_bwd_matches_torch_and_invariants():
    x = rng.standard_normal((2, 3, 8, 6))
    y, idx = O.relu_maxpool_fwd(x)
    dy = rng.standard_normal(y.shape)
    dx = O.relu_maxpool_bwd(dy, idx)
    xt = _t(x, True)
    torch.relu(F.max_pool2d(xt, 2, 2)).backward(_t(dy))
    np.testing.assert_array_equal(dx, xt.grad.numpy())
    win = dx.reshape(2, 3, 4, 2, 3, 2)
    nnz = (win != 0).sum(axis=(3, 5))
    assert nnz.max() <= 1
    np.testing.assert_allclose(dx.sum(), (dy * ((idx & 0x80) == 0)).sum(), rtol=1e-13)


def test_relu_maxpool_bwd_routes_to_code_position():
    dy = np.array([1.5, -2.0, 3.0, 4.0]).reshape(1, 4, 1, 1)
    idx = np.array([3, 0, 0x80 | 2, 1], dtype=np.uint8).reshape(1, 4, 1, 1)
    dx = O.relu_maxpool_bwd(dy, idx).reshape(4, 4)
    np.testing.assert_array_equal(dx, [[0, 0, 0, 1.5], [-2.0, 0, 0, 0], [0, 0, 0, 0], [0, 4.0, 0, 0]])


# -------------------------------------------------------------- FC shard --
def test_fc_fwd_matches_matmul():
    x = rng.standard_normal((7, 11))
    w = rng.standard_normal((11, 5))
    b = rng.standard_normal(5)
    np.testing.assert_allclose(O.fc_fwd(x, w, b), x @ w + b, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.fc_fwd(x, w, b, relu=True), np.maximum(x @ w + b, 0),
                               rtol=1e-12, atol=1e-12)


def test_fc_shards_concatenate_to_full_layer():
    """K column shards: Y concatenates, partial dX sums, dW concatenates."""
    m, kin, nf, K = 9, 12, 8, 4
    x = rng.standard_normal((m, kin))
    w = rng.standard_normal((kin, nf))
    b = rng.standard_normal(nf)
    dy = rng.standard_normal((m, nf))
    ns = nf // K
    ys, dxs, dws, dbs = [], [], [], []
    for q in range(K):
        sl = slice(q * ns, (q + 1) * ns)
        ys.append(O.fc_fwd(x, w[:, sl], b[sl]))
        dxp, dw, db = O.fc_bwd(x, w[:, sl], dy[:, sl])
        dxs.append(dxp); dws.append(dw); dbs.append(db)
    np.testing.assert_allclose(np.concatenate(ys, 1), x @ w + b, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(sum(dxs), dy @ w.T, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(np.concatenate(dws, 1), x.T @ dy, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(np.concatenate(dbs), dy.sum(0), rtol=1e-12, atol=1e-12)


def test_fc_bwd_matches_torch_autograd_with_mask():
    x = _t(rng.standard_normal((6, 10)), True)
    w = _t(rng.standard_normal((10, 4)), True)
    b = _t(rng.standard_normal(4), True)
    dy = rng.standard_normal((6, 4))
    y = torch.relu(x @ w + b)
    y.backward(_t(dy))
    dxp, dw, db = O.fc_bwd(x.detach().numpy(), w.detach().numpy(), dy,
                           mask_src=y.detach().numpy())
    np.testing.assert_allclose(dxp, x.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, w.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, b.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_fc_accumulate_over_row_blocks_equals_one_call():
    """Summing dW over the K modulo iterations (row blocks of the gathered
    batch) equals one call on all rows."""
    x = rng.standard_normal((12, 5))
    w = rng.standard_normal((5, 3))
    dy = rng.standard_normal((12, 3))
    _, dw_all, db_all = O.fc_bwd(x, w, dy)
    dw = np.zeros((5, 3)); db = np.zeros(3)
    for q in range(4):
        sl = slice(3 * q, 3 * q + 3)
        _, dw, db = O.fc_bwd(x[sl], w, dy[sl], dw_acc=dw, db_acc=db)
    np.testing.assert_allclose(dw, dw_all, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(db, db_all, rtol=1e-13, atol=1e-13)


def test_fc_at_matches_full():
    x = rng.standard_normal((6, 9))
    w = rng.standard_normal((9, 4))
    b = rng.standard_normal(4)
    dy = rng.standard_normal((6, 4))
    mask = np.maximum(rng.standard_normal((6, 4)), 0)
    y = O.fc_fwd(x, w, b, relu=True)
    f = rng.choice(y.size, 10, replace=False)
    np.testing.assert_array_equal(O.fc_fwd_at(x, w, f, b, relu=True), y.ravel()[f])
    dxp, dw, _ = O.fc_bwd(x, w, dy, mask_src=mask)
    f = rng.choice(dxp.size, 13, replace=False)
    np.testing.assert_array_equal(O.fc_bwd_dx_at(w, dy, f, mask_src=mask), dxp.ravel()[f])
    f = rng.choice(dw.size, 11, replace=False)
    np.testing.assert_array_equal(O.fc_bwd_dw_at(x, dy, f, mask_src=mask), dw.ravel()[f])


# ------------------------------------------------------------- bf16 -------
def test_round_bf16_matches_torch_and_halfway_cases():
    v = np.concatenate([rng.standard_normal(5000) * 10.0 ** rng.integers(-30, 30, 5000),
                        rng.standard_normal(100) * 1e-39])   # bf16 subnormals
    v32 = v.astype(np.float32)
    ref = torch.tensor(v32).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(O.round_bf16(v32), ref)
    q = 2.0 ** -8
    half = np.array([1 + q, 1 + 3 * q, -(1 + q), 2 + 2 * q * 1, 0.0, -0.0])
    np.testing.assert_array_equal(O.round_bf16(half), [1.0, 1 + 4 * q, -1.0, 2.0, 0.0, -0.0])


# ------------------------------------------------------------ composition --
def _torch_stack(x, ws, bs, pools, dy):
    xt = _t(x, True)
    wt = [_t(w, True) for w in ws]
    a = xt
    for l, w in enumerate(wt):
        z = F.conv2d(a, w, _t(bs[l]), padding=1)
        a = torch.relu(F.max_pool2d(z, 2, 2)) if pools[l] else torch.relu(z)
    a.backward(_t(dy))
    return a.detach().numpy(), xt.grad.numpy(), [w.grad.numpy() for w in wt]


def test_vgg_stack_matches_torch_autograd():
    sched = [(3, 4, False), (4, 5, True), (5, 6, False), (6, 6, True)]
    x = rng.standard_normal((2, 3, 8, 8))
    ws = [rng.standard_normal((k, c, 3, 3)) * 0.5 for c, k, _ in sched]
    bs = [rng.standard_normal(k) * 0.1 for _, k, _ in sched]
    pools = [p for *_, p in sched]
    dy = rng.standard_normal((2, 6, 2, 2))
    f, b = OS.vgg_step(x, ws, bs, pools, dy)
    out, dx, dws = _torch_stack(x, ws, bs, pools, dy)
    np.testing.assert_allclose(f["A"][-1], out, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(b["dX"], dx, rtol=1e-10, atol=1e-11)
    for l in range(len(ws)):
        np.testing.assert_allclose(b["dW"][l], dws[l], rtol=1e-10, atol=1e-11)


def test_hybrid_step_matches_torch_autograd():
    """Three FC shards (ReLU, ReLU, linear) after a two-conv stack, with
    remote rows and remote shard columns as constants: the oracle's chain of
    restricted partial gradients equals autograd of the same graph."""
    n, rep = 2, 3
    sched = [(3, 4, True), (4, 8, True)]          # 4x4 -> 2x2 -> 1x1, 8 features
    x = rng.standard_normal((n, 3, 4, 4))
    ws = [rng.standard_normal((k, c, 3, 3)) for c, k, _ in sched]
    bs = [np.zeros(k) for _, k, _ in sched]
    pools = [p for *_, p in sched]
    # FC j: local shard ns_j of the layer's outputs; the next layer's input is
    # ns_j local columns + remote columns.
    ns, remote = [5, 6, 4], [7, 3]
    ins = [8, ns[0] + remote[0], ns[1] + remote[1]]
    fw = [rng.standard_normal((ins[j], ns[j])) for j in range(3)]
    fb = [rng.standard_normal(ns[j]) for j in range(3)]
    rows = np.maximum(rng.standard_normal((n * (rep - 1), 8)), 0)
    cols = [np.maximum(rng.standard_normal((n * rep, remote[j])), 0) for j in range(2)]
    dy = rng.standard_normal((n * rep, ns[2]))
    r = OS.hybrid_step(x, ws, bs, pools, fw, fb, rows, cols, dy)
    # torch: the same graph, remote stand-ins as constants; gradients flow to
    # the local rows / local columns only, exactly as the restriction does.
    xt = _t(x, True); wt = [_t(w, True) for w in ws]
    a = xt
    for l, w in enumerate(wt):
        a = torch.relu(F.max_pool2d(F.conv2d(a, w, padding=1), 2, 2))
    h = torch.cat([a.reshape(n, 8), _t(rows)], 0)
    fwt = [_t(w, True) for w in fw]
    for j in range(3):
        h = h @ fwt[j] + _t(fb[j])
        if j < 2:
            h = torch.cat([torch.relu(h), _t(cols[j])], 1)
    h.backward(_t(dy))
    np.testing.assert_allclose(r["ys"][2], h.detach().numpy(), rtol=1e-11, atol=1e-12)
    for j in range(3):
        np.testing.assert_allclose(r["dw"][j], fwt[j].grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(r["bwd"]["dX"], xt.grad.numpy(), rtol=1e-10, atol=1e-11)
    for l in range(2):
        np.testing.assert_allclose(r["bwd"]["dW"][l], wt[l].grad.numpy(), rtol=1e-10, atol=1e-11)


def test_bf16_stack_rounds_at_storage_points():
    sched = [(3, 4, False), (4, 4, True)]
    x = O.round_bf16(rng.standard_normal((1, 3, 4, 4)))
    ws = [O.round_bf16(rng.standard_normal((k, c, 3, 3))) for c, k, _ in sched]
    bs = [np.zeros(k) for _, k, _ in sched]
    pools = [p for *_, p in sched]
    dy = O.round_bf16(rng.standard_normal((1, 4, 2, 2)))
    f, b = OS.vgg_step(x, ws, bs, pools, dy, bf16=True)
    for a in f["A"][1:] + list(f["Z"].values()) + [b["dX"]] + list(b["dZ"].values()):
        np.testing.assert_array_equal(a, O.round_bf16(a))


def test_round_f32_matches_torch_and_halfway_cases():
    a = rng.standard_normal(1000) * 10.0 ** rng.integers(-30, 30, 1000)
    np.testing.assert_array_equal(O.round_f32(a), torch.tensor(a).float().double().numpy())
    u = 2.0 ** -24                                   # half an ulp of 1 in float32
    half = np.array([1 + u, 1 + 3 * u, -(1 + u), 1 + u * 1.5])
    np.testing.assert_array_equal(O.round_f32(half), [1.0, 1 + 4 * u, -1.0, 1 + 2 * u])


@pytest.mark.parametrize("store", ["f32", "bf16"])
def test_stack_chain_rounds_at_storage_points(store):
    """The storage-rounded chain: every stored activation and activation
    gradient is representable in the storage type, and each stored tensor
    is the rounding of the exact layer function applied to the stored
    tensors before it (one layer checked by hand here)."""
    rnd = O.round_f32 if store == "f32" else O.round_bf16
    sched = [(3, 4, False), (4, 4, True)]
    x = rnd(rng.standard_normal((2, 3, 4, 4)))
    ws = [rnd(rng.standard_normal((k, c, 3, 3))) for c, k, _ in sched]
    bs = [np.zeros(k) for _, k, _ in sched]
    pools = [p for *_, p in sched]
    dy = rnd(rng.standard_normal((2, 4, 2, 2)))
    f, b = OS.vgg_step(x, ws, bs, pools, dy, store=store)
    for a in f["A"][1:] + list(f["Z"].values()) + [b["dX"]] + list(b["dZ"].values()):
        np.testing.assert_array_equal(a, rnd(a))
    np.testing.assert_array_equal(f["A"][1], rnd(np.maximum(
        F.conv2d(_t(x), _t(ws[0]), padding=1).numpy(), 0)))
    if store == "f32":
        f64, b64 = OS.vgg_step(x, ws, bs, pools, dy)
        for l in range(2):
            np.testing.assert_allclose(b["dW"][l], b64["dW"][l], rtol=1e-5, atol=1e-6)
