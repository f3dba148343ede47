"""GPU parity at the workloads' real shapes, and end-to-end through the stacks.

* Every distinct layer shape of the VGG-16 CIFAR stack (batch 128) runs each
  conv pass in the same launch configuration the benchmark times; the oracle
  evaluates a sample of outputs one by one.
* The whole VGG-16 stack and the hybrid worker step run end-to-end from the
  seeded inputs at a batch the oracle finishes in seconds; every forward
  tensor, pool code and gradient is compared layer by layer.
"""
import numpy as np
import pytest
import torch

import oracle as O
from oracle import stack as OS
from paper_2112_15317_amd import configs, sb, synth
from paper_2112_15317_amd.stack import ConvStack, HybridStep
from tests.helpers import TOL, print_case, rel_l2, sample_idx, to_dev, to_host

pytestmark = pytest.mark.gpu

VGG_CIFAR = configs.conv_layers(configs.VGG16, 3, 32)
SAMPLES = 3000


def _ws(nbytes):
    # The workspace needs no initialisation: hand it over full of NaN bytes.
    return torch.full((max(int(nbytes), 256),), 0xFF, dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("L", VGG_CIFAR, ids=lambda L: "conv%d_%dx%d_%d" % (L.index + 1, L.c, L.k, L.h))
def test_vgg_cifar_layer_full_size_sampled(L):
    n = 128
    print_case("layer_full", layer=L.index, c=L.c, k=L.k, h=L.h, n=n)
    seed = 100 + L.index
    x = np.maximum(synth.normal((n, L.c, L.h, L.w), seed, synth.TID.IMAGES), 0)
    if L.index == 0:
        x = synth.normal((n, L.c, L.h, L.w), seed, synth.TID.IMAGES)
    wt = synth.he_normal_conv3x3(L.k, L.c, seed, synth.TID.CONV_W)
    dy = synth.normal((n, L.k, L.h, L.w), seed, synth.TID.DY_TOP)
    relu = not L.pool_after
    mask = x if L.index > 0 else None
    xd, wd, dyd = to_dev(x), to_dev(wt), to_dev(dy)
    df = sb.conv_desc(n, L.c, L.h, L.w, L.k, sb.SB_F32, relu=relu)
    db_ = sb.conv_desc(n, L.c, L.h, L.w, L.k, sb.SB_F32)
    ws = _ws(max(sb.sb_conv3x3_workspace_bytes(df, 0), sb.sb_conv3x3_workspace_bytes(db_, 1),
                 sb.sb_conv3x3_workspace_bytes(db_, 2)))
    y = torch.empty((n, L.k, L.h, L.w), device="cuda")
    dx = torch.empty((n, L.c, L.h, L.w), device="cuda")
    dw = torch.empty((L.k, L.c, 3, 3), device="cuda")
    dbias = torch.empty((L.k,), device="cuda")
    sb.sb_conv3x3_fwd(df, xd, wd, None, y, ws)
    sb.sb_conv3x3_bwd_data(db_, dyd, wd, xd if mask is not None else None, dx, ws)
    sb.sb_conv3x3_bwd_weight(db_, xd, dyd, dw, dbias, ws)
    torch.cuda.synchronize()
    f = sample_idx(y.numel(), SAMPLES, seed)
    assert rel_l2(to_host(y).ravel()[f], O.conv3x3_fwd_at(x, wt, f, relu=relu)) <= TOL["f32"]
    f = sample_idx(dx.numel(), SAMPLES, seed + 1)
    ref = O.conv3x3_bwd_data_at(dy, wt, f, mask_src=mask)
    assert rel_l2(to_host(dx).ravel()[f], ref) <= TOL["f32"]
    f = sample_idx(dw.numel(), min(SAMPLES, 600), seed + 2)
    assert rel_l2(to_host(dw).ravel()[f], O.conv3x3_bwd_weight_at(x, dy, f)) <= TOL["f32"]
    assert rel_l2(to_host(dbias), dy.astype(np.float64).sum(axis=(0, 2, 3))) <= TOL["f32"]


def _distinct(layers):
    seen, out = set(), []
    for L in layers:
        key = (L.c, L.k, L.h, L.pool_after, L.index == 0)
        if key not in seen:
            seen.add(key)
            out.append(L)
    return out


VGG_IMAGENET = _distinct(configs.conv_layers(configs.VGG16, 3, 224))


@pytest.mark.parametrize("L", VGG_IMAGENET,
                         ids=lambda L: "conv%d_%dx%d_%d" % (L.index + 1, L.c, L.k, L.h))
def test_vgg_imagenet_bf16_layer_full_size_sampled(L):
    """bf16 activations / filters, fp32 accumulation, batch 32 at 224x224:
    each distinct layer shape of the ImageNet-shaped stack, sampled."""
    n = 32
    print_case("layer_full_bf16", layer=L.index, c=L.c, k=L.k, h=L.h, n=n)
    seed = 300 + L.index
    x = synth.normal((n, L.c, L.h, L.w), seed, synth.TID.IMAGES)
    if L.index > 0:
        x = np.maximum(x, 0)
    wt = synth.he_normal_conv3x3(L.k, L.c, seed, synth.TID.CONV_W)
    dy = synth.normal((n, L.k, L.h, L.w), seed, synth.TID.DY_TOP)
    relu = not L.pool_after
    xd, wd, dyd = to_dev(x, "bf16"), to_dev(wt, "bf16"), to_dev(dy, "bf16")
    del x, dy
    # The oracle sees the bf16 values the kernels read.
    x, wt, dy = to_host(xd), to_host(wd), to_host(dyd)
    mask = x if L.index > 0 else None
    df = sb.conv_desc(n, L.c, L.h, L.w, L.k, sb.SB_BF16, relu=relu)
    db_ = sb.conv_desc(n, L.c, L.h, L.w, L.k, sb.SB_BF16)
    ws = _ws(max(sb.sb_conv3x3_workspace_bytes(df, 0), sb.sb_conv3x3_workspace_bytes(db_, 1),
                 sb.sb_conv3x3_workspace_bytes(db_, 2)))
    y = torch.empty((n, L.k, L.h, L.w), dtype=torch.bfloat16, device="cuda")
    dx = torch.empty((n, L.c, L.h, L.w), dtype=torch.bfloat16, device="cuda")
    dw = torch.empty((L.k, L.c, 3, 3), device="cuda")
    dbias = torch.empty((L.k,), device="cuda")
    sb.sb_conv3x3_fwd(df, xd, wd, None, y, ws)
    sb.sb_conv3x3_bwd_data(db_, dyd, wd, xd if mask is not None else None, dx, ws)
    sb.sb_conv3x3_bwd_weight(db_, xd, dyd, dw, dbias, ws)
    torch.cuda.synchronize()
    f = sample_idx(y.numel(), SAMPLES, seed)
    assert rel_l2(to_host(y).ravel()[f], O.conv3x3_fwd_at(x, wt, f, relu=relu)) <= TOL["bf16"]
    f = sample_idx(dx.numel(), SAMPLES, seed + 1)
    ref = O.conv3x3_bwd_data_at(dy, wt, f, mask_src=mask)
    assert rel_l2(to_host(dx).ravel()[f], ref) <= TOL["bf16"]
    # Weight gradients are fp32 sums of exact bf16 products: fp32 bound.
    f = sample_idx(dw.numel(), 300, seed + 2)
    assert rel_l2(to_host(dw).ravel()[f], O.conv3x3_bwd_weight_at(x, dy, f)) <= TOL["f32"]
    assert rel_l2(to_host(dbias), dy.astype(np.float64).sum(axis=(0, 2, 3))) <= TOL["f32"]


def _vgg_inputs(n, hw, seed, layers):
    x = synth.normal((n, 3, hw, hw), seed, synth.TID.IMAGES)
    ws = [synth.he_normal_conv3x3(L.k, L.c, seed, synth.TID.CONV_W + L.index) for L in layers]
    bs = [synth.normal((L.k,), seed, synth.TID.CONV_B + L.index, std=0.05) for L in layers]
    return x, ws, bs


def _near_ties(z, ref_idx, got_idx, eps):
    """Windows whose codes differ must be near-ties in the oracle's values:
    the two candidates (or the max and zero, for the ReLU flag) within eps."""
    bad = np.nonzero(ref_idx.ravel() != got_idx.ravel())[0]
    if bad.size == 0:
        return 0
    n, c, h, w = z.shape
    zw = z.reshape(n, c, h // 2, 2, w // 2, 2).transpose(0, 1, 2, 4, 3, 5).reshape(-1, 4)
    for f in bad:
        a, b = ref_idx.ravel()[f], got_idx.ravel()[f]
        va, vb = zw[f, a & 3], zw[f, b & 3]
        gap = abs(va - vb) if (a & 3) != (b & 3) else 0.0
        flag_gap = abs(va) if (a & 0x80) != (b & 0x80) else 0.0
        assert max(gap, flag_gap) <= eps, "code mismatch at window %d is not a near-tie" % f
    return bad.size


def test_vgg16_cifar_stack_end_to_end():
    n, hw = 2, 32
    print_case("vgg16_stack", n=n, hw=hw)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 5, layers)
    dy_top = synth.normal((n, 512, 1, 1), 5, synth.TID.DY_TOP)
    st = ConvStack(configs.VGG16, n, 3, hw, "f32")
    st.load_inputs(x, wts, bs, dy_top)
    st.step()
    torch.cuda.synchronize()
    pools = [L.pool_after for L in layers]
    f, b = OS.vgg_step(x, wts, bs, pools, dy_top)
    flips = 0
    for L in layers:
        i = L.index
        if L.pool_after:
            z = f["Z"][i]
            assert rel_l2(to_host(st.Z[i]), z) <= TOL["f32"], "Z%d" % i
            eps = 1e-5 * np.sqrt(np.mean(z * z))
            flips += _near_ties(z, f["idx"][i], st.idx[i].cpu().numpy(), eps)
        assert rel_l2(to_host(st.A[i + 1]), f["A"][i + 1]) <= TOL["f32"], "A%d" % (i + 1)
    if flips == 0:
        # Identical ReLU / pool decisions: every gradient meets the bound.
        for L in layers:
            i = L.index
            assert rel_l2(to_host(st.grad_at_conv_output(i)), b["dZ"][i]) <= TOL["f32"], "dZ%d" % i
            assert rel_l2(to_host(st.dW[i]), b["dW"][i]) <= TOL["f32"], "dW%d" % i
            assert rel_l2(to_host(st.db[i]), b["db"][i]) <= TOL["f32"], "db%d" % i
        assert rel_l2(to_host(st.gA[0]), b["dX"]) <= TOL["f32"]
    else:
        pytest.fail("%d certified near-tie pool decisions differ; choose another seed" % flips)


def test_vgg16_stack_bf16_end_to_end():
    """The bf16 stack against the oracle that rounds to bf16 wherever the GPU
    path stores a tensor (activations, pool outputs, activation gradients).

    Forward: every tensor within the bf16 bound; pool codes may differ only at
    certified near-ties.  Such ties are common in bf16: the two sides round
    sums that differ in their last fp32 bits, so a few windows in a thousand
    hold two maxima that are equal on one side only.  Each such window sends
    its gradient to another pixel, which moves the gradients of every layer
    below by ~0.1-0.2 in relative L2 (measured), so the backward is held to the
    bf16 bound only above the deepest pool with a differing code, and below it
    to a gross-error bound that a wrong sign, index or transposition (relative
    error >= 1) fails.  Per-pass bf16 parity with identical inputs is tested
    layer by layer at full size."""
    n, hw = 2, 32
    print_case("vgg16_stack_bf16", n=n, hw=hw)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 15, layers)
    dy_top = synth.normal((n, 512, 1, 1), 15, synth.TID.DY_TOP)
    # The stack's inputs as the GPU holds them (bf16 values).
    x = O.round_bf16(x)
    wts = [O.round_bf16(w) for w in wts]
    dy_top = O.round_bf16(dy_top)
    st = ConvStack(configs.VGG16, n, 3, hw, "bf16")
    st.load_inputs(x, wts, bs, dy_top)
    st.step()
    torch.cuda.synchronize()
    pools = [L.pool_after for L in layers]
    f, b = OS.vgg_step(x, wts, bs, pools, dy_top, bf16=True)
    tol = TOL["bf16"]
    deepest_flip = -1
    for L in layers:
        i = L.index
        if L.pool_after:
            z = f["Z"][i]
            assert rel_l2(to_host(st.Z[i]), z) <= tol, "Z%d" % i
            # Differing codes must be near-ties: within two bf16 steps.
            eps = 2.0 ** -6 * np.max(np.abs(z))
            if _near_ties(z, f["idx"][i], st.idx[i].cpu().numpy(), eps):
                deepest_flip = i
        assert rel_l2(to_host(st.A[i + 1]), f["A"][i + 1]) <= tol, "A%d" % (i + 1)
    for L in layers:
        i = L.index
        bound = tol if i > deepest_flip else 0.5
        assert rel_l2(to_host(st.grad_at_conv_output(i)), b["dZ"][i]) <= bound, "dZ%d" % i
        assert rel_l2(to_host(st.dW[i]), b["dW"][i]) <= bound, "dW%d" % i
        assert rel_l2(to_host(st.db[i]), b["db"][i]) <= bound, "db%d" % i
    bound = tol if deepest_flip < 0 else 0.5
    assert rel_l2(to_host(st.gA[0]), b["dX"]) <= bound


def test_vgg16_imagenet_bf16_stack_full_size_properties():
    """The whole ImageNet-shaped bf16 stack (batch 32, 224x224) through one
    step: every pool output and code is consistent with the stored
    pre-activation (y = max(0, window max), first maximum, ReLU flag), the
    un-pooled gradient routes exactly, and every gradient is finite."""
    n, hw = 32, 224
    print_case("vgg16_imagenet_bf16_stack", n=n, hw=hw)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 21, layers)
    dy_top = synth.normal((n, 512, 7, 7), 21, synth.TID.DY_TOP)
    st = ConvStack(configs.VGG16, n, 3, hw, "bf16")
    st.load_inputs(x, wts, bs, dy_top)
    st.step()
    torch.cuda.synchronize()
    for L in layers:
        i = L.index
        assert torch.isfinite(st.dW[i]).all() and torch.isfinite(st.db[i]).all(), "dW%d" % i
        if not L.pool_after:
            continue
        z = st.Z[i].float()
        nn_, c, h, w = z.shape
        win = z.reshape(nn_, c, h // 2, 2, w // 2, 2).permute(0, 1, 2, 4, 3, 5).reshape(
            nn_, c, h // 2, w // 2, 4)
        mx = win.max(dim=-1).values
        is_max = win == mx.unsqueeze(-1)
        first = torch.argmax(is_max.to(torch.float32), dim=-1)
        code = first.to(torch.uint8) | ((mx <= 0).to(torch.uint8) << 7)
        assert torch.equal(st.idx[i], code), "pool code %d" % i
        assert torch.equal(st.A[i + 1].float(), torch.clamp(mx, min=0)), "pool value %d" % i
        del win, is_max, z
        g = st.gA[i + 1].float().unsqueeze(-1)
        sel = (torch.arange(4, device=g.device) == first.unsqueeze(-1)) & (mx > 0).unsqueeze(-1)
        dz = torch.where(sel, g, torch.zeros_like(g)).reshape(nn_, c, h // 2, w // 2, 2, 2)
        dz = dz.permute(0, 1, 2, 4, 3, 5).reshape(nn_, c, h, w)
        assert torch.equal(st.dZ[i].float(), dz), "pool gradient routing %d" % i
        del g, sel, dz


def _hybrid_inputs(n, hw, R, S, schedule, fc_shapes, seed):
    layers = configs.conv_layers(schedule, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, seed, layers)
    m = n * R
    ns = [fo // S for _, fo in fc_shapes]
    fw = [np.ascontiguousarray(synth.xavier_uniform(fi, fo, seed, synth.TID.FC_W + j)[:, :ns[j]])
          for j, (fi, fo) in enumerate(fc_shapes)]
    fb = [synth.normal((ns[j],), seed, synth.TID.FC_B + j, std=0.05) for j in range(len(ns))]
    rows = synth.relu_normal((m - n, fc_shapes[0][0]), seed, synth.TID.X0_REMOTE)
    cols = [synth.relu_normal((m, fc_shapes[j][0] - ns[j - 1]), seed,
                              synth.TID.X1_REMOTE if j == 1 else synth.TID.COLS_REMOTE + j)
            for j in range(1, len(fc_shapes))]
    dy = synth.normal((m, ns[-1]), seed, synth.TID.FC_DY)
    return layers, x, wts, bs, fw, fb, rows, cols, dy


def _check_hybrid(hs, r, layers):
    tol = TOL["f32"]
    for j in range(hs.L):
        assert rel_l2(to_host(hs.X[j]), r["xs"][j]) <= tol, "X%d" % j
        assert rel_l2(to_host(hs.dXp[j]), r["dxp"][j]) <= tol, "dXp%d" % j
        assert rel_l2(to_host(hs.fc[j].dW), r["dw"][j]) <= tol, "dW_fc%d" % j
        assert rel_l2(to_host(hs.fc[j].db), r["db"][j]) <= tol, "db_fc%d" % j
    assert rel_l2(to_host(hs.Y), r["ys"][-1]) <= tol
    for L in layers:
        i = L.index
        if L.pool_after:
            np.testing.assert_array_equal(hs.conv.idx[i].cpu().numpy(), r["fwd"]["idx"][i])
        assert rel_l2(to_host(hs.conv.dW[i]), r["bwd"]["dW"][i]) <= tol, "dW%d" % i
    assert rel_l2(to_host(hs.conv.gA[0]), r["bwd"]["dX"]) <= tol


def test_hybrid_worker_step_end_to_end():
    """VGG-16 conv stack, then FC0 512 -> 1024 (of 4096) and FC1 4096 -> 1024
    (of 4096) shards on the rows gathered from 4 replicas."""
    n, hw, R, S = 2, 32, 4, 4
    print_case("hybrid_step", n=n, replicas=R, shards=S)
    fc_shapes = configs.CONFIGS[4]["fc"]
    layers, x, wts, bs, fw, fb, rows, cols, dy = _hybrid_inputs(
        n, hw, R, S, configs.VGG16, fc_shapes, 6)
    hs = HybridStep(configs.VGG16, n, 3, hw, R, fc_shapes, S)
    hs.load_inputs(x, wts, bs, fw, fb, rows, cols, dy)
    hs.step()
    torch.cuda.synchronize()
    pools = [L.pool_after for L in layers]
    r = OS.hybrid_step(x, wts, bs, pools, fw, fb, rows, cols, dy)
    _check_hybrid(hs, r, layers)


def test_paper_variant_hybrid_step_end_to_end():
    """The paper's own VGG variant (Table 1: seven convs, three pools, FC
    4096 -> 1024 -> 1024 -> 10) as a worker of an MP group of 2: the flattened
    256x4x4 conv output feeds FC0, every FC layer is split in two column
    shards (512, 512 and 5 outputs here)."""
    n, hw, R, S = 3, 32, 2, 2
    print_case("paper_variant_hybrid", n=n, replicas=R, shards=S)
    fc_shapes = configs.PAPER_VARIANT_FC
    layers, x, wts, bs, fw, fb, rows, cols, dy = _hybrid_inputs(
        n, hw, R, S, configs.PAPER_VARIANT_CONV, fc_shapes, 7)
    hs = HybridStep(configs.PAPER_VARIANT_CONV, n, 3, hw, R, fc_shapes, S)
    hs.load_inputs(x, wts, bs, fw, fb, rows, cols, dy)
    hs.step()
    torch.cuda.synchronize()
    pools = [L.pool_after for L in layers]
    r = OS.hybrid_step(x, wts, bs, pools, fw, fb, rows, cols, dy)
    _check_hybrid(hs, r, layers)


def _group_inputs(n, K, fc_shapes, seed, schedule=configs.PAPER_VARIANT_CONV):
    layers = configs.conv_layers(schedule, 3, 32)
    x, wts, bs = _vgg_inputs(n, 32, seed, layers)
    F = fc_shapes[0][0]
    fw = [synth.xavier_uniform(fi, fo, seed, synth.TID.FC_W + j)
          for j, (fi, fo) in enumerate(fc_shapes)]
    fb = [synth.normal((fo,), seed, synth.TID.FC_B + j, std=0.05)
          for j, (_, fo) in enumerate(fc_shapes)]
    remote = synth.relu_normal((K - 1, n, F), seed, synth.TID.X0_REMOTE)
    labels = synth.labels(K * n, fc_shapes[-1][1], seed, synth.TID.LABELS).reshape(K, n)
    return layers, x, wts, bs, fw, fb, remote, labels


@pytest.mark.parametrize("K,n,fc_shapes", [
    (2, 4, configs.PAPER_VARIANT_FC),
    (4, 8, [(4096, 256), (256, 128), (128, 8)])], ids=["paper_variant_K2", "K4"])
def test_group_training_step_end_to_end(K, n, fc_shapes):
    """A training step of an MP group of K (the paper's VGG variant's conv
    stack on worker 0): K modulo iterations, each gathering B rows, running
    every worker's FC shards with shard layers between them, the loss of the
    full logits, the backward and an FC update with the gradient divided by
    K; then the conv backward and update.  Every iteration's gathered batch,
    logits, losses and shard gradients, and the step's updated parameters,
    against the oracle's group step (sec. 3.1, Modulo Layer)."""
    from paper_2112_15317_amd import partition as P
    from paper_2112_15317_amd.stack import GroupTrainStep
    lr = 0.05
    print_case("group_training_step", K=K, n=n, fc=fc_shapes)
    plan = P.fc_plan(P.partition(P.vgg_net(configs.PAPER_VARIANT_CONV, 3, 32, fc_shapes), K))
    layers, x, wts, bs, fw, fb, remote, labels = _group_inputs(n, K, fc_shapes, 9 + K)
    gs = GroupTrainStep(configs.PAPER_VARIANT_CONV, n, 3, 32, plan, lr=lr)
    gs.load_inputs(x, wts, bs, fw, fb, remote, labels)
    gs.conv.forward()
    snaps = []
    for k in range(K):
        gs.iteration(k)
        torch.cuda.synchronize()
        snaps.append({"gathered": to_host(gs.X[0]), "logits": to_host(gs.X[gs.L]),
                      "loss": to_host(gs.loss[k]),
                      "dW": [to_host(w) for w in gs.dW], "db": [to_host(b) for b in gs.db]})
    gs.finish()
    torch.cuda.synchronize()
    pools = [L.pool_after for L in layers]
    r = OS.group_train_step(x, wts, bs, pools, fw, fb, remote, labels, lr)
    tol = TOL["f32"]
    for L in layers:
        if L.pool_after:
            np.testing.assert_array_equal(gs.conv.idx[L.index].cpu().numpy(),
                                          r["fwd"]["idx"][L.index])
    for k, (sn, it) in enumerate(zip(snaps, r["iters"])):
        assert rel_l2(sn["gathered"], it["gathered"]) <= tol, "gathered, iteration %d" % k
        assert rel_l2(sn["logits"], it["logits"]) <= tol, "logits, iteration %d" % k
        assert rel_l2(sn["loss"], it["loss"]) <= tol, "loss, iteration %d" % k
        for j in range(gs.L):
            for w in range(K):
                assert rel_l2(sn["dW"][j][w], it["dw"][j][w]) <= tol, "dW fc%d w%d it%d" % (j, w, k)
                assert rel_l2(sn["db"][j][w], it["db"][j][w]) <= tol, "db fc%d w%d it%d" % (j, w, k)
    for j in range(gs.L):
        # The accumulated update of K steps (new minus initial parameters).
        assert rel_l2(gs.full_weights(j) - fw[j], r["fc_w_new"][j] - fw[j]) <= tol, "W_fc%d" % j
        assert rel_l2(gs.full_bias(j) - fb[j], r["fc_b_new"][j] - fb[j]) <= tol, "b_fc%d" % j
    assert rel_l2(to_host(gs.dlocal), r["dlocal"]) <= tol
    for L in layers:
        i = L.index
        assert rel_l2(to_host(gs.conv.dW[i]), r["bwd"]["dW"][i]) <= tol, "dW%d" % i
        assert rel_l2(to_host(gs.conv.W[i]) - wts[i], r["conv_w_new"][i] - wts[i]) <= tol, "W%d" % i
        assert rel_l2(to_host(gs.conv.b[i]) - bs[i], r["conv_b_new"][i] - bs[i]) <= tol, "b%d" % i


def test_graph_replay_matches_eager():
    """The benchmark replays the step from a captured HIP graph: every replay,
    with eager work and synchronisations in between, must reproduce the eager
    step bit for bit (all kernels have a fixed summation order)."""
    from paper_2112_15317_amd.stack import capture_graph
    n, hw = 4, 32
    print_case("graph_replay", n=n, hw=hw)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 9, layers)
    dy_top = synth.normal((n, 512, 1, 1), 9, synth.TID.DY_TOP)
    st = ConvStack(configs.VGG16, n, 3, hw, "f32")
    st.load_inputs(x, wts, bs, dy_top)
    st.step()
    torch.cuda.synchronize()
    watch = [st.A[-1], st.gA[0]] + st.dW + st.db + list(st.idx.values())
    ref = [t.clone() for t in watch]
    g = capture_graph(st.step, 1)
    for rep in range(3):
        for t in watch:
            t.zero_()                                  # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(watch, ref):
            assert torch.equal(a, b), "replay %d differs from the eager step" % rep


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_overlapped_backward_matches_single_stream(dtype):
    """The weight gradients run on a second stream beside the data-gradient
    chain; eagerly on a non-default torch stream and replayed from a graph,
    the step must equal, bit for bit, the same step on one stream."""
    from paper_2112_15317_amd.stack import capture_graph
    n, hw = 4, 32
    print_case("overlapped_backward", n=n, hw=hw, dtype=dtype)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 10, layers)
    dy_top = synth.normal((n, 512, 1, 1), 10, synth.TID.DY_TOP)
    one = ConvStack(configs.VGG16, n, 3, hw, dtype, overlap=False)
    two = ConvStack(configs.VGG16, n, 3, hw, dtype, overlap=True)
    for st in (one, two):
        st.load_inputs(x, wts, bs, dy_top)
    one.step()
    torch.cuda.synchronize()

    def watch(st):
        return [st.A[-1], st.gA[0]] + st.dW + st.db
    ref = [t.clone() for t in watch(one)]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        two.step(side)
    torch.cuda.synchronize()
    for a, b in zip(watch(two), ref):
        assert torch.equal(a, b), "eager overlapped step differs"
    g = capture_graph(two.step, 1)
    for rep in range(2):
        for t in watch(two):
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(watch(two), ref):
            assert torch.equal(a, b), "replay %d of the overlapped step differs" % rep


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_packed_filter_step_matches_unpacked(dtype):
    """The stack packs every layer's filters once per step on a side stream
    (SB_PACKED_FILTERS); the step must equal, bit for bit, a stack whose
    calls pack their filters themselves."""
    n, hw = 4, 32
    print_case("packed_step", n=n, hw=hw, dtype=dtype)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 10, layers)
    dy_top = synth.normal((n, 512, 1, 1), 10, synth.TID.DY_TOP)
    outs = []
    for packed in (True, False):
        st = ConvStack(configs.VGG16, n, 3, hw, dtype, packed=packed)
        st.load_inputs(x, wts, bs, dy_top)
        st.step()
        torch.cuda.synchronize()
        outs.append([st.A[-1], st.gA[0]] + st.dW + st.db + list(st.idx.values()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)
