"""GPU parity end to end through the stacks at small batches (nonzero
biases, the paper's VGG variant, the group training step), graph replays,
the overlapped backward and packed filters.  The workloads' own shapes are
checked call by call in test_gpu_full_size*.py."""
import numpy as np
import pytest
import torch

import oracle as O
from oracle import stack as OS
from paper_2112_15317_amd import configs, sb, synth
from paper_2112_15317_amd.stack import ConvStack, HybridStep
from tests.helpers import TOL, print_case, rel_l2, to_host

pytestmark = pytest.mark.gpu



def _vgg_inputs(n, hw, seed, layers):
    x = synth.normal((n, 3, hw, hw), seed, synth.TID.IMAGES)
    ws = [synth.he_normal_conv3x3(L.k, L.c, seed, synth.TID.CONV_W + L.index) for L in layers]
    bs = [synth.normal((L.k,), seed, synth.TID.CONV_B + L.index, std=0.05) for L in layers]
    return x, ws, bs


def test_vgg16_cifar_stack_end_to_end():
    """The stack with nonzero biases at a small batch, end to end from the
    seeded inputs (each side taking its own decisions; see
    test_gpu_full_size.independent_check)."""
    from tests.test_gpu_full_size import independent_check
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
    f, b = OS.vgg_step(x, wts, bs, pools, dy_top, store="f32")
    print(independent_check(st, f, b, "f32", 1e-5))


def test_vgg16_imagenet_bf16_stack_full_size_properties():
    """The whole ImageNet-shaped bf16 stack (batch 32, 224x224, the
    benchmark's channel-blocked layout, each pooled layer's forward and
    pooling as separate calls so that its pre-activation is stored) through
    one step: every pool output and code is consistent with the stored
    pre-activation (y = max(0, window max), first maximum, ReLU flag), the
    un-pooled gradient routes exactly, and every gradient is finite."""
    n, hw = 32, 224
    print_case("vgg16_imagenet_bf16_stack", n=n, hw=hw)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 21, layers)
    dy_top = synth.normal((n, 512, 7, 7), 21, synth.TID.DY_TOP)
    st = ConvStack(configs.VGG16, n, 3, hw, "bf16", layout="c8", fuse_pool=False)
    st.load_inputs(x, wts, bs, dy_top)
    st.step()
    torch.cuda.synchronize()
    nchw = st.nchw
    for L in layers:
        i = L.index
        assert torch.isfinite(st.dW[i]).all() and torch.isfinite(st.db[i]).all(), "dW%d" % i
        if not L.pool_after:
            continue
        z = nchw(st.Z[i]).float()
        nn_, c, h, w = z.shape
        win = z.reshape(nn_, c, h // 2, 2, w // 2, 2).permute(0, 1, 2, 4, 3, 5).reshape(
            nn_, c, h // 2, w // 2, 4)
        mx = win.max(dim=-1).values
        is_max = win == mx.unsqueeze(-1)
        first = torch.argmax(is_max.to(torch.float32), dim=-1)
        code = first.to(torch.uint8) | ((mx <= 0).to(torch.uint8) << 7)
        assert torch.equal(nchw(st.idx[i]), code), "pool code %d" % i
        assert torch.equal(nchw(st.A[i + 1]).float(), torch.clamp(mx, min=0)), \
            "pool value %d" % i
        del win, is_max, z
        g = nchw(st.gA[i + 1]).float().unsqueeze(-1)
        sel = (torch.arange(4, device=g.device) == first.unsqueeze(-1)) & (mx > 0).unsqueeze(-1)
        dz = torch.where(sel, g, torch.zeros_like(g)).reshape(nn_, c, h // 2, w // 2, 2, 2)
        dz = dz.permute(0, 1, 2, 4, 3, 5).reshape(nn_, c, h, w)
        assert torch.equal(nchw(st.dZ[i]).float(), dz), "pool gradient routing %d" % i
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


LAYOUTS = [("f32", "nchw"), ("bf16", "nchw"), ("bf16", "c8")]


def _small(layout):
    """(batch, image size) of the small-stack tests: the channel-blocked
    kernels need images at least 8 wide, so 128x128 (deepest layer 8x8)."""
    return (2, 128) if layout == "c8" else (4, 32)


@pytest.mark.parametrize("dtype,layout", LAYOUTS)
def test_overlapped_backward_matches_single_stream(dtype, layout):
    """The weight gradients run on a second stream beside the data-gradient
    chain; eagerly on a non-default torch stream and replayed from a graph,
    the step must equal, bit for bit, the same step on one stream."""
    from paper_2112_15317_amd.stack import capture_graph
    n, hw = _small(layout)
    print_case("overlapped_backward", n=n, hw=hw, dtype=dtype, layout=layout)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 10, layers)
    dy_top = synth.normal((n, 512, hw // 32, hw // 32), 10, synth.TID.DY_TOP)
    one = ConvStack(configs.VGG16, n, 3, hw, dtype, overlap=False, layout=layout)
    two = ConvStack(configs.VGG16, n, 3, hw, dtype, overlap=True, layout=layout)
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


@pytest.mark.parametrize("dtype,layout", LAYOUTS)
def test_packed_filter_step_matches_unpacked(dtype, layout):
    """The stack packs every layer's filters once per step on a side stream
    (SB_PACKED_FILTERS); the step must equal, bit for bit, a stack whose
    calls pack their filters themselves."""
    n, hw = _small(layout)
    print_case("packed_step", n=n, hw=hw, dtype=dtype, layout=layout)
    layers = configs.conv_layers(configs.VGG16, 3, hw)
    x, wts, bs = _vgg_inputs(n, hw, 10, layers)
    dy_top = synth.normal((n, 512, hw // 32, hw // 32), 10, synth.TID.DY_TOP)
    outs = []
    for packed in (True, False):
        st = ConvStack(configs.VGG16, n, 3, hw, dtype, packed=packed, layout=layout)
        st.load_inputs(x, wts, bs, dy_top)
        st.step()
        torch.cuda.synchronize()
        outs.append([st.A[-1], st.gA[0]] + st.dW + st.db + list(st.idx.values()))
    for a, b in zip(*outs):
        assert torch.equal(a, b)
