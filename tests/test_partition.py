"""The host-side layer partitioning (sec. 3.1, Layer Partitioning) on the
paper's VGG variant (Table 1) and on the cases its description covers:
modulo layer before the first split FC layer, shard layers before later ones
and before LOG_SOFTMAX, functional layers following the split width,
unsplittable layers rejecting a partitioned input.  No GPU."""
import pytest

from paper_2112_15317_amd import configs
from paper_2112_15317_amd import partition as P


def vgg_variant():
    """The paper's VGG variant on 3x32x32 images as a sequential CNN."""
    return P.vgg_net(configs.PAPER_VARIANT_CONV, 3, 32, configs.PAPER_VARIANT_FC)


def kinds(layers):
    return [l.kind for l in layers]


def test_vgg_variant_in_mp_groups_of_two():
    out = P.partition(vgg_variant(), 2)
    tail = out[kinds(out).index(P.RESHAPE):]
    assert kinds(tail) == [P.RESHAPE, P.MODULO, P.LINEAR, P.RELU, P.SHARD, P.LINEAR, P.RELU,
                           P.SHARD, P.LINEAR, P.SHARD, P.LOG_SOFTMAX]
    assert (tail[1].in_dim, tail[4].in_dim, tail[4].out_dim) == (4096, 512, 1024)
    assert (tail[9].in_dim, tail[9].out_dim) == (5, 10)
    # Convolutional and pooling layers are never split.
    assert all(l.kind != P.LINEAR or l.shards == 2 for l in out)
    assert sum(l.kind in (P.CONV, P.POOLING) for l in out) == 10
    # The shard shapes the training-step workload runs.
    assert P.fc_shards(out) == [(i, o // 2, o) for i, o in configs.PAPER_VARIANT_FC]


def test_vgg_variant_fc_weights_halve_per_worker():
    # Table 1: the three FC layers hold 5,253,120 of the 6,987,456 weights.
    out = P.partition(vgg_variant(), 2)
    fc_weights = sum(l.in_dim * l.out_dim for l in out if l.kind == P.LINEAR)
    assert fc_weights == 5253120 // 2
    full = sum(l.in_dim * (l.full_out or l.out_dim) for l in out if l.kind == P.LINEAR)
    assert full == 5253120


def test_no_model_parallelism_leaves_the_model_whole():
    net = vgg_variant()
    out = P.partition(net, 1)
    assert P.MODULO not in kinds(out) and P.SHARD not in kinds(out)
    assert all(l.shards == 1 for l in out if l.kind == P.LINEAR)
    assert len(out) == len(net.children)
    # A threshold above every layer's CCR does the same with K = 4.
    out4 = P.partition(net, 2, threshold=1e9)
    assert kinds(out4) == kinds(out)


def test_ccr_threshold_keeps_a_cheap_last_layer_whole():
    # FC2 (1024 -> 10) has the lowest CCR: above it but below the others,
    # FC2 runs unsplit on the full input a shard layer assembles, and the
    # output reaching LOG_SOFTMAX is whole (no shard layer before it).
    ccrs = [P.ccr(P.linear(i, o)) for i, o in configs.PAPER_VARIANT_FC]
    assert ccrs[2] < min(ccrs[:2])
    out = P.partition(vgg_variant(), 2, threshold=(ccrs[2] + min(ccrs[:2])) / 2)
    tail = out[kinds(out).index(P.MODULO):]
    assert kinds(tail) == [P.MODULO, P.LINEAR, P.RELU, P.SHARD, P.LINEAR, P.RELU, P.SHARD,
                           P.LINEAR, P.LOG_SOFTMAX]
    assert tail[-2].shards == 1 and tail[-2].out_dim == 10


def test_first_fc_kept_whole_moves_the_modulo_layer_down():
    # Only the second FC layer is worth splitting: its input is whole, so
    # it gets the modulo layer.
    net = P.seq(P.linear(2, 64), P.Layer(P.RELU), P.linear(64, 4096), P.Layer(P.LOG_SOFTMAX))
    assert P.ccr(P.linear(2, 64)) < 10 < P.ccr(P.linear(64, 4096))
    out = P.partition(net, 4, threshold=10)
    assert kinds(out) == [P.LINEAR, P.RELU, P.MODULO, P.LINEAR, P.SHARD, P.LOG_SOFTMAX]
    assert out[3].out_dim == 1024 and (out[4].in_dim, out[4].out_dim) == (1024, 4096)


def test_dropout_follows_the_split_width():
    net = P.seq(P.linear(64, 32), P.Layer(P.DROPOUT), P.linear(32, 16), P.Layer(P.LOG_SOFTMAX))
    out = P.partition(net, 4)
    assert kinds(out) == [P.MODULO, P.LINEAR, P.DROPOUT, P.SHARD, P.LINEAR, P.SHARD,
                          P.LOG_SOFTMAX]
    assert out[3].in_dim == 8 and out[5].in_dim == 4


def test_unsplittable_layer_after_a_split_layer_is_rejected():
    net = P.seq(P.linear(64, 32), P.Layer(P.RESHAPE, 32, 32))
    with pytest.raises(ValueError):
        P.partition(net, 2)
    with pytest.raises(ValueError):
        P.partition(P.seq(P.linear(64, 30)), 4)      # 30 outputs do not split in 4


def test_fc_plan_of_the_vgg_variant():
    """The call sequence of the training step's model-parallel part."""
    plan = P.fc_plan(P.partition(vgg_variant(), 2))
    assert plan == [("modulo", 4096),
                    ("linear", 4096, 512, 1024, True), ("shard", 512, 1024),
                    ("linear", 1024, 512, 1024, True), ("shard", 512, 1024),
                    ("linear", 1024, 5, 10, False), ("shard", 5, 10),
                    ("loss", 10)]
    with pytest.raises(ValueError):
        P.fc_plan(P.partition(vgg_variant(), 1))       # no model parallelism


def test_nested_containers_flatten_in_order():
    inner = P.seq(P.linear(64, 32), P.Layer(P.RELU))
    net = P.seq(inner, P.seq(P.linear(32, 16)), P.Layer(P.LOG_SOFTMAX))
    assert [l.kind for l in P.flatten(net)] == [P.LINEAR, P.RELU, P.LINEAR, P.LOG_SOFTMAX]
    assert kinds(P.partition(net, 4)) == [P.MODULO, P.LINEAR, P.RELU, P.SHARD, P.LINEAR,
                                          P.SHARD, P.LOG_SOFTMAX]
