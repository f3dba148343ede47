"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/sb.h declares, and rejects bad arguments before
enqueueing anything.  Only argument-validation paths are exercised here: each
call below fails its checks, so no kernel is launched."""
import ctypes
import os
import re

import pytest

from paper_2112_15317_amd import sb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sb.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sb_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported_and_bound():
    lib = sb.load()
    names = _declared()
    assert len(names) >= 11
    for name in names:
        assert hasattr(lib, name), name
        assert name in sb.SIGNATURES, name


def test_status_strings_and_version():
    assert sb.status_name(sb.SB_OK) == "SB_OK"
    assert sb.status_name(sb.SB_ERR_WORKSPACE) == "SB_ERR_WORKSPACE"
    assert sb.status_name(99) == "SB_ERR_UNKNOWN"
    assert sb.sb_version() >= 100


def _raw(name, *args):
    return getattr(sb.load(), name)(*args)


P = 0x10000000          # fake device addresses: never dereferenced (calls fail validation)


def test_conv_argument_validation():
    d = sb.conv_desc(2, 3, 8, 8, 4)
    bad = [sb.conv_desc(0, 3, 8, 8, 4), sb.conv_desc(2, -1, 8, 8, 4), sb.conv_desc(2, 3, 8, 8, 0),
           sb.sb_conv3x3_desc(2, 3, 8, 8, 4, 7, 0), sb.sb_conv3x3_desc(2, 3, 8, 8, 4, 0, 8)]
    for b in bad:
        assert _raw("sb_conv3x3_fwd", ctypes.byref(b), P, P + 4096, None, P + 8192, None, 0, None) == sb.SB_ERR_INVALID_ARG
        assert sb.sb_conv3x3_workspace_bytes(b, 0) == 2 ** 64 - 1
    # Null input / output pointers.
    assert _raw("sb_conv3x3_fwd", ctypes.byref(d), None, P, None, P + 8192, None, 0, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_conv3x3_bwd_data", ctypes.byref(d), P, P + 8192, None, None, None, 0, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_conv3x3_bwd_weight", ctypes.byref(d), P, P + 8192, None, None, None, 0, None) == sb.SB_ERR_INVALID_ARG
    # Output overlapping an input.
    assert _raw("sb_conv3x3_fwd", ctypes.byref(d), P, P + 1 << 20, None, P + 64, None, 0, None) == sb.SB_ERR_INVALID_ARG
    # ReLU flag is forward-only.
    dr = sb.conv_desc(2, 3, 8, 8, 4, relu=True)
    assert _raw("sb_conv3x3_bwd_data", ctypes.byref(dr), P, P + (1 << 20), None, P + (2 << 20), None, 0, None) == sb.SB_ERR_INVALID_ARG
    assert sb.sb_conv3x3_workspace_bytes(d, 4) == 2 ** 64 - 1
    assert sb.sb_conv3x3_workspace_bytes(d, -1) == 2 ** 64 - 1


def test_conv_workspace_is_checked_before_launch():
    d = sb.conv_desc(128, 512, 2, 2, 512)      # small output grid -> split reduction
    need = sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_FWD)
    assert need > 0
    x, w, y = P, P + (16 << 20), P + (64 << 20)
    assert _raw("sb_conv3x3_fwd", ctypes.byref(d), x, w, None, y, None, 0, None) == sb.SB_ERR_WORKSPACE
    assert _raw("sb_conv3x3_fwd", ctypes.byref(d), x, w, None, y, P + (128 << 20), need - 1, None) == sb.SB_ERR_WORKSPACE
    need = sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_WEIGHT)
    assert need > 0
    assert _raw("sb_conv3x3_bwd_weight", ctypes.byref(d), x, y, P + (96 << 20), None, None, 0, None) == sb.SB_ERR_WORKSPACE


def test_pool_argument_validation():
    for shape in [(0, 1, 2, 2), (1, 1, 3, 2), (1, 1, 2, 5), (1, -2, 2, 2)]:
        assert _raw("sb_relu_maxpool_fwd", *shape, 0, 0, P, P + 4096, P + 8192, None) == sb.SB_ERR_INVALID_ARG
        assert _raw("sb_relu_maxpool_bwd", *shape, 0, 0, P, P + 4096, P + 8192, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_relu_maxpool_fwd", 1, 1, 2, 2, 5, 0, P, P + 4096, P + 8192, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_relu_maxpool_fwd", 1, 1, 2, 2, 0, 0, None, P + 4096, P + 8192, None) == sb.SB_ERR_INVALID_ARG
    # Output aliasing the input.
    assert _raw("sb_relu_maxpool_fwd", 1, 4, 4, 4, 0, 0, P, P + 8, P + 8192, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_relu_maxpool_bwd", 1, 4, 4, 4, 0, 0, P, P + 8192, P + 16, None) == sb.SB_ERR_INVALID_ARG
    # Bad layout; channel-blocked needs whole 8-channel blocks.
    assert _raw("sb_relu_maxpool_fwd", 1, 8, 4, 4, 1, 2, P, P + 8192, P + 16384, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_relu_maxpool_fwd", 1, 12, 4, 4, 1, 1, P, P + 8192, P + 16384, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_relu_maxpool_bwd", 1, 12, 4, 4, 1, 1, P, P + 8192, P + 16384, None) == sb.SB_ERR_INVALID_ARG


def test_fc_argument_validation():
    ok = sb.fc_desc(16, 32, 8)
    assert sb.sb_fc_workspace_bytes(ok, sb.SB_FC_FWD) != 2 ** 64 - 1
    for bad in [sb.fc_desc(0, 32, 8), sb.fc_desc(16, 32, 8, ldx=16), sb.fc_desc(16, 32, 8, ldy=4),
                sb.sb_fc_desc(16, 32, 8, 0, 32, 8, 4), sb.sb_fc_desc(16, 32, 8, 7, 32, 8, 0)]:
        assert sb.sb_fc_workspace_bytes(bad, 0) == 2 ** 64 - 1
        assert _raw("sb_fc_shard_fwd", ctypes.byref(bad), P, P + 8192, None, P + 65536, None, 0, None) == sb.SB_ERR_INVALID_ARG
    # bf16 is validated like fp32 (element size 2): an output overlapping x.
    bf = sb.fc_desc(16, 32, 8, dtype=sb.SB_BF16)
    assert sb.sb_fc_workspace_bytes(bf, sb.SB_FC_FWD) != 2 ** 64 - 1
    assert _raw("sb_fc_shard_fwd", ctypes.byref(bf), P, P + 8192, None, P + 1000, None, 0, None) == sb.SB_ERR_INVALID_ARG
    # Missing dW, bad accumulate flag, overlapping outputs.
    assert _raw("sb_fc_shard_bwd", ctypes.byref(ok), P, P + 8192, P + 16384, None, None, None, None, 0, None, 0, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_fc_shard_bwd", ctypes.byref(ok), P, P + 8192, P + 16384, None, None, P + 65536, None, 2, None, 0, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_fc_shard_bwd", ctypes.byref(ok), P, P + 8192, P + 16384, None, P + 65536, P + 65536, None, 0, None, 0, None) == sb.SB_ERR_INVALID_ARG


def test_binding_refuses_host_tensors():
    import torch
    d = sb.conv_desc(1, 1, 2, 2, 1)
    with pytest.raises(ValueError):
        sb.sb_conv3x3_fwd(d, torch.zeros(1, 1, 2, 2), torch.zeros(1, 1, 3, 3), None,
                          torch.zeros(1, 1, 2, 2), None, stream=0)


def test_packed_filter_sizes_and_validation():
    d = sb.conv_desc(128, 512, 2, 2, 512)
    for pass_ in (sb.SB_PASS_FWD, sb.SB_PASS_BWD_DATA):
        pb = sb.sb_conv3x3_packed_bytes(d, pass_)
        assert pb >= 512 * 512 * 9 * 4        # every filter element, padded to whole slices
        # The workspace of a call with packed filters leaves out the packing room.
        dp = sb.conv_desc(128, 512, 2, 2, 512, packed=True)
        full = sb.sb_conv3x3_workspace_bytes(d, pass_)
        part = sb.sb_conv3x3_workspace_bytes(dp, pass_)
        assert part < full and full - part >= pb
    assert sb.sb_conv3x3_packed_bytes(d, sb.SB_PASS_BWD_WEIGHT) == 0
    assert sb.sb_conv3x3_packed_bytes(sb.conv_desc(0, 3, 8, 8, 4), 0) == 0
    # The flag is for the forward and data-gradient passes only, and ReLU
    # stays forward-only with it.
    dp = sb.conv_desc(2, 3, 8, 8, 4, packed=True)
    assert sb.sb_conv3x3_workspace_bytes(dp, sb.SB_PASS_BWD_WEIGHT) == 2 ** 64 - 1
    dpr = sb.conv_desc(2, 3, 8, 8, 4, relu=True, packed=True)
    assert sb.sb_conv3x3_workspace_bytes(dpr, sb.SB_PASS_FWD) != 2 ** 64 - 1
    assert sb.sb_conv3x3_workspace_bytes(dpr, sb.SB_PASS_BWD_DATA) == 2 ** 64 - 1
    small = sb.conv_desc(2, 3, 8, 8, 4)
    need = sb.sb_conv3x3_packed_bytes(small, sb.SB_PASS_FWD)
    pk = _raw
    # Bad pass, null pointers, a short buffer, a buffer overlapping the filters.
    assert pk("sb_conv3x3_pack_filters", ctypes.byref(small), 2, P, P + (1 << 20), need, None) == sb.SB_ERR_INVALID_ARG
    assert pk("sb_conv3x3_pack_filters", ctypes.byref(small), 0, None, P + (1 << 20), need, None) == sb.SB_ERR_INVALID_ARG
    assert pk("sb_conv3x3_pack_filters", ctypes.byref(small), 0, P, None, need, None) == sb.SB_ERR_INVALID_ARG
    assert pk("sb_conv3x3_pack_filters", ctypes.byref(small), 0, P, P + (1 << 20), need - 1, None) == sb.SB_ERR_INVALID_ARG
    assert pk("sb_conv3x3_pack_filters", ctypes.byref(small), 0, P, P + 8, need, None) == sb.SB_ERR_INVALID_ARG


def test_packed_filters_many_validation():
    d = sb.conv_desc(2, 3, 8, 8, 4)
    need = sb.sb_conv3x3_packed_bytes(d, sb.SB_PASS_FWD)

    def call(descs, passes, ws, outs, sizes):
        n = len(descs)
        return _raw("sb_conv3x3_pack_filters_many", n, (sb.sb_conv3x3_desc * n)(*descs),
                    (ctypes.c_int * n)(*passes), (ctypes.c_void_p * n)(*ws),
                    (ctypes.c_void_p * n)(*outs), (ctypes.c_size_t * n)(*sizes), None)
    w0, o0, o1 = P, P + (1 << 20), P + (2 << 20)
    assert _raw("sb_conv3x3_pack_filters_many", 0, None, None, None, None, None, None) == sb.SB_ERR_INVALID_ARG
    # More tasks than one launch takes.
    many = 65
    assert call([d] * many, [0] * many, [w0] * many, [o0 + (i << 16) for i in range(many)],
                [need] * many) == sb.SB_ERR_INVALID_ARG
    # Mixed dtypes, a bad pass, a short buffer, overlapping outputs.
    db = sb.conv_desc(2, 3, 8, 8, 4, sb.SB_BF16)
    assert call([d, db], [0, 0], [w0, w0], [o0, o1], [need, need]) == sb.SB_ERR_INVALID_ARG
    assert call([d], [2], [w0], [o0], [need]) == sb.SB_ERR_INVALID_ARG
    assert call([d], [0], [w0], [o0], [need - 1]) == sb.SB_ERR_INVALID_ARG
    assert call([d, d], [0, 1], [w0, w0], [o0, o0 + 4], [need, need]) == sb.SB_ERR_INVALID_ARG


def test_modulo_and_shard_argument_validation():
    E = sb.SB_ERR_INVALID_ARG
    good = sb.modulo_desc(4, 2, 8, 16)         # slots of 8 x 16 = 128 elements
    slot = 128
    bad_descs = [sb.modulo_desc(4, 0, 8, 16), sb.modulo_desc(3, 2, 8, 16),   # mp 0; N % mp
                 sb.modulo_desc(4, 2, 7, 16), sb.modulo_desc(4, 2, 8, 0),    # B % mp; F = 0
                 sb.modulo_desc(2, 4, 8, 16)]                                # mp > N
    for d in bad_descs:
        assert _raw("sb_modulo_fwd", ctypes.byref(d), 0, 0, P, slot, P + 1 << 24, None) == E
        assert _raw("sb_modulo_bwd", ctypes.byref(d), 0, 0, P, slot, P + 1 << 24, slot, None) == E
    g = ctypes.byref(good)
    # iproc and k out of range, null pointers, short strides.
    assert _raw("sb_modulo_fwd", g, 4, 0, P, slot, P + (1 << 24), None) == E
    assert _raw("sb_modulo_fwd", g, -1, 0, P, slot, P + (1 << 24), None) == E
    assert _raw("sb_modulo_fwd", g, 0, 2, P, slot, P + (1 << 24), None) == E
    assert _raw("sb_modulo_fwd", g, 0, 0, None, slot, P + (1 << 24), None) == E
    assert _raw("sb_modulo_fwd", g, 0, 0, P, slot - 1, P + (1 << 24), None) == E
    assert _raw("sb_modulo_bwd", g, 0, 0, P, slot, P + (1 << 24), slot - 1, None) == E
    assert _raw("sb_modulo_bwd", g, 0, 0, P, slot, None, slot, None) == E
    # Output overlapping the group's input slots (group of worker 3: slots 2, 3).
    assert _raw("sb_modulo_fwd", g, 3, 0, P, slot, P + 2 * slot * 4 + 64, None) == E
    assert _raw("sb_modulo_bwd", g, 1, 0, P, slot, P + 4 * slot, slot, None) == E

    sgood = sb.shard_desc(4, 2, 5, 8)          # slots of 5 x 8; full input 5 x 16
    s = ctypes.byref(sgood)
    for d in [sb.shard_desc(4, 3, 5, 8), sb.shard_desc(4, 2, 0, 8), sb.shard_desc(4, 2, 5, 0)]:
        assert _raw("sb_shard_fwd", ctypes.byref(d), 0, P, 40, P + (1 << 24), None) == E
        assert _raw("sb_shard_bwd", ctypes.byref(d), 0, P, 80, P + (1 << 24), 40, None) == E
    assert _raw("sb_shard_fwd", s, 4, P, 40, P + (1 << 24), None) == E
    assert _raw("sb_shard_fwd", s, 0, P, 39, P + (1 << 24), None) == E
    assert _raw("sb_shard_bwd", s, 0, P, 79, P + (1 << 24), 40, None) == E    # dfull slot is 80
    assert _raw("sb_shard_bwd", s, 0, P, 80, P + (1 << 24), 39, None) == E
    assert _raw("sb_shard_fwd", s, 0, P, 40, P + 100, None) == E               # overlap
    assert _raw("sb_shard_bwd", s, 2, P, 80, P + 2 * 80 * 4 + 8, 40, None) == E


def test_loss_and_sgd_argument_validation():
    f = ctypes.c_float
    # Bad sizes, null logits or labels, non-finite scale, too small row stride.
    assert _raw("sb_log_softmax_nll", -1, 10, 10, P, P + 4096, f(1.0), None, None, None, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_log_softmax_nll", 4, 0, 10, P, P + 4096, f(1.0), None, None, None, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_log_softmax_nll", 4, 10, 9, P, P + 4096, f(1.0), None, None, None, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_log_softmax_nll", 4, 10, 10, None, P + 4096, f(1.0), None, None, None, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_log_softmax_nll", 4, 10, 10, P, None, f(1.0), None, None, None, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_log_softmax_nll", 4, 10, 10, P, P + 4096, f(float("nan")), None, None, None, None) == sb.SB_ERR_INVALID_ARG
    # Outputs overlapping the logits, the labels or each other.
    assert _raw("sb_log_softmax_nll", 4, 10, 10, P, P + 4096, f(1.0), P + 8, None, None, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_log_softmax_nll", 4, 10, 10, P, P + 4096, f(1.0), None, P + 4100, None, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_log_softmax_nll", 4, 10, 10, P, P + 4096, f(1.0), P + 8192, None, P + 8200, None) == sb.SB_ERR_INVALID_ARG
    # No rows: nothing to do.
    assert _raw("sb_log_softmax_nll", 0, 10, 10, P, None, f(1.0), None, None, None, None) == sb.SB_OK

    def sgd(ws, gs, ns, scales, lr=0.1, count=None):
        n = len(ws)
        return _raw("sb_sgd_update", n if count is None else count,
                    (ctypes.c_void_p * max(n, 1))(*ws), (ctypes.c_void_p * max(n, 1))(*gs),
                    (ctypes.c_size_t * max(n, 1))(*ns), (ctypes.c_float * max(n, 1))(*scales),
                    f(lr), None)
    assert sgd([P], [P + 4096], [16], [1.0], count=0) == sb.SB_ERR_INVALID_ARG
    assert sgd([P], [P + 4096], [16], [1.0], count=sb.SB_SGD_MAX_TENSORS + 1) == sb.SB_ERR_INVALID_ARG
    assert sgd([None], [P + 4096], [16], [1.0]) == sb.SB_ERR_INVALID_ARG
    assert sgd([P], [None], [16], [1.0]) == sb.SB_ERR_INVALID_ARG
    assert sgd([P], [P + 4096], [16], [float("inf")]) == sb.SB_ERR_INVALID_ARG
    assert sgd([P], [P + 4096], [16], [1.0], lr=float("nan")) == sb.SB_ERR_INVALID_ARG
    # A gradient overlapping a parameter (its own or another's); parameters overlapping.
    assert sgd([P], [P + 32], [16], [1.0]) == sb.SB_ERR_INVALID_ARG
    assert sgd([P, P + 4096], [P + 8192, P + 4100], [16, 16], [1.0, 1.0]) == sb.SB_ERR_INVALID_ARG
    assert sgd([P, P + 32], [P + 8192, P + 12288], [16, 16], [1.0, 1.0]) == sb.SB_ERR_INVALID_ARG
    # Only empty tensors: nothing to do.
    assert sgd([None], [None], [0], [1.0]) == sb.SB_OK


def test_model_average_argument_validation():
    avg = lambda *a: _raw("sb_model_average", *a)
    assert avg(0, 1, 16, P, 16, None) == sb.SB_ERR_INVALID_ARG
    assert avg(4, 0, 16, P, 16, None) == sb.SB_ERR_INVALID_ARG
    assert avg(6, 4, 16, P, 16, None) == sb.SB_ERR_INVALID_ARG      # not whole groups
    assert avg(4, 1, 16, None, 16, None) == sb.SB_ERR_INVALID_ARG
    assert avg(4, 1, 16, P, 8, None) == sb.SB_ERR_INVALID_ARG       # slots would overlap
    assert avg(4, 1, 0, None, 0, None) == sb.SB_OK                  # nothing to average
    assert avg(4, 4, 16, P, 16, None) == sb.SB_OK                   # one worker per set


def test_model_average_replicas_argument_validation():
    ptrs = lambda *a: (ctypes.c_void_p * max(len(a), 1))(*a)
    avg = lambda k, n, p: _raw("sb_model_average_replicas", k, n, p, None)
    a, b = P, P + (1 << 20)
    assert avg(0, 16, ptrs(a)) == sb.SB_ERR_INVALID_ARG
    assert avg(sb.SB_MAX_REPLICAS + 1, 16, ptrs(*[P + (i << 20) for i in range(65)])) == \
        sb.SB_ERR_INVALID_ARG
    assert avg(2, 16, None) == sb.SB_ERR_INVALID_ARG
    assert avg(2, 16, ptrs(a, None)) == sb.SB_ERR_INVALID_ARG
    assert avg(2, 16, ptrs(a, a + 32)) == sb.SB_ERR_INVALID_ARG      # ranges overlap
    assert avg(3, 16, ptrs(a, b, b)) == sb.SB_ERR_INVALID_ARG
    assert avg(2, 0, ptrs(a, b)) == sb.SB_OK                          # nothing to average
    assert avg(1, 16, ptrs(a)) == sb.SB_OK                            # one replica


def test_fused_forward_pool_validation():
    """sb_conv3x3_fwd_pool: channel-blocked bf16 or NCHW fp32 with even
    sizes and an unsplit plan; the pass-3 workspace query says which
    descriptors it takes, with the forward's workspace; nothing is launched
    on an error."""
    c8 = lambda n, c, h, w, k, **kw: sb.conv_desc(n, c, h, w, k, sb.SB_BF16,
                                                  layout=sb.SB_NCHW8C, **kw)
    ok = c8(32, 64, 224, 224, 64)          # 6272 tiles: one split
    need = sb.sb_conv3x3_workspace_bytes(ok, sb.SB_PASS_FWD_POOL)
    assert need == sb.sb_conv3x3_workspace_bytes(ok, sb.SB_PASS_FWD)
    assert "pool" in sb.sb_conv3x3_plan_string(ok, sb.SB_PASS_FWD_POOL)
    fwd_pool = lambda d, x, w, y, idx, ws=None, nb=0: _raw(
        "sb_conv3x3_fwd_pool", ctypes.byref(d), x, w, None, y, idx, ws, nb, None)
    x, w, y, idx = P, P + (256 << 20), P + (512 << 20), P + (768 << 20)
    ws = P + (1024 << 20) if need else None
    for bad, status in ((sb.conv_desc(32, 64, 224, 224, 64, sb.SB_BF16), sb.SB_ERR_UNSUPPORTED),
                        (sb.conv_desc(32, 64, 224, 224, 64, sb.SB_F32, layout=sb.SB_NCHW8C),
                         sb.SB_ERR_UNSUPPORTED),
                        (c8(32, 64, 224, 223, 64), sb.SB_ERR_INVALID_ARG),
                        (c8(32, 64, 224, 224, 64, relu=True), sb.SB_ERR_INVALID_ARG),
                        (c8(2, 64, 32, 32, 64), sb.SB_ERR_UNSUPPORTED)):     # split plan
        assert sb.sb_conv3x3_workspace_bytes(bad, sb.SB_PASS_FWD_POOL) == sb.SIZE_MAX
        assert fwd_pool(bad, x, w, y, idx, ws, need) == status
    assert fwd_pool(ok, x, w, y, None, ws, need) == sb.SB_ERR_INVALID_ARG
    assert fwd_pool(ok, x, w, y, y + 64, ws, need) == sb.SB_ERR_INVALID_ARG   # idx over y
    assert fwd_pool(ok, x, w, x + 64, idx, ws, need) == sb.SB_ERR_INVALID_ARG  # y over x
    # NCHW fp32 pools in the call too: an unsplit plan in the kernel's
    # epilogue, a split one (small batches, the 4x4 and 2x2 images) in its
    # split reduction; not bf16 NCHW, not the few-output-channel kernel.
    f32 = sb.conv_desc(128, 64, 32, 32, 64, sb.SB_F32)
    assert sb.sb_conv3x3_workspace_bytes(f32, sb.SB_PASS_FWD_POOL) == \
        sb.sb_conv3x3_workspace_bytes(f32, sb.SB_PASS_FWD)
    assert sb.sb_conv3x3_plan_string(f32, sb.SB_PASS_FWD_POOL).split(" grid")[0].endswith(
        ", true>")
    for good in (sb.conv_desc(2, 64, 32, 32, 64, sb.SB_F32),
                 sb.conv_desc(128, 512, 4, 4, 512, sb.SB_F32),
                 sb.conv_desc(128, 512, 2, 2, 512, sb.SB_F32)):
        assert sb.sb_conv3x3_workspace_bytes(good, sb.SB_PASS_FWD_POOL) == \
            sb.sb_conv3x3_workspace_bytes(good, sb.SB_PASS_FWD)
    few = sb.conv_desc(2, 12, 6, 38, 3, sb.SB_F32)          # 3 outputs: vector-ALU kernel
    assert sb.sb_conv3x3_workspace_bytes(few, sb.SB_PASS_FWD_POOL) == sb.SIZE_MAX
    assert fwd_pool(few, x, w, y, idx, ws, need) == sb.SB_ERR_UNSUPPORTED
    # A plan that splits the channel loop cannot pool in the kernel.
    split = c8(1, 512, 14, 14, 512)
    splits = int(sb.sb_conv3x3_plan_string(split, sb.SB_PASS_FWD).rsplit("x", 1)[1])
    assert (sb.sb_conv3x3_workspace_bytes(split, sb.SB_PASS_FWD_POOL) == sb.SIZE_MAX) == \
        (splits > 1)


def test_pack_many_rejects_packing_over_another_tasks_filters():
    d = sb.conv_desc(2, 3, 8, 8, 4)
    need = sb.sb_conv3x3_packed_bytes(d, sb.SB_PASS_FWD)
    n = 2
    w0, w1, o0 = P, P + (1 << 20), P + (2 << 20)
    args = lambda outs: (n, (sb.sb_conv3x3_desc * n)(d, d), (ctypes.c_int * n)(0, 1),
                         (ctypes.c_void_p * n)(w0, w1), (ctypes.c_void_p * n)(*outs),
                         (ctypes.c_size_t * n)(need, need), None)
    # Task 0 packs into task 1's source filters (and the reverse): one launch
    # would read and write the same bytes.
    assert _raw("sb_conv3x3_pack_filters_many", *args([w1, o0])) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_conv3x3_pack_filters_many", *args([o0, w0 + 16])) == sb.SB_ERR_INVALID_ARG


def test_fc_workspace_must_not_overlap_operands():
    d = sb.fc_desc(512, 4096, 1024)            # few output tiles: the forward is split
    d2 = sb.fc_desc(4096, 64, 64)              # a 64 x 64 weight gradient over 4096 rows: split
    need_f = sb.sb_fc_workspace_bytes(d, sb.SB_FC_FWD)
    need_b = sb.sb_fc_workspace_bytes(d2, sb.SB_FC_BWD)
    assert need_f > 0 and need_b > 0
    x, w, y = P, P + (16 << 20), P + (96 << 20)
    ws = P + (128 << 20)
    fwd = lambda ws_: _raw("sb_fc_shard_fwd", ctypes.byref(d), x, w, None, y, ws_, need_f, None)
    assert fwd(x + 64) == sb.SB_ERR_INVALID_ARG          # over x
    assert fwd(w + 4096) == sb.SB_ERR_INVALID_ARG        # over w
    assert fwd(y - 1024) == sb.SB_ERR_INVALID_ARG        # over y
    dy, dx, dw = P + (200 << 20), P + (240 << 20), P + (300 << 20)
    ws = P + (400 << 20)
    bwd = lambda ws_: _raw("sb_fc_shard_bwd", ctypes.byref(d2), x, w, dy, None, dx, dw, None, 0,
                           ws_, need_b, None)
    for bad in (x, w, dy, dx, dw):
        assert bwd(bad + 256) == sb.SB_ERR_INVALID_ARG


def _noalloc(d, x, dy, dw, db):
    return _raw("sb_conv3x3_bwd_weight_noalloc", ctypes.byref(d), x, dy, dw, db, None)


def test_noalloc_weight_gradient_validation():
    """The no-allocation weight gradient validates like sb_conv3x3_bwd_weight
    and refuses, before touching any device, a call whose split partials
    would not fit its fixed scratch array."""
    d = sb.conv_desc(2, 3, 8, 8, 4)
    assert _noalloc(d, None, P, P + (1 << 20), None) == sb.SB_ERR_INVALID_ARG
    assert _noalloc(d, P, P + 8192, None, None) == sb.SB_ERR_INVALID_ARG
    assert _noalloc(sb.conv_desc(2, 3, 8, 8, 4, relu=True), P, P + 8192, P + (1 << 20),
                    None) == sb.SB_ERR_INVALID_ARG
    assert _noalloc(d, P, P + 8192, P + 64, None) == sb.SB_ERR_INVALID_ARG    # dw over x
    # A shape whose split partials exceed the scratch array: 511 blocks of
    # 64 k x 32 c in bf16 give two splits of 448 x 2336 x 9 fp32 each.
    big = sb.conv_desc(8, 2336, 32, 32, 448, sb.SB_BF16)
    need = sb.sb_conv3x3_workspace_bytes(big, sb.SB_PASS_BWD_WEIGHT)
    assert need > sb.SB_NOALLOC_SCRATCH_BYTES
    assert _noalloc(big, P, P + (1 << 30), P + (2 << 30), None) == sb.SB_ERR_WORKSPACE
    # Every VGG-16 layer of both workloads fits.
    from paper_2112_15317_amd import configs
    for hw, n, dt in ((32, 128, sb.SB_F32), (224, 32, sb.SB_BF16)):
        for L in configs.conv_layers(configs.VGG16, 3, hw):
            q = sb.conv_desc(n, L.c, L.h, L.w, L.k, dt)
            assert sb.sb_conv3x3_workspace_bytes(q, 2) <= sb.SB_NOALLOC_SCRATCH_BYTES


def test_channel_blocked_layout_validation():
    """SB_NCHW8C: bf16 only (fp32 is unsupported), whole 8-channel blocks,
    images at least 8 wide; an unknown layout is rejected."""
    ok = sb.conv_desc(2, 16, 16, 16, 32, sb.SB_BF16, layout=sb.SB_NCHW8C)
    for p in range(3):
        assert sb.sb_conv3x3_workspace_bytes(ok, p) != 2 ** 64 - 1
        assert "c8" in sb.sb_conv3x3_plan_string(ok, p)
    bad_layout = sb.conv_desc(2, 16, 16, 16, 32, sb.SB_BF16, layout=3)
    ragged = sb.conv_desc(2, 12, 16, 16, 32, sb.SB_BF16, layout=sb.SB_NCHW8C)
    f32 = sb.conv_desc(2, 16, 16, 16, 32, sb.SB_F32, layout=sb.SB_NCHW8C)
    narrow = sb.conv_desc(2, 16, 4, 4, 32, sb.SB_BF16, layout=sb.SB_NCHW8C)
    x, w, y = P, P + (1 << 20), P + (2 << 20)
    for d, status in ((bad_layout, sb.SB_ERR_INVALID_ARG), (ragged, sb.SB_ERR_INVALID_ARG),
                      (f32, sb.SB_ERR_UNSUPPORTED), (narrow, sb.SB_ERR_UNSUPPORTED)):
        assert _raw("sb_conv3x3_fwd", ctypes.byref(d), x, w, None, y, None, 0, None) == status
        assert _raw("sb_conv3x3_bwd_weight", ctypes.byref(d), x, y, P + (3 << 20), None, None, 0,
                    None) == status
        assert sb.sb_conv3x3_workspace_bytes(d, 0) == 2 ** 64 - 1


def test_bwd_weight_many_validation():
    d8 = sb.conv_desc(8, 256, 8, 8, 256)
    d16 = sb.conv_desc(8, 128, 16, 16, 128)
    n = 2

    def call(descs, xs, dys, dws, dbs, ws, wsb):
        k = len(descs)
        arr = lambda v: (ctypes.c_void_p * k)(*v) if v is not None else None
        return _raw("sb_conv3x3_bwd_weight_many", k, (sb.sb_conv3x3_desc * k)(*descs),
                    arr(xs), arr(dys), arr(dws), arr(dbs), ws, wsb, None)
    x0, y0, x1, y1 = P, P + (64 << 20), P + (128 << 20), P + (192 << 20)
    w0, w1, b0, b1 = P + (256 << 20), P + (264 << 20), P + (272 << 20), P + (273 << 20)
    ws = P + (320 << 20)
    need = sb.load().sb_conv3x3_bwd_weight_many_workspace_bytes(
        n, (sb.sb_conv3x3_desc * n)(d8, d16))
    one = [sb.sb_conv3x3_workspace_bytes(d, sb.SB_PASS_BWD_WEIGHT) for d in (d8, d16)]
    assert need == sum((b + 255) // 256 * 256 for b in one)
    assert sb.load().sb_conv3x3_bwd_weight_many_workspace_bytes(0, None) == ctypes.c_size_t(-1).value
    ok = lambda **kw: call(**dict(dict(descs=[d8, d16], xs=[x0, x1], dys=[y0, y1], dws=[w0, w1],
                                       dbs=[b0, b1], ws=ws, wsb=need), **kw))
    E, W = sb.SB_ERR_INVALID_ARG, sb.SB_ERR_WORKSPACE
    assert _raw("sb_conv3x3_bwd_weight_many", 0, None, None, None, None, None, None, 0,
                None) == E
    assert ok(xs=None) == E                                   # null arrays
    assert ok(dws=[w0, None]) == E                            # a null output
    assert ok(dws=[w0, x1 + 64]) == E                         # dW over another layer's input
    assert ok(dws=[w0, w0 + 4]) == E                          # two layers' dW overlap
    assert ok(dbs=[b0, w0]) == E                              # a db over another layer's dW
    assert ok(ws=y1) == E                                     # workspace over an input
    assert ok(wsb=need - 1) == W                              # short workspace
    assert ok(descs=[d8, sb.conv_desc(8, 128, 16, 16, 0)]) == E   # a bad descriptor
