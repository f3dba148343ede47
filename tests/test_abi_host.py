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
    assert sb.sb_conv3x3_workspace_bytes(d, 3) == 2 ** 64 - 1


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
        assert _raw("sb_relu_maxpool_fwd", *shape, 0, P, P + 4096, P + 8192, None) == sb.SB_ERR_INVALID_ARG
        assert _raw("sb_relu_maxpool_bwd", *shape, 0, P, P + 4096, P + 8192, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_relu_maxpool_fwd", 1, 1, 2, 2, 5, P, P + 4096, P + 8192, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_relu_maxpool_fwd", 1, 1, 2, 2, 0, None, P + 4096, P + 8192, None) == sb.SB_ERR_INVALID_ARG
    # Output aliasing the input.
    assert _raw("sb_relu_maxpool_fwd", 1, 4, 4, 4, 0, P, P + 8, P + 8192, None) == sb.SB_ERR_INVALID_ARG
    assert _raw("sb_relu_maxpool_bwd", 1, 4, 4, 4, 0, P, P + 8192, P + 16, None) == sb.SB_ERR_INVALID_ARG


def test_fc_argument_validation():
    ok = sb.fc_desc(16, 32, 8)
    assert sb.sb_fc_workspace_bytes(ok, sb.SB_FC_FWD) != 2 ** 64 - 1
    for bad in [sb.fc_desc(0, 32, 8), sb.fc_desc(16, 32, 8, ldx=16), sb.fc_desc(16, 32, 8, ldy=4),
                sb.sb_fc_desc(16, 32, 8, 0, 32, 8, 4)]:
        assert sb.sb_fc_workspace_bytes(bad, 0) == 2 ** 64 - 1
        assert _raw("sb_fc_shard_fwd", ctypes.byref(bad), P, P + 8192, None, P + 65536, None, 0, None) == sb.SB_ERR_INVALID_ARG
    bf = sb.fc_desc(16, 32, 8, dtype=sb.SB_BF16)
    assert _raw("sb_fc_shard_fwd", ctypes.byref(bf), P, P + 8192, None, P + 65536, None, 0, None) == sb.SB_ERR_UNSUPPORTED
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
