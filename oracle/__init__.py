"""fp64 CPU oracle for one SplitBrain worker's compute share (arXiv 2112.15317).

TEST INFRASTRUCTURE.  Only the test suite (``tests/``), the smoke check in
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` import
this package.  The product (``paper_2112_15317_amd``) never imports, loads or
calls it, and this package never touches the HIP library: the two share no
code.  The arithmetic lives in ``sb_oracle.c`` (plain fp64 loops over each
layer's definition, sec. 2.2 and sec. 3.1 of the paper); this module only
builds that file with gcc and marshals numpy arrays into it.

All functions take and return numpy arrays.  Inputs of any float dtype are
converted exactly to float64 (every float32 and bfloat16 value is a float64
value), so the oracle sees the very numbers the GPU library is given.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sb_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

_D = ctypes.POINTER(ctypes.c_double)
_U8 = ctypes.POINTER(ctypes.c_uint8)
_I64 = ctypes.POINTER(ctypes.c_int64)
_i = ctypes.c_int
_i64 = ctypes.c_int64


def build(force: bool = True) -> str:
    """Compile sb_oracle.c into liboracle.so next to it (gcc, OpenMP)."""
    if not force and os.path.exists(_LIB_PATH) and (
            os.path.getmtime(_LIB_PATH) >= os.path.getmtime(_SRC)):
        return _LIB_PATH
    tmp = _LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-std=c11", "-O2", "-fno-fast-math", "-ffp-contract=off",
           "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build(force=False)
            lib = ctypes.CDLL(_LIB_PATH)
            sig = {
                "or_conv3x3_fwd": [_i, _i, _i, _i, _i, _D, _D, _D, _i, _D],
                "or_conv3x3_fwd_at": [_i, _i, _i, _i, _i, _D, _D, _D, _i, _i64, _I64, _D],
                "or_conv3x3_bwd_data": [_i, _i, _i, _i, _i, _D, _D, _D, _D],
                "or_conv3x3_bwd_data_at": [_i, _i, _i, _i, _i, _D, _D, _D, _i64, _I64, _D],
                "or_conv3x3_bwd_weight": [_i, _i, _i, _i, _i, _D, _D, _D, _D],
                "or_conv3x3_bwd_weight_at": [_i, _i, _i, _i, _i, _D, _D, _i64, _I64, _D],
                "or_relu_maxpool_fwd": [_i, _i, _i, _i, _D, _D, _U8],
                "or_relu_maxpool_bwd": [_i, _i, _i, _i, _D, _U8, _D],
                "or_fc_fwd": [_i, _i, _i, _D, _D, _D, _i, _D],
                "or_fc_fwd_at": [_i, _i, _i, _D, _D, _D, _i, _i64, _I64, _D],
                "or_fc_bwd": [_i, _i, _i, _D, _D, _D, _D, _D, _D, _D, _i],
                "or_fc_bwd_dx_at": [_i, _i, _i, _D, _D, _D, _i64, _I64, _D],
                "or_fc_bwd_dw_at": [_i, _i, _i, _D, _D, _D, _i64, _I64, _D],
                "or_round_bf16": [_D, _i64],
            }
            lib.or_num_threads.argtypes = []
            lib.or_num_threads.restype = _i
            for name, args in sig.items():
                fn = getattr(lib, name)
                fn.argtypes = args
                fn.restype = None
            _lib = lib
    return _lib


def _f64(a):
    """Exact float64 copy (C-contiguous) of any float array, incl. torch bf16."""
    if a is None:
        return None
    if hasattr(a, "detach"):                      # torch tensor (CPU)
        import torch
        a = a.detach().to("cpu", torch.float64).numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _p(a):
    return None if a is None else a.ctypes.data_as(_D)


def _flat(idx):
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int64).ravel())
    return idx, idx.ctypes.data_as(_I64)


# ------------------------------------------------------------------ conv --
def conv3x3_fwd(x, w, bias=None, relu=False):
    """Z = b + X (*) W, 3x3, stride 1, zero pad 1 (cross-correlation); NCHW/KCRS."""
    x, w, b = _f64(x), _f64(w), _f64(bias)
    n, c, h, wd = x.shape
    k = w.shape[0]
    assert w.shape == (k, c, 3, 3)
    y = np.empty((n, k, h, wd))
    _load().or_conv3x3_fwd(n, c, h, wd, k, _p(x), _p(w), _p(b), int(relu), _p(y))
    return y


def conv3x3_fwd_at(x, w, flat, bias=None, relu=False):
    """conv3x3_fwd evaluated only at the given flat NKHW output indices."""
    x, w, b = _f64(x), _f64(w), _f64(bias)
    n, c, h, wd = x.shape
    k = w.shape[0]
    idx, pidx = _flat(flat)
    out = np.empty(idx.size)
    _load().or_conv3x3_fwd_at(n, c, h, wd, k, _p(x), _p(w), _p(b), int(relu),
                              idx.size, pidx, _p(out))
    return out


def conv3x3_bwd_data(dz, w, mask_src=None):
    """dX = dZ (*)^T W; zeroed where mask_src <= 0 when a mask source is given."""
    dz, w, m = _f64(dz), _f64(w), _f64(mask_src)
    n, k, h, wd = dz.shape
    c = w.shape[1]
    assert w.shape == (k, c, 3, 3)
    if m is not None:
        assert m.shape == (n, c, h, wd)
    dx = np.empty((n, c, h, wd))
    _load().or_conv3x3_bwd_data(n, c, h, wd, k, _p(dz), _p(w), _p(m), _p(dx))
    return dx


def conv3x3_bwd_data_at(dz, w, flat, mask_src=None):
    dz, w, m = _f64(dz), _f64(w), _f64(mask_src)
    n, k, h, wd = dz.shape
    c = w.shape[1]
    idx, pidx = _flat(flat)
    out = np.empty(idx.size)
    _load().or_conv3x3_bwd_data_at(n, c, h, wd, k, _p(dz), _p(w), _p(m),
                                   idx.size, pidx, _p(out))
    return out


def conv3x3_bwd_weight(x, dz, want_db=True):
    """(dW[K,C,3,3], db[K]) for Z = X (*) W + b."""
    x, dz = _f64(x), _f64(dz)
    n, c, h, wd = x.shape
    k = dz.shape[1]
    assert dz.shape == (n, k, h, wd)
    dw = np.empty((k, c, 3, 3))
    db = np.empty(k) if want_db else None
    _load().or_conv3x3_bwd_weight(n, c, h, wd, k, _p(x), _p(dz), _p(dw), _p(db))
    return dw, db


def conv3x3_bwd_weight_at(x, dz, flat):
    x, dz = _f64(x), _f64(dz)
    n, c, h, wd = x.shape
    k = dz.shape[1]
    idx, pidx = _flat(flat)
    out = np.empty(idx.size)
    _load().or_conv3x3_bwd_weight_at(n, c, h, wd, k, _p(x), _p(dz),
                                     idx.size, pidx, _p(out))
    return out


# ------------------------------------------------------- relu + maxpool --
def relu_maxpool_fwd(x):
    """(Y, idx) of ReLU(maxpool2x2/2(X)); idx codes as documented in sb_oracle.c."""
    x = _f64(x)
    n, c, h, wd = x.shape
    assert h % 2 == 0 and wd % 2 == 0
    y = np.empty((n, c, h // 2, wd // 2))
    idx = np.empty((n, c, h // 2, wd // 2), dtype=np.uint8)
    _load().or_relu_maxpool_fwd(n, c, h, wd, _p(x), _p(y), idx.ctypes.data_as(_U8))
    return y, idx


def relu_maxpool_bwd(dy, idx):
    """dX (un-pooled shape) from the pooled gradient and the window codes."""
    dy = _f64(dy)
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.uint8))
    n, c, ho, wo = dy.shape
    assert idx.shape == dy.shape
    dx = np.empty((n, c, 2 * ho, 2 * wo))
    _load().or_relu_maxpool_bwd(n, c, 2 * ho, 2 * wo, _p(dy),
                                idx.ctypes.data_as(_U8), _p(dx))
    return dx


# -------------------------------------------------------------- FC shard --
def fc_fwd(x, w, b=None, relu=False):
    """Y = X W_shard + b_shard (ReLU optional); X [M,Kin], W_shard [Kin,Ns]."""
    x, w, b = _f64(x), _f64(w), _f64(b)
    m, kin = x.shape
    ns = w.shape[1]
    assert w.shape[0] == kin
    y = np.empty((m, ns))
    _load().or_fc_fwd(m, kin, ns, _p(x), _p(w), _p(b), int(relu), _p(y))
    return y


def fc_fwd_at(x, w, flat, b=None, relu=False):
    x, w, b = _f64(x), _f64(w), _f64(b)
    m, kin = x.shape
    ns = w.shape[1]
    idx, pidx = _flat(flat)
    out = np.empty(idx.size)
    _load().or_fc_fwd_at(m, kin, ns, _p(x), _p(w), _p(b), int(relu),
                         idx.size, pidx, _p(out))
    return out


def fc_bwd(x, w, dy, mask_src=None, dw_acc=None, db_acc=None, want_dx=True):
    """(dX_partial, dW_shard, db_shard) of the shard; dW/db added to the given
    accumulators when dw_acc is passed (the K modulo iterations)."""
    x, w, dy, m = _f64(x), _f64(w), _f64(dy), _f64(mask_src)
    mm, kin = x.shape
    ns = w.shape[1]
    assert dy.shape == (mm, ns)
    accumulate = dw_acc is not None
    dw = _f64(dw_acc).copy() if accumulate else np.empty((kin, ns))
    db = (_f64(db_acc).copy() if db_acc is not None else np.zeros(ns)) if accumulate \
        else np.empty(ns)
    dxp = np.empty((mm, kin)) if want_dx else None
    _load().or_fc_bwd(mm, kin, ns, _p(x), _p(w), _p(dy), _p(m), _p(dxp), _p(dw),
                      _p(db), int(accumulate))
    return dxp, dw, db


def fc_bwd_dx_at(w, dy, flat, mask_src=None):
    w, dy, m = _f64(w), _f64(dy), _f64(mask_src)
    kin, ns = w.shape
    mm = dy.shape[0]
    idx, pidx = _flat(flat)
    out = np.empty(idx.size)
    _load().or_fc_bwd_dx_at(mm, kin, ns, _p(w), _p(dy), _p(m), idx.size, pidx, _p(out))
    return out


def fc_bwd_dw_at(x, dy, flat, mask_src=None):
    x, dy, m = _f64(x), _f64(dy), _f64(mask_src)
    mm, kin = x.shape
    ns = dy.shape[1]
    idx, pidx = _flat(flat)
    out = np.empty(idx.size)
    _load().or_fc_bwd_dw_at(mm, kin, ns, _p(x), _p(dy), _p(m), idx.size, pidx, _p(out))
    return out


def num_threads() -> int:
    """OpenMP threads the oracle's loops use."""
    return int(_load().or_num_threads())


# ------------------------------------------------------------- rounding --
def round_f32(a):
    """Nearest float32 value (ties to even) of each element, as float64."""
    return np.asarray(_f64(a), np.float64).astype(np.float32).astype(np.float64)


def round_bf16(a):
    """Nearest bfloat16 value (ties to even) of each element, as float64."""
    a = _f64(a).copy()
    _load().or_round_bf16(_p(a), a.size)
    return a
