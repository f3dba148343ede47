"""Thin Python binding of libsb (include/sb.h): argument marshalling only.

Every function has the name of the C entry point it calls and takes torch
tensors that live on the GPU (torch provides device memory and streams, and
nothing else here): the tensor's dtype selects SB_F32 / SB_BF16, its data
pointer is passed through, and the current torch stream is the HIP stream
unless one is given.  Every step of the computation runs in libsb's HIP
kernels.  A non-OK status raises ``SBError``.

The library must have been built (``python -m paper_2112_15317_amd.build``);
if ``libsb.so`` is missing, loading fails loudly: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import threading

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsb.so")

SB_OK, SB_ERR_INVALID_ARG, SB_ERR_UNSUPPORTED, SB_ERR_WORKSPACE, SB_ERR_HIP = range(5)
SB_F32, SB_BF16 = 0, 1
SB_NCHW, SB_NCHW8C = 0, 1
SB_FUSE_RELU = 1
SB_PACKED_FILTERS = 2
SB_PASS_FWD, SB_PASS_BWD_DATA, SB_PASS_BWD_WEIGHT, SB_PASS_FWD_POOL = 0, 1, 2, 3
SIZE_MAX = 2 ** 64 - 1          # (size_t)-1: the workspace queries' "not supported"
SB_FC_FWD, SB_FC_BWD = 0, 1
SB_SGD_MAX_TENSORS = 64
SB_NOALLOC_SCRATCH_BYTES = 40 << 20

_vp = ctypes.c_void_p
_i = ctypes.c_int
_sz = ctypes.c_size_t


class sb_conv3x3_desc(ctypes.Structure):
    _fields_ = [("n", _i), ("c", _i), ("h", _i), ("w", _i), ("k", _i),
                ("dtype", _i), ("flags", ctypes.c_uint), ("layout", _i)]


class sb_fc_desc(ctypes.Structure):
    _fields_ = [("m", _i), ("k_in", _i), ("n_shard", _i), ("dtype", _i),
                ("ldx", _i), ("ldy", _i), ("flags", ctypes.c_uint)]


class sb_modulo_desc(ctypes.Structure):
    _fields_ = [("workers", _i), ("mp", _i), ("batch", _i), ("features", _i)]


class sb_shard_desc(ctypes.Structure):
    _fields_ = [("workers", _i), ("mp", _i), ("rows", _i), ("shard", _i)]


# Every exported symbol of include/sb.h with its ctypes signature.
SIGNATURES = {
    "sb_status_string": (ctypes.c_char_p, [_i]),
    "sb_version": (_i, []),
    "sb_conv3x3_workspace_bytes": (_sz, [ctypes.POINTER(sb_conv3x3_desc), _i]),
    "sb_conv3x3_packed_bytes": (_sz, [ctypes.POINTER(sb_conv3x3_desc), _i]),
    "sb_conv3x3_pack_filters": (_i, [ctypes.POINTER(sb_conv3x3_desc), _i, _vp, _vp, _sz, _vp]),
    "sb_conv3x3_pack_filters_many": (_i, [_i, ctypes.POINTER(sb_conv3x3_desc),
                                          ctypes.POINTER(_i), ctypes.POINTER(_vp),
                                          ctypes.POINTER(_vp), ctypes.POINTER(_sz), _vp]),
    "sb_conv3x3_plan_string": (_sz, [ctypes.POINTER(sb_conv3x3_desc), _i, ctypes.c_char_p, _sz]),
    "sb_conv3x3_fwd": (_i, [ctypes.POINTER(sb_conv3x3_desc), _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "sb_conv3x3_fwd_pool": (_i, [ctypes.POINTER(sb_conv3x3_desc), _vp, _vp, _vp, _vp, _vp, _vp,
                                 _sz, _vp]),
    "sb_conv3x3_bwd_data": (_i, [ctypes.POINTER(sb_conv3x3_desc), _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "sb_conv3x3_bwd_weight": (_i, [ctypes.POINTER(sb_conv3x3_desc), _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "sb_conv3x3_bwd_weight_noalloc": (_i, [ctypes.POINTER(sb_conv3x3_desc), _vp, _vp, _vp, _vp,
                                           _vp]),
    "sb_conv3x3_bwd_weight_many_workspace_bytes": (_sz, [_i, ctypes.POINTER(sb_conv3x3_desc)]),
    "sb_conv3x3_bwd_weight_many": (_i, [_i, ctypes.POINTER(sb_conv3x3_desc), ctypes.POINTER(_vp),
                                        ctypes.POINTER(_vp), ctypes.POINTER(_vp),
                                        ctypes.POINTER(_vp), _vp, _sz, _vp]),
    "sb_relu_maxpool_fwd": (_i, [_i, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp]),
    "sb_relu_maxpool_bwd": (_i, [_i, _i, _i, _i, _i, _i, _vp, _vp, _vp, _vp]),
    "sb_fc_workspace_bytes": (_sz, [ctypes.POINTER(sb_fc_desc), _i]),
    "sb_fc_shard_fwd": (_i, [ctypes.POINTER(sb_fc_desc), _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "sb_fc_shard_bwd": (_i, [ctypes.POINTER(sb_fc_desc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _i,
                             _vp, _sz, _vp]),
    "sb_modulo_fwd": (_i, [ctypes.POINTER(sb_modulo_desc), _i, _i, _vp, _sz, _vp, _vp]),
    "sb_modulo_bwd": (_i, [ctypes.POINTER(sb_modulo_desc), _i, _i, _vp, _sz, _vp, _sz, _vp]),
    "sb_shard_fwd": (_i, [ctypes.POINTER(sb_shard_desc), _i, _vp, _sz, _vp, _vp]),
    "sb_shard_bwd": (_i, [ctypes.POINTER(sb_shard_desc), _i, _vp, _sz, _vp, _sz, _vp]),
    "sb_model_average": (_i, [_i, _i, _sz, _vp, _sz, _vp]),
    "sb_model_average_replicas": (_i, [_i, _sz, ctypes.POINTER(_vp), _vp]),
    "sb_log_softmax_nll": (_i, [_i, _i, _i, _vp, _vp, ctypes.c_float, _vp, _vp, _vp, _vp]),
    "sb_sgd_update": (_i, [_i, ctypes.POINTER(_vp), ctypes.POINTER(_vp), ctypes.POINTER(_sz),
                           ctypes.POINTER(ctypes.c_float), ctypes.c_float, _vp]),
}

_lock = threading.Lock()
_lib = None


class SBError(RuntimeError):
    def __init__(self, fn, status):
        self.status = status
        super().__init__("%s failed: %s" % (fn, status_name(status)))


def load():
    """Load libsb.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    "libsb.so not found at %s: build it with "
                    "`python -m paper_2112_15317_amd.build` (no fallback exists)" % LIB_PATH)
            lib = ctypes.CDLL(LIB_PATH)
            for name, (res, args) in SIGNATURES.items():
                fn = getattr(lib, name)
                fn.restype = res
                fn.argtypes = args
            _lib = lib
    return _lib


def status_name(status: int) -> str:
    return load().sb_status_string(int(status)).decode()


def _check(fn, status):
    if status != SB_OK:
        raise SBError(fn, status)


# ----------------------------------------------------------- marshalling --
def _dtype_code(t):
    import torch
    if t.dtype == torch.float32:
        return SB_F32
    if t.dtype == torch.bfloat16:
        return SB_BF16
    raise TypeError("libsb takes float32 or bfloat16 tensors, got %s" % t.dtype)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("libsb takes device tensors")
    if not t.is_contiguous():
        raise ValueError("libsb takes contiguous tensors (strides go in the descriptor)")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ws(ws):
    if ws is None:
        return None, 0
    return ws.data_ptr(), ws.numel() * ws.element_size()


def conv_desc(n, c, h, w, k, dtype=SB_F32, relu=False, packed=False, layout=SB_NCHW):
    return sb_conv3x3_desc(n, c, h, w, k, dtype,
                           (SB_FUSE_RELU if relu else 0) | (SB_PACKED_FILTERS if packed else 0),
                           layout)


def fc_desc(m, k_in, n_shard, dtype=SB_F32, ldx=None, ldy=None, relu=False):
    return sb_fc_desc(m, k_in, n_shard, dtype, ldx or k_in, ldy or n_shard,
                      SB_FUSE_RELU if relu else 0)


# --------------------------------------------------------- entry points --
def sb_version():
    return load().sb_version()


def sb_conv3x3_workspace_bytes(desc, pass_):
    return load().sb_conv3x3_workspace_bytes(ctypes.byref(desc), pass_)


def sb_conv3x3_plan_string(desc, pass_):
    buf = ctypes.create_string_buffer(512)
    n = load().sb_conv3x3_plan_string(ctypes.byref(desc), pass_, buf, 512)
    if n == 0:
        raise SBError("sb_conv3x3_plan_string", SB_ERR_INVALID_ARG)
    return buf.value.decode()


def sb_conv3x3_packed_bytes(desc, pass_):
    return load().sb_conv3x3_packed_bytes(ctypes.byref(desc), pass_)


def sb_conv3x3_pack_filters(desc, pass_, w, packed, stream=None):
    _check("sb_conv3x3_pack_filters", load().sb_conv3x3_pack_filters(
        ctypes.byref(desc), pass_, _ptr(w), _ptr(packed),
        packed.numel() * packed.element_size(), _stream(stream)))


class PackList:
    """Marshalled arguments of sb_conv3x3_pack_filters_many for a fixed list
    of (desc, pass, filters, packed buffer): built once, passed to every
    call (the buffers must stay alive)."""

    def __init__(self, items):
        n = len(items)
        self.count = n
        self.descs = (sb_conv3x3_desc * n)(*[d for d, _, _, _ in items])
        self.passes = (_i * n)(*[p for _, p, _, _ in items])
        self.w = (_vp * n)(*[_ptr(w) for _, _, w, _ in items])
        self.packed = (_vp * n)(*[_ptr(o) for _, _, _, o in items])
        self.nbytes = (_sz * n)(*[o.numel() * o.element_size() for _, _, _, o in items])


def sb_conv3x3_pack_filters_many(plist, stream=None):
    _check("sb_conv3x3_pack_filters_many", load().sb_conv3x3_pack_filters_many(
        plist.count, plist.descs, plist.passes, plist.w, plist.packed, plist.nbytes,
        _stream(stream)))


def sb_conv3x3_fwd(desc, x, w, bias, y, ws=None, stream=None):
    p, nb = _ws(ws)
    _check("sb_conv3x3_fwd", load().sb_conv3x3_fwd(
        ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(bias), _ptr(y), p, nb, _stream(stream)))


def sb_conv3x3_fwd_pool(desc, x, w, bias, y, idx, ws=None, stream=None):
    p, nb = _ws(ws)
    _check("sb_conv3x3_fwd_pool", load().sb_conv3x3_fwd_pool(
        ctypes.byref(desc), _ptr(x), _ptr(w), _ptr(bias), _ptr(y), _ptr(idx), p, nb,
        _stream(stream)))


def sb_conv3x3_bwd_data(desc, dy, w, relu_mask_src, dx, ws=None, stream=None):
    p, nb = _ws(ws)
    _check("sb_conv3x3_bwd_data", load().sb_conv3x3_bwd_data(
        ctypes.byref(desc), _ptr(dy), _ptr(w), _ptr(relu_mask_src), _ptr(dx), p, nb,
        _stream(stream)))


def sb_conv3x3_bwd_weight(desc, x, dy, dw, db, ws=None, stream=None):
    p, nb = _ws(ws)
    _check("sb_conv3x3_bwd_weight", load().sb_conv3x3_bwd_weight(
        ctypes.byref(desc), _ptr(x), _ptr(dy), _ptr(dw), _ptr(db), p, nb, _stream(stream)))


class WgradList:
    """Host arrays of a sb_conv3x3_bwd_weight_many call (kept alive with the
    object, so a recorded call can be issued again)."""

    def __init__(self, descs, x, dy, dw, db):
        n = len(descs)
        self.count = n
        self.descs = (sb_conv3x3_desc * n)(*descs)
        self.x = (_vp * n)(*[_ptr(t) for t in x])
        self.dy = (_vp * n)(*[_ptr(t) for t in dy])
        self.dw = (_vp * n)(*[_ptr(t) for t in dw])
        self.db = (_vp * n)(*[_ptr(t) for t in db])

    def workspace_bytes(self):
        return load().sb_conv3x3_bwd_weight_many_workspace_bytes(self.count, self.descs)


def sb_conv3x3_bwd_weight_many(wlist, ws=None, stream=None):
    p, nb = _ws(ws)
    _check("sb_conv3x3_bwd_weight_many", load().sb_conv3x3_bwd_weight_many(
        wlist.count, wlist.descs, wlist.x, wlist.dy, wlist.dw, wlist.db, p, nb,
        _stream(stream)))


def sb_conv3x3_bwd_weight_noalloc(desc, x, dy, dw, db, stream=None):
    _check("sb_conv3x3_bwd_weight_noalloc", load().sb_conv3x3_bwd_weight_noalloc(
        ctypes.byref(desc), _ptr(x), _ptr(dy), _ptr(dw), _ptr(db), _stream(stream)))


def sb_relu_maxpool_fwd(n, c, h, w, dtype, layout, x, y, idx, stream=None):
    _check("sb_relu_maxpool_fwd", load().sb_relu_maxpool_fwd(
        n, c, h, w, dtype, layout, _ptr(x), _ptr(y), _ptr(idx), _stream(stream)))


def sb_relu_maxpool_bwd(n, c, h, w, dtype, layout, dy, idx, dx, stream=None):
    _check("sb_relu_maxpool_bwd", load().sb_relu_maxpool_bwd(
        n, c, h, w, dtype, layout, _ptr(dy), _ptr(idx), _ptr(dx), _stream(stream)))


def sb_fc_workspace_bytes(desc, pass_):
    return load().sb_fc_workspace_bytes(ctypes.byref(desc), pass_)


def sb_fc_shard_fwd(desc, x, w_shard, b_shard, y, ws=None, stream=None):
    p, nb = _ws(ws)
    _check("sb_fc_shard_fwd", load().sb_fc_shard_fwd(
        ctypes.byref(desc), _ptr(x), _ptr(w_shard), _ptr(b_shard), _ptr(y), p, nb,
        _stream(stream)))


def sb_fc_shard_bwd(desc, x, w_shard, dy, relu_mask_src, dx_partial, dw_shard, db_shard,
                    accumulate=False, ws=None, stream=None):
    p, nb = _ws(ws)
    _check("sb_fc_shard_bwd", load().sb_fc_shard_bwd(
        ctypes.byref(desc), _ptr(x), _ptr(w_shard), _ptr(dy), _ptr(relu_mask_src),
        _ptr(dx_partial), _ptr(dw_shard), _ptr(db_shard), 1 if accumulate else 0, p, nb,
        _stream(stream)))


# ------------------------------------------------ modulo and shard layers --
# Slotted buffers: worker w's slot starts at w * stride elements; by default
# the stride is the tensor's element count divided by the number of workers
# (a contiguous [workers][...] tensor).
def modulo_desc(workers, mp, batch, features):
    return sb_modulo_desc(workers, mp, batch, features)


def shard_desc(workers, mp, rows, shard):
    return sb_shard_desc(workers, mp, rows, shard)


def _slot_stride(t, workers, stride):
    if stride is not None:
        return int(stride)
    if t is None or isinstance(t, int):
        raise ValueError("give the slot stride for a raw pointer")
    return t.numel() // workers


def sb_modulo_fwd(desc, iproc, k, local, gathered, local_stride=None, stream=None):
    _check("sb_modulo_fwd", load().sb_modulo_fwd(
        ctypes.byref(desc), int(iproc), int(k), _ptr(local),
        _slot_stride(local, desc.workers, local_stride), _ptr(gathered), _stream(stream)))


def sb_modulo_bwd(desc, iproc, k, dgathered, dlocal, dg_stride=None, dl_stride=None,
                  stream=None):
    _check("sb_modulo_bwd", load().sb_modulo_bwd(
        ctypes.byref(desc), int(iproc), int(k), _ptr(dgathered),
        _slot_stride(dgathered, desc.workers, dg_stride), _ptr(dlocal),
        _slot_stride(dlocal, desc.workers, dl_stride), _stream(stream)))


def sb_shard_fwd(desc, iproc, parts, full, parts_stride=None, stream=None):
    _check("sb_shard_fwd", load().sb_shard_fwd(
        ctypes.byref(desc), int(iproc), _ptr(parts),
        _slot_stride(parts, desc.workers, parts_stride), _ptr(full), _stream(stream)))


def sb_shard_bwd(desc, iproc, dfull, dparts, df_stride=None, dp_stride=None, stream=None):
    _check("sb_shard_bwd", load().sb_shard_bwd(
        ctypes.byref(desc), int(iproc), _ptr(dfull),
        _slot_stride(dfull, desc.workers, df_stride), _ptr(dparts),
        _slot_stride(dparts, desc.workers, dp_stride), _stream(stream)))


def sb_model_average(workers, mp, params, n=None, stride=None, stream=None):
    """params: `workers` slots of fp32 parameters (a contiguous
    [workers][...] tensor by default: n = stride = numel / workers)."""
    st = _slot_stride(params, workers, stride)
    _check("sb_model_average", load().sb_model_average(
        int(workers), int(mp), int(st if n is None else n), _ptr(params), st, _stream(stream)))


SB_MAX_REPLICAS = 64


def sb_model_average_replicas(replicas, n=None, stream=None):
    """replicas: one fp32 tensor (or device pointer) per replica; each is
    replaced by the mean of all.  n defaults to the first tensor's numel."""
    k = len(replicas)
    if n is None:
        n = replicas[0].numel()
    for t in replicas:
        if not isinstance(t, int) and (str(t.dtype) != "torch.float32" or t.numel() < n):
            raise ValueError("replicas must be fp32 tensors of at least n elements")
    ptrs = (_vp * max(k, 1))(*[_ptr(t) for t in replicas])
    _check("sb_model_average_replicas", load().sb_model_average_replicas(
        int(k), int(n), ptrs, _stream(stream)))


# --------------------------------------------------- loss and SGD update --
def sb_log_softmax_nll(m, classes, z, labels, scale, logp=None, loss=None, dz=None, ldz=None,
                       stream=None):
    """z, logp, dz: fp32 [m][ldz] (ldz defaults to classes); labels: int32 [m]."""
    _check("sb_log_softmax_nll", load().sb_log_softmax_nll(
        int(m), int(classes), int(ldz or classes), _ptr(z), _ptr(labels), float(scale),
        _ptr(logp), _ptr(loss), _ptr(dz), _stream(stream)))


class SgdList:
    """Marshalled arguments of sb_sgd_update for a fixed list of
    (parameter, gradient, scale) fp32 tensors: built once, passed to every
    call (the tensors must stay alive)."""

    def __init__(self, items):
        import torch
        n = len(items)
        if not 1 <= n <= SB_SGD_MAX_TENSORS:
            raise ValueError("1 to %d tensors per update" % SB_SGD_MAX_TENSORS)
        for w, g, _ in items:
            if w.dtype != torch.float32 or g.dtype != torch.float32 or w.numel() != g.numel():
                raise ValueError("fp32 parameter and gradient of equal size")
        self.count = n
        self.w = (_vp * n)(*[_ptr(w) for w, _, _ in items])
        self.g = (_vp * n)(*[_ptr(g) for _, g, _ in items])
        self.n = (_sz * n)(*[w.numel() for w, _, _ in items])
        self.scale = (ctypes.c_float * n)(*[float(sc) for _, _, sc in items])


def sb_sgd_update(slist, lr, stream=None):
    _check("sb_sgd_update", load().sb_sgd_update(
        slist.count, slist.w, slist.g, slist.n, slist.scale, float(lr), _stream(stream)))
