"""Per-call parity on the oracle's chain: helpers shared by the full-size
GPU tests.

Every call of a step reads tensors the calls before it produced.  The
oracle's storage-rounded chain (``oracle.stack`` with ``store=``) holds each
of those tensors exactly in the GPU's storage type, so a call can be run on
the GPU with *the oracle's* inputs (uploaded into the step's own buffers,
with the step's own descriptors and workspaces: the launch configuration
the benchmark times) and its outputs compared, in full, with the oracle's
outputs of the same call.  No GPU result ever feeds the oracle, and every
decision (a ReLU mask, a pool window's first maximum) is taken on the same
values on both sides, so pool codes and routed gradients must match bit for
bit and every other output meets the dtype's tolerance.
"""
import numpy as np
import torch

from tests.helpers import TOL, rel_l2, to_host

EXACT = "exact"
# Pool codes decided on the GPU's own sums: ("near_tie", z_ref, rel); a
# differing code must be a near-tie within rel x max |z_ref| (2^-6 for bf16
# sums rounded to bf16, 2^-12 for fp32 sums).
NEAR_TIE = "near_tie"
NEAR_TIE_REL = {"bf16": 2.0 ** -6, "f32": 2.0 ** -12}


def put(buf, arr):
    """Upload a host array into a device buffer (any view), exactly."""
    t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).reshape(buf.shape)
    if buf.dtype == torch.uint8:
        t = torch.from_numpy(np.ascontiguousarray(arr, dtype=np.uint8)).reshape(buf.shape)
    buf.copy_(t.to(buf.dtype))


def in_layout(st, buf, arr):
    """An NCHW oracle array in the layout and shape of one of st's buffers:
    channel-blocked for an activation of a c8 stack, and zero-padded along
    the channels where the stack pads them (the first layer's input, its
    data gradient and its filters' gradient)."""
    arr = np.asarray(arr)
    if tuple(arr.shape) == tuple(buf.shape):
        return arr
    if buf.dim() == 5:
        return st.to_layout(torch.from_numpy(np.ascontiguousarray(arr)),
                            buf.shape[1] * buf.shape[4]).numpy()
    pad = [(0, 0)] * arr.ndim
    pad[1] = (0, buf.shape[1] - arr.shape[1])
    return np.pad(arr, pad)


def host_nchw(st, buf, ref_shape):
    """A buffer of st on the host as NCHW, cut to the oracle's channels."""
    got = to_host(st.nchw(buf) if buf.dim() == 5 else buf)
    if got.ndim > 1 and got.shape[1] != ref_shape[1]:
        got = got[:, :ref_shape[1]]
    return got


def conv_io(st, f, b, key):
    """(uploads, checks) of one ConvStack call on the oracle chain (f, b),
    every array already in the buffer's layout.
    uploads: [(buffer, host array)]; checks: [(name, buffer, ref, tol|EXACT)]."""
    ups, checks = _conv_io(st, f, b, key)
    out = []
    for name, buf, r, t in checks:
        if isinstance(t, tuple) and t[0] == NEAR_TIE:
            # Compared as NCHW arrays (the windows of z are NCHW windows).
            out.append((name, (lambda bb=buf, rr=r: host_nchw(st, bb, np.shape(rr))), r, t))
        else:
            out.append((name, buf, in_layout(st, buf, r), t))
    return [(buf, in_layout(st, buf, a)) for buf, a in ups], out


def _conv_io(st, f, b, key):
    kind, i = key
    L = st.layers
    pool = L[i].pool_after if kind != "pack" else False
    tol = TOL[st.dtype]
    if kind == "pack":
        return [], []
    if kind == "fwd":
        out, ref = (st.Z[i], f["Z"][i]) if pool else (st.A[i + 1], f["A"][i + 1])
        return [(st.A[i], f["A"][i])], [("fwd%d" % i, out, ref, tol)]
    if kind == "fwd_pool":
        # The pooling decisions are taken on the GPU's own rounded sums.
        return [(st.A[i], f["A"][i])], [("fwd_pool%d.y" % i, st.A[i + 1], f["A"][i + 1], tol),
                                         ("fwd_pool%d.idx" % i, st.idx[i], f["idx"][i],
                                          (NEAR_TIE, f["Z"][i], NEAR_TIE_REL[st.dtype]))]
    if kind == "pool_fwd":
        return [(st.Z[i], f["Z"][i])], [("pool_fwd%d.y" % i, st.A[i + 1], f["A"][i + 1], EXACT),
                                         ("pool_fwd%d.idx" % i, st.idx[i], f["idx"][i], EXACT)]
    if kind == "pool_bwd":
        return ([(st.gA[i + 1], b["dA"][i]), (st.idx[i], f["idx"][i])],
                [("pool_bwd%d" % i, st.dZ[i], b["dZ"][i], EXACT)])
    g = st.dZ[i] if pool else st.gA[i + 1]
    if kind == "wgrad_many":
        # Every layer of the group, each on its own oracle inputs.
        ups, checks = [], []
        for j in st.wg_group_of[i]:
            gj = st.grad_at_conv_output(j)
            ups += [(st.A[j], f["A"][j]), (gj, b["dZ"][j])]
            checks += [("wgrad%d.dw" % j, st.dW[j], b["dW"][j], TOL["f32"]),
                       ("wgrad%d.db" % j, st.db[j], b["db"][j], TOL["f32"])]
        return ups, checks
    if kind == "wgrad":
        # fp32 weight and bias gradients (sums of exact products in bf16 too).
        return ([(st.A[i], f["A"][i]), (g, b["dZ"][i])],
                [("wgrad%d.dw" % i, st.dW[i], b["dW"][i], TOL["f32"]),
                 ("wgrad%d.db" % i, st.db[i], b["db"][i], TOL["f32"])])
    if kind == "dgrad":
        ups = [(g, b["dZ"][i])]
        if i == 0:
            ref = b["dX"]
        elif L[i - 1].pool_after:
            ref = b["dA"][i - 1]
        else:
            ups.append((st.A[i], f["A"][i]))      # the ReLU mask of layer i-1
            ref = b["dZ"][i - 1]
        return ups, [("dgrad%d" % i, st.gA[i], ref, tol)]
    raise KeyError(key)


def run_and_check(call, uploads, checks):
    """Upload, run the one call, compare every output in full."""
    _, fn, args = call
    for buf, arr in uploads:
        put(buf, arr)
    torch.cuda.synchronize()
    fn(*args)
    torch.cuda.synchronize()
    worst = {}
    for name, buf, ref, tol in checks:
        got = buf() if callable(buf) else to_host(buf)
        if isinstance(tol, tuple) and tol[0] == NEAR_TIE:
            z = np.asarray(tol[1])
            worst[name] = near_tie_flips(z, ref, got, tol[2] * np.max(np.abs(z)))
            continue
        ref = np.asarray(ref).reshape(got.shape)
        if tol == EXACT:
            bad = int(np.count_nonzero(got != ref))
            assert bad == 0, "%s: %d elements differ" % (name, bad)
            worst[name] = 0.0
        else:
            e = rel_l2(got, ref)
            worst[name] = e
            assert e <= tol, "%s: relative L2 %.3g > %.3g" % (name, e, tol)
    return worst


def near_tie_flips(z, ref_idx, got_idx, eps):
    """Windows whose codes differ; each must be a near-tie of the oracle's
    values (the two candidates, or the maximum and zero for the ReLU flag,
    within eps).  Returns the number of such windows."""
    bad = np.nonzero(np.asarray(ref_idx).ravel() != np.asarray(got_idx).ravel())[0]
    if bad.size == 0:
        return 0
    n, c, h, w = z.shape
    zw = z.reshape(n, c, h // 2, 2, w // 2, 2).transpose(0, 1, 2, 4, 3, 5).reshape(-1, 4)
    r, g = np.asarray(ref_idx).ravel(), np.asarray(got_idx).ravel()
    for f in bad:
        a, bb = r[f], g[f]
        va, vb = zw[f, a & 3], zw[f, bb & 3]
        gap = abs(va - vb) if (a & 3) != (bb & 3) else 0.0
        flag_gap = abs(va) if (a & 0x80) != (bb & 0x80) else 0.0
        assert max(gap, flag_gap) <= eps, "code mismatch at window %d is not a near-tie" % f
    return int(bad.size)
