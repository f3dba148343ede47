"""Shared helpers of the parity tests: comparison metrics and device plumbing."""
import numpy as np

# Tolerances on the relative L2 error of every output tensor (fp32 path, bf16
# path); argmax codes must match exactly.
TOL = {"f32": 1e-4, "bf16": 2e-2}


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.float64).ravel()
    ref = np.asarray(ref, dtype=np.float64).ravel()
    den = np.linalg.norm(ref)
    num = np.linalg.norm(got - ref)
    if den == 0.0:
        return num if num > 1e-30 else 0.0
    return num / den


def to_dev(a, dtype="f32"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    return t.cuda()


def to_host(t):
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


def sample_idx(total, count, seed):
    rng = np.random.default_rng(seed)
    count = min(count, total)
    idx = rng.choice(total, size=count, replace=False)
    # Always include the first and last elements (borders / ragged tails).
    return np.unique(np.concatenate([idx, [0, total - 1]])).astype(np.int64)


def print_case(name, **kw):
    """Name the case before a GPU step, so a failure can be attributed."""
    print("CASE", name, " ".join("%s=%s" % kv for kv in kw.items()), flush=True)
