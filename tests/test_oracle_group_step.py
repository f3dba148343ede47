"""Pins of the oracle's training step of an MP group (oracle/stack.py,
group_train_step) against torch autograd in float64, written from sec. 3.1
(Modulo Layer) directly: a full (unsharded) model, the gathered batch of
each modulo iteration built here from the paper's index map (gathered
example b comes from worker b // (B/K), local row k*(B/K) + b % (B/K)), the
mean cross-entropy of the B gathered rows, an SGD step of the FC layers at
lr / K after every iteration, and the conv layers' gradient accumulated over
the K iterations and applied once at the end.  The averaged training of
several MP groups (sec. 4: the models averaged every few steps) is pinned
against torch groups stepping on their own data and torch means of their
parameters.  No GPU."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import stack as OS

rng = np.random.default_rng(20211231)


def _t(a, grad=False):
    return torch.tensor(np.asarray(a, np.float64), requires_grad=grad)


def _setup(K, B, seed):
    g = np.random.default_rng(seed)
    sched = [(3, 4, True), (4, 8, True)]          # 4x4 -> 2x2 -> 1x1, 8 features
    x = g.standard_normal((B, 3, 4, 4))
    ws = [g.standard_normal((k, c, 3, 3)) * 0.7 for c, k, _ in sched]
    bs = [g.standard_normal(k) * 0.1 for _, k, _ in sched]
    pools = [p for *_, p in sched]
    classes = 3 * K
    shapes = [(8, 4 * K), (4 * K, 2 * K), (2 * K, classes)]
    fw = [g.standard_normal(s) * 0.6 for s in shapes]
    fb = [g.standard_normal(s[1]) * 0.1 for s in shapes]
    remote = np.maximum(g.standard_normal((K - 1, B, 8)), 0)
    labels = g.integers(0, classes, size=(K, B))
    return x, ws, bs, pools, fw, fb, remote, labels


def _torch_group_step(x, ws, bs, fw, fb, remote, labels, lr, update_between=True):
    """The same step as plain autograd on the unsharded model."""
    K, B = len(remote) + 1, x.shape[0]
    s = B // K
    xt = _t(x, True)
    wt = [_t(w, True) for w in ws]
    bt = [_t(b, True) for b in bs]
    a = xt
    for l in range(len(ws)):
        a = torch.relu(F.max_pool2d(F.conv2d(a, wt[l], bt[l], padding=1), 2, 2))
    top = a.reshape(B, -1)
    top.retain_grad()
    rem = [_t(r, True) for r in remote]
    local = [top] + rem
    W = [_t(w) for w in fw]
    bb = [_t(b) for b in fb]
    losses, grads_sum = [], [torch.zeros_like(w) for w in W]
    for k in range(K):
        rows = [local[b // s][k * s + b % s] for b in range(B)]
        h = torch.stack(rows)
        Wk = [w.clone().requires_grad_(True) for w in W]
        bk = [b.clone().requires_grad_(True) for b in bb]
        for j in range(len(W)):
            h = h @ Wk[j] + bk[j]
            if j < len(W) - 1:
                h = torch.relu(h)
        loss = F.cross_entropy(h, torch.tensor(labels[k]), reduction="mean")
        loss.backward(retain_graph=True)
        losses.append(loss.item())
        with torch.no_grad():
            for j in range(len(W)):
                if update_between:
                    W[j] = W[j] - lr / K * Wk[j].grad
                    bb[j] = bb[j] - lr / K * bk[j].grad
                else:
                    grads_sum[j] = grads_sum[j] + Wk[j].grad
    if not update_between:
        W = [w - lr / K * gsum for w, gsum in zip(W, grads_sum)]
    return {"loss": losses, "W": [w.numpy() for w in W], "b": [b.detach().numpy() for b in bb],
            "conv_w": [w.detach().numpy() - lr * w.grad.numpy() for w in wt],
            "conv_b": [b.detach().numpy() - lr * b.grad.numpy() for b in bt],
            "dtop": top.grad.numpy(), "drem": [r.grad.numpy() for r in rem]}


@pytest.mark.parametrize("K,B", [(1, 3), (2, 4), (3, 6), (4, 4)])
def test_group_step_matches_torch_loop_with_sgd_between_iterations(K, B):
    lr = 0.4
    x, ws, bs, pools, fw, fb, remote, labels = _setup(K, B, 100 + K)
    r = OS.group_train_step(x, ws, bs, pools, fw, fb, remote, labels, lr)
    t = _torch_group_step(x, ws, bs, fw, fb, remote, labels, lr)
    for k in range(K):
        assert abs(r["iters"][k]["loss"].mean() - t["loss"][k]) < 1e-12
    for j in range(3):
        np.testing.assert_allclose(r["fc_w_new"][j], t["W"][j], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(r["fc_b_new"][j], t["b"][j], rtol=1e-10, atol=1e-12)
    for l in range(2):
        np.testing.assert_allclose(r["conv_w_new"][l], t["conv_w"][l], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(r["conv_b_new"][l], t["conv_b"][l], rtol=1e-10, atol=1e-12)
    # The modulo layer's backward hands every worker the gradient of its own
    # local rows, summed over the group's shards.
    np.testing.assert_allclose(r["dlocal"][0], t["dtop"], rtol=1e-10, atol=1e-13)
    for w in range(1, K):
        np.testing.assert_allclose(r["dlocal"][w], t["drem"][w - 1], rtol=1e-10, atol=1e-13)


def test_updates_between_iterations_change_the_step():
    """The K per-iteration FC updates are not one update with the summed
    gradient: the two differ at first order in lr (iteration k's gradient is
    taken at the weights after k updates), far above the pins' tolerance."""
    K, B, lr = 2, 4, 0.4
    x, ws, bs, pools, fw, fb, remote, labels = _setup(K, B, 7)
    r = OS.group_train_step(x, ws, bs, pools, fw, fb, remote, labels, lr)
    once = _torch_group_step(x, ws, bs, fw, fb, remote, labels, lr, update_between=False)
    step = [r["fc_w_new"][j] - fw[j] for j in range(3)]
    diff = [np.linalg.norm(r["fc_w_new"][j] - once["W"][j]) / np.linalg.norm(step[j])
            for j in range(3)]
    assert max(diff) > 1e-3


def test_group_step_iteration_records():
    """Every iteration gathers B rows; the shards of each layer side by side
    are the full layer's output at the weights of that iteration; one
    worker's block of local rows is written per iteration."""
    K, B, lr = 2, 4, 0.25
    x, ws, bs, pools, fw, fb, remote, labels = _setup(K, B, 9)
    r = OS.group_train_step(x, ws, bs, pools, fw, fb, remote, labels, lr)
    for k, it in enumerate(r["iters"]):
        assert it["gathered"].shape == (B, 8)
        h = it["gathered"]
        for j in range(3):
            full = h @ it["w_before"][j] + it["b_before"][j]
            if j < 2:
                full = np.maximum(full, 0)
            np.testing.assert_allclose(it["xs"][j + 1], full, rtol=1e-12, atol=1e-13)
            h = full
        # Iteration 0 runs on the initial weights.
        if k == 0:
            for j in range(3):
                np.testing.assert_array_equal(it["w_before"][j], fw[j])


def _torch_averaged_training(groups, ws, bs, fw, fb, steps, period, lr):
    """G groups stepping independently, their models replaced by the torch
    mean over the groups every `period` steps."""
    state = [{"conv_w": list(ws), "conv_b": list(bs), "fc_w": list(fw), "fc_b": list(fb)}
             for _ in groups]
    for s in range(steps):
        for g, (x, remote, labels) in enumerate(groups):
            p = state[g]
            t = _torch_group_step(x, p["conv_w"], p["conv_b"], p["fc_w"], p["fc_b"], remote,
                                  labels, lr)
            state[g] = {"conv_w": t["conv_w"], "conv_b": t["conv_b"], "fc_w": t["W"],
                        "fc_b": t["b"]}
        if (s + 1) % period == 0:
            for key in state[0]:
                for i in range(len(state[0][key])):
                    m = torch.stack([torch.from_numpy(np.asarray(st[key][i])) for st in state])
                    m = m.mean(dim=0).numpy()
                    for st in state:
                        st[key][i] = m
    return state


def _groups(K, B, G, seed):
    base = _setup(K, B, seed)
    out = []
    for g in range(G):
        x, *_, remote, labels = _setup(K, B, seed + 1 + g)
        out.append((x, remote, labels))
    return base, out


@pytest.mark.parametrize("G,steps,period", [(2, 3, 2), (3, 2, 1)])
def test_averaged_training_matches_torch(G, steps, period):
    """Groups with different data, averaged every `period` steps (sec. 4):
    the oracle against torch autograd groups and torch means."""
    K, B, lr = 2, 4, 0.3
    (_, ws, bs, pools, fw, fb, _, _), groups = _groups(K, B, G, 300 + G)
    r = OS.averaged_group_training(groups, ws, bs, pools, fw, fb, steps, period, lr)
    t = _torch_averaged_training(groups, ws, bs, fw, fb, steps, period, lr)
    for g in range(G):
        for key in ("conv_w", "conv_b", "fc_w", "fc_b"):
            for a, b in zip(r[g][key], t[g][key]):
                np.testing.assert_allclose(a, b, rtol=1e-10, atol=1e-12)


def test_averaging_schedule_invariants():
    """Averaged steps leave every group with the same model; steps between
    averages let groups with different data drift apart; groups that see
    the same data never differ, so their training is one group's."""
    K, B, lr = 2, 4, 0.3
    (x, ws, bs, pools, fw, fb, remote, labels), groups = _groups(K, B, 2, 77)
    after1 = OS.averaged_group_training(groups, ws, bs, pools, fw, fb, 1, 2, lr)
    after2 = OS.averaged_group_training(groups, ws, bs, pools, fw, fb, 2, 2, lr)
    for key in ("conv_w", "fc_w"):
        assert any(np.abs(a - b).max() > 1e-6 for a, b in zip(after1[0][key], after1[1][key]))
        for a, b in zip(after2[0][key], after2[1][key]):
            np.testing.assert_array_equal(a, b)
    same = [(x, remote, labels)] * 3
    avg = OS.averaged_group_training(same, ws, bs, pools, fw, fb, 2, 1, lr)
    one = OS.group_train_step(x, ws, bs, pools, fw, fb, remote, labels, lr)
    two = OS.group_train_step(x, one["conv_w_new"], one["conv_b_new"], pools, one["fc_w_new"],
                              one["fc_b_new"], remote, labels, lr)
    for g in range(3):
        for a, b in zip(avg[g]["fc_w"], two["fc_w_new"]):
            np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-15)
        for a, b in zip(avg[g]["conv_w"], two["conv_w_new"]):
            np.testing.assert_allclose(a, b, rtol=1e-13, atol=1e-15)
