"""Pins of the Child-Sum TreeLSTM oracle (oracle/childsum.py) against what
does not depend on it: torch autograd in float64 over the same recursion;
chain-shaped trees, where the cell is exactly an LSTM step per node, against
torch.nn.LSTM run from the leaf to the root; central finite differences; and
invariance to the order of each node's children."""
import numpy as np
import pytest
import torch

from oracle import childsum, steps
from paper_1812_01329_amd import workloads as wl


def _small(seed=3, n_trees=4, E=5, H=4, V=30, sizes=None, chain=False):
    return wl.sst_childsum(n_trees=n_trees, E=E, H=H, V=V, min_nodes=1, max_nodes=9, seed=seed, sizes=sizes,
                           chain=chain)


def _torch_step(w):
    t = w.trees
    f64 = dict(dtype=torch.float64)
    emb = torch.tensor(w.emb, requires_grad=True, **f64)
    W = torch.tensor(w.W, requires_grad=True, **f64)
    U = torch.tensor(w.U, requires_grad=True, **f64)
    b = torch.tensor(w.b, requires_grad=True, **f64)
    H = w.H

    def visit(n):
        kids = [int(c) for c in t.children[int(t.child_offsets[n]):int(t.child_offsets[n + 1])]]
        res = [visit(k) for k in kids]
        a = W @ emb[int(t.word[n])] + b
        ht = sum((r[0] for r in res), torch.zeros(H, **f64))
        z = U[:3 * H] @ ht
        i, o, u = torch.sigmoid(a[:H] + z[:H]), torch.sigmoid(a[H:2 * H] + z[H:2 * H]), torch.tanh(a[2 * H:3 * H] + z[2 * H:])
        c = i * u
        for hk, ck in res:
            c = c + torch.sigmoid(a[3 * H:] + U[3 * H:] @ hk) * ck
        return o * torch.tanh(c), c

    roots = torch.stack([visit(int(r))[0] for r in t.root])
    logits = roots @ torch.tensor(w.Ws, **f64).T + torch.tensor(w.bs, **f64)
    loss = torch.nn.functional.cross_entropy(logits, torch.tensor(w.labels, dtype=torch.int64))
    loss.backward()
    return float(loss.detach()), roots.detach().numpy(), emb.grad.numpy(), W.grad.numpy(), U.grad.numpy(), b.grad.numpy()


@pytest.mark.parametrize("seed", [3, 4, 5])
def test_matches_torch_autograd(seed):
    w = _small(seed)
    r = steps.childsum_step(w)
    loss, roots, demb, dW, dU, db = _torch_step(w)
    assert r["loss"] == pytest.approx(loss, rel=1e-13)
    np.testing.assert_allclose(r["h_root"], roots, rtol=0, atol=1e-14)
    for got, ref in ((r["demb"], demb), (r["dW"], dW), (r["dU"], dU), (r["db"], db)):
        np.testing.assert_allclose(got, ref, rtol=0, atol=1e-13)


def test_chain_is_an_lstm():
    """A chain (every node has one child) is an LSTM over its nodes from the
    leaf up; torch's gate blocks are (i, f, g, o), these are (i, o, u, f)."""
    w = _small(6, n_trees=2, sizes=[7, 4], chain=True)
    h_root, _ = childsum.forward_recursive(w.trees, w.emb, w.W, w.U, w.b)
    H = w.H
    perm = np.concatenate([np.arange(0, H), np.arange(3 * H, 4 * H), np.arange(2 * H, 3 * H), np.arange(H, 2 * H)])
    lstm = torch.nn.LSTM(w.E_dim, H).double()
    with torch.no_grad():
        lstm.weight_ih_l0.copy_(torch.tensor(w.W[perm], dtype=torch.float64))
        lstm.weight_hh_l0.copy_(torch.tensor(w.U[perm], dtype=torch.float64))
        lstm.bias_ih_l0.copy_(torch.tensor(w.b[perm], dtype=torch.float64))
        lstm.bias_hh_l0.zero_()
    t = w.trees
    for k, root in enumerate(t.root):
        nodes, n = [], int(root)
        while True:
            nodes.append(n)
            kids = t.children[int(t.child_offsets[n]):int(t.child_offsets[n + 1])]
            if len(kids) == 0:
                break
            n = int(kids[0])
        x = torch.tensor(np.stack([w.emb[int(t.word[m])] for m in reversed(nodes)]), dtype=torch.float64)
        y, _ = lstm(x[:, None, :])
        np.testing.assert_allclose(h_root[k], y[-1, 0].detach().numpy(), rtol=0, atol=1e-14)


def test_finite_differences():
    w = _small(7, n_trees=3, E=3, H=3, V=12)
    w.W, w.U, w.b, w.emb = (np.asarray(a, np.float64) for a in (w.W, w.U, w.b, w.emb))
    r = steps.childsum_step(w)
    rng = np.random.default_rng(1)
    for name, grad in (("W", r["dW"]), ("U", r["dU"]), ("b", r["db"]), ("emb", r["demb"])):
        arr = getattr(w, name)
        for _ in range(6):
            idx = tuple(int(rng.integers(0, s)) for s in arr.shape)
            saved = arr[idx]
            arr[idx] = saved + 1e-6
            lp = steps.childsum_step(w)["loss"]
            arr[idx] = saved - 1e-6
            lm = steps.childsum_step(w)["loss"]
            arr[idx] = saved
            assert (lp - lm) / 2e-6 == pytest.approx(grad[idx], abs=1e-7)


def test_child_order_does_not_matter():
    w = _small(8)
    t = w.trees
    rng = np.random.default_rng(2)
    kids = t.children.copy()
    for n in range(t.num_nodes):
        a, b = int(t.child_offsets[n]), int(t.child_offsets[n + 1])
        kids[a:b] = rng.permutation(kids[a:b])
    t2 = wl.NaryTreeBatch(t.child_offsets, kids, t.word, t.root)
    h1, _ = childsum.forward_recursive(t, w.emb, w.W, w.U, w.b)
    h2, _ = childsum.forward_recursive(t2, w.emb, w.W, w.U, w.b)
    np.testing.assert_allclose(h1, h2, rtol=0, atol=1e-15)
