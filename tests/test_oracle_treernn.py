"""Pins of the TreeRNN oracle (oracle/treernn.py) against what does not
depend on it: torch autograd in float64 over the same recursion (gradients),
central finite differences of the loss, a one-leaf tree (h = its word
vector), a two-leaf tree against torch's linear layer and tanh, and the
symmetry of swapping every node's children together with W's two column
blocks."""
import numpy as np
import pytest
import torch

from oracle import heads, steps, treernn
from paper_1812_01329_amd import workloads as wl


def _small(seed=3, n_trees=4, H=6, V=30, sizes=None):
    return wl.sst_treernn(n_trees=n_trees, H=H, V=V, min_leaves=1, max_leaves=7, seed=seed, sizes=sizes)


def _torch_loss(w, emb, W, b):
    t = w.trees
    memo = {}

    def visit(n):
        l, r = int(t.left[n]), int(t.right[n])
        if l < 0:
            v = emb[int(t.word[n])]
        else:
            v = torch.tanh(W @ torch.cat([visit(l), visit(r)]) + b)
        memo[n] = v
        return v

    roots = torch.stack([visit(int(r)) for r in t.root])
    logits = roots @ torch.tensor(w.Ws, dtype=torch.float64).T + torch.tensor(w.bs, dtype=torch.float64)
    return torch.nn.functional.cross_entropy(logits, torch.tensor(w.labels, dtype=torch.int64)), roots


@pytest.mark.parametrize("seed", [3, 4])
def test_gradients_match_torch_autograd(seed):
    w = _small(seed)
    r = steps.treernn_step(w)
    emb = torch.tensor(w.emb, dtype=torch.float64, requires_grad=True)
    W = torch.tensor(w.W, dtype=torch.float64, requires_grad=True)
    b = torch.tensor(w.b, dtype=torch.float64, requires_grad=True)
    loss, roots = _torch_loss(w, emb, W, b)
    loss.backward()
    assert r["loss"] == pytest.approx(float(loss.detach()), rel=1e-13)
    np.testing.assert_allclose(r["h_root"], roots.detach().numpy(), rtol=0, atol=1e-14)
    np.testing.assert_allclose(r["demb"], emb.grad.numpy(), rtol=0, atol=1e-13)
    np.testing.assert_allclose(r["dW"], W.grad.numpy(), rtol=0, atol=1e-13)
    np.testing.assert_allclose(r["db"], b.grad.numpy(), rtol=0, atol=1e-13)


def test_finite_differences():
    w = _small(5, n_trees=3, H=4, V=12)
    # perturb in float64: a float32 array would quantize the step
    w.W, w.b, w.emb = (np.asarray(a, np.float64) for a in (w.W, w.b, w.emb))
    r = steps.treernn_step(w)
    rng = np.random.default_rng(0)
    for name, grad in (("W", r["dW"]), ("b", r["db"]), ("emb", r["demb"])):
        for _ in range(6):
            arr = getattr(w, name)
            idx = tuple(int(rng.integers(0, s)) for s in arr.shape)
            eps = 1e-6
            saved = arr[idx]
            arr[idx] = saved + eps
            lp = steps.treernn_step(w)["loss"]
            arr[idx] = saved - eps
            lm = steps.treernn_step(w)["loss"]
            arr[idx] = saved
            assert (lp - lm) / (2 * eps) == pytest.approx(grad[idx], abs=1e-7)


def test_one_leaf_tree_is_its_word_vector():
    w = _small(6, n_trees=2, sizes=[1, 1])
    h_root, _ = treernn.forward_recursive(w.trees, w.emb, w.W, w.b)
    for k in range(2):
        assert np.array_equal(h_root[k], np.asarray(w.emb[int(w.trees.word[int(w.trees.root[k])])], np.float64))


def test_two_leaf_tree_against_torch_linear():
    w = _small(7, n_trees=1, sizes=[2])
    t = w.trees
    root = int(t.root[0])
    l, r = int(t.left[root]), int(t.right[root])
    x = torch.tensor(np.concatenate([w.emb[int(t.word[l])], w.emb[int(t.word[r])]]), dtype=torch.float64)
    ref = torch.tanh(torch.nn.functional.linear(x, torch.tensor(w.W, dtype=torch.float64),
                                                torch.tensor(w.b, dtype=torch.float64)))
    h_root, _ = treernn.forward_recursive(t, w.emb, w.W, w.b)
    np.testing.assert_allclose(h_root[0], ref.numpy(), rtol=0, atol=1e-15)


def test_children_swap_symmetry():
    w = _small(8)
    t = w.trees
    swapped = wl.TreeBatch(left=t.right.copy(), right=t.left.copy(), word=t.word, root=t.root)
    H = w.H
    W2 = np.concatenate([w.W[:, H:], w.W[:, :H]], axis=1)
    a, _ = treernn.forward_recursive(t, w.emb, w.W, w.b)
    c, _ = treernn.forward_recursive(swapped, w.emb, W2, w.b)
    np.testing.assert_allclose(a, c, rtol=0, atol=1e-15)
