"""Pins of the TreeLSTM oracle: finite differences, brute force (recursive
evaluation equals a level-by-level evaluation bit for bit), closed forms on
hand-built trees, and invariants."""
import copy

import numpy as np
import pytest

from oracle import schedule, steps, treelstm
from paper_1812_01329_amd import workloads as wl


def build(spec, words_iter):
    """Build a TreeBatch from nested tuples: a leaf is None, an internal node
    is (left, right).  Post-order numbering, trees concatenated."""
    left, right, word, roots = [], [], [], []

    def rec(s):
        if s is None:
            left.append(-1); right.append(-1); word.append(next(words_iter))
            return len(left) - 1
        l = rec(s[0]); r = rec(s[1])
        left.append(l); right.append(r); word.append(-1)
        return len(left) - 1

    for s in spec:
        roots.append(rec(s))
    return wl.TreeBatch(np.asarray(left, np.int32), np.asarray(right, np.int32),
                        np.asarray(word, np.int32), np.asarray(roots, np.int32))


LEAF = None
CHAIN_L = (((((LEAF, LEAF), LEAF), LEAF), LEAF), LEAF)
CHAIN_R = (LEAF, (LEAF, (LEAF, (LEAF, (LEAF, LEAF)))))
BAL8 = (((LEAF, LEAF), (LEAF, LEAF)), ((LEAF, LEAF), (LEAF, LEAF)))
HAND_BUILT = [[LEAF], [(LEAF, LEAF)], [((LEAF, LEAF), LEAF)], [(LEAF, (LEAF, LEAF))],
              [CHAIN_L], [CHAIN_R], [BAL8], [BAL8, LEAF, CHAIN_L, (LEAF, LEAF)]]


def small_tree(spec, E=3, H=2, V=7, C=3, seed=0, scale=0.8):
    rng = np.random.default_rng(seed)
    trees = build(spec, iter(rng.integers(0, V, 1000).tolist()))
    return wl.TreeWorkload("t", E, H, V, C, trees, rng.integers(0, C, trees.num_trees).astype(np.int32),
                           rng.uniform(-1, 1, (V, E)), rng.uniform(-scale, scale, (5 * H, E)),
                           rng.uniform(-scale, scale, (5 * H, 2 * H)), rng.uniform(-scale, scale, 5 * H),
                           rng.uniform(-1, 1, (C, H)), rng.uniform(-1, 1, C))


@pytest.mark.parametrize("spec", HAND_BUILT)
def test_recursive_equals_levelwise_bitwise(spec):
    w = small_tree(spec, E=4, H=3)
    hr, st = treelstm.forward_recursive(w.trees, w.emb, w.W, w.U, w.b)
    _, off, order, _ = schedule.tree_schedule(w.trees.left, w.trees.right, w.trees.word, w.trees.root, w.V)
    hl, sl = treelstm.forward_by_levels(w.trees, w.emb, w.W, w.U, w.b, order, off)
    assert np.array_equal(hr, hl)
    assert np.array_equal(st.h, sl.h) and np.array_equal(st.c, sl.c)


def test_recursive_equals_levelwise_random_batch():
    w = wl.sst_treelstm(n_trees=6, E=5, H=4, V=50, seed=11)
    hr, st = treelstm.forward_recursive(w.trees, w.emb, w.W, w.U, w.b)
    _, off, order, _ = schedule.tree_schedule(w.trees.left, w.trees.right, w.trees.word, w.trees.root, w.V)
    hl, sl = treelstm.forward_by_levels(w.trees, w.emb, w.W, w.U, w.b, order, off)
    assert np.array_equal(hr, hl) and np.array_equal(st.c, sl.c)


@pytest.mark.parametrize("spec", HAND_BUILT[:7])
def test_finite_differences(spec):
    w = small_tree(spec)
    base = steps.tree_step(w)
    eps = 1e-5
    for name, key in (("W", "dW"), ("U", "dU"), ("b", "db"), ("emb", "demb"), ("Ws", "dWs"), ("bs", "dbs")):
        arr = getattr(w, name)
        fd = np.zeros(arr.shape)
        flat = arr.reshape(-1)
        for k in range(flat.size):
            old = flat[k]
            flat[k] = old + eps; lp = steps.tree_step(w)["loss"]
            flat[k] = old - eps; lm = steps.tree_step(w)["loss"]
            flat[k] = old
            fd.reshape(-1)[k] = (lp - lm) / (2 * eps)
        an = base[key]
        err = np.abs(fd - an).max() / max(np.abs(an).max(), 1e-30)
        assert err < 1e-6, (name, err)


def test_closed_form_perfect_trees():
    """W = U = 0, b = 0 except b_u = beta: every gate is 1/2, a leaf has
    c = tanh(beta)/2 and a node c = tanh(beta)/2 + (c_L + c_R)/2, so the root
    of a perfect tree of height k has c = (k + 1) tanh(beta) / 2."""
    beta, H, E = 0.7, 3, 2
    for k, spec in enumerate([LEAF, (LEAF, LEAF), ((LEAF, LEAF), (LEAF, LEAF)), BAL8]):
        w = small_tree([spec], E=E, H=H)
        b = np.zeros(5 * H); b[4 * H:] = beta
        hr, st = treelstm.forward_recursive(w.trees, w.emb, np.zeros((5 * H, E)), np.zeros((5 * H, 2 * H)), b)
        c = (k + 1) * np.tanh(beta) / 2
        np.testing.assert_allclose(st.c[w.trees.root[0]], c, atol=1e-15)
        np.testing.assert_allclose(hr[0], 0.5 * np.tanh(c), atol=1e-15)


def test_closed_form_left_forget_gate_follows_left_child():
    """W = U = 0; f_L saturated open (b = 40), f_R shut (b = -40): the cell
    memory of a node is s(b_i) tanh(b_u) times the number of nodes on its
    leftmost path, and h = s(b_o) tanh(c).  Pins which child each forget gate
    reads and the order of the gate blocks."""
    H, E = 2, 2
    bi, bo, bu = 0.3, -0.6, 0.9
    b = np.concatenate([np.full(H, v) for v in (bi, 40.0, -40.0, bo, bu)])
    s = lambda z: 1 / (1 + np.exp(-z))
    unit = s(bi) * np.tanh(bu)
    for spec, m in ((CHAIN_L, 6), (CHAIN_R, 2), (BAL8, 4), ((LEAF, CHAIN_L), 2), ((CHAIN_L, LEAF), 7)):
        w = small_tree([spec], E=E, H=H)
        hr, st = treelstm.forward_recursive(w.trees, w.emb, np.zeros((5 * H, E)), np.zeros((5 * H, 2 * H)), b)
        np.testing.assert_allclose(st.c[w.trees.root[0]], m * unit, atol=1e-12)
        np.testing.assert_allclose(hr[0], s(bo) * np.tanh(m * unit), atol=1e-12)


def test_one_leaf_tree_is_one_cell_step():
    """A one-leaf tree: a = W x + b, c = s(a_i) tanh(a_u), h = s(a_o) tanh(c),
    evaluated elementwise."""
    w = small_tree([LEAF], E=4, H=3)
    hr, st = treelstm.forward_recursive(w.trees, w.emb, w.W, w.U, w.b)
    x = w.emb[w.trees.word[0]]
    H = 3
    for j in range(H):
        a = [w.b[g * H + j] + sum(w.W[g * H + j, k] * x[k] for k in range(4)) for g in range(5)]
        c = 1 / (1 + np.exp(-a[0])) * np.tanh(a[4])
        assert abs(st.c[0, j] - c) < 1e-15
        assert abs(hr[0, j] - 1 / (1 + np.exp(-a[3])) * np.tanh(c)) < 1e-15


def test_forget_rows_of_W_get_zero_gradient():
    """Only leaves read W and their children's memory is 0, so the f_L and
    f_R rows of dW are exactly zero."""
    w = wl.sst_treelstm(n_trees=4, E=6, H=5, V=30, seed=3)
    r = steps.tree_step(w)
    H = 5
    assert np.all(r["dW"][H:3 * H] == 0)
    assert np.abs(r["dW"][:H]).max() > 0


def test_node_numbering_invariance():
    """Renumbering the nodes (and remapping child ids) changes nothing."""
    w = wl.sst_treelstm(n_trees=3, E=4, H=3, V=20, seed=5)
    r0 = steps.tree_step(w)
    N = w.trees.num_nodes
    p = np.random.default_rng(0).permutation(N)       # new id of old node n is p[n]
    inv = np.argsort(p)
    t = w.trees
    remap = lambda a: np.where(a >= 0, p[np.maximum(a, 0)], -1).astype(np.int32)
    w2 = copy.deepcopy(w)
    w2.trees = wl.TreeBatch(remap(t.left)[inv], remap(t.right)[inv], t.word[inv], p[t.root].astype(np.int32))
    r1 = steps.tree_step(w2)
    np.testing.assert_allclose(r1["h_root"], r0["h_root"], atol=1e-15)
    for k in ("dW", "dU", "db", "demb"):
        np.testing.assert_allclose(r1[k], r0[k], atol=1e-14)
