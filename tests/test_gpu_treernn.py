"""GPU parity of the binary TreeRNN step (janus_treernn_fwd/bwd plus the
5-class softmax cross-entropy at the roots) against the float64 oracle
(oracle/treernn.py), element by element, at the float32 tolerances."""
import numpy as np
import pytest

from oracle import steps as oracle_steps
from paper_1812_01329_amd import workloads as wl
from tests.parity import TOL, check

pytestmark = pytest.mark.gpu


def _run_and_check(w):
    import torch
    from paper_1812_01329_amd.train_step import make_step
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    print(f"[treernn] trees={w.trees.num_trees} nodes={w.trees.num_nodes} H={w.H}", flush=True)
    step = make_step(w)
    step.run()
    g = step.results()
    r = oracle_steps.treernn_step(w)
    t = TOL["f32"]
    check("loss", np.array([g["loss"]]), np.array([r["loss"]]), t["out"])
    check("h_root", g["h_root"], r["h_root"], t["out"])
    for k in ("dh_root", "dWs", "dbs", "dW", "db", "demb"):
        check(k, g[k], r[k], t["grad"])
    return g, r


def test_treernn_sst_fp32():
    """The SST-sized batch: 25 trees of 5-50 leaves, H = 300."""
    _run_and_check(wl.sst_treernn())


def test_treernn_edge_trees():
    """One-leaf trees (a root that is a leaf: h is its word vector and its
    gradient goes straight to the embedding), two-leaf trees, and one deep
    50-leaf tree, in one batch."""
    w = wl.sst_treernn(n_trees=6, H=48, V=40, seed=71, sizes=[1, 2, 50, 1, 3, 17])
    g, r = _run_and_check(w)
    t = w.trees
    for k in (0, 3):   # the one-leaf trees
        word = int(t.word[int(t.root[k])])
        assert np.array_equal(g["h_root"][k], w.emb[word].astype(np.float64))


def test_treernn_wide_hidden():
    """H = 640: the forward contraction's K = 2H = 1280 walks the LDS slab in
    two chunks."""
    _run_and_check(wl.sst_treernn(n_trees=5, H=640, V=64, seed=72))


def test_treernn_only_leaves():
    """A batch of one-leaf trees: no internal level at all, dW and db are 0."""
    w = wl.sst_treernn(n_trees=4, H=32, V=20, seed=73, sizes=[1, 1, 1, 1])
    g, _ = _run_and_check(w)
    assert not g["dW"].any() and not g["db"].any()


def test_treernn_many_leaves():
    """More than 16384 leaves in one batch (700 trees of 25-31 leaves): the
    embedding gradient groups the leaves by word on the host, with no row
    limit."""
    w = wl.sst_treernn(n_trees=700, H=8, V=500, seed=74, min_leaves=25, max_leaves=31)
    assert int((w.trees.left < 0).sum()) > 16384
    _run_and_check(w)
