"""GPU parity of the binary TreeRNN step (janus_treernn_fwd/bwd plus the
5-class softmax cross-entropy at the roots) against the float64 oracle
(oracle/treernn.py), element by element, at the float32 tolerances."""
import numpy as np
import pytest

from oracle import steps as oracle_steps
from paper_1812_01329_amd import workloads as wl
from tests.parity import TOL, check

pytestmark = pytest.mark.gpu


def _run_and_check(w, labels=None):
    import torch
    from paper_1812_01329_amd import janus as J
    from paper_1812_01329_amd.train_step import make_step
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    print(f"[treernn] trees={w.trees.num_trees} nodes={w.trees.num_nodes} H={w.H}", flush=True)
    step = make_step(w)
    J.janus_trace_begin()
    step.run()
    g = step.results()
    if labels is not None:
        labels.update(r["label"] for r in J.janus_trace_end())
    else:
        J.janus_trace_end()
    assert J.janus_treernn_device_report(step.desc, w.trees, step.ws) == 0
    r = oracle_steps.treernn_step(w)
    t = TOL["f32"]
    check("loss", np.array([g["loss"]]), np.array([r["loss"]]), t["out"])
    check("h_root", g["h_root"], r["h_root"], t["out"])
    for k in ("dh_root", "dWs", "dbs", "dW", "db", "demb"):
        check(k, g[k], r[k], t["grad"])
    used = np.zeros(w.V, bool)
    used[w.trees.word[w.trees.word >= 0]] = True
    assert np.all(g["demb"][~used] == 0.0)   # rows of words not in the batch are zero
    # a second step on the same workspace gives the same bits
    step.run()
    g2 = step.results()
    for k in ("h_root", "dW", "db", "demb"):
        assert np.array_equal(g[k], g2[k]), k
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


def _batch(case):
    if case == "sst":
        return wl.sst_treernn()
    if case == "edge":
        return wl.sst_treernn(n_trees=6, H=48, V=40, seed=71, sizes=[1, 2, 50, 1, 3, 17])
    if case == "leaves":
        return wl.sst_treernn(n_trees=4, H=32, V=20, seed=73, sizes=[1, 1, 1, 1])
    if case == "odd":   # H = 29: 2H is not a multiple of 4, partial column tiles
        return wl.sst_treernn(n_trees=9, H=29, V=77, seed=75)
    # H = 304: the widest forward operand slab that fits a CU's LDS
    return wl.sst_treernn(n_trees=12, H=304, V=300, seed=76)


@pytest.mark.parametrize("persist", ["1", "0"])
@pytest.mark.parametrize("case", ["sst", "edge", "leaves", "odd", "wide"])
def test_treernn_persistent_levels(persist, case, monkeypatch):
    """The TreeRNN step with each direction as one persistent launch (a grid
    barrier between levels, fp32 MFMA contractions, dW, db and the embedding
    gradient in the backward's launch) and with the level-by-level kernels
    (JANUS_TREE_PERSIST=0), each against the oracle: the SST-sized batch,
    one-leaf, two-leaf and deep trees, one-leaf trees only, an odd H and the
    widest H the persistent forward takes."""
    monkeypatch.setenv("JANUS_TREE_PERSIST", persist)
    w = _batch(case)
    print(f"[treernn-persist] case={case} persist={persist} N={w.trees.num_nodes}", flush=True)
    labels = set()
    _run_and_check(w, labels)
    if persist == "1":
        assert {"treernn_fwd_persistent", "treernn_bwd_persistent"} <= labels, labels
        assert not labels & {"treernn_level", "treernn_level_bwd", "treernn_dW_gemm"}, labels
    else:
        assert not labels & {"treernn_fwd_persistent", "treernn_bwd_persistent"}, labels


def test_treernn_wide_hidden_runs_levels():
    """H = 640 does not fit the persistent forward's LDS slabs: both
    directions run the level-by-level kernels (checked against the oracle by
    test_treernn_wide_hidden)."""
    from paper_1812_01329_amd import janus as J
    from paper_1812_01329_amd.train_step import make_step
    w = wl.sst_treernn(n_trees=2, H=640, V=64, seed=77)
    step = make_step(w)
    J.janus_trace_begin()
    step.run()
    labels = {r["label"] for r in J.janus_trace_end()}
    assert "treernn_fwd_persistent" not in labels and "treernn_level" in labels, labels

