"""GPU parity of the Child-Sum TreeLSTM step (janus_childsum_fwd/bwd plus the
5-class softmax cross-entropy at the roots) against the float64 oracle
(oracle/childsum.py), element by element, at the float32 tolerances."""
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
    t = w.trees
    print(f"[childsum] trees={t.num_trees} nodes={t.num_nodes} E={w.E_dim} H={w.H}", flush=True)
    step = make_step(w)
    J.janus_trace_begin()
    step.run()
    g = step.results()
    traced = J.janus_trace_end()
    if labels is not None:
        labels.update(r["label"] for r in traced)
    assert J.janus_childsum_device_report(step.desc, t, step.ws) == 0
    r = oracle_steps.childsum_step(w)
    tol = TOL["f32"]
    check("loss", np.array([g["loss"]]), np.array([r["loss"]]), tol["out"])
    check("h_root", g["h_root"], r["h_root"], tol["out"])
    for k in ("dh_root", "dWs", "dbs", "dW", "dU", "db", "demb"):
        check(k, g[k], r[k], tol["grad"])
    used = np.zeros(w.V, bool)
    used[np.asarray(t.word)] = True
    assert np.all(g["demb"][~used] == 0.0)   # rows of words not in the batch are zero
    # a second step on the same workspace gives the same bits
    step.run()
    g2 = step.results()
    for k in ("h_root", "dW", "dU", "db", "demb"):
        assert np.array_equal(g[k], g2[k]), k
    return g, r


def test_childsum_sst_fp32():
    """25 random trees of 5-50 nodes, a word at every node, E 300, H 150:
    the dh contraction's K = 4H = 600, the weight contractions' K = the node
    count."""
    _run_and_check(wl.sst_childsum())


def test_childsum_chains_stars_and_single_nodes():
    """Chains (one child per node, 40 levels), a star (one root over 40
    leaves: one level of 40 children), and single-node trees in one batch."""
    ch = wl.sst_childsum(n_trees=2, E=24, H=32, V=50, seed=81, sizes=[40, 3], chain=True).trees
    rt = wl.sst_childsum(n_trees=3, E=24, H=32, V=50, seed=82, sizes=[41, 1, 1]).trees
    # make the first tree of rt a star: every node under the root
    n = 41
    kids = list(range(1, n))
    off = [0, n - 1] + [n - 1] * (n - 1) + [n - 1 + 0, n - 1 + 0]
    star = wl.NaryTreeBatch(np.asarray(off, np.int32), np.asarray(kids, np.int32), rt.word, rt.root)
    # concatenate the chain batch after the star batch
    base = star.num_nodes
    off2 = np.concatenate([star.child_offsets[:-1], ch.child_offsets + star.child_offsets[-1]]).astype(np.int32)
    trees = wl.NaryTreeBatch(off2, np.concatenate([star.children, ch.children + base]).astype(np.int32),
                             np.concatenate([star.word, ch.word]).astype(np.int32),
                             np.concatenate([star.root, ch.root + base]).astype(np.int32))
    w = wl.sst_childsum(n_trees=5, E=24, H=32, V=50, seed=83, sizes=[1, 1, 1, 1, 1])
    labels = np.arange(trees.num_trees, dtype=np.int32) % w.C
    w = wl.ChildSumWorkload("childsum-edges", w.E_dim, w.H, w.V, w.C, trees, labels, w.emb, w.W, w.U, w.b,
                            w.Ws, w.bs)
    _run_and_check(w)


def test_childsum_wide_hidden():
    """H = 320: the level contraction's N = 4H = 1280 columns in 20 blocks,
    the dh contraction's K = 1280 in two LDS chunks."""
    _run_and_check(wl.sst_childsum(n_trees=5, E=40, H=320, V=64, seed=84))


def test_childsum_many_nodes():
    """More than 16384 nodes, each with a word (520 trees of 35-45 nodes):
    the embedding gradient has no row limit."""
    w = wl.sst_childsum(n_trees=520, E=8, H=8, V=300, min_nodes=35, max_nodes=45, seed=75)
    assert w.trees.num_nodes > 16384
    _run_and_check(w)


def _with_star(w, k):
    """The batch of w with a tree of one root over k leaves put first."""
    t = w.trees
    n = k + 1
    off = np.asarray([0, k] + [k] * k, np.int32)          # node 0 is the root, nodes 1..k its leaves
    rng = np.random.default_rng(k)
    off2 = np.concatenate([off, t.child_offsets[1:] + k]).astype(np.int32)
    kids = np.concatenate([np.arange(1, n, dtype=np.int32), t.children + n]).astype(np.int32)
    word = np.concatenate([rng.integers(0, w.V, n), t.word]).astype(np.int32)
    root = np.concatenate([[0], t.root + n]).astype(np.int32)
    trees = wl.NaryTreeBatch(off2, kids, word, root)
    labels = np.arange(trees.num_trees, dtype=np.int32) % w.C
    return wl.ChildSumWorkload(w.name + "-star", w.E_dim, w.H, w.V, w.C, trees, labels, w.emb, w.W, w.U, w.b,
                               w.Ws, w.bs)


def _cs_batch(case):
    if case == "sst":
        return wl.sst_childsum()
    if case == "chains":   # a 40-node chain and a 3-node chain: one level per node
        return wl.sst_childsum(n_trees=2, E=24, H=32, V=50, seed=81, sizes=[40, 3], chain=True)
    if case == "singles":  # one-node trees only: a single level, no child
        return wl.sst_childsum(n_trees=5, E=24, H=32, V=50, seed=83, sizes=[1, 1, 1, 1, 1])
    if case == "odd":      # E = 37, H = 29: partial column tiles, scalar staging
        return wl.sst_childsum(n_trees=7, E=37, H=29, V=61, seed=85)
    if case == "bigstar":  # a root over 600 leaves beside ordinary trees: a node with 600 children
        return _with_star(wl.sst_childsum(n_trees=6, E=24, H=32, V=50, seed=87), 600)
    # H = 156: the widest the persistent backward takes (two 32 x 4H slabs in LDS)
    return wl.sst_childsum(n_trees=9, E=300, H=156, V=300, seed=86)


@pytest.mark.parametrize("persist", ["1", "0"])
@pytest.mark.parametrize("case", ["sst", "chains", "singles", "odd", "bigstar", "wide"])
def test_childsum_persistent_levels(persist, case, monkeypatch):
    """The Child-Sum step with each direction as one persistent launch (device
    barriers between the levels' cells and contractions, fp32 MFMA tiles) and
    with the level-by-level kernels (JANUS_TREE_PERSIST=0), each against the
    oracle: the SST-sized batch, chains, one-node trees, odd sizes, a root
    over 600 leaves beside ordinary trees (one level holds a node with 600
    children), and the widest H the persistent backward takes."""
    monkeypatch.setenv("JANUS_TREE_PERSIST", persist)
    w = _cs_batch(case)
    print(f"[childsum-persist] case={case} persist={persist} N={w.trees.num_nodes}", flush=True)
    labels = set()
    _run_and_check(w, labels)
    if persist == "1":
        assert {"childsum_fwd_persistent", "childsum_bwd_persistent"} <= labels, labels
        assert not labels & {"childsum_fwd_cell", "childsum_bwd_cell", "childsum_level_gemm"}, labels
    else:
        assert not labels & {"childsum_fwd_persistent", "childsum_bwd_persistent"}, labels


def test_childsum_wide_hidden_runs_levels():
    """H = 320 does not fit the persistent backward's LDS slabs: both
    directions run the level-by-level kernels (checked against the oracle by
    test_childsum_wide_hidden)."""
    from paper_1812_01329_amd import janus as J
    from paper_1812_01329_amd.train_step import make_step
    w = wl.sst_childsum(n_trees=2, E=40, H=320, V=64, seed=87)
    step = make_step(w)
    J.janus_trace_begin()
    step.run()
    labels = {r["label"] for r in J.janus_trace_end()}
    assert "childsum_fwd_persistent" not in labels and "childsum_fwd_cell" in labels, labels

