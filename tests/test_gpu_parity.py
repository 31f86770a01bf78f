"""GPU parity: the HIP path through the C ABI against the float64 oracle on
the same seeded inputs, element by element, at the path's tolerances."""
import sys

import numpy as np
import pytest

from oracle import steps as oracle_steps
from paper_1812_01329_amd import workloads as wl
from tests.parity import TOL, check, compare_lstm

pytestmark = pytest.mark.gpu


def _run(w):
    import torch
    from paper_1812_01329_amd.train_step import make_step
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    print(f"[parity] {w.name} dtype={w.dtype}", flush=True)
    step = make_step(w)
    step.run()
    return step, step.results()


def _lstm(head, dtype, L, I, H, B, T, lengths=None, seed=0, h0=False, V=50, P=24, scale=None):
    rng = np.random.default_rng(seed)
    a = scale if scale is not None else 1.0 / np.sqrt(H)
    rnd = lambda shape, s: wl.bf16_round(rng.uniform(-s, s, shape).astype(np.float32)) if dtype == "bf16" \
        else rng.uniform(-s, s, shape).astype(np.float32)
    Wx = [rnd((4 * H, I if l == 0 else H), a) for l in range(L)]
    Wh = [rnd((4 * H, H), a) for l in range(L)]
    b = [rnd((4 * H,), a) for l in range(L)]
    x = rnd((T, B, I), 1.0)
    w = wl.LSTMWorkload(f"lstm-{head}-{dtype}-L{L}I{I}H{H}B{B}T{T}", dtype, L, I, H, B, T, x,
                        None if lengths is None else np.asarray(lengths, np.int32), Wx, Wh, b, head)
    if head == "xent":
        w.V = V
        w.tokens = rng.integers(0, V, (B, T + 1)).astype(np.int32)
        w.E = rnd((V, I), 0.5)
        w.Wout = rnd((V, H), 0.5)
        w.bout = rnd((V,), 0.5)
        w.x = None
    if head == "mse":
        w.Wout = rnd((P, H), a)
        w.bout = rnd((P,), a)
        w.target = rnd((T, B, P), 1.0)
    if h0:
        w.h0 = rng.uniform(-0.5, 0.5, (L, B, H)).astype(np.float32)
        w.c0 = rng.uniform(-0.5, 0.5, (L, B, H)).astype(np.float32)
    return w


# ---------------------------------------------------------------- the five workloads
def test_tiny_fixed_length_fp32():
    w = wl.tiny_lstm()
    _, g = _run(w)
    compare_lstm(g, oracle_steps.lstm_step(w), "f32")


def test_ptb_language_model_bf16():
    w = wl.ptb_lstm()
    _, g = _run(w)
    r = oracle_steps.lstm_step(w)
    compare_lstm(g, r, "bf16", with_dx=False)


def test_varlen_masked_loop_bf16():
    w = wl.varlen_lstm()
    _, g = _run(w)
    r = oracle_steps.lstm_step(w)
    compare_lstm(g, r, "bf16")
    # positions past each sequence's end are exactly zero
    T = w.T
    mask = np.arange(T)[:, None] >= w.lengths[None, :]
    assert np.all(g["y"][mask] == 0.0)
    assert np.all(g["dx"][mask] == 0.0)


def test_treelstm_fp32():
    w = wl.sst_treelstm()
    _, g = _run(w)
    r = oracle_steps.tree_step(w)
    t = TOL["f32"]
    check("loss", np.array([g["loss"]]), np.array([r["loss"]]), t["out"])
    check("h_root", g["h_root"], r["h_root"], t["out"])
    for k in ("dh_root", "dWs", "dbs", "dW", "dU", "db", "demb"):
        check(k, g[k], r[k], t["grad"])
    H = w.H
    assert np.all(g["dW"][H:3 * H] == 0.0)   # forget rows of W see no gradient


def test_treelstm_wide_hidden_fp32():
    """H = 240: the five gate blocks (5H = 1200) exceed one LDS slab of the
    fused backward level kernel, so the levels take the separate pointwise
    kernel and contraction, and the contractions walk K in two chunks."""
    w = wl.sst_treelstm(n_trees=6, E=40, H=240, V=64, seed=13)
    _, g = _run(w)
    r = oracle_steps.tree_step(w)
    t = TOL["f32"]
    check("loss", np.array([g["loss"]]), np.array([r["loss"]]), t["out"])
    check("h_root", g["h_root"], r["h_root"], t["out"])
    for k in ("dh_root", "dW", "dU", "db", "demb"):
        check(k, g[k], r[k], t["grad"])


def test_treelstm_many_leaves_fp32():
    """More than 16384 leaves in one batch (700 trees of 25-31 leaves): the
    embedding gradient groups the leaves by word on the host, with no row
    limit."""
    w = wl.sst_treelstm(n_trees=700, E=8, H=8, V=500, min_leaves=25, max_leaves=31, seed=14)
    assert int((w.trees.left < 0).sum()) > 16384
    _, g = _run(w)
    r = oracle_steps.tree_step(w)
    t = TOL["f32"]
    check("h_root", g["h_root"], r["h_root"], t["out"])
    for k in ("dW", "dU", "db", "demb"):
        check(k, g[k], r[k], t["grad"])


def _chain_and_leaf_batch():
    """A one-leaf tree, a left chain of 12 leaves and a balanced 16-leaf tree."""
    left, right, word, roots = [], [], [], []
    rng = np.random.default_rng(1)
    roots.append(wl.random_bracketing(rng, 1, np.array([3]), left, right, word))
    prev = None
    for k in range(12):
        left.append(-1); right.append(-1); word.append(int(rng.integers(0, 40)))
        leaf = len(left) - 1
        if prev is None:
            prev = leaf
        else:
            left.append(prev); right.append(leaf); word.append(-1)
            prev = len(left) - 1
    roots.append(prev)
    roots.append(wl.random_bracketing(rng, 16, rng.integers(0, 40, 16), left, right, word))
    trees = wl.TreeBatch(np.asarray(left, np.int32), np.asarray(right, np.int32), np.asarray(word, np.int32),
                         np.asarray(roots, np.int32))
    base = wl.sst_treelstm(n_trees=2, E=24, H=20, V=40, seed=9)
    base.trees = trees
    base.labels = rng.integers(0, base.C, trees.num_trees).astype(np.int32)
    return base


def _leaves_only_batch():
    """Seven trees of one leaf each: a single level, no internal node."""
    base = wl.sst_treelstm(n_trees=2, E=24, H=20, V=40, seed=10)
    n = 7
    base.trees = wl.TreeBatch(np.full(n, -1, np.int32), np.full(n, -1, np.int32),
                              np.arange(3, 3 + n, dtype=np.int32) * 5 % 40, np.arange(n, dtype=np.int32))
    base.labels = np.random.default_rng(10).integers(0, base.C, n).astype(np.int32)
    return base


@pytest.mark.parametrize("persist", ["1", "0"])
@pytest.mark.parametrize("case", ["sst", "chains", "leaves", "odd", "wide"])
def test_treelstm_persistent_levels(persist, case, monkeypatch):
    """The TreeLSTM step with each direction as one persistent launch (a
    grid barrier between levels, fp32 MFMA contractions) and with the
    level-by-level kernels (JANUS_TREE_PERSIST=0), each against the oracle:
    the SST-sized batch, a one-leaf tree with a 12-leaf chain and a balanced
    tree, a batch of one-leaf trees only, odd sizes (E = 37, H = 29:
    partial unit groups and column tiles), and H = 184 over 120 trees (six
    32-unit chunks per row, the last partial, the backward's widest LDS
    layout, and levels of more 16-row tiles than a column tile has
    workgroups)."""
    from paper_1812_01329_amd import janus as J
    monkeypatch.setenv("JANUS_TREE_PERSIST", persist)
    if case == "sst":
        w = wl.sst_treelstm()
    elif case == "chains":
        w = _chain_and_leaf_batch()
    elif case == "leaves":
        w = _leaves_only_batch()
    elif case == "odd":
        w = wl.sst_treelstm(n_trees=9, E=37, H=29, V=77, seed=15)
    else:
        w = wl.sst_treelstm(n_trees=120, E=32, H=184, V=90, seed=16)
    print(f"[tree-persist] case={case} persist={persist} N={w.trees.num_nodes}", flush=True)
    J.janus_trace_begin()
    step, g = _run(w)
    labels = {r["label"] for r in J.janus_trace_end()}
    if persist == "1":
        assert {"treelstm_fwd_persistent", "treelstm_bwd_persistent"} <= labels, labels
        assert not labels & {"tree_level_gemm", "tree_fwd_point", "tree_bwd_level"}, labels
    else:
        assert "treelstm_fwd_persistent" not in labels, labels
    assert J.janus_treelstm_device_report(step.desc, w.trees, step.ws) == 0
    r = oracle_steps.tree_step(w)
    t = TOL["f32"]
    check("loss", np.array([g["loss"]]), np.array([r["loss"]]), t["out"])
    check("h_root", g["h_root"], r["h_root"], t["out"])
    for k in ("dh_root", "dWs", "dbs", "dW", "dU", "db", "demb"):
        check(k, g[k], r[k], t["grad"])
    H = w.H
    assert np.all(g["dW"][H:3 * H] == 0.0)   # forget rows of W see no gradient
    used = np.zeros(w.V, bool)
    used[w.trees.word[w.trees.word >= 0]] = True
    assert np.all(g["demb"][~used] == 0.0)   # rows of words not in the batch are zero
    # a second step on the same workspace gives the same bits
    step.run()
    g2 = step.results()
    for k in ("h_root", "dW", "dU", "db", "demb"):
        assert np.array_equal(g[k], g2[k]), k


def test_lm2048_reduced_shape_bf16():
    """The regression workload's structure (2 layers, projection + MSE) at a
    shape the oracle runs in seconds, spanning several tiles with ragged tails."""
    w = wl.lm2048_lstm(T=12, B=70, H=200, I=136, P=72)
    _, g = _run(w)
    compare_lstm(g, oracle_steps.lstm_step(w), "bf16", with_dx=False)


# ---------------------------------------------------------------- edge cases
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("head,lengths", [
    ("sumsq", None),
    ("mean_final", [7, 0, 3, 7, 1]),
    ("mse", [1, 1, 1, 1, 1]),
    ("sumsq", [0, 0, 0, 0, 0]),
    ("xent", None),
])
def test_ragged_shapes(dtype, head, lengths):
    w = _lstm(head, dtype, L=2, I=13, H=37, B=5, T=7, lengths=lengths, seed=7, h0=(head != "xent"))
    _, g = _run(w)
    compare_lstm(g, oracle_steps.lstm_step(w), dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_multi_tile_varlen(dtype):
    """Rows and hidden units spanning several tiles, with a ragged tail."""
    rng = np.random.default_rng(3)
    lengths = rng.integers(0, 20, 150)
    w = _lstm("mean_final", dtype, L=2, I=72, H=104, B=150, T=19, lengths=lengths, seed=3, h0=True)
    _, g = _run(w)
    compare_lstm(g, oracle_steps.lstm_step(w), dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_one_step_sequences(dtype):
    w = _lstm("sumsq", dtype, L=1, I=8, H=16, B=3, T=1, seed=5, h0=True)
    _, g = _run(w)
    compare_lstm(g, oracle_steps.lstm_step(w), dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_zero_steps(dtype):
    """T = 0: no step runs, hT = h0 and cT = c0; the loss gradient passes
    straight back to dh0, dc0 is 0 and every weight gradient is 0."""
    w = _lstm("sumsq", dtype, L=2, I=8, H=32, B=4, T=0, seed=6, h0=True)
    _, g = _run(w)
    r = oracle_steps.lstm_step(w)
    compare_lstm(g, r, dtype, with_dx=False)
    assert np.array_equal(g["hT"], w.h0.astype(np.float64)) and np.array_equal(g["cT"], w.c0.astype(np.float64))
    for k in ("dWx", "dWh", "db"):
        for t in g[k]:
            assert not t.any()


@pytest.mark.parametrize("B,H,ragged,persist", [(300, 64, True, "1"), (300, 64, True, "0"), (512, 128, False, "1"),
                                                 (544, 128, True, "1")])
def test_large_batch_bf16(B, H, ragged, persist, monkeypatch):
    """Batches of more than 256 rows: the persistent kernels run the sorted
    rows in parts of 256, one launch each (rows are independent sequences),
    the backward adding each part's bias gradient to the earlier parts'.
    B = 300 and 544 with ragged lengths (the last part partial, rows of
    length 0), B = 512 fixed length; B = 300 also through the per-step
    kernels (JANUS_PERSIST=0).  Each against the oracle."""
    from paper_1812_01329_amd import janus as J
    monkeypatch.setenv("JANUS_PERSIST", persist)
    rng = np.random.default_rng(B + H)
    lens = rng.integers(0, 7, B) if ragged else None
    w = _lstm("mean_final" if ragged else "mse", "bf16", L=2, I=40, H=H, B=B, T=6, lengths=lens, seed=8, h0=True,
              P=24)
    print(f"[large-batch] B={B} H={H} ragged={ragged} persist={persist}", flush=True)
    J.janus_trace_begin()
    step, g = _run(w)
    stats = J.janus_trace_end()
    labels = {r["label"]: r["launches"] for r in stats}
    if persist == "1":
        parts = (B + 255) // 256
        assert labels.get("lstm_fwd_persistent") == 2 * parts, labels   # two layers
        assert labels.get("lstm_bwd_persistent") == 2 * parts, labels
        assert J.janus_lstm_device_report(step.desc, step.ws)["timed_out"] == 0
    else:
        assert "lstm_fwd_persistent" not in labels, labels
    compare_lstm(g, oracle_steps.lstm_step(w), "bf16")


def test_single_leaf_and_chain_trees():
    left, right, word, roots = [], [], [], []
    rng = np.random.default_rng(1)
    # a one-leaf tree, a left chain of 12 leaves and a balanced 16-leaf tree
    roots.append(wl.random_bracketing(rng, 1, np.array([3]), left, right, word))
    n0 = len(left)
    prev = None
    for k in range(12):
        left.append(-1); right.append(-1); word.append(int(rng.integers(0, 40)))
        leaf = len(left) - 1
        if prev is None:
            prev = leaf
        else:
            left.append(prev); right.append(leaf); word.append(-1)
            prev = len(left) - 1
    roots.append(prev)
    roots.append(wl.random_bracketing(rng, 16, rng.integers(0, 40, 16), left, right, word))
    trees = wl.TreeBatch(np.asarray(left, np.int32), np.asarray(right, np.int32), np.asarray(word, np.int32),
                         np.asarray(roots, np.int32))
    base = wl.sst_treelstm(n_trees=2, E=24, H=20, V=40, seed=9)
    base.trees = trees
    base.labels = rng.integers(0, base.C, trees.num_trees).astype(np.int32)
    _, g = _run(base)
    r = oracle_steps.tree_step(base)
    check("h_root", g["h_root"], r["h_root"], 1e-4)
    for k in ("dW", "dU", "db", "demb"):
        check(k, g[k], r[k], 1e-3)


def test_deterministic_repeat():
    """Two runs of the same step give identical bits."""
    w = wl.varlen_lstm(T=30, B=40, I=64, H=96)
    step, g1 = _run(w)
    step.run()
    g2 = step.results()
    for k in ("y", "hT", "dx", "dh0"):
        assert np.array_equal(g1[k], g2[k]), k
    for k in ("dWx", "dWh", "db"):
        for a, b in zip(g1[k], g2[k]):
            assert np.array_equal(a, b), k


@pytest.mark.parametrize("H,B,ragged", [(1024, 256, False), (2048, 256, True)])
def test_deterministic_repeat_persistent(H, B, ragged):
    """The persistent kernels in the configurations of the large workloads:
    the backward in 8 slices with its readiness counters (dG slot of 2 MB
    and more) and, at H = 2048 (h slot of 1 MB), the forward in 2 slices.  Without a grid
    barrier a workgroup may run a step ahead of others; four runs of the
    same step must still give identical bits (a race on a partial-sum slot
    or on a dG slot would show here), and the first matches the oracle."""
    from paper_1812_01329_amd import janus as J
    lens = None
    if ragged:
        lens = [int(v) for v in np.random.default_rng(H + B).integers(1, 7, B)]
        lens[0] = 6
    w = _lstm("mse", "bf16", L=2, I=64, H=H, B=B, T=6, lengths=lens, seed=41, h0=True, P=32)
    step, g1 = _run(w)
    rep = J.janus_lstm_device_report(step.desc, step.ws)
    print(f"[repeat] H={H} B={B} report {rep}", flush=True)
    assert rep["timed_out"] == 0
    assert rep["bwd_groups"] == 2 * (H // 64)   # 8 slices: groups of 64 units, two layers
    compare_lstm(g1, oracle_steps.lstm_step(w), "bf16")
    for _ in range(3):
        step.run()
        g2 = step.results()
        for k in ("y", "hT", "cT", "dh0", "dc0"):
            assert np.array_equal(g1[k], g2[k]), k
        for k in ("dWx", "dWh", "db"):
            for a, b in zip(g1[k], g2[k]):
                assert np.array_equal(a, b), k


@pytest.mark.parametrize("ragged", [False, True])
def test_persistent_contraction_tiles(ragged, monkeypatch):
    """Contractions of 512 tiles and more can run as a persistent grid (one
    workgroup per CU walking the tiles, the next tile's first K block loaded
    during the current tile's epilogue; JANUS_GEMM_PERSIST=1).  The input
    projection here has 8192 x 4096 outputs (512 tiles of 256 x 256), or,
    with ragged lengths, about 8300 packed rows (528 tiles, the last M tile
    partial): with the persistent grid and without (JANUS_GEMM_PERSIST=0,
    the default) the step gives identical bits, and matches the oracle."""
    T, lens = 32, None
    if ragged:
        T = 64
        lens = [int(v) for v in np.random.default_rng(44).integers(1, T + 1, 256)]
        lens[0] = T
    w = _lstm("mse", "bf16", L=1, I=1024 if not ragged else 256, H=1024, B=256, T=T, lengths=lens, seed=43,
              h0=True, P=64)
    res = {}
    for mode in ("1", "0"):
        monkeypatch.setenv("JANUS_GEMM_PERSIST", mode)
        _, res[mode] = _run(w)
    for k in ("y", "hT", "cT", "dh0", "dc0"):
        assert np.array_equal(res["1"][k], res["0"][k]), k
    for k in ("dWx", "dWh", "db"):
        for a, b in zip(res["1"][k], res["0"][k]):
            assert np.array_equal(a, b), k
    compare_lstm(res["1"], oracle_steps.lstm_step(w), "bf16")


def test_batch_permutation_on_device():
    w = _lstm("mse", "bf16", L=1, I=32, H=64, B=9, T=6, lengths=[6, 2, 5, 0, 3, 6, 1, 4, 2], seed=2, h0=True)
    _, g1 = _run(w)
    p = np.array([3, 8, 0, 2, 7, 1, 5, 6, 4])
    w.x = w.x[:, p]; w.lengths = w.lengths[p]; w.target = w.target[:, p]; w.h0 = w.h0[:, p]; w.c0 = w.c0[:, p]
    _, g2 = _run(w)
    np.testing.assert_allclose(g2["y"], g1["y"][:, p], rtol=0, atol=1e-6)
    assert abs(g1["loss"] - g2["loss"]) <= 1e-4 * abs(g1["loss"])
    assert check("dWh-perm", g2["dWh"][0], g1["dWh"][0], 1e-3) <= 1e-3


@pytest.mark.parametrize("persist", ["0", "1"])
@pytest.mark.parametrize("lengths", [None, "ragged"])
def test_both_recurrence_paths(persist, lengths, monkeypatch):
    """bf16 LSTM through the per-step kernels (JANUS_PERSIST=0) and through the
    persistent kernels, each against the oracle."""
    monkeypatch.setenv("JANUS_PERSIST", persist)
    rng = np.random.default_rng(11)
    B = 96
    lens = None if lengths is None else rng.integers(0, 13, B)
    w = _lstm("mse", "bf16", L=2, I=64, H=128, B=B, T=12, lengths=lens, seed=11, h0=True, P=40)
    _, g = _run(w)
    compare_lstm(g, oracle_steps.lstm_step(w), "bf16")


def test_long_ragged_batch_split_contractions():
    """Enough packed rows (ragged count) that the weight-gradient
    contractions split K and the input projection gathers rows."""
    rng = np.random.default_rng(21)
    B = 100
    lengths = rng.integers(0, 49, B)
    w = _lstm("mse", "bf16", L=1, I=64, H=128, B=B, T=48, lengths=lengths, seed=21, h0=True, P=136)
    _, g = _run(w)
    compare_lstm(g, oracle_steps.lstm_step(w), "bf16")


@pytest.mark.parametrize("slices", ["4", "8"])
@pytest.mark.parametrize("H,B,ragged", [(512, 256, False), (200, 70, True)])
def test_backward_slices(slices, H, B, ragged, monkeypatch):
    """The persistent backward with its K = 4H gate columns in 4 and in 8
    slices (JANUS_BWD_SLICES): unit groups of 32 or 64, one or two weight
    tiles per wave, full and split-K waves (B = 256, 70).  With H = 512 every
    XCD holds whole groups (partial sums kept in the L2); with H = 200
    (padded to 208, last group partial) the workgroup count is not a multiple
    of 8 slices per XCD, so some groups straddle two XCDs and write their
    partial sums through to memory."""
    from paper_1812_01329_amd import janus as J
    monkeypatch.setenv("JANUS_BWD_SLICES", slices)
    rng = np.random.default_rng(31)
    lens = rng.integers(0, 11, B) if ragged else None
    w = _lstm("mse", "bf16", L=2, I=64, H=H, B=B, T=10, lengths=lens, seed=31, h0=True, P=40)
    J.janus_trace_begin()
    step, g = _run(w)
    labels = {r["label"] for r in J.janus_trace_end()}
    assert "lstm_bwd_persistent" in labels, labels
    rep = J.janus_lstm_device_report(step.desc, step.ws)
    print(f"[slices] H={H} B={B} NS={slices} report {rep}", flush=True)
    units = 8 * int(slices)
    assert rep["timed_out"] == 0
    hp = (H + 15) // 16 * 16   # H padded to 16
    assert rep["bwd_groups"] == 2 * ((hp + units - 1) // units)   # two layers
    assert 0 <= rep["bwd_local_groups"] <= rep["bwd_groups"]
    if H == 512:   # 64 workgroups: whole groups fit on the XCDs of an even placement
        assert rep["bwd_local_groups"] > 0, rep
    compare_lstm(g, oracle_steps.lstm_step(w), "bf16")


@pytest.mark.parametrize("slices", ["1", "2", "4"])
@pytest.mark.parametrize("H,B,ragged", [(512, 256, False), (200, 70, True), (256, 24, True)])
def test_forward_slices(slices, H, B, ragged, monkeypatch):
    """The persistent forward with the columns of Wh in 1, 2 and 4 slices
    (JANUS_FWD_SLICES): unit groups of 16 or 32 exchange partial
    pre-activations.  H = 512 places whole groups on the XCDs (partial sums
    kept in the L2); H = 200 (padded to 208) has 26 or 28 workgroups, so some
    groups straddle two XCDs and use per-step slots; B = 24 splits each
    slice's k-groups over 8 waves, some of which get none."""
    import torch
    from paper_1812_01329_amd import janus as J
    from paper_1812_01329_amd.train_step import make_step
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    monkeypatch.setenv("JANUS_FWD_SLICES", slices)
    rng = np.random.default_rng(37)
    lens = rng.integers(0, 11, B) if ragged else None
    w = _lstm("mse", "bf16", L=2, I=64, H=H, B=B, T=10, lengths=lens, seed=37, h0=True, P=40)
    print(f"[fwd-slices] H={H} B={B} NS={slices}", flush=True)
    step = make_step(w)
    J.janus_trace_begin()
    J.janus_lstm_seq_fwd(step.desc, step.x, step.lengths, step.Wx, step.Wh, step.b, step.h0, step.c0,
                         step.y, step.hT, step.cT, step.ws)
    labels = {r["label"] for r in J.janus_trace_end()}
    assert "lstm_fwd_persistent" in labels, labels
    rep = J.janus_lstm_device_report(step.desc, step.ws)
    print(f"[fwd-slices] report {rep}", flush=True)
    ns = int(slices)
    assert rep["timed_out"] == 0
    hp = (H + 15) // 16 * 16   # H padded to 16
    assert rep["fwd_groups"] == (0 if ns == 1 else 2 * ((hp + 8 * ns - 1) // (8 * ns)))   # two layers
    assert 0 <= rep["fwd_local_groups"] <= rep["fwd_groups"]
    if H == 512 and ns > 1:   # 64 workgroups: whole groups fit on the XCDs of an even placement
        assert rep["fwd_local_groups"] > 0, rep
    step.run()
    g = step.results()
    assert J.janus_lstm_device_report(step.desc, step.ws)["timed_out"] == 0
    compare_lstm(g, oracle_steps.lstm_step(w), "bf16")


@pytest.mark.parametrize("small", ["1", "0"])
@pytest.mark.parametrize("dtype,ragged", [("f32", False), ("f32", True), ("bf16", True)])
@pytest.mark.parametrize("B,H", [(6, 48), (1, 65), (40, 48)])
def test_one_workgroup_recurrence(small, dtype, ragged, B, H, monkeypatch):
    """Small problems run each layer's time loop in one workgroup (weights,
    state and dG in LDS, steps separated by workgroup barriers); with
    JANUS_SMALL=0 the per-step kernels run instead.  Both against the
    oracle, with fixed and ragged lengths (zero-length rows included), the
    loss on y so dy enters every step, and h0, c0 given.  Lanes per cell
    (forward, backward): (1, 2); (2, 8), both splitting K unevenly (65 and
    260 terms); (1, 1) with two cells per thread."""
    from paper_1812_01329_amd import janus as J
    monkeypatch.setenv("JANUS_SMALL", small)
    monkeypatch.setenv("JANUS_PERSIST", "0")
    lengths = None
    if ragged:
        lengths = [int(v) for v in np.random.default_rng(B * 100 + H).integers(0, 10, B)]
        lengths[-1] = 0
        lengths[0] = 9
    print(f"[small] S={small} {dtype} B={B} H={H} lengths={lengths}", flush=True)
    w = _lstm("mse", dtype, L=2, I=24, H=H, B=B, T=9, lengths=lengths, seed=12, h0=True, P=20)
    J.janus_trace_begin()
    _, g = _run(w)
    labels = {r["label"] for r in J.janus_trace_end()}
    want = ("lstm_fwd_small", "lstm_bwd_small") if small == "1" else ("lstm_fwd_step", "lstm_bwd_step")
    for lab in want:
        assert any(x.startswith(lab) for x in labels), labels
    compare_lstm(g, oracle_steps.lstm_step(w), dtype)
