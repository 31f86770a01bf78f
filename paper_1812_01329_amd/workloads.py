"""Seeded synthetic inputs for the five training-step workloads.

This module holds input generation only: random draws, bf16 rounding of the
drawn values, random tree shapes and token ids.  It contains none of the
method's arithmetic (no cell, no loss, no schedule), so that the CPU oracle
and the HIP path can both be fed from it without sharing any computation.

The paper measures on PTB, One Billion Words and SST (Section 6.1, Table 2).
None of those datasets is used: every workload below is a seeded stand-in
with the shapes, sizes and value distributions of the corresponding model
(LSTM on PTB with batch 20, LM on 1B with batch 256, TreeLSTM on SST with
batch 25).

Seeding: one ``numpy.random.Generator(PCG64)`` tree per workload, rooted at
``SeedSequence(1812 + index)`` and split with ``spawn(4)`` into the streams
[parameters, inputs, lengths/trees, labels/targets].  Values are drawn in
float32; bf16 workloads then round every drawn value to bf16 with
round-to-nearest-even, and the float64 oracle receives those rounded values.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"


# --------------------------------------------------------------------------
# bf16 helpers (input preparation only)
# --------------------------------------------------------------------------
def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest-even) and return the uint16 bit
    patterns.  NaN inputs are not expected (all draws are finite)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def bf16_round(a: np.ndarray) -> np.ndarray:
    """float32 array whose values are exactly representable in bf16."""
    return bf16_to_f32(bf16_bits(a))


def _round_if(a: np.ndarray, dtype: str) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    return bf16_round(a) if dtype == BF16 else a


# --------------------------------------------------------------------------
# Distributions
# --------------------------------------------------------------------------
def zipf_truncated(rng: np.random.Generator, s: float, V: int, size) -> np.ndarray:
    """Token ids in [0, V) with p(r) proportional to (r+1)^-s, drawn by the
    inverse CDF.  Returns int32."""
    ranks = np.arange(1, V + 1, dtype=np.float64)
    p = ranks ** (-s)
    cdf = np.cumsum(p)
    cdf /= cdf[-1]
    u = rng.random(size)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def uniform(rng: np.random.Generator, a: float, shape) -> np.ndarray:
    return rng.uniform(-a, a, size=shape).astype(np.float32)


def normal(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(size=shape, dtype=np.float32)


def _streams(index: int, seed: Optional[int] = None):
    ss = np.random.SeedSequence(1812 + index if seed is None else seed)
    return [np.random.Generator(np.random.PCG64(s)) for s in ss.spawn(4)]


# --------------------------------------------------------------------------
# LSTM workloads
# --------------------------------------------------------------------------
@dataclasses.dataclass
class LSTMWorkload:
    """Inputs of one LSTM training step.

    Parameters follow the per-layer layout of ``torch.nn.LSTM``:
    ``Wx[l]`` is [4H, I_l], ``Wh[l]`` is [4H, H], ``b[l]`` is [4H], gate
    blocks in the order (i, f, g, o), one bias per layer.
    """
    name: str
    dtype: str
    L: int
    I: int
    H: int
    B: int
    T: int
    x: Optional[np.ndarray]            # [T, B, I] float32 (bf16-exact for bf16)
    lengths: Optional[np.ndarray]      # [B] int32, or None for all == T
    Wx: List[np.ndarray]
    Wh: List[np.ndarray]
    b: List[np.ndarray]
    head: str                          # "sumsq", "mean_final", "xent", "mse"
    # language-model head (xent): token ids and embedding / output layer
    V: int = 0
    tokens: Optional[np.ndarray] = None  # [B, T+1] int32
    E: Optional[np.ndarray] = None       # [V, I]
    Wout: Optional[np.ndarray] = None    # [V, H] (xent) or [P, H] (mse)
    bout: Optional[np.ndarray] = None
    target: Optional[np.ndarray] = None  # [T, B, P] for mse
    h0: Optional[np.ndarray] = None      # [L, B, H] float32 or None = 0
    c0: Optional[np.ndarray] = None

    @property
    def input_ids(self) -> np.ndarray:
        """[T, B] ids fed to the embedding (time-major)."""
        return np.ascontiguousarray(self.tokens[:, : self.T].T)

    @property
    def target_ids(self) -> np.ndarray:
        """[T, B] next-token targets (time-major)."""
        return np.ascontiguousarray(self.tokens[:, 1:].T)


def _lstm_params(rng, L, I, H, a, dtype):
    Wx, Wh, b = [], [], []
    for layer in range(L):
        Il = I if layer == 0 else H
        Wx.append(_round_if(uniform(rng, a, (4 * H, Il)), dtype))
        Wh.append(_round_if(uniform(rng, a, (4 * H, H)), dtype))
        b.append(_round_if(uniform(rng, a, (4 * H,)), dtype))
    return Wx, Wh, b


def tiny_lstm(T=16, B=4, I=32, H=64, seed=None) -> LSTMWorkload:
    """1-layer LSTM, input 32, hidden 64, batch 4, fixed length 16, fp32;
    inputs N(0,1), weights U(-0.1, 0.1), zero initial state, loss = sum of
    squares of the final h."""
    rp, ri, _, _ = _streams(1, seed)
    Wx, Wh, b = _lstm_params(rp, 1, I, H, 0.1, F32)
    x = normal(ri, (T, B, I))
    return LSTMWorkload("tiny", F32, 1, I, H, B, T, x, None, Wx, Wh, b, "sumsq")


def ptb_lstm(T=35, B=20, H=650, V=10000, L=2, seed=None) -> LSTMWorkload:
    """2-layer LSTM language model: vocabulary 10000 with Zipf(1.1) ids,
    embedding 650, hidden 650, batch 20, 35 steps, bf16 parameters
    U(-0.05, 0.05); embedding gather and next-token softmax cross-entropy."""
    rp, _, _, rt = _streams(2, seed)
    E = _round_if(uniform(rp, 0.05, (V, H)), BF16)
    Wx, Wh, b = _lstm_params(rp, L, H, H, 0.05, BF16)
    Wout = _round_if(uniform(rp, 0.05, (V, H)), BF16)
    bout = _round_if(uniform(rp, 0.05, (V,)), BF16)
    tokens = zipf_truncated(rt, 1.1, V, (B, T + 1))
    return LSTMWorkload("ptb", BF16, L, H, H, B, T, None, None, Wx, Wh, b, "xent",
                        V=V, tokens=tokens, E=E, Wout=Wout, bout=bout)


def varlen_lstm(T=200, B=128, I=512, H=1024, seed=None) -> LSTMWorkload:
    """1-layer LSTM, input 512, hidden 1024, batch 128, lengths uniform in
    [1, T] (data-dependent loop exit), bf16 inputs N(0,1), weights
    U(-1/sqrt(H), 1/sqrt(H)); loss = mean of the final h of each sequence."""
    rp, ri, rl, _ = _streams(3, seed)
    a = 1.0 / np.sqrt(H)
    Wx, Wh, b = _lstm_params(rp, 1, I, H, a, BF16)
    x = _round_if(normal(ri, (T, B, I)), BF16)
    lengths = rl.integers(1, T + 1, size=B).astype(np.int32)
    return LSTMWorkload("varlen", BF16, 1, I, H, B, T, x, lengths, Wx, Wh, b, "mean_final")


def lm2048_lstm(T=256, B=256, H=2048, I=2048, P=2048, L=2, seed=None) -> LSTMWorkload:
    """2-layer LSTM, input 2048, hidden 2048, batch 256, length 256, bf16
    with fp32 accumulation; inputs N(0,1), weights U(-0.02, 0.02); per-step
    linear projection to 2048 and MSE against N(0,1) targets."""
    rp, ri, _, rt = _streams(5, seed)
    Wx, Wh, b = _lstm_params(rp, L, I, H, 0.02, BF16)
    Wp = _round_if(uniform(rp, 0.02, (P, H)), BF16)
    bp = _round_if(uniform(rp, 0.02, (P,)), BF16)
    x = _round_if(normal(ri, (T, B, I)), BF16)
    tgt = _round_if(normal(rt, (T, B, P)), BF16)
    return LSTMWorkload("lm2048", BF16, L, I, H, B, T, x, None, Wx, Wh, b, "mse",
                        Wout=Wp, bout=bp, target=tgt)


# --------------------------------------------------------------------------
# Tree workloads
# --------------------------------------------------------------------------
@dataclasses.dataclass
class TreeBatch:
    """A batch of binary trees stored as flat int32 arrays.

    Nodes are numbered in post-order within each tree and the trees are
    concatenated, so the root of a tree is its last node.  ``left[n]`` and
    ``right[n]`` are child node ids or -1 for a leaf; ``word[n]`` is the
    token id of a leaf or -1 for an internal node; ``root[k]`` is the root
    node id of tree k.
    """
    left: np.ndarray
    right: np.ndarray
    word: np.ndarray
    root: np.ndarray

    @property
    def num_nodes(self) -> int:
        return int(self.left.shape[0])

    @property
    def num_trees(self) -> int:
        return int(self.root.shape[0])


def random_bracketing(rng: np.random.Generator, n_leaves: int, words: np.ndarray,
                      left: list, right: list, word: list) -> int:
    """Append a random full binary tree over ``n_leaves`` leaves (each span of
    n > 1 leaves splits at k ~ U{1..n-1}) in post-order; return the root id."""
    # iterative post-order construction to avoid deep Python recursion
    stack = [("build", 0, n_leaves)]
    results: list = []
    while stack:
        item = stack.pop()
        if item[0] == "build":
            _, lo, n = item
            if n == 1:
                nid = len(left)
                left.append(-1); right.append(-1); word.append(int(words[lo]))
                results.append(nid)
            else:
                k = int(rng.integers(1, n))
                stack.append(("join",))
                stack.append(("build", lo + k, n - k))
                stack.append(("build", lo, k))
        else:
            r = results.pop(); l = results.pop()
            nid = len(left)
            left.append(l); right.append(r); word.append(-1)
            results.append(nid)
    assert len(results) == 1
    return results[0]


@dataclasses.dataclass
class TreeWorkload:
    """Inputs of one binary TreeLSTM training step (fp32)."""
    name: str
    E_dim: int
    H: int
    V: int
    C: int
    trees: TreeBatch
    labels: np.ndarray     # [num_trees] int32 in [0, C)
    emb: np.ndarray        # [V, E]
    W: np.ndarray          # [5H, E]   gate blocks (i, f_L, f_R, o, u)
    U: np.ndarray          # [5H, 2H]
    b: np.ndarray          # [5H]
    Ws: np.ndarray         # [C, H]
    bs: np.ndarray         # [C]
    dtype: str = F32


def make_trees(rng: np.random.Generator, n_trees: int, min_leaves: int, max_leaves: int,
               V: int, zipf_s: float = 1.1, sizes: Optional[List[int]] = None) -> TreeBatch:
    left: list = []; right: list = []; word: list = []; roots = []
    if sizes is None:
        sizes = [int(s) for s in rng.integers(min_leaves, max_leaves + 1, size=n_trees)]
    for n in sizes:
        words = zipf_truncated(rng, zipf_s, V, n)
        roots.append(random_bracketing(rng, n, words, left, right, word))
    return TreeBatch(np.asarray(left, np.int32), np.asarray(right, np.int32),
                     np.asarray(word, np.int32), np.asarray(roots, np.int32))


def sst_treelstm(n_trees=25, E=300, H=150, V=20000, C=5, min_leaves=5, max_leaves=50,
                 seed=None, sizes=None) -> TreeWorkload:
    """Binary TreeLSTM, embedding 300, hidden 150, batch 25 random full binary
    trees over sentences of 5-50 leaves with Zipf(1.1) leaf ids over a 20000
    vocabulary, 5-class softmax at the root with uniform labels, fp32,
    all parameters U(-0.1, 0.1)."""
    rp, _, rtree, rl = _streams(4, seed)
    emb = uniform(rp, 0.1, (V, E))
    W = uniform(rp, 0.1, (5 * H, E))
    U = uniform(rp, 0.1, (5 * H, 2 * H))
    b = uniform(rp, 0.1, (5 * H,))
    Ws = uniform(rp, 0.1, (C, H))
    bs = uniform(rp, 0.1, (C,))
    trees = make_trees(rtree, n_trees, min_leaves, max_leaves, V, sizes=sizes)
    labels = rl.integers(0, C, size=trees.num_trees).astype(np.int32)
    return TreeWorkload("treelstm", E, H, V, C, trees, labels, emb, W, U, b, Ws, bs)


@dataclasses.dataclass
class TreeRNNWorkload:
    """Inputs of one binary TreeRNN training step (fp32): leaves take their
    word vector as h (embedding width = H), internal nodes
    h = tanh(W [h_L; h_R] + b)."""
    name: str
    H: int
    V: int
    C: int
    trees: TreeBatch
    labels: np.ndarray     # [num_trees] int32 in [0, C)
    emb: np.ndarray        # [V, H]
    W: np.ndarray          # [H, 2H]
    b: np.ndarray          # [H]
    Ws: np.ndarray         # [C, H]
    bs: np.ndarray         # [C]
    dtype: str = F32


def sst_treernn(n_trees=25, H=300, V=20000, C=5, min_leaves=5, max_leaves=50, seed=None,
                sizes=None) -> TreeRNNWorkload:
    """Binary TreeRNN with 300-wide word vectors and hidden state, batch 25
    random full binary trees over sentences of 5-50 leaves with Zipf(1.1)
    leaf ids over a 20000 vocabulary (the trees of the TreeLSTM workload),
    5-class softmax at the root with uniform labels, fp32, all parameters
    U(-0.1, 0.1)."""
    rp, _, rtree, rl = _streams(4, seed)
    emb = uniform(rp, 0.1, (V, H))
    W = uniform(rp, 0.1, (H, 2 * H))
    b = uniform(rp, 0.1, (H,))
    Ws = uniform(rp, 0.1, (C, H))
    bs = uniform(rp, 0.1, (C,))
    trees = make_trees(rtree, n_trees, min_leaves, max_leaves, V, sizes=sizes)
    labels = rl.integers(0, C, size=trees.num_trees).astype(np.int32)
    return TreeRNNWorkload("treernn", H, V, C, trees, labels, emb, W, b, Ws, bs)


@dataclasses.dataclass
class NaryTreeBatch:
    """A batch of trees of any arity as flat int32 arrays: the children of
    node n are ``children[child_offsets[n]:child_offsets[n + 1]]`` (none for
    a leaf); every node has a token id ``word[n]`` (dependency-tree style);
    ``root[k]`` is the root of tree k.  Trees are concatenated, each
    numbered from its root."""
    child_offsets: np.ndarray
    children: np.ndarray
    word: np.ndarray
    root: np.ndarray

    @property
    def num_nodes(self) -> int:
        return int(self.word.shape[0])

    @property
    def num_trees(self) -> int:
        return int(self.root.shape[0])


def make_nary_trees(rng: np.random.Generator, n_trees: int, min_nodes: int, max_nodes: int, V: int,
                    zipf_s: float = 1.1, sizes: Optional[List[int]] = None,
                    chain: bool = False) -> NaryTreeBatch:
    """Random recursive trees: node i > 0 of a tree hangs under a uniformly
    drawn earlier node (under node i - 1 when ``chain``), so arities vary and
    depth grows like log n.  Words Zipf(s) over [0, V)."""
    if sizes is None:
        sizes = [int(s) for s in rng.integers(min_nodes, max_nodes + 1, size=n_trees)]
    kids: list = []
    roots = []
    base = 0
    for n in sizes:
        par = [-1] + [(i - 1 if chain else int(rng.integers(0, i))) for i in range(1, n)]
        lists = [[] for _ in range(n)]
        for i in range(1, n):
            lists[par[i]].append(base + i)
        kids += lists
        roots.append(base)
        base += n
    off = np.zeros(base + 1, np.int32)
    off[1:] = np.cumsum([len(c) for c in kids])
    children = np.asarray([c for cl in kids for c in cl], np.int32)
    words = zipf_truncated(rng, zipf_s, V, base).astype(np.int32)
    return NaryTreeBatch(off, children, words, np.asarray(roots, np.int32))


@dataclasses.dataclass
class ChildSumWorkload:
    """Inputs of one Child-Sum TreeLSTM training step (fp32).  Gate blocks of
    W [4H, E], U [4H, H] and b [4H] are (i, o, u, f)."""
    name: str
    E_dim: int
    H: int
    V: int
    C: int
    trees: NaryTreeBatch
    labels: np.ndarray
    emb: np.ndarray
    W: np.ndarray
    U: np.ndarray
    b: np.ndarray
    Ws: np.ndarray
    bs: np.ndarray
    dtype: str = F32


def sst_childsum(n_trees=25, E=300, H=150, V=20000, C=5, min_nodes=5, max_nodes=50, seed=None, sizes=None,
                 chain=False) -> ChildSumWorkload:
    """Child-Sum TreeLSTM, embedding 300, hidden 150, batch 25 random
    recursive trees (dependency-tree stand-ins) of 5-50 nodes, a Zipf(1.1)
    word at every node over a 20000 vocabulary, 5-class softmax at the root
    with uniform labels, fp32, all parameters U(-0.1, 0.1)."""
    rp, _, rtree, rl = _streams(6, seed)
    emb = uniform(rp, 0.1, (V, E))
    W = uniform(rp, 0.1, (4 * H, E))
    U = uniform(rp, 0.1, (4 * H, H))
    b = uniform(rp, 0.1, (4 * H,))
    Ws = uniform(rp, 0.1, (C, H))
    bs = uniform(rp, 0.1, (C,))
    trees = make_nary_trees(rtree, n_trees, min_nodes, max_nodes, V, sizes=sizes, chain=chain)
    labels = rl.integers(0, C, size=trees.num_trees).astype(np.int32)
    return ChildSumWorkload("childsum", E, H, V, C, trees, labels, emb, W, U, b, Ws, bs)


# Named full-size workloads, in the order of the five configurations.
FULL: Dict[str, callable] = {
    "tiny": tiny_lstm,
    "ptb": ptb_lstm,
    "varlen": varlen_lstm,
    "treelstm": sst_treelstm,
    "lm2048": lm2048_lstm,
    "treernn": sst_treernn,
    "childsum": sst_childsum,
}
