"""Binary TreeRNN (recursive neural network) evaluated by recursion over the
tree, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper trains a TreeRNN on SST ([37], Table 2) with the same recursive
program shape as the TreeLSTM: a function called on the two subtrees of a
node, a conditional separating leaves (Section 6.1, footnote 6).  It gives
no equations; the form used is the standard one of the cited recursive
neural network: a leaf's vector is its word vector, and an internal node
composes its children,

    h = emb[word]                       (leaf; width H = embedding width)
    h = tanh(W [h_L; h_R] + b)          (internal node; W is H x 2H)

Every node has at most one parent, so the backward pass sends each gradient
to exactly one child slot.
"""
from __future__ import annotations

import numpy as np


def forward_recursive(trees, emb, W, b):
    """Returns (h_root [num_trees, H], h [num_nodes, H])."""
    H = b.shape[0]
    h = np.zeros((trees.num_nodes, H))

    def visit(n):
        l, r = int(trees.left[n]), int(trees.right[n])
        if l < 0:
            h[n] = np.asarray(emb[int(trees.word[n])], dtype=np.float64)
        else:
            visit(l)
            visit(r)
            h[n] = np.tanh(W @ np.concatenate([h[l], h[r]]) + b)

    for root in trees.root:
        visit(int(root))
    return h[np.asarray(trees.root, dtype=np.int64)].copy(), h


def backward_recursive(trees, h, emb_shape, W, dh_root):
    """Backward from dL/dh_root [num_trees, H].

    Returns (demb [V, H] dense, dW, db)."""
    H = W.shape[0]
    demb = np.zeros(emb_shape)
    dW = np.zeros(W.shape)
    db = np.zeros(H)

    def visit(n, dh):
        l, r = int(trees.left[n]), int(trees.right[n])
        if l < 0:
            demb[int(trees.word[n])] += dh
            return
        da = dh * (1.0 - h[n] * h[n])
        db[:] += da
        dW[:] += np.outer(da, np.concatenate([h[l], h[r]]))
        dlr = W.T @ da
        visit(l, dlr[:H])
        visit(r, dlr[H:])

    for k, root in enumerate(trees.root):
        visit(int(root), np.asarray(dh_root[k], dtype=np.float64))
    return demb, dW, db
