"""Binary TreeLSTM evaluated by recursion over the tree, forward and backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The TreeNN programs of the paper call a function recursively on the two
subtrees of a node, with a conditional separating leaves from internal nodes
(Section 6.1, footnote 6; converted to recursive graph invocations,
Section 4.2.1).  The cell is the binary (N-ary, N = 2) TreeLSTM of the model
the paper trains on SST ([40], Table 2), in its constituency form where only
leaves read a word vector:

    a = b + (leaf ? W x_n : U [h_L; h_R])     5H values, blocks (i, f_L, f_R, o, u)
    i, f_L, f_R, o = sigma(.),  u = tanh(.)
    c = i u + f_L c_L + f_R c_R,   h = o tanh(c)

A leaf has h_L = h_R = c_L = c_R = 0.  Every node has at most one parent, so
the backward pass sends each gradient to exactly one child slot.
"""
from __future__ import annotations

import numpy as np

from .lstm import sigmoid


def _gates(a, H):
    i = sigmoid(a[0:H])
    fl = sigmoid(a[H:2 * H])
    fr = sigmoid(a[2 * H:3 * H])
    o = sigmoid(a[3 * H:4 * H])
    u = np.tanh(a[4 * H:5 * H])
    return i, fl, fr, o, u


def node_cell(is_leaf, x, hl, cl, hr, cr, W, U, b):
    """Cell of one node.  Returns (h, c, gates)."""
    H = b.shape[0] // 5
    if is_leaf:
        a = W @ x + b
    else:
        a = U @ np.concatenate([hl, hr]) + b
    i, fl, fr, o, u = _gates(a, H)
    c = i * u + fl * cl + fr * cr
    h = o * np.tanh(c)
    return h, c, (i, fl, fr, o, u)


class TreeState:
    """Per-node values saved by the forward pass (indexed by node id)."""
    def __init__(self, N, H):
        self.h = np.zeros((N, H))
        self.c = np.zeros((N, H))
        self.gates = [None] * N
        self.x = [None] * N


def forward_recursive(trees, emb, W, U, b):
    """Evaluate every tree from its root by recursion.

    Returns (h_root [num_trees, H], state)."""
    H = b.shape[0] // 5
    N = trees.num_nodes
    st = TreeState(N, H)
    zero = np.zeros(H)

    def visit(n):
        l, r = int(trees.left[n]), int(trees.right[n])
        if l < 0:
            x = np.asarray(emb[int(trees.word[n])], dtype=np.float64)
            h, c, g = node_cell(True, x, zero, zero, zero, zero, W, U, b)
            st.x[n] = x
        else:
            visit(l)
            visit(r)
            h, c, g = node_cell(False, None, st.h[l], st.c[l], st.h[r], st.c[r], W, U, b)
        st.h[n], st.c[n], st.gates[n] = h, c, g

    for root in trees.root:
        visit(int(root))
    return st.h[np.asarray(trees.root, dtype=np.int64)].copy(), st


def forward_by_levels(trees, emb, W, U, b, level_nodes, level_offsets):
    """The same per-node cell, visited level by level in a given order.

    Used only to pin that a frontier schedule evaluates every node after its
    children: the result must equal ``forward_recursive`` bit for bit."""
    H = b.shape[0] // 5
    st = TreeState(trees.num_nodes, H)
    zero = np.zeros(H)
    for k in range(len(level_offsets) - 1):
        for n in level_nodes[level_offsets[k]:level_offsets[k + 1]]:
            n = int(n)
            l, r = int(trees.left[n]), int(trees.right[n])
            if l < 0:
                x = np.asarray(emb[int(trees.word[n])], dtype=np.float64)
                h, c, g = node_cell(True, x, zero, zero, zero, zero, W, U, b)
                st.x[n] = x
            else:
                assert st.gates[l] is not None and st.gates[r] is not None
                h, c, g = node_cell(False, None, st.h[l], st.c[l], st.h[r], st.c[r], W, U, b)
            st.h[n], st.c[n], st.gates[n] = h, c, g
    return st.h[np.asarray(trees.root, dtype=np.int64)].copy(), st


def backward_recursive(trees, st, emb_shape, W, U, dh_root):
    """Backward from dL/dh_root [num_trees, H] (dL/dc_root = 0).

    Returns (demb [V, E] dense, dW, dU, db)."""
    H = W.shape[0] // 5
    demb = np.zeros(emb_shape)
    dW = np.zeros(W.shape)
    dU = np.zeros(U.shape)
    db = np.zeros(5 * H)
    zero = np.zeros(H)

    def visit(n, dh, dc):
        l, r = int(trees.left[n]), int(trees.right[n])
        i, fl, fr, o, u = st.gates[n]
        cl = st.c[l] if l >= 0 else zero
        cr = st.c[r] if r >= 0 else zero
        tau = np.tanh(st.c[n])
        do = dh * tau
        dct = dc + dh * o * (1.0 - tau * tau)
        da = np.concatenate([dct * u * i * (1.0 - i),
                             dct * cl * fl * (1.0 - fl),
                             dct * cr * fr * (1.0 - fr),
                             do * o * (1.0 - o),
                             dct * i * (1.0 - u * u)])
        db[:] += da
        if l < 0:
            dW[:] += np.outer(da, st.x[n])
            demb[int(trees.word[n])] += W.T @ da
        else:
            hlr = np.concatenate([st.h[l], st.h[r]])
            dU[:] += np.outer(da, hlr)
            dhlr = U.T @ da
            visit(l, dhlr[:H], dct * fl)
            visit(r, dhlr[H:], dct * fr)

    for k, root in enumerate(trees.root):
        visit(int(root), np.asarray(dh_root[k], dtype=np.float64), np.zeros(H))
    return demb, dW, dU, db
