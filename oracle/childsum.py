"""Child-Sum TreeLSTM over trees of any arity, by recursion, forward and
backward.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The TreeLSTM the paper trains ([40], Table 2) comes from a paper that
defines two variants; the binary one is in oracle/treelstm.py.  This is the
other, for nodes with any number of children, every node reading its word
vector x (dependency trees).  With h~ the sum of the children's h:

    i = s(W_i x + U_i h~ + b_i)    o = s(W_o x + U_o h~ + b_o)
    u = tanh(W_u x + U_u h~ + b_u)
    f_k = s(W_f x + U_f h_k + b_f)            one forget gate per child k
    c = i u + sum_k f_k c_k,   h = o tanh(c)

Gate blocks of W [4H, E], U [4H, H] and b [4H] are (i, o, u, f).  A leaf
has no children (h~ = 0, no forget gate).  Each node has at most one parent,
so every gradient goes to exactly one child slot.
"""
from __future__ import annotations

import numpy as np

from .lstm import sigmoid


def _children(t, n):
    return [int(c) for c in t.children[int(t.child_offsets[n]):int(t.child_offsets[n + 1])]]


def forward_recursive(trees, emb, W, U, b):
    """Returns (h_root [num_trees, H], state dict of per-node arrays)."""
    H = U.shape[1]
    N = trees.num_nodes
    st = dict(h=np.zeros((N, H)), c=np.zeros((N, H)), i=np.zeros((N, H)), o=np.zeros((N, H)),
              u=np.zeros((N, H)), f=np.zeros((N, H)), x=np.zeros((N, W.shape[1])))

    def visit(n):
        kids = _children(trees, n)
        for k in kids:
            visit(k)
        x = np.asarray(emb[int(trees.word[n])], dtype=np.float64)
        ht = sum((st["h"][k] for k in kids), np.zeros(H))
        a = W @ x + b
        z = U[:3 * H] @ ht
        i = sigmoid(a[:H] + z[:H])
        o = sigmoid(a[H:2 * H] + z[H:2 * H])
        u = np.tanh(a[2 * H:3 * H] + z[2 * H:])
        c = i * u
        for k in kids:
            fk = sigmoid(a[3 * H:] + U[3 * H:] @ st["h"][k])
            st["f"][k] = fk          # the forget gate of child k, kept in k's row
            c = c + fk * st["c"][k]
        st["h"][n], st["c"][n] = o * np.tanh(c), c
        st["i"][n], st["o"][n], st["u"][n], st["x"][n] = i, o, u, x

    for r in trees.root:
        visit(int(r))
    return st["h"][np.asarray(trees.root, dtype=np.int64)].copy(), st


def backward_recursive(trees, st, emb_shape, W, U, dh_root):
    """Backward from dL/dh_root (dL/dc_root = 0).  Returns (demb, dW, dU, db)."""
    H = U.shape[1]
    demb = np.zeros(emb_shape)
    dW = np.zeros(W.shape)
    dU = np.zeros(U.shape)
    db = np.zeros(4 * H)

    def visit(n, dh, dc):
        kids = _children(trees, n)
        i, o, u, c = st["i"][n], st["o"][n], st["u"][n], st["c"][n]
        tau = np.tanh(c)
        dct = dc + dh * o * (1.0 - tau * tau)
        da_i = dct * u * i * (1.0 - i)
        da_o = dh * tau * o * (1.0 - o)
        da_u = dct * i * (1.0 - u * u)
        da_iou = np.concatenate([da_i, da_o, da_u])
        ht = sum((st["h"][k] for k in kids), np.zeros(H))
        dU[:3 * H] += np.outer(da_iou, ht)
        dh_tilde = U[:3 * H].T @ da_iou
        da_f_sum = np.zeros(H)
        child_grads = []
        for k in kids:
            fk = st["f"][k]
            da_f = dct * st["c"][k] * fk * (1.0 - fk)
            da_f_sum += da_f
            dU[3 * H:] += np.outer(da_f, st["h"][k])
            child_grads.append((k, dh_tilde + U[3 * H:].T @ da_f, dct * fk))
        da = np.concatenate([da_iou, da_f_sum])
        db[:] += da
        dW[:] += np.outer(da, st["x"][n])
        demb[int(trees.word[n])] += W.T @ da
        for k, dhk, dck in child_grads:
            visit(k, dhk, dck)

    for kk, r in enumerate(trees.root):
        visit(int(r), np.asarray(dh_root[kk], dtype=np.float64), np.zeros(H))
    return demb, dW, dU, db
