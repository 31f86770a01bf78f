"""One whole training step (forward + backward) for each workload.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Each function takes a workload from ``paper_1812_01329_amd.workloads`` (the
seeded inputs, already rounded to bf16 where the workload is bf16) and
returns a dict with the loss, the forward outputs and every gradient, all in
float64.  The composition is the imperative program: embedding lookup, the
recurrence or the tree recursion, the loss, then the hand-derived backward
in reverse order.
"""
from __future__ import annotations

import numpy as np

from . import childsum, heads, lstm, treelstm, treernn


def _f64(a):
    return None if a is None else np.asarray(a, dtype=np.float64)


def lstm_step(w, batch_rows=None):
    """Training step of an LSTM workload (heads: sumsq, mean_final, xent, mse).

    ``batch_rows`` restricts the step to a subset of the sequences.  Every
    output and the input gradients of a sequence depend only on that
    sequence (the losses are sums over sequences, scaled by a count that is
    passed in unchanged), so a subset reproduces those values exactly."""
    Wx = [_f64(a) for a in w.Wx]
    Wh = [_f64(a) for a in w.Wh]
    b = [_f64(a) for a in w.b]
    rows = np.arange(w.B) if batch_rows is None else np.asarray(batch_rows)
    B = len(rows)
    lengths = None if w.lengths is None else np.asarray(w.lengths)[rows]
    out = {}
    if w.head == "xent":
        ids = w.input_ids[:, rows]
        x = heads.embed_forward(w.E, ids)                    # [T, B, I]
    else:
        x = _f64(w.x)[:, rows]
    h0 = None if w.h0 is None else _f64(w.h0)[:, rows]
    c0 = None if w.c0 is None else _f64(w.c0)[:, rows]
    y, hT, cT, caches, ys = lstm.stack_forward(x, lengths, Wx, Wh, b, h0, c0)
    out.update(y=y, hT=hT, cT=cT)
    dy = dhT = None
    if w.head == "sumsq":
        loss, dtop = heads.sumsq(hT[-1])
        dhT = np.zeros_like(hT); dhT[-1] = dtop
    elif w.head == "mean_final":
        # mean over B and H of the final h of every sequence (count = full B * H)
        top = hT[-1]
        loss = float(top.sum() / (w.B * w.H))
        dhT = np.zeros_like(hT); dhT[-1] = 1.0 / (w.B * w.H)
    elif w.head == "xent":
        T = w.T
        tgt = w.target_ids[:, rows].reshape(-1)
        hflat = y.reshape(T * B, w.H)
        # mean over all B * T positions of the full batch
        loss_sub, dh, dWo, dbo, logits = heads.softmax_xent(hflat, w.Wout, _f64(w.bout), tgt)
        scale = (T * B) / (T * w.B)
        loss = loss_sub * scale
        dy = (dh * scale).reshape(T, B, w.H)
        out.update(dWout=dWo * scale, dbout=dbo * scale, logits=logits)
    elif w.head == "mse":
        T, P = w.T, w.Wout.shape[0]
        hflat = y.reshape(T * B, w.H)
        tgt = _f64(w.target)[:, rows].reshape(T * B, P)
        loss_sub, dh, dWp, dbp, yp = heads.linear_mse(hflat, w.Wout, _f64(w.bout), tgt)
        scale = (T * B) / (T * w.B)
        loss = loss_sub * scale
        dy = (dh * scale).reshape(T, B, w.H)
        out.update(dWout=dWp * scale, dbout=dbp * scale, proj=yp)
    else:
        raise ValueError(w.head)
    dx, dh0, dc0, dWx, dWh, db = lstm.stack_backward(caches, ys, Wx, Wh, dy, dhT, None)
    out.update(loss=loss, dx=dx, dh0=dh0, dc0=dc0, dWx=dWx, dWh=dWh, db=db)
    if w.head == "xent":
        out["dE"] = heads.embed_backward(w.V, dx, w.input_ids[:, rows])
    return out


def tree_step(w):
    """Training step of the TreeLSTM workload: recursion from every root,
    5-class softmax cross-entropy at the roots (mean over trees), backward."""
    W, U, b = _f64(w.W), _f64(w.U), _f64(w.b)
    h_root, st = treelstm.forward_recursive(w.trees, _f64(w.emb), W, U, b)
    loss, dh_root, dWs, dbs, logits = heads.softmax_xent(h_root, w.Ws, _f64(w.bs), w.labels)
    demb, dW, dU, db = treelstm.backward_recursive(w.trees, st, w.emb.shape, W, U, dh_root)
    return dict(loss=loss, h_root=h_root, logits=logits, dh_root=dh_root, dWs=dWs, dbs=dbs,
                demb=demb, dW=dW, dU=dU, db=db, h=st.h, c=st.c)


def treernn_step(w):
    """Training step of the TreeRNN workload: recursion from every root,
    5-class softmax cross-entropy at the roots (mean over trees), backward."""
    W, b = _f64(w.W), _f64(w.b)
    h_root, h = treernn.forward_recursive(w.trees, _f64(w.emb), W, b)
    loss, dh_root, dWs, dbs, logits = heads.softmax_xent(h_root, w.Ws, _f64(w.bs), w.labels)
    demb, dW, db = treernn.backward_recursive(w.trees, h, w.emb.shape, W, dh_root)
    return dict(loss=loss, h_root=h_root, logits=logits, dh_root=dh_root, dWs=dWs, dbs=dbs,
                demb=demb, dW=dW, db=db, h=h)


def childsum_step(w):
    """Training step of the Child-Sum TreeLSTM workload: recursion from every
    root, 5-class softmax cross-entropy at the roots (mean over trees),
    backward."""
    W, U, b = _f64(w.W), _f64(w.U), _f64(w.b)
    h_root, st = childsum.forward_recursive(w.trees, _f64(w.emb), W, U, b)
    loss, dh_root, dWs, dbs, logits = heads.softmax_xent(h_root, w.Ws, _f64(w.bs), w.labels)
    demb, dW, dU, db = childsum.backward_recursive(w.trees, st, w.emb.shape, W, U, dh_root)
    return dict(loss=loss, h_root=h_root, logits=logits, dh_root=dh_root, dWs=dWs, dbs=dbs,
                demb=demb, dW=dW, dU=dU, db=db, h=st["h"], c=st["c"])
