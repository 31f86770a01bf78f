"""One training step (forward + backward) of each workload, as a sequence of
calls through the C ABI.

This module only allocates device buffers (through torch) and orders the
library calls the way the imperative program orders its operations
(Figure 1: embedding lookup, the recurrence, the loss, then the backward in
reverse).  All arithmetic happens inside libjanus.so.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence, Tuple

import numpy as np
import torch

from . import janus as J
from . import workloads as wl


def _tdt(dtype: str):
    return torch.bfloat16 if dtype == wl.BF16 else torch.float32


def _cdt(dtype: str) -> int:
    return J.BF16 if dtype == wl.BF16 else J.F32


def _dev(a: np.ndarray, dtype, device) -> torch.Tensor:
    """Upload a float32 array (bf16-exact for bf16) in the given torch dtype."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device=device).to(dtype)


def _f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


class SgdUpdate:
    """The parameter update that ends a training step (janus_sgd_clip_update):
    every parameter tensor with its float32 gradient, one call."""

    def __init__(self, params: Sequence[torch.Tensor], grads: Sequence[torch.Tensor], lr: float, max_norm: float):
        dts = {p.dtype for p in params}
        assert len(dts) == 1, "one parameter dtype per update"
        self.params = [p.view(-1) for p in params]
        self.grads = [g.view(-1) for g in grads]
        dt = J.BF16 if params[0].dtype == torch.bfloat16 else J.F32
        self.desc = J.SgdDesc(len(self.params), dt, lr, max_norm)
        dev = params[0].device
        self.ws = torch.empty(J.sgd_workspace_bytes(self.desc), dtype=torch.uint8, device=dev)
        self.stats = torch.zeros(2, dtype=torch.float32, device=dev)   # [norm before clipping, scale]

    def apply(self, hold: Optional[int] = None):
        """``hold``: device address of a uint32 that, when non-zero at run
        time, leaves every parameter unchanged (a failed step)."""
        J.janus_sgd_clip_update(self.desc, self.params, self.grads, stats=self.stats, ws=self.ws, hold=hold)


class LSTMStep:
    """Device state and call sequence of an LSTM training step.

    ``skip_dx``: do not form the gradient of the (non-embedding) input x,
    as in the regression workload where x is data.  ``update`` = (lr,
    max_norm) appends the parameter update to the step."""

    def __init__(self, w: wl.LSTMWorkload, device="cuda", skip_dx: Optional[bool] = None,
                 update: Optional[Tuple[float, float]] = None):
        self.w = w
        self.device = device
        tdt = _tdt(w.dtype)
        self.tdt = tdt
        L, I, H, B, T = w.L, w.I, w.H, w.B, w.T
        self.desc = J.LstmDesc(L, I, H, B, T, _cdt(w.dtype))
        self.Wx = [_dev(a, tdt, device) for a in w.Wx]
        self.Wh = [_dev(a, tdt, device) for a in w.Wh]
        self.b = [_dev(a, tdt, device) for a in w.b]
        self.lengths = None if w.lengths is None else np.ascontiguousarray(w.lengths, np.int32)
        zeros = lambda *s, dt=torch.float32: torch.zeros(*s, dtype=dt, device=device)
        self.h0 = None if w.h0 is None else _dev(w.h0, torch.float32, device)
        self.c0 = None if w.c0 is None else _dev(w.c0, torch.float32, device)
        self.y = zeros(T, B, H, dt=tdt)
        self.hT = zeros(L, B, H)
        self.cT = zeros(L, B, H)
        self.dWx = [torch.empty_like(a, dtype=torch.float32) for a in self.Wx]
        self.dWh = [torch.empty_like(a, dtype=torch.float32) for a in self.Wh]
        self.db = [torch.empty_like(a, dtype=torch.float32) for a in self.b]
        self.dh0 = zeros(L, B, H)
        self.dc0 = zeros(L, B, H)
        self.loss = zeros(1)
        ws = J.janus_lstm_workspace_bytes(L, I, H, B, T, self.desc.dtype)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        self.skip_dx = (w.head == "mse") if skip_dx is None else skip_dx
        if w.head == "xent":
            self.ids_host = np.ascontiguousarray(w.input_ids.reshape(-1), np.int32)       # [T*B]
            self.tgt_host = np.ascontiguousarray(w.target_ids.reshape(-1), np.int32)
            self.ids = torch.from_numpy(self.ids_host).to(device)
            self.tgt = torch.from_numpy(self.tgt_host).to(device)
            self.E = _dev(w.E, tdt, device)
            self.Wout = _dev(w.Wout, tdt, device)
            self.bout = _dev(w.bout, tdt, device)
            self.x = zeros(T, B, I, dt=tdt)
            self.dx = zeros(T, B, I, dt=tdt)
            self.dy = zeros(T, B, H, dt=tdt)
            self.dE = zeros(w.V, I)
            self.dWout = torch.empty_like(self.Wout, dtype=torch.float32)
            self.dbout = torch.empty_like(self.bout, dtype=torch.float32)
            self.xdesc = J.XentDesc(w.V, H, T * B, self.desc.dtype)
            self.edesc = J.XentDesc(w.V, I, T * B, self.desc.dtype)
            xw = J.janus_xent_workspace_bytes(w.V, H, T * B, self.desc.dtype, J.XENT_FWD_BWD)
            self.xws = torch.empty(xw, dtype=torch.uint8, device=device)
            ew = J.janus_xent_workspace_bytes(w.V, I, T * B, self.desc.dtype, J.EMBED_BWD)
            self.ews = torch.empty(ew, dtype=torch.uint8, device=device)
        else:
            self.x = _dev(w.x, tdt, device)
            self.dx = None if self.skip_dx else zeros(T, B, I, dt=tdt)
        if w.head == "mse":
            P = w.Wout.shape[0]
            self.Wout = _dev(w.Wout, tdt, device)
            self.bout = _dev(w.bout, tdt, device)
            self.tgt = _dev(w.target.reshape(T * B, P), tdt, device)
            self.dy = zeros(T, B, H, dt=tdt)
            self.dWout = torch.empty_like(self.Wout, dtype=torch.float32)
            self.dbout = torch.empty_like(self.bout, dtype=torch.float32)
            self.mdesc = J.MseDesc(T * B, H, P, self.desc.dtype)
            mw = J.janus_mse_workspace_bytes(T * B, H, P, self.desc.dtype)
            self.mws = torch.empty(mw, dtype=torch.uint8, device=device)
        if w.head in ("sumsq", "mean_final"):
            self.dhT = zeros(L, B, H)
            self.dy = None
        self.update = None
        if update is not None:
            P, G = self.parameters()
            self.update = SgdUpdate(P, G, *update)
        # the timeout word of the step's recurrences: a step whose forward or
        # backward wait ran out leaves the parameters unchanged
        self.fault = J.janus_lstm_fault_flag(self.desc, self.ws)

    def carry_from(self, prev: "LSTMStep"):
        """Seeds this step's initial state with the final state of the step
        that ran before it (run after that step's backward call)."""
        L, B, H = self.w.L, self.w.B, self.w.H
        if self.h0 is None:
            self.h0 = torch.zeros(L, B, H, dtype=torch.float32, device=self.device)
            self.c0 = torch.zeros(L, B, H, dtype=torch.float32, device=self.device)
        J.janus_lstm_state_carry(self.desc, prev.w.B, prev.hT, prev.cT, self.h0, self.c0)

    def parameters(self):
        """(parameters, their gradients) in a fixed order: per layer Wx, Wh,
        b, then the head's table and bias, then the embedding."""
        P, G = [], []
        for l in range(self.w.L):
            P += [self.Wx[l], self.Wh[l], self.b[l]]
            G += [self.dWx[l], self.dWh[l], self.db[l]]
        if self.w.head in ("xent", "mse"):
            P += [self.Wout, self.bout]
            G += [self.dWout, self.dbout]
        if self.w.head == "xent":
            P.append(self.E)
            G.append(self.dE)
        return P, G

    def run(self):
        w = self.w
        T, B, H = w.T, w.B, w.H
        if w.head == "xent":
            J.janus_embed_softmax_xent(self.edesc, J.EMBED_FWD, self.ids_host, self.ids, table=self.E, out=self.x)
        J.janus_lstm_seq_fwd(self.desc, self.x, self.lengths, self.Wx, self.Wh, self.b, self.h0, self.c0,
                             self.y, self.hT, self.cT, self.ws)
        dhT = None
        if w.head == "xent":
            J.janus_embed_softmax_xent(self.xdesc, J.XENT_FWD_BWD, self.tgt_host, self.tgt, table=self.Wout,
                                       bias=self.bout, inp=self.y, out=self.dy, dtable=self.dWout,
                                       dbias=self.dbout, loss=self.loss, ws=self.xws)
        elif w.head == "mse":
            J.janus_linear_mse(self.mdesc, self.y, self.Wout, self.bout, self.tgt, self.dy, self.dWout,
                               self.dbout, self.loss, self.mws)
        else:
            kind = J.LOSS_SUMSQ if w.head == "sumsq" else J.LOSS_MEAN
            top = self.hT[w.L - 1]
            J.janus_loss_reduce(kind, top, B * H, self.loss, self.dhT[w.L - 1])
            dhT = self.dhT
        J.janus_lstm_seq_bwd(self.desc, self.x, self.lengths, self.Wx, self.Wh, self.ws, self.dy, dhT, None,
                             self.dx, self.dh0, self.dc0, self.dWx, self.dWh, self.db)
        if w.head == "xent":
            J.janus_embed_softmax_xent(self.edesc, J.EMBED_BWD, self.ids_host, self.ids, inp=self.dx,
                                       dtable=self.dE, ws=self.ews)
        if self.update is not None:
            self.update.apply(hold=self.fault)

    def results(self) -> Dict[str, object]:
        torch.cuda.synchronize()
        r = dict(loss=float(self.loss.item()), y=_f64(self.y), hT=_f64(self.hT), cT=_f64(self.cT),
                 dh0=_f64(self.dh0), dc0=_f64(self.dc0),
                 dWx=[_f64(t) for t in self.dWx], dWh=[_f64(t) for t in self.dWh], db=[_f64(t) for t in self.db])
        if self.dx is not None:
            r["dx"] = _f64(self.dx)
        if self.w.head in ("xent", "mse"):
            r["dWout"] = _f64(self.dWout)
            r["dbout"] = _f64(self.dbout)
        if self.w.head == "xent":
            r["dE"] = _f64(self.dE)
        return r


class TreeStep:
    """Device state and call sequence of a TreeLSTM training step."""

    def __init__(self, w: wl.TreeWorkload, device="cuda", update: Optional[Tuple[float, float]] = None):
        self.w = w
        self.device = device
        f = torch.float32
        self.desc = J.TreeDesc(w.E_dim, w.H, w.V, J.F32)
        self.emb = _dev(w.emb, f, device)
        self.W = _dev(w.W, f, device)
        self.U = _dev(w.U, f, device)
        self.b = _dev(w.b, f, device)
        self.Ws = _dev(w.Ws, f, device)
        self.bs = _dev(w.bs, f, device)
        K = w.trees.num_trees
        self.labels_host = np.ascontiguousarray(w.labels, np.int32)
        self.labels = torch.from_numpy(self.labels_host).to(device)
        self.h_root = torch.zeros(K, w.H, dtype=f, device=device)
        self.dh_root = torch.zeros(K, w.H, dtype=f, device=device)
        self.demb = torch.zeros(w.V, w.E_dim, dtype=f, device=device)
        self.dW = torch.empty_like(self.W)
        self.dU = torch.empty_like(self.U)
        self.db = torch.empty_like(self.b)
        self.dWs = torch.empty_like(self.Ws)
        self.dbs = torch.empty_like(self.bs)
        self.loss = torch.zeros(1, dtype=f, device=device)
        ws = J.janus_treelstm_workspace_bytes(w.E_dim, w.H, w.V, J.F32, w.trees.num_nodes, K)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        self.xdesc = J.XentDesc(w.C, w.H, K, J.F32)
        self.xws = torch.empty(J.janus_xent_workspace_bytes(w.C, w.H, K, J.F32, J.XENT_FWD_BWD),
                               dtype=torch.uint8, device=device)
        self.update = None
        if update is not None:
            self.update = SgdUpdate([self.emb, self.W, self.U, self.b, self.Ws, self.bs],
                                    [self.demb, self.dW, self.dU, self.db, self.dWs, self.dbs], *update)

    def run(self):
        w = self.w
        J.janus_treelstm_fwd(self.desc, w.trees, self.emb, self.W, self.U, self.b, self.h_root, self.ws)
        J.janus_embed_softmax_xent(self.xdesc, J.XENT_FWD_BWD, self.labels_host, self.labels, table=self.Ws,
                                   bias=self.bs, inp=self.h_root, out=self.dh_root, dtable=self.dWs,
                                   dbias=self.dbs, loss=self.loss, ws=self.xws)
        J.janus_treelstm_bwd(self.desc, w.trees, self.emb, self.W, self.U, self.ws, self.dh_root, self.demb,
                             self.dW, self.dU, self.db)
        if self.update is not None:
            self.update.apply()

    def results(self) -> Dict[str, object]:
        torch.cuda.synchronize()
        return dict(loss=float(self.loss.item()), h_root=_f64(self.h_root), dh_root=_f64(self.dh_root),
                    demb=_f64(self.demb), dW=_f64(self.dW), dU=_f64(self.dU), db=_f64(self.db),
                    dWs=_f64(self.dWs), dbs=_f64(self.dbs))


class TreeRNNStep:
    """Device state and call sequence of a TreeRNN training step."""

    def __init__(self, w: wl.TreeRNNWorkload, device="cuda", update: Optional[Tuple[float, float]] = None):
        self.w = w
        self.device = device
        f = torch.float32
        self.desc = J.TreeDesc(w.H, w.H, w.V, J.F32)
        self.emb = _dev(w.emb, f, device)
        self.W = _dev(w.W, f, device)
        self.b = _dev(w.b, f, device)
        self.Ws = _dev(w.Ws, f, device)
        self.bs = _dev(w.bs, f, device)
        K = w.trees.num_trees
        self.labels_host = np.ascontiguousarray(w.labels, np.int32)
        self.labels = torch.from_numpy(self.labels_host).to(device)
        self.h_root = torch.zeros(K, w.H, dtype=f, device=device)
        self.dh_root = torch.zeros(K, w.H, dtype=f, device=device)
        self.demb = torch.zeros(w.V, w.H, dtype=f, device=device)
        self.dW = torch.empty_like(self.W)
        self.db = torch.empty_like(self.b)
        self.dWs = torch.empty_like(self.Ws)
        self.dbs = torch.empty_like(self.bs)
        self.loss = torch.zeros(1, dtype=f, device=device)
        ws = J.janus_treernn_workspace_bytes(w.H, w.V, w.trees.num_nodes, K)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        self.xdesc = J.XentDesc(w.C, w.H, K, J.F32)
        self.xws = torch.empty(J.janus_xent_workspace_bytes(w.C, w.H, K, J.F32, J.XENT_FWD_BWD),
                               dtype=torch.uint8, device=device)
        self.update = None
        if update is not None:
            self.update = SgdUpdate([self.emb, self.W, self.b, self.Ws, self.bs],
                                    [self.demb, self.dW, self.db, self.dWs, self.dbs], *update)

    def run(self):
        w = self.w
        J.janus_treernn_fwd(self.desc, w.trees, self.emb, self.W, self.b, self.h_root, self.ws)
        J.janus_embed_softmax_xent(self.xdesc, J.XENT_FWD_BWD, self.labels_host, self.labels, table=self.Ws,
                                   bias=self.bs, inp=self.h_root, out=self.dh_root, dtable=self.dWs,
                                   dbias=self.dbs, loss=self.loss, ws=self.xws)
        J.janus_treernn_bwd(self.desc, w.trees, self.W, self.ws, self.dh_root, self.demb, self.dW, self.db)
        if self.update is not None:
            self.update.apply()

    def results(self) -> Dict[str, object]:
        torch.cuda.synchronize()
        return dict(loss=float(self.loss.item()), h_root=_f64(self.h_root), dh_root=_f64(self.dh_root),
                    demb=_f64(self.demb), dW=_f64(self.dW), db=_f64(self.db), dWs=_f64(self.dWs),
                    dbs=_f64(self.dbs))


class ChildSumStep:
    """Device state and call sequence of a Child-Sum TreeLSTM training step."""

    def __init__(self, w: wl.ChildSumWorkload, device="cuda", update: Optional[Tuple[float, float]] = None):
        self.w = w
        self.device = device
        f = torch.float32
        self.desc = J.TreeDesc(w.E_dim, w.H, w.V, J.F32)
        self.emb = _dev(w.emb, f, device)
        self.W = _dev(w.W, f, device)
        self.U = _dev(w.U, f, device)
        self.b = _dev(w.b, f, device)
        self.Ws = _dev(w.Ws, f, device)
        self.bs = _dev(w.bs, f, device)
        K = w.trees.num_trees
        self.labels_host = np.ascontiguousarray(w.labels, np.int32)
        self.labels = torch.from_numpy(self.labels_host).to(device)
        self.h_root = torch.zeros(K, w.H, dtype=f, device=device)
        self.dh_root = torch.zeros(K, w.H, dtype=f, device=device)
        self.demb = torch.zeros(w.V, w.E_dim, dtype=f, device=device)
        self.dW = torch.empty_like(self.W)
        self.dU = torch.empty_like(self.U)
        self.db = torch.empty_like(self.b)
        self.dWs = torch.empty_like(self.Ws)
        self.dbs = torch.empty_like(self.bs)
        self.loss = torch.zeros(1, dtype=f, device=device)
        ws = J.janus_childsum_workspace_bytes(w.E_dim, w.H, w.V, w.trees.num_nodes)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        self.xdesc = J.XentDesc(w.C, w.H, K, J.F32)
        self.xws = torch.empty(J.janus_xent_workspace_bytes(w.C, w.H, K, J.F32, J.XENT_FWD_BWD),
                               dtype=torch.uint8, device=device)
        self.update = None
        if update is not None:
            self.update = SgdUpdate([self.emb, self.W, self.U, self.b, self.Ws, self.bs],
                                    [self.demb, self.dW, self.dU, self.db, self.dWs, self.dbs], *update)

    def run(self):
        w = self.w
        J.janus_childsum_fwd(self.desc, w.trees, self.emb, self.W, self.U, self.b, self.h_root, self.ws)
        J.janus_embed_softmax_xent(self.xdesc, J.XENT_FWD_BWD, self.labels_host, self.labels, table=self.Ws,
                                   bias=self.bs, inp=self.h_root, out=self.dh_root, dtable=self.dWs,
                                   dbias=self.dbs, loss=self.loss, ws=self.xws)
        J.janus_childsum_bwd(self.desc, w.trees, self.emb, self.W, self.U, self.ws, self.dh_root, self.demb,
                             self.dW, self.dU, self.db)
        if self.update is not None:
            self.update.apply()

    def results(self) -> Dict[str, object]:
        torch.cuda.synchronize()
        return dict(loss=float(self.loss.item()), h_root=_f64(self.h_root), dh_root=_f64(self.dh_root),
                    demb=_f64(self.demb), dW=_f64(self.dW), dU=_f64(self.dU), db=_f64(self.db),
                    dWs=_f64(self.dWs), dbs=_f64(self.dbs))


def make_step(w, device="cuda", update: Optional[Tuple[float, float]] = None):
    """The training step of a workload; ``update`` = (lr, max_norm) appends
    the SGD update with global-norm clipping."""
    if isinstance(w, wl.TreeRNNWorkload):
        return TreeRNNStep(w, device, update=update)
    if isinstance(w, wl.ChildSumWorkload):
        return ChildSumStep(w, device, update=update)
    if isinstance(w, wl.TreeWorkload):
        return TreeStep(w, device, update=update)
    return LSTMStep(w, device, update=update)
