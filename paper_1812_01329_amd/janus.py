"""ctypes binding of libjanus.so (declared in include/janus.h).

Argument marshalling only: every function passes device pointers taken from
torch tensors (``tensor.data_ptr()``), host int32 arrays and the current HIP
stream to the C entry point of the same name, and raises ``JanusError`` on a
non-OK status.  Nothing here computes any part of the training step.

The shared library is loaded from the package directory; if it is missing
or fails to load, every call raises immediately (there is no fallback).
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libjanus.so")

OK, ERR_INVALID_ARG, ERR_LENGTH, ERR_TREE, ERR_TOKEN, ERR_WORKSPACE, ERR_UNSUPPORTED, ERR_DEVICE = range(8)
F32, BF16 = 0, 1
EMBED_FWD, XENT_FWD_BWD, EMBED_BWD = 0, 1, 2
LOSS_SUMSQ, LOSS_MEAN = 0, 1

EXPORTS = [
    "janus_lstm_workspace_bytes", "janus_lstm_seq_fwd", "janus_lstm_seq_bwd", "janus_lstm_device_report",
    "janus_lstm_fault_flag", "janus_lstm_schedule",
    "janus_treelstm_workspace_bytes", "janus_tree_schedule_build", "janus_treelstm_fwd",
    "janus_treelstm_bwd", "janus_treelstm_device_report", "janus_xent_workspace_bytes", "janus_embed_softmax_xent",
    "janus_mse_workspace_bytes", "janus_linear_mse", "janus_loss_reduce", "janus_trace_begin",
    "janus_trace_end", "janus_status_string", "janus_version", "janus_last_error",
    "janus_sgd_workspace_bytes", "janus_sgd_clip_update", "janus_sgd_clip_update_noalloc",
    "janus_lstm_state_carry",
    "janus_treernn_workspace_bytes", "janus_treernn_fwd", "janus_treernn_bwd", "janus_treernn_device_report",
    "janus_childsum_workspace_bytes", "janus_childsum_fwd", "janus_childsum_bwd", "janus_childsum_device_report",
]


class JanusError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        self.detail = detail
        super().__init__(f"{where}: {status_string(status)} (status {status})" + (f": {detail}" if detail else ""))


class LstmDesc(C.Structure):
    _fields_ = [("L", C.c_int32), ("I", C.c_int32), ("H", C.c_int32), ("B", C.c_int32),
                ("T", C.c_int32), ("dtype", C.c_int)]


class TreeDesc(C.Structure):
    _fields_ = [("E", C.c_int32), ("H", C.c_int32), ("V", C.c_int32), ("dtype", C.c_int)]


class TreeBatchC(C.Structure):
    _fields_ = [("num_trees", C.c_int32), ("num_nodes", C.c_int32),
                ("left", C.POINTER(C.c_int32)), ("right", C.POINTER(C.c_int32)),
                ("word", C.POINTER(C.c_int32)), ("root", C.POINTER(C.c_int32))]


class NaryBatchC(C.Structure):
    _fields_ = [("num_trees", C.c_int32), ("num_nodes", C.c_int32),
                ("child_offsets", C.POINTER(C.c_int32)), ("children", C.POINTER(C.c_int32)),
                ("word", C.POINTER(C.c_int32)), ("root", C.POINTER(C.c_int32))]


class XentDesc(C.Structure):
    _fields_ = [("V", C.c_int32), ("H", C.c_int32), ("rows", C.c_int32), ("dtype", C.c_int)]


class TraceStat(C.Structure):
    _fields_ = [("label", C.c_char * 48), ("launches", C.c_int64), ("total_ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


class LstmReport(C.Structure):
    _fields_ = [("timed_out", C.c_int32), ("bwd_groups", C.c_int32), ("bwd_local_groups", C.c_int32),
                ("fwd_groups", C.c_int32), ("fwd_local_groups", C.c_int32)]


class MseDesc(C.Structure):
    _fields_ = [("rows", C.c_int32), ("H", C.c_int32), ("P", C.c_int32), ("dtype", C.c_int)]


class SgdDesc(C.Structure):
    _fields_ = [("n", C.c_int32), ("dtype", C.c_int), ("lr", C.c_float), ("max_norm", C.c_float)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_1812_01329_amd.build`")
        # torch brings its own HIP runtime.  Loaded first, it is the one the
        # library binds to; loaded after the library, a second runtime would
        # come up beside the system one, and the library's launches would fail
        # (hipErrorNoDevice) on buffers torch allocated.
        import torch  # noqa: F401
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_size_t
        pi32 = C.POINTER(C.c_int32)
        L.janus_status_string.restype = C.c_char_p
        L.janus_status_string.argtypes = [C.c_int]
        L.janus_version.restype = C.c_char_p
        L.janus_last_error.restype = C.c_char_p
        L.janus_lstm_workspace_bytes.restype = sz
        L.janus_lstm_workspace_bytes.argtypes = [C.POINTER(LstmDesc)]
        L.janus_lstm_seq_fwd.argtypes = [C.POINTER(LstmDesc), vp, pi32, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.janus_lstm_seq_bwd.argtypes = [C.POINTER(LstmDesc), vp, pi32, vp, vp, vp, sz, vp, vp, vp, vp, vp, vp,
                                         vp, vp, vp, vp]
        L.janus_lstm_schedule.argtypes = [i32, i32, pi32, pi32, pi32, pi32, pi32]
        L.janus_lstm_device_report.argtypes = [C.POINTER(LstmDesc), vp, sz, C.POINTER(LstmReport), vp]
        L.janus_lstm_fault_flag.argtypes = [C.POINTER(LstmDesc), vp, sz, C.POINTER(vp)]
        L.janus_treelstm_workspace_bytes.restype = sz
        L.janus_treelstm_workspace_bytes.argtypes = [C.POINTER(TreeDesc), i32, i32]
        L.janus_tree_schedule_build.argtypes = [C.POINTER(TreeBatchC), i32, pi32, pi32, pi32, pi32]
        L.janus_treelstm_fwd.argtypes = [C.POINTER(TreeDesc), C.POINTER(TreeBatchC), vp, vp, vp, vp, vp, vp, sz, vp]
        L.janus_treelstm_bwd.argtypes = [C.POINTER(TreeDesc), C.POINTER(TreeBatchC), vp, vp, vp, vp, sz, vp, vp, vp,
                                         vp, vp, vp]
        L.janus_treelstm_device_report.argtypes = [C.POINTER(TreeDesc), C.POINTER(TreeBatchC), vp, sz,
                                                   C.POINTER(i32), vp]
        L.janus_treernn_workspace_bytes.restype = sz
        L.janus_treernn_workspace_bytes.argtypes = [C.POINTER(TreeDesc), i32, i32]
        L.janus_treernn_fwd.argtypes = [C.POINTER(TreeDesc), C.POINTER(TreeBatchC), vp, vp, vp, vp, vp, sz, vp]
        L.janus_treernn_bwd.argtypes = [C.POINTER(TreeDesc), C.POINTER(TreeBatchC), vp, vp, sz, vp, vp, vp, vp, vp]
        L.janus_treernn_device_report.argtypes = [C.POINTER(TreeDesc), C.POINTER(TreeBatchC), vp, sz,
                                                  C.POINTER(i32), vp]
        L.janus_childsum_workspace_bytes.restype = sz
        L.janus_childsum_workspace_bytes.argtypes = [C.POINTER(TreeDesc), i32]
        L.janus_childsum_fwd.argtypes = [C.POINTER(TreeDesc), C.POINTER(NaryBatchC), vp, vp, vp, vp, vp, vp, sz, vp]
        L.janus_childsum_bwd.argtypes = [C.POINTER(TreeDesc), C.POINTER(NaryBatchC), vp, vp, vp, vp, sz, vp, vp, vp,
                                         vp, vp, vp]
        L.janus_childsum_device_report.argtypes = [C.POINTER(TreeDesc), C.POINTER(NaryBatchC), vp, sz,
                                                   C.POINTER(i32), vp]
        L.janus_xent_workspace_bytes.restype = sz
        L.janus_xent_workspace_bytes.argtypes = [C.POINTER(XentDesc), C.c_int]
        L.janus_embed_softmax_xent.argtypes = [C.POINTER(XentDesc), C.c_int, pi32, vp, vp, vp, vp, vp, vp, vp, vp,
                                               vp, sz, vp]
        L.janus_lstm_state_carry.argtypes = [C.POINTER(LstmDesc), i32, vp, vp, vp, vp, vp]
        L.janus_sgd_workspace_bytes.restype = sz
        L.janus_sgd_workspace_bytes.argtypes = [C.POINTER(SgdDesc)]
        L.janus_sgd_clip_update.argtypes = [C.POINTER(SgdDesc), C.POINTER(vp), C.POINTER(vp),
                                            C.POINTER(C.c_int64), vp, vp, vp, sz, vp]
        L.janus_sgd_clip_update_noalloc.argtypes = [C.POINTER(SgdDesc), C.POINTER(vp), C.POINTER(vp),
                                                    C.POINTER(C.c_int64), vp, vp, vp]
        L.janus_mse_workspace_bytes.restype = sz
        L.janus_mse_workspace_bytes.argtypes = [C.POINTER(MseDesc)]
        L.janus_linear_mse.argtypes = [C.POINTER(MseDesc), vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.janus_loss_reduce.argtypes = [C.c_int, vp, i64, vp, vp, vp]
        L.janus_trace_begin.argtypes = []
        L.janus_trace_end.argtypes = [C.POINTER(TraceStat), i32, C.POINTER(C.c_int32)]
        for name in EXPORTS:
            if name not in ("janus_status_string", "janus_version", "janus_last_error") and "workspace_bytes" not in name:
                getattr(L, name).restype = C.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().janus_status_string(status).decode()


def version() -> str:
    return lib().janus_version().decode()


# ---------------------------------------------------------------- helpers
def _p(t) -> Optional[int]:
    """Device pointer of a tensor (or None)."""
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> Optional[int]:
    if stream is not None:
        return stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _ptr_array(tensors: Sequence) -> C.Array:
    arr = (C.c_void_p * len(tensors))()
    for i, t in enumerate(tensors):
        arr[i] = _p(t)
    return arr


def _i32(a) -> Optional[np.ndarray]:
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


def _i32p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.POINTER(C.c_int32))


def last_error() -> str:
    """Which HIP call failed behind the last DEVICE status on this thread."""
    return lib().janus_last_error().decode()


def _check(st: int, where: str):
    if st != OK:
        raise JanusError(st, where, last_error() if st == ERR_DEVICE else "")


def _tree_c(left, right, word, root):
    arrs = [_i32(a) for a in (left, right, word, root)]
    tb = TreeBatchC(len(arrs[3]), len(arrs[0]), *[_i32p(a) for a in arrs])
    return tb, arrs   # keep the arrays alive with the struct


# ---------------------------------------------------------------- LSTM
def janus_lstm_workspace_bytes(L, I, H, B, T, dtype) -> int:
    return int(lib().janus_lstm_workspace_bytes(C.byref(LstmDesc(L, I, H, B, T, dtype))))


def janus_lstm_seq_fwd(desc: LstmDesc, x, lengths, Wx, Wh, b, h0, c0, y, hT, cT, ws, stream=None):
    lens = _i32(lengths)
    st = lib().janus_lstm_seq_fwd(C.byref(desc), _p(x), _i32p(lens), _ptr_array(Wx), _ptr_array(Wh),
                                  _ptr_array(b), _p(h0), _p(c0), _p(y), _p(hT), _p(cT), _p(ws),
                                  ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "janus_lstm_seq_fwd")


def janus_lstm_seq_bwd(desc: LstmDesc, x, lengths, Wx, Wh, ws, dy, dhT, dcT, dx, dh0, dc0, dWx, dWh, db,
                       stream=None):
    lens = _i32(lengths)
    st = lib().janus_lstm_seq_bwd(C.byref(desc), _p(x), _i32p(lens), _ptr_array(Wx), _ptr_array(Wh), _p(ws),
                                  ws.numel() * ws.element_size(), _p(dy), _p(dhT), _p(dcT), _p(dx), _p(dh0),
                                  _p(dc0), _ptr_array(dWx), _ptr_array(dWh), _ptr_array(db), _stream(stream))
    _check(st, "janus_lstm_seq_bwd")


def janus_lstm_device_report(desc: LstmDesc, ws, stream=None) -> dict:
    """Synchronises the stream and returns the report of the current step on
    this workspace (the last forward and the backward after it); raises
    JanusError(DEVICE) if a barrier wait ran out."""
    rep = LstmReport()
    st = lib().janus_lstm_device_report(C.byref(desc), _p(ws), ws.numel() * ws.element_size(), C.byref(rep),
                                        _stream(stream))
    _check(st, "janus_lstm_device_report")
    return dict(timed_out=int(rep.timed_out), bwd_groups=int(rep.bwd_groups),
                bwd_local_groups=int(rep.bwd_local_groups), fwd_groups=int(rep.fwd_groups),
                fwd_local_groups=int(rep.fwd_local_groups))


def janus_lstm_fault_flag(desc: LstmDesc, ws) -> int:
    """Device address of the workspace's timeout word (see janus.h)."""
    out = C.c_void_p(0)
    st = lib().janus_lstm_fault_flag(C.byref(desc), _p(ws), ws.numel() * ws.element_size(), C.byref(out))
    _check(st, "janus_lstm_fault_flag")
    return int(out.value)


def janus_lstm_schedule(B: int, T: int, lengths):
    """Host-only schedule: returns (perm, active[T], offsets[T+1], t_eff)."""
    lens = _i32(lengths)
    perm = np.zeros(B, np.int32)
    active = np.zeros(max(T, 1), np.int32)
    offsets = np.zeros(T + 1, np.int32)
    t_eff = C.c_int32(0)
    st = lib().janus_lstm_schedule(B, T, _i32p(lens), _i32p(perm), _i32p(active), _i32p(offsets), C.byref(t_eff))
    _check(st, "janus_lstm_schedule")
    return perm, active[:T], offsets, int(t_eff.value)


# ---------------------------------------------------------------- TreeLSTM
def janus_treelstm_workspace_bytes(E, H, V, dtype, max_nodes, max_trees) -> int:
    return int(lib().janus_treelstm_workspace_bytes(C.byref(TreeDesc(E, H, V, dtype)), max_nodes, max_trees))


def janus_tree_schedule_build(left, right, word, root, V):
    """Host-only frontier schedule: returns (node_level, level_offsets, level_nodes, num_levels)."""
    tb, keep = _tree_c(left, right, word, root)
    N = tb.num_nodes
    level = np.zeros(max(N, 1), np.int32)
    offsets = np.zeros(N + 1, np.int32)
    nodes = np.zeros(max(N, 1), np.int32)
    L = C.c_int32(0)
    st = lib().janus_tree_schedule_build(C.byref(tb), V, _i32p(level), _i32p(offsets), _i32p(nodes), C.byref(L))
    _check(st, "janus_tree_schedule_build")
    L = int(L.value)
    return level[:N], offsets[:L + 1], nodes[:N], L


def janus_treelstm_fwd(desc: TreeDesc, trees, emb, W, U, b, h_root, ws, stream=None):
    tb, keep = _tree_c(trees.left, trees.right, trees.word, trees.root)
    st = lib().janus_treelstm_fwd(C.byref(desc), C.byref(tb), _p(emb), _p(W), _p(U), _p(b), _p(h_root), _p(ws),
                                  ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "janus_treelstm_fwd")


def janus_treelstm_bwd(desc: TreeDesc, trees, emb, W, U, ws, dh_root, demb, dW, dU, db, stream=None):
    tb, keep = _tree_c(trees.left, trees.right, trees.word, trees.root)
    st = lib().janus_treelstm_bwd(C.byref(desc), C.byref(tb), _p(emb), _p(W), _p(U), _p(ws),
                                  ws.numel() * ws.element_size(), _p(dh_root), _p(demb), _p(dW), _p(dU), _p(db),
                                  _stream(stream))
    _check(st, "janus_treelstm_bwd")


def janus_treelstm_device_report(desc: TreeDesc, trees, ws, stream=None) -> int:
    """Synchronises the stream and returns 1 if a level barrier of the last
    TreeLSTM forward or backward on this workspace ran out of its wait (the
    call then raises JanusError(DEVICE)), else 0."""
    tb, keep = _tree_c(trees.left, trees.right, trees.word, trees.root)
    out = C.c_int32(0)
    st = lib().janus_treelstm_device_report(C.byref(desc), C.byref(tb), _p(ws), ws.numel() * ws.element_size(),
                                            C.byref(out), _stream(stream))
    _check(st, "janus_treelstm_device_report")
    return int(out.value)


def janus_treernn_device_report(desc: TreeDesc, trees, ws, stream=None) -> int:
    """Synchronises the stream and returns 1 if a level barrier of the last
    TreeRNN forward or backward on this workspace ran out of its wait (the
    call then raises JanusError(DEVICE)), else 0."""
    tb, keep = _tree_c(trees.left, trees.right, trees.word, trees.root)
    out = C.c_int32(0)
    st = lib().janus_treernn_device_report(C.byref(desc), C.byref(tb), _p(ws), ws.numel() * ws.element_size(),
                                           C.byref(out), _stream(stream))
    _check(st, "janus_treernn_device_report")
    return int(out.value)


def janus_treernn_workspace_bytes(H, V, max_nodes, max_trees) -> int:
    return int(lib().janus_treernn_workspace_bytes(C.byref(TreeDesc(H, H, V, F32)), max_nodes, max_trees))


def janus_treernn_fwd(desc: TreeDesc, trees, emb, W, b, h_root, ws, stream=None):
    tb, keep = _tree_c(trees.left, trees.right, trees.word, trees.root)
    st = lib().janus_treernn_fwd(C.byref(desc), C.byref(tb), _p(emb), _p(W), _p(b), _p(h_root), _p(ws),
                                 ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "janus_treernn_fwd")


def janus_treernn_bwd(desc: TreeDesc, trees, W, ws, dh_root, demb, dW, db, stream=None):
    tb, keep = _tree_c(trees.left, trees.right, trees.word, trees.root)
    st = lib().janus_treernn_bwd(C.byref(desc), C.byref(tb), _p(W), _p(ws), ws.numel() * ws.element_size(),
                                 _p(dh_root), _p(demb), _p(dW), _p(db), _stream(stream))
    _check(st, "janus_treernn_bwd")


def _nary_c(trees):
    arrs = [np.ascontiguousarray(a, dtype=np.int32) for a in
            (trees.child_offsets, trees.children, trees.word, trees.root)]
    tb = NaryBatchC(len(arrs[3]), len(arrs[2]), *[_i32p(a) for a in arrs])
    return tb, arrs   # keep the arrays alive with the struct


def janus_childsum_workspace_bytes(E, H, V, max_nodes) -> int:
    return int(lib().janus_childsum_workspace_bytes(C.byref(TreeDesc(E, H, V, F32)), max_nodes))


def janus_childsum_fwd(desc: TreeDesc, trees, emb, W, U, b, h_root, ws, stream=None):
    tb, keep = _nary_c(trees)
    st = lib().janus_childsum_fwd(C.byref(desc), C.byref(tb), _p(emb), _p(W), _p(U), _p(b), _p(h_root), _p(ws),
                                  ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "janus_childsum_fwd")


def janus_childsum_bwd(desc: TreeDesc, trees, emb, W, U, ws, dh_root, demb, dW, dU, db, stream=None):
    tb, keep = _nary_c(trees)
    st = lib().janus_childsum_bwd(C.byref(desc), C.byref(tb), _p(emb), _p(W), _p(U), _p(ws),
                                  ws.numel() * ws.element_size(), _p(dh_root), _p(demb), _p(dW), _p(dU), _p(db),
                                  _stream(stream))
    _check(st, "janus_childsum_bwd")


def janus_childsum_device_report(desc: TreeDesc, trees, ws, stream=None) -> int:
    """Synchronises the stream and returns 1 if a level barrier of the last
    Child-Sum forward or backward on this workspace ran out of its wait (the
    call then raises JanusError(DEVICE)), else 0."""
    tb, keep = _nary_c(trees)
    out = C.c_int32(0)
    st = lib().janus_childsum_device_report(C.byref(desc), C.byref(tb), _p(ws), ws.numel() * ws.element_size(),
                                            C.byref(out), _stream(stream))
    _check(st, "janus_childsum_device_report")
    return int(out.value)


# ---------------------------------------------------------------- heads
def janus_xent_workspace_bytes(V, H, rows, dtype, op) -> int:
    return int(lib().janus_xent_workspace_bytes(C.byref(XentDesc(V, H, rows, dtype)), op))


def janus_embed_softmax_xent(desc: XentDesc, op, ids_host, ids_dev, table=None, bias=None, inp=None, out=None,
                             dtable=None, dbias=None, loss=None, ws=None, stream=None):
    ids = _i32(ids_host)
    st = lib().janus_embed_softmax_xent(C.byref(desc), op, _i32p(ids), _p(ids_dev), _p(table), _p(bias), _p(inp),
                                        _p(out), _p(dtable), _p(dbias), _p(loss), _p(ws),
                                        0 if ws is None else ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "janus_embed_softmax_xent")


def janus_mse_workspace_bytes(rows, H, P, dtype) -> int:
    return int(lib().janus_mse_workspace_bytes(C.byref(MseDesc(rows, H, P, dtype))))


def janus_linear_mse(desc: MseDesc, h, W, b, target, dh, dW, db, loss, ws, stream=None):
    st = lib().janus_linear_mse(C.byref(desc), _p(h), _p(W), _p(b), _p(target), _p(dh), _p(dW), _p(db), _p(loss),
                                _p(ws), ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "janus_linear_mse")


def janus_loss_reduce(kind, h, n, loss, dh, stream=None):
    st = lib().janus_loss_reduce(kind, _p(h), n, _p(loss), _p(dh), _stream(stream))
    _check(st, "janus_loss_reduce")


def janus_lstm_state_carry(desc: LstmDesc, B_prev: int, hT, cT, h0, c0, stream=None):
    """Initial state of the next batch (desc.B rows) from the final state of
    the previous one (B_prev rows)."""
    st = lib().janus_lstm_state_carry(C.byref(desc), int(B_prev), _p(hT), _p(cT), _p(h0), _p(c0), _stream(stream))
    _check(st, "janus_lstm_state_carry")


# ---------------------------------------------------------------- update
def sgd_workspace_bytes(desc: SgdDesc) -> int:
    return int(lib().janus_sgd_workspace_bytes(C.byref(desc)))


def janus_sgd_clip_update(desc: SgdDesc, params, grads, stats=None, ws=None, stream=None, hold=None):
    """SGD step with global-norm clipping on lists of flat device tensors
    (parameters updated in place; float32 gradients).  ``hold``: a device
    address (int) of a uint32 that, when non-zero, keeps the update from
    writing anything (janus_lstm_fault_flag's word)."""
    n = len(params)
    S = (C.c_int64 * n)(*[int(t.numel()) for t in params])
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    st = lib().janus_sgd_clip_update(C.byref(desc), _ptr_array(params), _ptr_array(grads), S, _p(stats),
                                     None if hold is None else C.c_void_p(int(hold)), _p(ws), wsb, _stream(stream))
    _check(st, "janus_sgd_clip_update")


SGD_NOALLOC_MAX_TENSORS = 256   # JANUS_SGD_NOALLOC_MAX_TENSORS


def janus_sgd_clip_update_noalloc(desc: SgdDesc, params, grads, stats=None, stream=None, hold=None):
    """janus_sgd_clip_update without a workspace (the library's fixed
    per-device array; at most SGD_NOALLOC_MAX_TENSORS tensors)."""
    n = len(params)
    S = (C.c_int64 * n)(*[int(t.numel()) for t in params])
    st = lib().janus_sgd_clip_update_noalloc(C.byref(desc), _ptr_array(params), _ptr_array(grads), S, _p(stats),
                                             None if hold is None else C.c_void_p(int(hold)), _stream(stream))
    _check(st, "janus_sgd_clip_update_noalloc")


# ---------------------------------------------------------------- tracing
def janus_trace_begin():
    _check(lib().janus_trace_begin(), "janus_trace_begin")


def janus_trace_end(max_out: int = 128):
    """Per-label kernel statistics of the launches since janus_trace_begin."""
    out = (TraceStat * max_out)()
    n = C.c_int32(0)
    _check(lib().janus_trace_end(out, max_out, C.byref(n)), "janus_trace_end")
    return [dict(label=out[i].label.decode(), launches=int(out[i].launches), total_ms=float(out[i].total_ms),
                 flops=float(out[i].flops), bytes=float(out[i].bytes)) for i in range(min(n.value, max_out))]
