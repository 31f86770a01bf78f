"""Host-side tests of the C ABI (no GPU needed): the library loads and
exports every declared symbol, the integer schedules match the oracle's bit
for bit, and invalid calls are rejected before any device work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle import schedule as osched
from paper_1812_01329_amd import janus as J
from paper_1812_01329_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    src = open(os.path.join(ROOT, "include", "janus.h")).read()
    return sorted(set(re.findall(r"\b(janus_[a-z_0-9]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = J.lib()
    decl = declared_symbols()
    assert len(decl) >= 15
    for name in decl:
        assert hasattr(lib, name), name
    assert set(decl) == set(J.EXPORTS)
    assert "gfx950" in J.version()
    for s in range(8):
        assert J.status_string(s)


@pytest.mark.parametrize("seed", range(8))
def test_seq_schedule_bit_exact(seed):
    rng = np.random.default_rng(seed)
    for _ in range(250):
        B = int(rng.integers(1, 300)); T = int(rng.integers(0, 260))
        mode = rng.integers(0, 3)
        if mode == 0:
            lengths = rng.integers(0, T + 1, B)
        elif mode == 1:
            lengths = np.full(B, T)
        else:
            lengths = rng.choice([0, T, T // 2], B)
        perm, active, offsets, t_eff = J.janus_lstm_schedule(B, T, lengths)
        operm, oactive, ooffsets, ot_eff = osched.seq_schedule(lengths, T)
        assert t_eff == ot_eff
        assert np.array_equal(perm, operm)
        assert np.array_equal(active[:t_eff], oactive)
        assert np.all(active[t_eff:] == 0)
        assert np.array_equal(offsets[:t_eff + 1], ooffsets)
        assert np.all(offsets[t_eff:] == offsets[t_eff])


@pytest.mark.parametrize("seed", range(8))
def test_tree_schedule_bit_exact(seed):
    rng = np.random.default_rng(100 + seed)
    for _ in range(150):
        t = wl.make_trees(rng, int(rng.integers(1, 30)), 1, int(rng.integers(1, 60)), 500)
        if rng.random() < 0.5:   # arbitrary node numbering
            N = t.num_nodes
            p = rng.permutation(N)
            inv = np.argsort(p)
            remap = lambda a: np.where(a >= 0, p[np.maximum(a, 0)], -1).astype(np.int32)
            t = wl.TreeBatch(remap(t.left)[inv], remap(t.right)[inv], t.word[inv], p[t.root].astype(np.int32))
        lev, off, nodes, L = J.janus_tree_schedule_build(t.left, t.right, t.word, t.root, 500)
        olev, ooff, onodes, oL = osched.tree_schedule(t.left, t.right, t.word, t.root, 500)
        assert L == oL
        assert np.array_equal(lev, olev)
        assert np.array_equal(off, ooff)
        assert np.array_equal(nodes, onodes)


def _tree(left, right, word, root):
    return [np.asarray(a, np.int32) for a in (left, right, word, root)]


@pytest.mark.parametrize("case,status", [
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 2, -1], [2]), J.OK),
    (_tree([-1, -1, 0], [-1, -1, -1], [1, 2, -1], [2]), J.ERR_TREE),
    (_tree([-1, -1, 0], [-1, -1, 0], [1, 2, -1], [2]), J.ERR_TREE),
    (_tree([-1, -1, 0, 0], [-1, -1, 1, 1], [1, 2, -1, -1], [2, 3]), J.ERR_TREE),
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 9, -1], [2]), J.ERR_TOKEN),
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 2, 4], [2]), J.ERR_TREE),
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 2, -1], [1]), J.ERR_TREE),
    (_tree([-1, 2, 1], [-1, 0, 0], [1, -1, -1], [0]), J.ERR_TREE),
    (_tree([-1, -1, 0], [-1, -1, 5], [1, 2, -1], [2]), J.ERR_TREE),
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 2, -1], [2, 2]), J.ERR_TREE),
])
def test_tree_validation_status(case, status):
    kind = {J.OK: None, J.ERR_TREE: "tree", J.ERR_TOKEN: "token"}[status]
    if status == J.OK:
        J.janus_tree_schedule_build(*case, 5)
        osched.tree_schedule(*case, 5)
    else:
        with pytest.raises(J.JanusError) as e:
            J.janus_tree_schedule_build(*case, 5)
        assert e.value.status == status
        with pytest.raises(osched.ScheduleError) as oe:
            osched.tree_schedule(*case, 5)
        assert oe.value.kind == kind


class _HostBuf:
    """A host buffer standing in for a device tensor in calls that must be
    rejected before any device access; filled with a sentinel."""
    def __init__(self, nbytes, fill=0x5A):
        self.a = np.full(max(nbytes, 1), fill, np.uint8)

    def data_ptr(self):
        return self.a.ctypes.data

    def numel(self):
        return self.a.size

    def element_size(self):
        return 1

    def untouched(self, fill=0x5A):
        return bool(np.all(self.a == fill))


def _lstm_args(L=1, I=4, H=8, B=3, T=5, dtype=J.F32, ws_bytes=None):
    d = J.LstmDesc(L, I, H, B, T, dtype)
    need = J.janus_lstm_workspace_bytes(L, I, H, B, T, dtype)
    es = 2 if dtype == J.BF16 else 4
    bufs = dict(x=_HostBuf(T * B * I * es), y=_HostBuf(T * B * H * es), hT=_HostBuf(L * B * H * 4),
                cT=_HostBuf(L * B * H * 4), ws=_HostBuf(need if ws_bytes is None else ws_bytes))
    W = [_HostBuf(4 * H * I * es) for _ in range(L)]
    U = [_HostBuf(4 * H * H * es) for _ in range(L)]
    b = [_HostBuf(4 * H * es) for _ in range(L)]
    return d, bufs, W, U, b


@pytest.mark.parametrize("lengths,status", [
    ([5, -1, 2], J.ERR_LENGTH),
    ([6, 1, 2], J.ERR_LENGTH),
])
def test_lstm_rejects_bad_lengths_untouched(lengths, status):
    d, bf, W, U, b = _lstm_args()
    with pytest.raises(J.JanusError) as e:
        J.janus_lstm_seq_fwd(d, bf["x"], lengths, W, U, b, None, None, bf["y"], bf["hT"], bf["cT"], bf["ws"],
                             stream=0)
    assert e.value.status == status
    assert all(v.untouched() for v in bf.values())


def test_lstm_rejects_small_workspace_and_bad_desc():
    d, bf, W, U, b = _lstm_args(ws_bytes=1024)
    with pytest.raises(J.JanusError) as e:
        J.janus_lstm_seq_fwd(d, bf["x"], None, W, U, b, None, None, bf["y"], bf["hT"], bf["cT"], bf["ws"], stream=0)
    assert e.value.status == J.ERR_WORKSPACE
    assert all(v.untouched() for v in bf.values())
    for bad in (J.LstmDesc(0, 4, 8, 3, 5, J.F32), J.LstmDesc(1, 4, -8, 3, 5, J.F32), J.LstmDesc(1, 4, 8, 3, -1, J.F32)):
        with pytest.raises(J.JanusError) as e:
            J.janus_lstm_seq_fwd(bad, bf["x"], None, W, U, b, None, None, bf["y"], bf["hT"], bf["cT"], bf["ws"],
                                 stream=0)
        assert e.value.status == J.ERR_INVALID_ARG
    with pytest.raises(J.JanusError) as e:
        J.janus_lstm_seq_fwd(J.LstmDesc(1, 4, 8, 3, 5, 7), bf["x"], None, W, U, b, None, None, bf["y"], bf["hT"],
                             bf["cT"], bf["ws"], stream=0)
    assert e.value.status == J.ERR_UNSUPPORTED
    with pytest.raises(J.JanusError) as e:
        J.janus_lstm_seq_fwd(d, None, None, W, U, b, None, None, bf["y"], bf["hT"], bf["cT"], bf["ws"], stream=0)
    assert e.value.status == J.ERR_INVALID_ARG
    assert all(v.untouched() for v in bf.values())


def test_lstm_device_report_rejects_bad_arguments():
    """The report call validates before it touches the device."""
    import ctypes as C
    d, bf, W, U, b = _lstm_args(ws_bytes=1024)
    rep = J.LstmReport()
    L = J.lib()
    assert L.janus_lstm_device_report(C.byref(d), None, 0, None, None) == J.ERR_INVALID_ARG
    assert L.janus_lstm_device_report(C.byref(d), None, 0, C.byref(rep), None) == J.ERR_WORKSPACE
    with pytest.raises(J.JanusError) as e:
        J.janus_lstm_device_report(d, bf["ws"], stream=0)
    assert e.value.status == J.ERR_WORKSPACE
    with pytest.raises(J.JanusError) as e:
        J.janus_lstm_device_report(J.LstmDesc(1, 4, 8, 3, 5, 7), bf["ws"], stream=0)
    assert e.value.status == J.ERR_UNSUPPORTED


def test_lstm_fault_flag_address():
    """The timeout word is a 4-byte-aligned word inside the workspace; the
    call validates like the report and reads or writes no memory (a host
    buffer stands in for the workspace)."""
    import ctypes as C
    L = J.lib()
    for (nl, I, H, B, T, dt) in [(2, 64, 256, 32, 8, J.BF16), (1, 4, 8, 3, 5, J.F32), (2, 650, 650, 20, 35, J.BF16)]:
        d = J.LstmDesc(nl, I, H, B, T, dt)
        need = J.janus_lstm_workspace_bytes(nl, I, H, B, T, dt)
        raw = np.full(need + 512, 0x5A, np.uint8)
        base = raw.ctypes.data + (-raw.ctypes.data) % 256
        out = C.c_void_p(0)
        assert L.janus_lstm_fault_flag(C.byref(d), C.c_void_p(base), need, C.byref(out)) == J.OK
        assert base <= out.value <= base + need - 4 and out.value % 4 == 0
        assert np.all(raw == 0x5A)
        assert L.janus_lstm_fault_flag(C.byref(d), C.c_void_p(base), need, None) == J.ERR_INVALID_ARG
        assert L.janus_lstm_fault_flag(C.byref(d), None, need, C.byref(out)) == J.ERR_WORKSPACE
        assert L.janus_lstm_fault_flag(C.byref(d), C.c_void_p(base), need - 1, C.byref(out)) == J.ERR_WORKSPACE
        assert L.janus_lstm_fault_flag(C.byref(d), C.c_void_p(base + 16), need, C.byref(out)) == J.ERR_WORKSPACE
    bad = J.LstmDesc(1, 4, 8, 3, 5, 7)
    assert L.janus_lstm_fault_flag(C.byref(bad), C.c_void_p(base), need, C.byref(out)) == J.ERR_UNSUPPORTED


def test_lstm_bwd_rejects_bad_lengths_untouched():
    d, bf, W, U, b = _lstm_args()
    g = [_HostBuf(4 * 8 * 4 * 4) for _ in range(3)]
    with pytest.raises(J.JanusError) as e:
        J.janus_lstm_seq_bwd(d, bf["x"], [1, 2, 9], W, U, bf["ws"], bf["y"], None, None, None, None, None,
                             [g[0]], [g[1]], [g[2]], stream=0)
    assert e.value.status == J.ERR_LENGTH
    assert all(v.untouched() for v in bf.values()) and all(v.untouched() for v in g)


def test_tree_calls_reject_malformed_trees_untouched():
    left, right, word, root = _tree([-1, -1, 0], [-1, -1, -1], [1, 2, -1], [2])
    t = wl.TreeBatch(left, right, word, root)
    E, H, V = 4, 3, 5
    need = J.janus_treelstm_workspace_bytes(E, H, V, J.F32, 3, 1)
    bufs = [_HostBuf(n) for n in (V * E * 4, 5 * H * E * 4, 5 * H * 2 * H * 4, 5 * H * 4, H * 4, need)]
    with pytest.raises(J.JanusError) as e:
        J.janus_treelstm_fwd(J.TreeDesc(E, H, V, J.F32), t, *bufs, stream=0)
    assert e.value.status == J.ERR_TREE
    assert all(v.untouched() for v in bufs)
    t2 = wl.TreeBatch(*_tree([-1, -1, 0], [-1, -1, 1], [1, 7, -1], [2]))
    with pytest.raises(J.JanusError) as e:
        J.janus_treelstm_fwd(J.TreeDesc(E, H, V, J.F32), t2, *bufs, stream=0)
    assert e.value.status == J.ERR_TOKEN
    with pytest.raises(J.JanusError) as e:
        J.janus_treelstm_fwd(J.TreeDesc(E, H, V, J.BF16), wl.TreeBatch(*_tree([-1], [-1], [1], [0])), *bufs, stream=0)
    assert e.value.status == J.ERR_UNSUPPORTED
    assert all(v.untouched() for v in bufs)


def test_xent_rejects_bad_ids_untouched():
    V, H, R = 10, 4, 6
    d = J.XentDesc(V, H, R, J.F32)
    bufs = dict(table=_HostBuf(V * H * 4), bias=_HostBuf(V * 4), inp=_HostBuf(R * H * 4), out=_HostBuf(R * H * 4),
                dtable=_HostBuf(V * H * 4), dbias=_HostBuf(V * 4), loss=_HostBuf(4),
                ws=_HostBuf(J.janus_xent_workspace_bytes(V, H, R, J.F32, J.XENT_FWD_BWD)))
    ids_dev = _HostBuf(R * 4)
    for op in (J.EMBED_FWD, J.XENT_FWD_BWD, J.EMBED_BWD):
        with pytest.raises(J.JanusError) as e:
            J.janus_embed_softmax_xent(d, op, np.array([0, 1, 2, 10, 3, 4]), ids_dev, stream=0, **bufs)
        assert e.value.status == J.ERR_TOKEN
        with pytest.raises(J.JanusError) as e:
            J.janus_embed_softmax_xent(d, op, np.array([0, 1, -2, 1, 3, 4]), ids_dev, stream=0, **bufs)
        assert e.value.status == J.ERR_TOKEN
    assert all(v.untouched() for v in bufs.values()) and ids_dev.untouched()


def test_workspace_sizes_monotone():
    a = J.janus_lstm_workspace_bytes(1, 32, 64, 4, 16, J.F32)
    b = J.janus_lstm_workspace_bytes(1, 32, 64, 4, 32, J.F32)
    c = J.janus_lstm_workspace_bytes(2, 32, 64, 4, 32, J.F32)
    assert 0 < a < b < c
    assert J.janus_lstm_workspace_bytes(0, 32, 64, 4, 16, J.F32) == 0


def test_one_hip_runtime_whatever_the_import_order():
    """torch ships its own HIP runtime.  Using the binding before torch is
    imported must still leave one runtime in the process (the library binds
    to torch's); two runtimes made the library's launches fail with
    hipErrorNoDevice on tensors torch allocated."""
    import subprocess
    import sys
    code = (
        "from paper_1812_01329_amd import janus as J\n"
        "J.janus_trace_begin()\n"
        "import torch\n"
        "maps = [l.split()[-1] for l in open('/proc/self/maps') if 'amdhip64' in l and 'r-xp' in l]\n"
        "print(len(set(maps)))\n"
    )
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=600)
    assert out.returncode == 0, out.stderr[-2000:]
    assert out.stdout.strip().splitlines()[-1] == "1", out.stdout


def test_last_error_text_is_readable():
    """janus_last_error names the failing HIP call after a DEVICE status; it
    is a plain (possibly empty) string otherwise."""
    assert isinstance(J.last_error(), str)


def _sgd_call(desc, params, grads, sizes, ws, ws_bytes):
    L = J.lib()
    n = len(sizes)
    P = (C.c_void_p * max(n, 1))(*params)
    G = (C.c_void_p * max(n, 1))(*grads)
    S = (C.c_int64 * max(n, 1))(*sizes)
    return L.janus_sgd_clip_update(None if desc is None else C.byref(desc), P, G, S, None, None, ws, ws_bytes, None)


def test_sgd_workspace_bytes():
    d = J.SgdDesc(1, J.F32, 0.1, 1.0)
    one = J.sgd_workspace_bytes(d)
    assert one > 0 and one % 256 == 0
    d.n = 65   # a second table of tensors needs its own block sums
    assert J.sgd_workspace_bytes(d) > one
    d.n = 0
    assert J.sgd_workspace_bytes(d) == 0


@pytest.mark.parametrize("case,status", [
    ("null_desc", J.ERR_INVALID_ARG), ("n0", J.ERR_INVALID_ARG), ("dtype", J.ERR_UNSUPPORTED),
    ("lr_nan", J.ERR_INVALID_ARG), ("lr_inf", J.ERR_INVALID_ARG), ("max_norm_nan", J.ERR_INVALID_ARG),
    ("neg_size", J.ERR_INVALID_ARG), ("null_ptr", J.ERR_INVALID_ARG), ("grad_unaligned", J.ERR_INVALID_ARG),
    ("param_unaligned", J.ERR_INVALID_ARG), ("ws_null", J.ERR_WORKSPACE), ("ws_small", J.ERR_WORKSPACE),
    ("ws_unaligned", J.ERR_WORKSPACE)])
def test_sgd_rejects_bad_arguments(case, status):
    """Every error is found before the first device operation (fake device
    pointers, never dereferenced)."""
    d = J.SgdDesc(2, J.BF16, 0.1, 1.0)
    params, grads, sizes = [0x100000, 0x200000], [0x300000, 0x400000], [10, 0]
    ws = 0x500000
    wsb = J.sgd_workspace_bytes(d)
    if case == "null_desc":
        d = None
    elif case == "n0":
        d.n = 0
    elif case == "dtype":
        d.dtype = 7
    elif case == "lr_nan":
        d.lr = float("nan")
    elif case == "lr_inf":
        d.lr = float("inf")
    elif case == "max_norm_nan":
        d.max_norm = float("nan")
    elif case == "neg_size":
        sizes[1] = -1
    elif case == "null_ptr":
        grads[0] = 0
    elif case == "grad_unaligned":
        grads[0] += 2
    elif case == "param_unaligned":
        params[0] += 1
    elif case == "ws_null":
        ws = 0
    elif case == "ws_small":
        wsb -= 256
    elif case == "ws_unaligned":
        ws += 64
    assert _sgd_call(d, params, grads, sizes, ws, wsb) == status


@pytest.mark.parametrize("case", ["neg", "null_h0", "null_hT", "overlap"])
def test_state_carry_rejects_bad_arguments(case):
    """Checked before any device operation (fake pointers, never used)."""
    L = J.lib()
    d = J.LstmDesc(2, 8, 16, 4, 3, J.F32)
    n = 2 * 4 * 16 * 4
    Bp, hT, cT, h0, c0 = 4, 0x100000, 0x200000, 0x300000, 0x400000
    if case == "neg":
        Bp = -1
    elif case == "null_h0":
        h0 = 0
    elif case == "null_hT":
        hT = 0
    elif case == "overlap":
        c0 = h0 + n // 2
    st = L.janus_lstm_state_carry(C.byref(d), Bp, hT, cT, h0, c0, None)
    assert st == J.ERR_INVALID_ARG


def test_treernn_needs_equal_embedding_and_hidden_width():
    L = J.lib()
    d = J.TreeDesc(300, 150, 100, J.F32)
    assert L.janus_treernn_workspace_bytes(C.byref(d), 10, 2) == 0
    d.E = 150
    assert L.janus_treernn_workspace_bytes(C.byref(d), 10, 2) > 0
    left, right, word, root = (np.array(v, np.int32) for v in ([-1, -1, 0], [-1, -1, 1], [3, 4, -1], [2]))
    tb, keep = J._tree_c(left, right, word, root)
    d.E = 300
    st = L.janus_treernn_fwd(C.byref(d), C.byref(tb), 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 1 << 20, None)
    assert st == J.ERR_INVALID_ARG
    d.E = 150
    bad = J._tree_c(np.array([-1, 0, 1], np.int32), np.array([-1, -1, 0], np.int32),
                    np.array([3, -1, -1], np.int32), np.array([2], np.int32))[0]   # a node with one child
    st = L.janus_treernn_fwd(C.byref(d), C.byref(bad), 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, 1 << 20, None)
    assert st == J.ERR_TREE


@pytest.mark.parametrize("case,status", [
    ("ok_but_no_ws", J.ERR_WORKSPACE), ("offset0", J.ERR_TREE), ("decreasing", J.ERR_TREE),
    ("child_range", J.ERR_TREE), ("two_parents", J.ERR_TREE), ("root_has_parent", J.ERR_TREE),
    ("cycle", J.ERR_TREE), ("unreachable", J.ERR_TREE), ("word", J.ERR_TOKEN), ("empty", J.ERR_INVALID_ARG)])
def test_childsum_rejects_malformed_batches(case, status):
    """Validation of the child-list trees happens before any device work."""
    L = J.lib()
    d = J.TreeDesc(8, 4, 10, J.F32)
    # tree 0: 0 -> (1, 2), 2 -> (3);  tree 1: 4 (a single node)
    off, kids, word, root = [0, 2, 2, 3, 3, 3], [1, 2, 3], [1, 2, 3, 4, 5], [0, 4]
    if case == "offset0":
        off = [1, 2, 2, 3, 3, 4]
    elif case == "decreasing":
        off = [0, 2, 1, 3, 3, 3]
    elif case == "child_range":
        kids = [1, 9, 3]
    elif case == "two_parents":
        kids = [1, 2, 1]
    elif case == "root_has_parent":
        kids = [1, 2, 4]
    elif case == "cycle":
        off, kids, word, root = [0, 1, 2, 3], [1, 2, 1], [1, 2, 3], [0]   # 1 -> 2 -> 1 hangs off the root
    elif case == "unreachable":
        root = [0]
    elif case == "word":
        word = [1, 2, 3, 10, 5]
    elif case == "empty":
        off, kids, word, root = [0], [], [], []
    arrs = [np.ascontiguousarray(a, dtype=np.int32) for a in (off, kids or [0], word or [0], root or [0])]
    tb = J.NaryBatchC(len(root), len(word), *[a.ctypes.data_as(C.POINTER(C.c_int32)) for a in arrs])
    st = L.janus_childsum_fwd(C.byref(d), C.byref(tb), 0x1000, 0x2000, 0x3000, 0x4000, 0x5000, None, 0, None)
    assert st == status


def test_childsum_workspace_bytes():
    L = J.lib()
    d = J.TreeDesc(300, 150, 20000, J.F32)
    a = L.janus_childsum_workspace_bytes(C.byref(d), 100)
    assert a > 0 and L.janus_childsum_workspace_bytes(C.byref(d), 200) > a
    d.dtype = J.BF16
    assert L.janus_childsum_workspace_bytes(C.byref(d), 100) == 0
