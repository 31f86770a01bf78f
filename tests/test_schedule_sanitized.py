"""The library's host schedule code (paper_1812_01329_amd/csrc/schedule.cpp)
built on its own with AddressSanitizer and UndefinedBehaviorSanitizer (a host
program, no device code) and run on random and malformed inputs: length
vectors, binary tree batches and trees of any arity, with cycles, shared
children, out-of-range ids, bad roots and bad offsets.  Every status and
every schedule must equal the oracle's (oracle/schedule.py), and the
sanitizers must report nothing (any report aborts the program)."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import schedule as osch
from paper_1812_01329_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "tests", "sanitize", "schedule_fuzz.cpp")
SOURCE = os.path.join(ROOT, "paper_1812_01329_amd", "csrc", "schedule.cpp")

OK, ERR_INVALID_ARG, ERR_LENGTH, ERR_TREE, ERR_TOKEN = 0, 1, 2, 3, 4
KIND = {"length": ERR_LENGTH, "tree": ERR_TREE, "token": ERR_TOKEN}


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("g++ not found")
    out = str(tmp_path_factory.mktemp("san") / "schedule_fuzz")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           f"-I{os.path.join(ROOT, 'include')}", DRIVER, SOURCE, "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return out


def _run(driver, tmp_path, lines):
    cases, res = tmp_path / "cases.txt", tmp_path / "results.txt"
    cases.write_text("\n".join(lines) + "\n")
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([driver, str(cases), str(res)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    out = [l.split(" |") for l in res.read_text().splitlines()]
    assert len(out) == len(lines)
    return out


def _ints(s):
    return [int(v) for v in s.split()]


def _line(tag, *parts):
    """One input line: the tag, then every integer of the parts in order."""
    vals = [int(v) for p in parts for v in (p if hasattr(p, "__len__") else [p])]
    return " ".join([tag] + [str(v) for v in vals])


def test_sequence_schedules(driver, tmp_path):
    rng = np.random.default_rng(901)
    lines, expect = [], []
    for i in range(800):
        B, T = int(rng.integers(1, 40)), int(rng.integers(0, 30))
        lengths = rng.integers(0, T + 1, B)
        mode = i % 8
        if mode == 1:
            lengths[rng.integers(0, B)] = -int(rng.integers(1, 5))
        elif mode == 2:
            lengths[rng.integers(0, B)] = T + int(rng.integers(1, 5))
        elif mode == 3:
            lengths[:] = T
        has = 0 if mode == 4 else 1
        if mode == 5:
            B = -int(rng.integers(0, 3))    # B <= 0
            lengths = lengths[:0]
        if mode == 6:
            T = -1
        lines.append(_line("S", B, T, has, lengths if has else []))
        if B <= 0 or T < 0:
            expect.append((ERR_INVALID_ARG, None))
            continue
        try:
            expect.append((OK, osch.seq_schedule(lengths if has else [T] * B, T)))
        except osch.ScheduleError as e:
            expect.append((KIND[e.kind], None))
    out = _run(driver, tmp_path, lines)
    for (st, ref), got in zip(expect, out):
        assert int(got[0]) == st, (got, st)
        if st == OK:
            perm, active, offsets, t_eff = ref
            assert _ints(got[1]) == perm.tolist()
            assert _ints(got[2]) == active.tolist()
            assert _ints(got[3]) == offsets.tolist()
            assert int(got[4]) == t_eff


def _mutate_binary(rng, t):
    left, right, word, root = (a.copy() for a in (t.left, t.right, t.word, t.root))
    N = len(left)
    k = int(rng.integers(0, 7))
    n = int(rng.integers(0, N))
    if k == 0:
        left[n] = int(rng.integers(-3, N + 3))           # any child id, also out of range
    elif k == 1:
        right[n] = int(rng.integers(-3, N + 3))
    elif k == 2:
        word[n] = int(rng.integers(-3, 60))              # words outside [0, V) too
    elif k == 3:
        root[int(rng.integers(0, len(root)))] = int(rng.integers(-2, N + 2))
    elif k == 4 and N >= 3:
        internal = np.nonzero(left >= 0)[0]
        if len(internal):
            p = int(rng.choice(internal))
            left[p] = int(rng.integers(0, N))            # a shared child or a cycle
    elif k == 5:
        root = np.concatenate([root, root[:1]])          # a repeated root
    return left, right, word, root


def test_binary_tree_schedules(driver, tmp_path):
    rng = np.random.default_rng(902)
    V = 50
    lines, expect = [], []
    for i in range(800):
        t = wl.make_trees(rng, int(rng.integers(1, 6)), 1, 12, V)
        left, right, word, root = (t.left, t.right, t.word, t.root) if i % 3 == 0 else _mutate_binary(rng, t)
        lines.append(_line("T", V, len(left), len(root), left, right, word, root))
        try:
            expect.append((OK, osch.tree_schedule(left, right, word, root, V)))
        except osch.ScheduleError as e:
            expect.append((KIND[e.kind], None))
    out = _run(driver, tmp_path, lines)
    n_ok = 0
    for (st, ref), got in zip(expect, out):
        assert int(got[0]) == st, (got[0], st)
        if st == OK:
            n_ok += 1
            level, offsets, order, L = ref
            assert _ints(got[1]) == level.tolist()
            assert _ints(got[2]) == offsets.tolist()
            assert _ints(got[3]) == order.tolist()
    assert 200 < n_ok < 800   # both valid and rejected batches were exercised


def _mutate_nary(rng, t):
    off, ch, word, root = (a.copy() for a in (t.child_offsets, t.children, t.word, t.root))
    N = len(word)
    k = int(rng.integers(0, 7))
    if k == 0 and len(ch):
        ch[int(rng.integers(0, len(ch)))] = int(rng.integers(-2, N + 2))   # bad, shared or cyclic child
    elif k == 1:
        off[int(rng.integers(1, N + 1))] -= int(rng.integers(1, 3))        # decreasing offsets
        off[-1] = max(off[-1], 0)
    elif k == 2:
        off[0] = 1
    elif k == 3:
        word[int(rng.integers(0, N))] = int(rng.integers(-3, 60))
    elif k == 4:
        root[int(rng.integers(0, len(root)))] = int(rng.integers(-2, N + 2))
    elif k == 5:
        root = np.concatenate([root, root[-1:]])
    # the children array always holds off[N] entries (the caller's contract)
    E = max(int(off[-1]), 0)
    ch = np.concatenate([ch, np.zeros(max(E - len(ch), 0), np.int32)])[:E] if off[0] == 0 else ch
    return off, ch, word, root


def test_nary_tree_schedules(driver, tmp_path):
    rng = np.random.default_rng(903)
    V = 50
    lines, expect = [], []
    for i in range(800):
        t = wl.make_nary_trees(rng, int(rng.integers(1, 6)), 1, 15, V, chain=(i % 11 == 0))
        if i % 3 == 0:
            off, ch, word, root = t.child_offsets, t.children, t.word, t.root
        else:
            off, ch, word, root = _mutate_nary(rng, t)
        N = len(word)
        lines.append(_line("N", V, N, len(root), len(ch), off, ch, word, root))
        try:
            ref = osch.nary_schedule(off, ch, word, root, V)
            expect.append((OK, ref, off, ch, word, root))
        except osch.ScheduleError as e:
            expect.append((KIND[e.kind], None, None, None, None, None))
    out = _run(driver, tmp_path, lines)
    n_ok = 0
    for (st, ref, off, ch, word, root), got in zip(expect, out):
        assert int(got[0]) == st, (got[0], st)
        if st != OK:
            continue
        n_ok += 1
        level, loff, order, L = ref
        N = len(word)
        pos = np.empty(N, np.int64)
        pos[order] = np.arange(N)
        kids = [[int(c) for c in ch[off[n]:off[n + 1]]] for n in range(N)]
        pcoff = np.concatenate([[0], np.cumsum([len(kids[n]) for n in order])]).astype(int)
        pkids = [int(pos[c]) for n in order for c in kids[n]]
        rootk = [-1] * N
        for k, r in enumerate(root):
            rootk[pos[r]] = k
        assert _ints(got[1]) == loff.tolist()
        assert _ints(got[2]) == [int(word[n]) for n in order]
        assert _ints(got[3]) == pcoff.tolist()
        assert _ints(got[4]) == pkids
        assert _ints(got[5]) == rootk
        assert _ints(got[6]) == [int(pos[r]) for r in root]
    assert 200 < n_ok < 800
