"""Pins of the oracle's integer schedules against library routines and
brute-force properties."""
import numpy as np
import pytest

from oracle import schedule
from paper_1812_01329_amd import workloads as wl


@pytest.mark.parametrize("seed", range(20))
def test_seq_schedule_against_numpy(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 40)); T = int(rng.integers(0, 30))
    lengths = rng.integers(0, T + 1, B)
    perm, active, offset, t_eff = schedule.seq_schedule(lengths, T)
    assert np.array_equal(perm, np.argsort(-lengths, kind="stable"))
    assert t_eff == (lengths.max() if B else 0)
    assert np.array_equal(active, np.array([(lengths > t).sum() for t in range(t_eff)], dtype=np.int32))
    assert offset[-1] == lengths.sum()
    # the running rows of step t are a prefix of perm
    for t in range(t_eff):
        assert set(perm[:active[t]].tolist()) == set(np.nonzero(lengths > t)[0].tolist())


def test_seq_schedule_rejects_bad_lengths():
    with pytest.raises(schedule.ScheduleError):
        schedule.seq_schedule([3, -1], 5)
    with pytest.raises(schedule.ScheduleError):
        schedule.seq_schedule([6, 1], 5)


@pytest.mark.parametrize("seed", range(10))
def test_tree_schedule_properties(seed):
    rng = np.random.default_rng(seed)
    t = wl.make_trees(rng, int(rng.integers(1, 8)), 1, 30, 100)
    level, off, order, L = schedule.tree_schedule(t.left, t.right, t.word, t.root, 100)
    N = t.num_nodes
    for n in range(N):
        if t.left[n] < 0:
            assert level[n] == 0
        else:
            assert level[n] == 1 + max(level[t.left[n]], level[t.right[n]])
    assert sorted(order.tolist()) == list(range(N))
    keys = [(level[n], n) for n in order]
    assert keys == sorted(keys)
    assert off[0] == 0 and off[-1] == N and len(off) == L + 1
    assert np.array_equal(np.diff(off), np.bincount(level, minlength=L))


def _tree(left, right, word, root):
    return [np.asarray(a, np.int32) for a in (left, right, word, root)]


@pytest.mark.parametrize("case,kind", [
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 2, -1], [2]), None),
    (_tree([-1, -1, 0], [-1, -1, -1], [1, 2, -1], [2]), "tree"),       # one child
    (_tree([-1, -1, 0], [-1, -1, 0], [1, 2, -1], [2]), "tree"),        # same child twice
    (_tree([-1, -1, 0, 0], [-1, -1, 1, 1], [1, 2, -1, -1], [2, 3]), "tree"),  # two parents
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 9, -1], [2]), "token"),       # word out of range
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 2, 4], [2]), "tree"),         # internal with word
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 2, -1], [1]), "tree"),        # root has a parent
    (_tree([-1, 2, 1], [-1, 0, 0], [1, -1, -1], [0]), "tree"),         # cycle / unreachable
    (_tree([-1, -1, 0], [-1, -1, 5], [1, 2, -1], [2]), "tree"),        # child id out of range
    (_tree([-1, -1, 0], [-1, -1, 1], [1, 2, -1], [2, 2]), "tree"),     # repeated root
])
def test_tree_validation(case, kind):
    if kind is None:
        schedule.tree_schedule(*case, 5)
    else:
        with pytest.raises(schedule.ScheduleError) as e:
            schedule.tree_schedule(*case, 5)
        assert e.value.kind == kind


def _child_lists(left, right):
    """Binary trees as child lists (left child first)."""
    offsets, children = [0], []
    for l, r in zip(left, right):
        if l >= 0:
            children += [int(l), int(r)]
        offsets.append(len(children))
    return np.asarray(offsets, np.int32), np.asarray(children, np.int32)


@pytest.mark.parametrize("seed", range(10))
def test_nary_schedule_equals_binary_schedule_on_binary_trees(seed):
    """A binary tree is a tree of any arity: as child lists it gets the same
    levels and the same level order as the binary schedule."""
    rng = np.random.default_rng(100 + seed)
    t = wl.make_trees(rng, int(rng.integers(1, 8)), 1, 30, 100)
    lb, ob, nb, Lb = schedule.tree_schedule(t.left, t.right, t.word, t.root, 100)
    off, ch = _child_lists(t.left, t.right)
    words = np.where(t.word >= 0, t.word, 0)
    la, oa, na, La = schedule.nary_schedule(off, ch, words, t.root, 100)
    assert La == Lb and np.array_equal(la, lb) and np.array_equal(oa, ob) and np.array_equal(na, nb)


def test_nary_schedule_chains_and_stars():
    """A chain of n nodes (each the child of the next) has levels 0 .. n-1;
    a star has its leaves at 0 and its root at 1; a lone node is level 0."""
    n = 9
    off = np.array([0] + [k for k in range(n)], np.int32)   # node k > 0 has the one child k - 1
    ch = np.arange(n - 1, dtype=np.int32)
    level, loff, order, L = schedule.nary_schedule(off, ch, np.zeros(n, np.int32), [n - 1], 3)
    assert np.array_equal(level, np.arange(n)) and L == n and np.array_equal(order, np.arange(n))
    m = 6   # star: node m is the root over nodes 0 .. m-1
    off = np.array([0] * (m + 1) + [m], np.int32)
    level, loff, order, L = schedule.nary_schedule(off, np.arange(m, dtype=np.int32),
                                                   np.zeros(m + 1, np.int32), [m], 3)
    assert L == 2 and np.array_equal(loff, [0, m, m + 1]) and level[m] == 1 and not level[:m].any()
    level, loff, order, L = schedule.nary_schedule([0, 0], [], [2], [0], 3)
    assert L == 1 and level[0] == 0


@pytest.mark.parametrize("off,ch,word,root,kind", [
    ([0, 0, 0, 2], [0, 1], [1, 2, 0], [2], None),
    ([1, 1, 1, 3], [0, 1, 0], [1, 2, 0], [2], "tree"),          # offsets do not start at 0
    ([0, 2, 1, 2], [0, 1], [1, 2, 0], [2], "tree"),             # offsets decrease
    ([0, 0, 0, 2], [0, 5], [1, 2, 0], [2], "tree"),             # child out of range
    ([0, 0, 1, 3], [0, 0, 1], [1, 2, 0], [2], "tree"),          # shared child
    ([0, 1, 2, 2], [1, 0], [1, 2, 0], [2], "tree"),             # cycle, node 2 alone
    ([0, 0, 0, 2], [0, 1], [1, 9, 0], [2], "token"),            # word out of range
    ([0, 0, 0, 2], [0, 1], [1, 2, 0], [1], "tree"),             # root has a parent
    ([0, 0, 0, 2], [0, 1], [1, 2, 0], [2, 2], "tree"),          # repeated root
    ([0, 0, 0, 1], [0], [1, 2, 0], [2], "tree"),                # node 1 unreachable
])
def test_nary_validation(off, ch, word, root, kind):
    args = [np.asarray(a, np.int32) for a in (off, ch, word, root)]
    if kind is None:
        schedule.nary_schedule(*args, 5)
    else:
        with pytest.raises(schedule.ScheduleError) as e:
            schedule.nary_schedule(*args, 5)
        assert e.value.kind == kind
