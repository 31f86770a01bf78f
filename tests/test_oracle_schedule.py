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
