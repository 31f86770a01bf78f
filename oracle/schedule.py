"""Integer schedules of the data-dependent loop and of the tree recursion.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sequences (the loop of Figure 1 with per-sequence trip counts, Section 4.2.1):
    perm    = batch indices sorted by (-len_b, b)      (stable, longest first)
    active[t] = #{b : len_b > t} for t < T_eff,  T_eff = max len
    offset[t] = sum of active[t'] for t' < t          (start of step t when the
                                                        running rows are packed)
Trees (recursion over subtrees, Section 4.2.1 / Section 6.1):
    level(leaf) = 0,  level(n) = 1 + max(level(left), level(right))
    level_nodes = node ids sorted by (level, id),  level_offsets[k] = #{n : level(n) < k}
Nodes of one level depend only on nodes of lower levels, so every level is a
batch of independent cell applications (the parallel execution of independent
operations that the paper measures, Section 6.3.1 "+PARL").

Validation mirrors what the library rejects before touching any output
(all-or-nothing updates, Section 3.2 and Section 4.2.3).
"""
from __future__ import annotations

import sys

import numpy as np


class ScheduleError(ValueError):
    def __init__(self, kind, msg):
        super().__init__(msg)
        self.kind = kind          # "length", "tree" or "token"


def seq_schedule(lengths, T):
    lengths = [int(v) for v in lengths]
    for v in lengths:
        if v < 0 or v > T:
            raise ScheduleError("length", f"length {v} outside [0, {T}]")
    B = len(lengths)
    perm = sorted(range(B), key=lambda b: (-lengths[b], b))
    t_eff = max(lengths) if B else 0
    active = []
    for t in range(t_eff):
        active.append(sum(1 for b in range(B) if lengths[b] > t))
    offset = [0]
    for a in active:
        offset.append(offset[-1] + a)
    return (np.asarray(perm, np.int32), np.asarray(active, np.int32),
            np.asarray(offset, np.int32), t_eff)


def validate_trees(left, right, word, root, V):
    N = len(left)
    if N == 0 or len(root) == 0:
        raise ScheduleError("tree", "empty batch")
    parents = [0] * N
    for n in range(N):
        l, r = int(left[n]), int(right[n])
        if (l < 0) != (r < 0):
            raise ScheduleError("tree", f"node {n} has one child")
        if l < 0:
            if l != -1 or r != -1:
                raise ScheduleError("tree", f"node {n}: bad child id")
            if not (0 <= int(word[n]) < V):
                raise ScheduleError("token", f"leaf {n}: word {word[n]} outside [0, {V})")
        else:
            if not (0 <= l < N and 0 <= r < N) or l == r:
                raise ScheduleError("tree", f"node {n}: bad child ids")
            if int(word[n]) != -1:
                raise ScheduleError("tree", f"internal node {n} carries a word")
            parents[l] += 1
            parents[r] += 1
    for n in range(N):
        if parents[n] > 1:
            raise ScheduleError("tree", f"node {n} has two parents")
    seen_root = set()
    for k in root:
        k = int(k)
        if not (0 <= k < N) or parents[k] != 0 or k in seen_root:
            raise ScheduleError("tree", f"bad root {k}")
        seen_root.add(k)
    # every node reachable from exactly one root (no cycles, no strays)
    reached = 0
    stack = [int(k) for k in root]
    while stack:
        n = stack.pop()
        reached += 1
        if int(left[n]) >= 0:
            stack.append(int(left[n]))
            stack.append(int(right[n]))
        if reached > N:
            raise ScheduleError("tree", "cycle")
    if reached != N:
        raise ScheduleError("tree", "node not reachable from a root")


def tree_schedule(left, right, word, root, V):
    validate_trees(left, right, word, root, V)
    N = len(left)
    level = [None] * N
    sys.setrecursionlimit(max(10000, 4 * N + 100))

    def height(n):
        if level[n] is None:
            if int(left[n]) < 0:
                level[n] = 0
            else:
                level[n] = 1 + max(height(int(left[n])), height(int(right[n])))
        return level[n]

    for k in root:
        height(int(k))
    num_levels = max(level) + 1
    order = sorted(range(N), key=lambda n: (level[n], n))
    offsets = [sum(1 for n in range(N) if level[n] < k) for k in range(num_levels + 1)]
    return (np.asarray(level, np.int32), np.asarray(offsets, np.int32),
            np.asarray(order, np.int32), num_levels)


def nary_schedule(offsets, children, word, root, V):
    """Trees of any arity given as child lists: node n's children are
    children[offsets[n]:offsets[n + 1]].  Every node carries a word (the
    Child-Sum TreeLSTM reads x at every node).

        level(n) = 0 without children, else 1 + max over its children
        order    = node ids sorted by (level, id)

    Checks, in this order: offsets start at 0 and never decrease; every
    child id is in range and has one parent; every word lies in [0, V);
    roots are in range, parentless and distinct, and every node is reached
    from exactly one root (no cycles, no strays).  Returns (level,
    level_offsets, order, num_levels)."""
    offsets = [int(v) for v in offsets]
    N = len(offsets) - 1
    if N <= 0 or len(root) == 0:
        raise ScheduleError("tree", "empty batch")
    if offsets[0] != 0:
        raise ScheduleError("tree", "offsets do not start at 0")
    for n in range(N):
        if offsets[n + 1] < offsets[n]:
            raise ScheduleError("tree", f"offsets decrease at node {n}")
    kids = [int(children[e]) for e in range(offsets[N])]
    has_parent = [False] * N
    for c in kids:
        if not (0 <= c < N) or has_parent[c]:
            raise ScheduleError("tree", f"bad or shared child {c}")
        has_parent[c] = True
    for n in range(N):
        if not (0 <= int(word[n]) < V):
            raise ScheduleError("token", f"node {n}: word {word[n]} outside [0, {V})")
    seen = set()
    for k in root:
        k = int(k)
        if not (0 <= k < N) or has_parent[k] or k in seen:
            raise ScheduleError("tree", f"bad root {k}")
        seen.add(k)
    reached = [False] * N
    stack = [int(k) for k in root]
    while stack:
        n = stack.pop()
        if reached[n]:
            raise ScheduleError("tree", "node reached twice")
        reached[n] = True
        stack.extend(kids[offsets[n]:offsets[n + 1]])
    if not all(reached):
        raise ScheduleError("tree", "node not reachable from a root")
    level = [None] * N
    sys.setrecursionlimit(max(10000, 4 * N + 100))

    def height(n):
        if level[n] is None:
            ch = kids[offsets[n]:offsets[n + 1]]
            level[n] = 0 if not ch else 1 + max(height(c) for c in ch)
        return level[n]

    for k in root:
        height(int(k))
    num_levels = max(level) + 1
    order = sorted(range(N), key=lambda n: (level[n], n))
    level_offsets = [sum(1 for n in range(N) if level[n] < k) for k in range(num_levels + 1)]
    return (np.asarray(level, np.int32), np.asarray(level_offsets, np.int32),
            np.asarray(order, np.int32), num_levels)
