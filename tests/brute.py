"""Brute-force and alternative formulations used to pin the oracle.

Each function is written straight from a definition, independent of the
oracle's C code, and is only practical on tiny graphs.
"""
from __future__ import annotations

import itertools
from functools import lru_cache

import numpy as np


def succs(wl):
    return [list(wl.out_idx[wl.out_ptr[v]:wl.out_ptr[v + 1]]) for v in range(wl.n)]


def preds(wl):
    return [list(wl.in_idx[wl.in_ptr[v]:wl.in_ptr[v + 1]]) for v in range(wl.n)]


def comm(wl):
    return [int(-(-int(o) // int(wl.bw)) + int(wl.lat)) for o in wl.ob]


def all_paths_from(wl, v):
    """Every maximal path starting at v (to a sink), as node lists."""
    S = succs(wl)
    out = []

    def rec(path):
        u = path[-1]
        if not S[u]:
            out.append(list(path))
            return
        for s in S[u]:
            path.append(s)
            rec(path)
            path.pop()

    rec([v])
    return out


def all_paths_to(wl, v):
    """Every maximal path ending at v (from a source)."""
    P = preds(wl)
    out = []

    def rec(path):
        u = path[0]
        if not P[u]:
            out.append(list(path))
            return
        for p in P[u]:
            path.insert(0, p)
            rec(path)
            path.pop(0)

    rec([v])
    return out


def hop_levels(wl):
    """level(v) = number of edges on the longest source -> v path."""
    return [max(len(p) - 1 for p in all_paths_to(wl, v)) for v in range(wl.n)]


def path_weight(wl, path, c):
    """sum of w over the path's nodes + c[u] for every edge u -> next."""
    return sum(int(wl.w[u]) for u in path) + sum(c[u] for u in path[:-1])


def blevel_brute(wl, comm_off=False):
    c = [0] * wl.n if comm_off else comm(wl)
    return [max(path_weight(wl, p, c) for p in all_paths_from(wl, v)) for v in range(wl.n)]


def tlevel_brute(wl):
    c = comm(wl)
    return [max(path_weight(wl, p, c) - int(wl.w[v]) for p in all_paths_to(wl, v))
            for v in range(wl.n)]


def interval_partitions(n):
    """All ways to cut 0..n into consecutive intervals: lists of breakpoints."""
    for mask in range(1 << max(n - 1, 0)):
        bps = [0] + [i + 1 for i in range(n - 1) if mask >> i & 1] + [n]
        yield bps


def cut_of(wl, order, bps, c):
    pos = np.empty(wl.n, np.int64)
    pos[np.asarray(order)] = np.arange(wl.n)
    cl = np.searchsorted(np.asarray(bps[1:]), pos, side="right")
    tot = 0
    S = succs(wl)
    for u in range(wl.n):
        for v in S[u]:
            if cl[u] != cl[v]:
                tot += c[u]
    return tot


def feasible(wl, order, bps, R, M):
    mem = [int(wl.mem[v]) for v in order]
    for a, b in zip(bps[:-1], bps[1:]):
        if b - a > R:
            return False
        if b - a > 1 and sum(mem[a:b]) > M:
            return False
    return True


def makespan_augmented(wl, order, dev):
    """Makespan as a longest path in the DAG augmented with device-order edges.

    finish(v) = w_v + max(0, max over graph preds p of finish(p) + [dev differs] c_p,
    finish(previous op on the same device in ``order``)), evaluated by memoised
    recursion (an independent formulation of the list schedule).
    """
    c = comm(wl)
    P = preds(wl)
    prev_on_dev = {}
    last = {}
    for v in order:
        prev_on_dev[int(v)] = last.get(int(dev[v]))
        last[int(dev[v])] = int(v)

    import sys
    sys.setrecursionlimit(max(10000, 4 * wl.n + 100))

    @lru_cache(maxsize=None)
    def fin(v):
        t = 0
        for p in P[v]:
            t = max(t, fin(int(p)) + (c[p] if dev[p] != dev[v] else 0))
        q = prev_on_dev[v]
        if q is not None:
            t = max(t, fin(q))
        return t + int(wl.w[v])

    f = [fin(v) for v in range(wl.n)]
    return (max(f) if f else 0), f


def all_placements(n, D):
    return itertools.product(range(D), repeat=n)


def makespan_blocking_transfers(wl, order, dev):
    """Makespan when every transfer occupies the compute queues of both the
    sending and the receiving device, as a longest path in a task DAG.

    Tasks: the nodes, plus one transfer task (u, b) of length c[u] for each
    producer u and each other device b holding a successor of u.  Walking
    ``order``, each node is appended to its device's queue, then its transfer
    tasks (increasing b) to the queues of both its device and b.  Edges: u ->
    (u, b) -> every successor of u on b; u -> successors on u's own device;
    consecutive tasks of each device queue.  A task finishes at its length
    plus the latest finish among its predecessors (0 if none): a formulation
    independent of the oracle's time-stepping.  Returns (makespan, finish by
    node id).
    """
    c = comm(wl)
    S = succs(wl)
    queue = {}  # device -> list of tasks in queue order
    length = {}
    preds_of = {}
    for v in order:
        v = int(v)
        d = int(dev[v])
        length[("n", v)] = int(wl.w[v])
        queue.setdefault(d, []).append(("n", v))
        for b in sorted({int(dev[s]) for s in S[v]} - {d}):
            t = ("t", v, b)
            length[t] = c[v]
            preds_of.setdefault(t, set()).add(("n", v))
            queue[d].append(t)
            queue.setdefault(b, []).append(t)
    for v in range(wl.n):
        for s in S[v]:
            src = ("n", v) if dev[s] == dev[v] else ("t", v, int(dev[s]))
            preds_of.setdefault(("n", int(s)), set()).add(src)
    for q in queue.values():
        for a, b in zip(q, q[1:]):
            preds_of.setdefault(b, set()).add(a)

    import sys
    sys.setrecursionlimit(max(10000, 8 * len(length) + 100))

    @lru_cache(maxsize=None)
    def fin(t):
        return length[t] + max([fin(p) for p in preds_of.get(t, ())] + [0])

    f = [fin(("n", v)) for v in range(wl.n)]
    return (max(f) if f else 0), f
