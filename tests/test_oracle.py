"""Pins for the CPU oracle: hand-traced fixtures, brute force, closed forms and
invariants.  CPU only; the GPU path is not involved."""
from __future__ import annotations

import json
import math
import os

import numpy as np
import pytest

from oracle import oracle as O
from tests import brute as B
from workloads import from_edges, make_config, make_random_dag

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def hand6(D=2, cap=(60, 60)):
    g = load("hand6.json")["graph"]
    return from_edges(g["n"], g["edges"], g["w"], g["ob"], D, cap, g["bw"], g["lat"],
                      mem=g["mem"])


def small_dags(count=40, n_lo=1, n_hi=11):
    for s in range(count):
        n = n_lo + s % (n_hi - n_lo + 1)
        yield make_random_dag(s, n, p_edge=0.25 + 0.05 * (s % 5), D=2 + s % 3,
                              multi=(s % 4 == 0), zero_frac=0.2 if s % 6 == 0 else 0.0)


# ------------------------------------------------------------------ fixtures


def test_hand6_levels_blevel():
    gd = load("hand6.json")
    wl = hand6()
    assert list(O.comm(wl)) == gd["comm"]
    lev, oid, lp, L = O.topo_levels(wl)
    e = gd["levels"]
    assert list(lev) == e["level"] and list(oid) == e["order_id"]
    assert list(lp) == e["level_ptr"] and L == e["L"]
    bl, tl, pr, cp = O.blevel(wl, lev, oid)
    e = gd["blevel"]
    assert list(bl) == e["blevel"] and list(tl) == e["tlevel"] and cp == e["cp"]
    assert list(pr) == e["prio_order"]
    bl0, _, _, cp0 = O.blevel(wl, lev, oid, comm_off=True)
    assert list(bl0) == e["blevel_comm_off"] and cp0 == e["cp0"]


def test_hand6_cluster():
    e = load("hand6.json")["cluster"]
    wl = hand6()
    for mode in (O.DP, O.DP_DIRECT):
        cid, C, cut = O.cluster(wl, e["order"], e["R"], e["M"], mode)
        assert list(cid) == e["cluster_id"] and C == e["n_clusters"] and cut == e["cut_cost"]
    cid, C, cut = O.cluster(wl, e["order"], e["R"], e["M"], O.GREEDY)
    assert list(cid) == e["greedy_cluster_id"] and cut == e["greedy_cut_cost"]


def test_hand6_place():
    gd = load("hand6.json")
    e = gd["place"]
    wl = hand6(e["D"], e["cap"])
    cdev, ndev, span, be, fin = O.place(wl, gd["cluster"]["cluster_id"], 3, want_fin=True)
    assert list(cdev) == e["cluster_dev"] and list(ndev) == e["node_dev"]
    assert list(fin) == e["cluster_fin"] and span == e["coarse_makespan"]
    assert be == e["best_effort_count"]


def test_hand6_makespan():
    e = load("hand6.json")["makespan"]
    for case in e["cases"]:
        wl = hand6(case["D"], [10 ** 6] * case["D"])
        ms, st, fi = O.makespan(wl, e["order"], np.array(case["node_dev"], np.uint8))
        assert ms[0] == case["makespan"], case["derivation"]
        assert list(st[0]) == case["start"] and list(fi[0]) == case["finish"]


@pytest.mark.parametrize("case", load("place_hand.json")["cases"], ids=lambda c: c["name"])
def test_place_hand_cases(case):
    n = case["n"]
    wl = from_edges(n, case["edges"], case["w"], case["ob"], case["D"], case["cap"],
                    case["bw"], case["lat"], mem=case["mem"])
    cid = np.array(case.get("cluster_id", range(n)), np.int32)
    C = int(cid.max()) + 1
    cdev, ndev, span, be, fin = O.place(wl, cid, C, want_fin=True)
    assert list(cdev) == case["cluster_dev"], case["derivation"]
    assert list(fin) == case["cluster_fin"]
    assert span == case["coarse_makespan"] and be == case["best_effort_count"]


# ------------------------------------------------------------------- levels


def check_level_characterisation(wl, lev, oid, lp, L):
    """The three properties that determine the level function uniquely."""
    n = wl.n
    src, dst = wl.edges()
    assert np.all(lev[src] < lev[dst])
    indeg = np.diff(wl.in_ptr)
    assert np.array_equal(lev == 0, indeg == 0)
    # every node above level 0 has a predecessor exactly one level below
    has = np.zeros(n, bool)
    np.logical_or.at(has, dst, lev[src] == lev[dst] - 1)
    assert np.all(has[lev > 0])
    # order_id = ids sorted by (level, id); level_ptr = bucket offsets
    assert np.array_equal(oid, np.lexsort((np.arange(n), lev)))
    assert L == (int(lev.max()) + 1 if n else 0)
    assert np.array_equal(lp, np.concatenate([[0], np.cumsum(np.bincount(lev, minlength=L))]))


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_levels_configs(cfg):
    wl = make_config(cfg, 0)
    check_level_characterisation(wl, *O.topo_levels(wl))


def test_levels_brute():
    for wl in small_dags():
        lev, oid, lp, L = O.topo_levels(wl)
        assert list(lev) == B.hop_levels(wl)
        check_level_characterisation(wl, lev, oid, lp, L)


def test_levels_degenerate():
    wl = from_edges(0, [], [], [], 1, [1], 1, 0)
    lev, oid, lp, L = O.topo_levels(wl)
    assert L == 0 and list(lp) == [0]
    wl = from_edges(1, [], [5], [3], 1, [1], 1, 0)
    lev, oid, lp, L = O.topo_levels(wl)
    assert L == 1 and list(lev) == [0] and list(lp) == [0, 1]


@pytest.mark.parametrize("edges", [[(0, 0)], [(0, 1), (1, 0)], [(0, 1), (1, 2), (2, 1)]])
def test_levels_cycle(edges):
    n = 1 + max(max(e) for e in edges)
    wl = from_edges(n, edges, [1] * n, [1] * n, 1, [1], 1, 0)
    with pytest.raises(O.OracleError) as ei:
        O.topo_levels(wl)
    assert ei.value.code == O.E_CYCLE


def test_bad_graph_rejected():
    wl = hand6()
    wl.in_idx = wl.in_idx.copy()
    wl.in_idx[0] = (wl.in_idx[0] + 1) % wl.n  # CSC no longer matches CSR
    with pytest.raises(O.OracleError) as ei:
        O.topo_levels(wl)
    assert ei.value.code == O.E_ARG
    wl = hand6()
    wl.w = wl.w.copy(); wl.w[2] = -1
    with pytest.raises(O.OracleError):
        O.topo_levels(wl)


def test_overflow_rejected():
    wl = from_edges(2, [(0, 1)], [5, 6], [2 ** 62 - 10, 0], 1, [1], 1, 0, mem=[1, 1])
    lev, oid, _, _ = O.topo_levels(wl)
    with pytest.raises(O.OracleError) as ei:
        O.blevel(wl, lev, oid)
    assert ei.value.code == O.E_OVERFLOW


# ------------------------------------------------------------ b/t-level, CP


def test_blevel_brute():
    for wl in small_dags():
        lev, oid, _, _ = O.topo_levels(wl)
        bl, tl, pr, cp = O.blevel(wl, lev, oid)
        assert list(bl) == B.blevel_brute(wl)
        assert list(tl) == B.tlevel_brute(wl)
        assert cp == (max(bl) if wl.n else 0)
        bl0, _, _, cp0 = O.blevel(wl, lev, oid, comm_off=True)
        assert list(bl0) == B.blevel_brute(wl, comm_off=True)
        if wl.n:  # longest path through any node equals the critical path
            assert int(np.max(tl + bl)) == cp


def test_blevel_chain_closed_form():
    n = 7
    w = [5, 1, 8, 2, 9, 3, 4]
    ob = [10, 0, 33, 7, 1, 2, 50]
    wl = from_edges(n, [(i, i + 1) for i in range(n - 1)], w, ob, 1, [1], 4, 6)
    lev, oid, _, _ = O.topo_levels(wl)
    bl, tl, pr, cp = O.blevel(wl, lev, oid)
    c = [math.ceil(o / 4) + 6 for o in ob]
    assert cp == sum(w) + sum(c[:-1])
    assert tl[-1] == sum(w[:-1]) + sum(c[:-1])


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_prio_order_properties(cfg):
    wl = make_config(cfg, 1)
    lev, oid, _, _ = O.topo_levels(wl)
    bl, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
    assert np.array_equal(np.sort(pr), np.arange(wl.n))
    key = np.lexsort((pr, -bl[pr], lev[pr]))  # already sorted iff identity
    assert np.array_equal(key, np.arange(wl.n))
    assert np.all(np.diff(lev[pr]) >= 0)


# ---------------------------------------------------------------- clustering


def test_cluster_brute_force():
    rng = np.random.default_rng(7)
    for s in range(30):
        n = 2 + s % 11
        wl = make_random_dag(100 + s, n, p_edge=0.35, D=2, multi=(s % 3 == 0))
        lev, oid, _, _ = O.topo_levels(wl)
        _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
        R = int(rng.integers(1, n + 1))
        tot = int(wl.mem.sum())
        M = int(rng.integers(0, tot + 1))
        c = B.comm(wl)
        cid, C, cut = O.cluster(wl, pr, R, M, O.DP)
        best = min(B.cut_of(wl, pr, bps, c) for bps in B.interval_partitions(n)
                   if B.feasible(wl, pr, bps, R, M))
        assert cut == best
        # the returned partition is contiguous in the order, feasible, and attains S(n)
        seq = cid[pr]
        assert seq[0] == 0 and np.all(np.diff(seq) >= 0) and np.all(np.diff(seq) <= 1)
        bps = [0] + list(np.nonzero(np.diff(seq))[0] + 1) + [n]
        assert B.feasible(wl, pr, bps, R, M) and B.cut_of(wl, pr, bps, c) == cut
        assert C == len(bps) - 1
        # tie reading: each cluster [a, b) starts at the smallest i for which
        # S(i) + cost(i, b) = S(b), with S from brute force over prefixes
        pos = np.empty(n, np.int64); pos[pr] = np.arange(n)

        def leave(a, b):  # eq. 4: comm leaving [a, b) for positions >= b
            return sum(c[pr[p]] for p in range(a, b)
                       for v in wl.out_idx[wl.out_ptr[pr[p]]:wl.out_ptr[pr[p] + 1]]
                       if pos[v] >= b)

        S = {0: 0}
        for j in range(1, n + 1):
            vals = [S[bp[-2]] + leave(bp[-2], j) for bp in ([i, j] for i in range(j))
                    if B.feasible(wl, pr, bp, R, M)]
            S[j] = min(vals)
        assert S[n] == cut
        for a, b in zip(bps[:-1], bps[1:]):
            cands = [i for i in range(max(0, b - R), b)
                     if B.feasible(wl, pr, [i, b], R, M) and S[i] + leave(i, b) == S[b]]
            assert a == min(cands)


def test_cluster_paths_agree():
    """eq. 4 evaluated directly vs the eq. 5 recursion."""
    for s in range(25):
        wl = make_random_dag(300 + s, 4 + s % 20, p_edge=0.3, D=3, multi=(s % 2 == 0))
        lev, oid, _, _ = O.topo_levels(wl)
        _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
        for R, M in ((3, -1), (7, int(wl.mem.sum()) // 3), (50, 10 ** 12)):
            a = O.cluster(wl, pr, R, M, O.DP)
            b = O.cluster(wl, pr, R, M, O.DP_DIRECT)
            assert np.array_equal(a[0], b[0]) and a[1:] == b[1:]


def test_cluster_special_cases():
    wl = make_random_dag(5, 12, p_edge=0.4, D=2)
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
    c = O.comm(wl)
    src, _ = wl.edges()
    cid, C, cut = O.cluster(wl, pr, 1, 10 ** 15, O.DP)
    assert C == wl.n and cut == int(c[src].sum())
    cid, C, cut = O.cluster(wl, pr, wl.n, int(wl.mem.sum()), O.DP)
    assert C == 1 and cut == 0 and np.all(cid == 0)
    cid, C, cut = O.cluster(wl, pr, 5, 0, O.DP)  # M = 0: singletons unless mem is 0
    assert C == wl.n or np.any(wl.mem == 0)


def check_cluster_invariants(wl, order, cid, C, cut, R, M):
    seq = cid[order]
    assert seq[0] == 0 and seq[-1] == C - 1
    assert np.all(np.diff(seq) >= 0) and np.all(np.diff(seq) <= 1)
    sizes = np.bincount(seq, minlength=C)
    memsum = np.bincount(seq, weights=wl.mem[order].astype(np.float64), minlength=C)
    assert sizes.max() <= R
    assert np.all((memsum <= M) | (sizes == 1))
    src, dst = wl.edges()
    crossing = cid[src] != cid[dst]
    assert cut == int(O.comm(wl)[src[crossing]].sum())
    assert np.all(cid[src[crossing]] < cid[dst[crossing]])  # coarse graph is a DAG


@pytest.mark.parametrize("cfg", [1, 2, 3])
@pytest.mark.parametrize("mode", [O.DP, O.GREEDY])
def test_cluster_invariants_configs(cfg, mode):
    wl = make_config(cfg, 0)
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
    M = int(wl.cap.min()) // 4
    cid, C, cut = O.cluster(wl, pr, 200, -1, mode)
    check_cluster_invariants(wl, pr, cid, C, cut, 200, M)
    if mode == O.GREEDY:  # every greedy cluster is maximal
        seq = cid[pr]
        ends = np.nonzero(np.diff(seq))[0] + 1
        PM = np.concatenate([[0], np.cumsum(wl.mem[pr])])
        starts = np.concatenate([[0], ends])
        for a, b in zip(starts[:-1], ends):
            assert b + 1 - a > 200 or PM[b + 1] - PM[a] > M


def test_cluster_rejects_bad_order():
    wl = hand6()
    with pytest.raises(O.OracleError) as ei:
        O.cluster(wl, [4, 0, 1, 2, 3, 5], 3, 40)
    assert ei.value.code == O.E_ORDER
    with pytest.raises(O.OracleError) as ei:
        O.cluster(wl, [0, 0, 1, 2, 3, 5], 3, 40)
    assert ei.value.code == O.E_ORDER


# ----------------------------------------------------------------- placement


def coarse_edges(wl, cid):
    c = O.comm(wl)
    src, dst = wl.edges()
    a, b = cid[src], cid[dst]
    keep = a != b
    d = {}
    for x, y, cc in zip(a[keep], b[keep], c[src[keep]]):
        d[(int(x), int(y))] = d.get((int(x), int(y)), 0) + int(cc)
    return d


def check_schedule(wl, cid, C, cdev, fin, be):
    W = np.bincount(cid, weights=wl.w.astype(np.float64), minlength=C).astype(np.int64)
    MEM = np.bincount(cid, weights=wl.mem.astype(np.float64), minlength=C).astype(np.int64)
    start = fin - W
    assert np.all(start >= 0)
    for (a, b), cc in coarse_edges(wl, cid).items():  # precedence + comm (eq. 7)
        assert start[b] >= fin[a] + (cc if cdev[a] != cdev[b] else 0)
    for d in range(wl.D):  # a device runs one cluster at a time
        on = np.nonzero((cdev == d) & (W > 0))[0]
        iv = sorted(zip(start[on], fin[on]))
        for (s0, f0), (s1, f1) in zip(iv[:-1], iv[1:]):
            assert f0 <= s1
        if be == 0:  # memory caps respected
            assert MEM[cdev == d].sum() <= wl.cap[d]


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_place_invariants_configs(cfg):
    wl = make_config(cfg, 2)
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
    cid, C, _ = O.cluster(wl, pr, 200, -1)
    cdev, ndev, span, be, fin = O.place(wl, cid, C, want_fin=True)
    check_schedule(wl, cid, C, cdev, fin, be)
    assert span == fin.max()
    assert np.array_equal(ndev, cdev[cid])


def test_place_random_invariants():
    for s in range(30):
        wl = make_random_dag(500 + s, 6 + s % 25, p_edge=0.3, D=1 + s % 4,
                             cap_frac=(1, 1 + s % 5), multi=(s % 3 == 0),
                             zero_frac=0.25 if s % 5 == 0 else 0.0)
        cid = np.arange(wl.n, dtype=np.int32)
        # cluster ids must follow a topological order: use the levels order
        lev, oid, _, _ = O.topo_levels(wl)
        cid[oid] = np.arange(wl.n)
        cdev, ndev, span, be, fin = O.place(wl, cid, wl.n, want_fin=True)
        check_schedule(wl, cid, wl.n, cdev, fin, be)


def test_place_single_device_closed_form():
    wl = make_config(1, 0)
    wl.D = 1; wl.cap = np.array([10 ** 15], np.int64)
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
    cid, C, _ = O.cluster(wl, pr, 50, -1)
    cdev, ndev, span, be, fin = O.place(wl, cid, C, want_fin=True)
    assert np.all(cdev == 0) and span == int(wl.w.sum()) and be == 0


def test_place_no_move_when_comm_dominates():
    """With huge link latency every move test fails, so nothing leaves device 0."""
    wl = make_config(1, 3)
    wl.lat = 10 ** 12
    wl.cap = np.full(wl.D, 10 ** 15, np.int64)
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
    cid, C, _ = O.cluster(wl, pr, 30, -1)
    cdev, _, span, be, _ = O.place(wl, cid, C, want_fin=True)
    src, dst = wl.edges()
    linked = set(cid[src[cid[src] != cid[dst]]]) | set(cid[dst[cid[src] != cid[dst]]])
    assert be == 0 and all(cdev[t] == 0 for t in linked)


def test_place_graham_bound_independent_tasks():
    """No edges and no comm: Adjusting Placement is a list schedule, so the
    makespan obeys Graham's bound sum(W)/D + (1 - 1/D) max(W)."""
    rng = np.random.default_rng(11)
    for s in range(20):
        n = int(rng.integers(1, 60)); D = int(rng.integers(1, 6))
        w = rng.integers(0, 100, n)
        wl = from_edges(n, [], w, np.zeros(n, np.int64), D, [10 ** 9] * D, 1, 0)
        cdev, _, span, be, fin = O.place(wl, np.arange(n, dtype=np.int32), n, want_fin=True)
        assert span * D <= int(w.sum()) + (D - 1) * int(w.max())
        # every task starts at the earliest time some device is free (list schedule)
        assert be == 0


# ------------------------------------------------------------------ makespan


def lower_upper(wl, ndev):
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, _, cp0 = O.blevel(wl, lev, oid, comm_off=True, want_tlevel=False, want_prio=False)
    sw = int(wl.w.sum())
    lb = max(cp0, -(-sw // wl.D))
    src, dst = wl.edges()
    ub = sw + int(O.comm(wl)[src[ndev[src] != ndev[dst]]].sum())
    return lb, ub


def test_makespan_augmented_and_bounds():
    rng = np.random.default_rng(3)
    for wl in small_dags(60, 1, 40):
        lev, oid, _, _ = O.topo_levels(wl)
        _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
        for _ in range(3):
            ndev = rng.integers(0, wl.D, wl.n).astype(np.uint8)
            ms, st, fi = O.makespan(wl, pr, ndev)
            ref, f = B.makespan_augmented(wl, pr, ndev)
            assert ms[0] == ref and list(fi[0]) == f
            assert np.array_equal(st[0], fi[0] - wl.w)
            lb, ub = lower_upper(wl, ndev)
            assert lb <= ms[0] <= ub


def test_makespan_closed_forms():
    for wl in small_dags(30, 2, 30):
        lev, oid, _, _ = O.topo_levels(wl)
        bl, tl, pr, cp = O.blevel(wl, lev, oid)
        ms, _, _ = O.makespan(wl, pr, np.zeros(wl.n, np.uint8))
        assert ms[0] == int(wl.w.sum())  # one device: no comm, no idle time
        if wl.n <= 255:  # every op on its own device: the critical path
            wl.D = wl.n; wl.cap = np.full(wl.n, 10 ** 12, np.int64)
            ms, st, fi = O.makespan(wl, pr, np.arange(wl.n, dtype=np.uint8))
            assert ms[0] == cp and np.array_equal(fi[0], tl + wl.w)


def test_makespan_alternating_chain():
    n = 9
    w = np.arange(1, n + 1) * 3
    ob = np.arange(n) * 11
    wl = from_edges(n, [(i, i + 1) for i in range(n - 1)], w, ob, 2, [1, 1], 5, 2)
    ms, _, _ = O.makespan(wl, np.arange(n), (np.arange(n) % 2).astype(np.uint8))
    c = -(-ob // 5) + 2
    assert ms[0] == w.sum() + c[:-1].sum()


def test_makespan_brute_force_opt_bound():
    for s in range(12):
        n = 3 + s % 5
        wl = make_random_dag(700 + s, n, p_edge=0.4, D=2 + s % 2)
        lev, oid, _, _ = O.topo_levels(wl)
        _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
        P = np.array(list(B.all_placements(n, wl.D)), np.uint8)
        ms, _, _ = O.makespan(wl, pr, P, want_times=False)
        lb = lower_upper(wl, P[0])[0]
        assert ms.min() >= lb
        for k in range(0, len(P), max(1, len(P) // 7)):  # batched row == single call
            assert O.makespan(wl, pr, P[k], want_times=False)[0][0] == ms[k]
        cid = np.empty(n, np.int32); cid[pr] = np.arange(n)
        _, ndev, _, _ = O.place(wl, cid, n)
        assert ms.min() <= O.makespan(wl, pr, ndev, want_times=False)[0][0]


def test_makespan_rejects_bad_device():
    wl = hand6()
    with pytest.raises(O.OracleError) as ei:
        O.makespan(wl, [1, 0, 3, 2, 4, 5], np.array([0, 1, 2, 0, 0, 0], np.uint8))
    assert ei.value.code == O.E_ARG


# ------------------------------------------------------------- CPD-TOPO order


def cpd_of(wl):
    lev, oid, lp, L = O.topo_levels(wl)
    bl, tl, _, _ = O.blevel(wl, lev, oid, want_prio=False)
    return O.cpd_topo(wl, bl, tl), bl + tl


def test_hand6_cpd():
    gd = load("hand6.json")
    order, cpath = cpd_of(hand6())
    assert list(cpath) == [17, 18, 16, 18, 18, 15]
    assert list(order) == gd["cpd"]["cpd_order"]


def test_cpd_two_chains_and_ties():
    # one source, two chains; the heavier chain (cpath 11) is finished first
    wl = from_edges(5, [(0, 1), (1, 2), (0, 3), (3, 4)], [1, 1, 1, 5, 5], [0] * 5, 2,
                    [10 ** 9] * 2, 1, 0)
    assert list(cpd_of(wl)[0]) == [0, 3, 4, 1, 2]
    # equal chains: the lower id goes first, depth first
    wl = from_edges(5, [(0, 1), (1, 3), (0, 2), (2, 4)], [1] * 5, [0] * 5, 2, [10 ** 9] * 2, 1, 0)
    assert list(cpd_of(wl)[0]) == [0, 1, 3, 2, 4]
    # sources by decreasing cpath, each followed by what it frees
    wl = from_edges(4, [(0, 2), (1, 3)], [1, 4, 1, 1], [0] * 4, 2, [10 ** 9] * 2, 1, 0)
    assert list(cpd_of(wl)[0]) == [1, 3, 0, 2]


def preorder(wl, cpath):
    """Textbook recursive preorder DFS of a forest (every node has at most one
    parent), children visited by decreasing cpath, then increasing id."""
    kids = [[] for _ in range(wl.n)]
    has_parent = np.zeros(wl.n, bool)
    for u, v in zip(*wl.edges()):
        kids[int(u)].append(int(v))
        has_parent[v] = True
    key = lambda v: (-int(cpath[v]), v)  # noqa: E731
    out = []

    def visit(v):
        out.append(v)
        for c in sorted(kids[v], key=key):
            visit(c)

    for r in sorted((v for v in range(wl.n) if not has_parent[v]), key=key):
        visit(r)
    return out


def test_cpd_forest_is_preorder_dfs():
    """On a forest, CPD-TOPO reduces to a preorder depth-first traversal."""
    rng = np.random.default_rng(21)
    for s in range(30):
        n = 1 + int(rng.integers(1, 300))
        parent = [-1 if (v == 0 or rng.random() < 0.1) else int(rng.integers(0, v))
                  for v in range(n)]
        edges = [(p, v) for v, p in enumerate(parent) if p >= 0]
        w = rng.integers(0, 30, n) if s % 3 else np.ones(n, np.int64)  # ties in some cases
        wl = from_edges(n, edges, w, rng.integers(0, 60, n), 2, [10 ** 12] * 2, 7, 3)
        order, cpath = cpd_of(wl)
        assert list(order) == preorder(wl, cpath)


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_cpd_topological_configs(cfg):
    wl = make_config(cfg, 0)
    order, _ = cpd_of(wl)
    pos = np.empty(wl.n, np.int64)
    pos[order] = np.arange(wl.n)
    assert sorted(order.tolist()) == list(range(wl.n))
    src = np.repeat(np.arange(wl.n), np.diff(np.asarray(wl.out_ptr)))
    assert np.all(pos[src] < pos[np.asarray(wl.out_idx)])


def test_cpd_small_dags_and_edge_cases():
    for wl in small_dags():
        order, _ = cpd_of(wl)
        pos = {v: k for k, v in enumerate(order)}
        assert sorted(order.tolist()) == list(range(wl.n))
        assert all(pos[int(u)] < pos[int(v)] for u, v in zip(*wl.edges()))
    wl = from_edges(0, [], [], [], 2, [5, 5], 3, 1)
    assert len(cpd_of(wl)[0]) == 0
    wl = from_edges(6, [(k, k + 1) for k in range(5)], [2] * 6, [1] * 6, 2, [50, 50], 1, 1)
    assert list(cpd_of(wl)[0]) == list(range(6))  # a chain stays a chain
    wl = from_edges(3, [(0, 1), (1, 2), (2, 0)], [1] * 3, [0] * 3, 2, [5, 5], 1, 0)
    with pytest.raises(O.OracleError):
        O.cpd_topo(wl, np.zeros(3, np.int64), np.zeros(3, np.int64))


# ------------------------------------------------------------- DFS-TOPO order


def dfs_by_freed_step(wl):
    """DFS-TOPO restated without a queue: the next node is the ready one freed
    most recently (sources count as freed before the first step), the lowest
    id among those freed by the same step.  Brute force, O(n^2)."""
    n = wl.n
    indeg = np.zeros(n, np.int64)
    us, vs = wl.edges()
    succ = [[] for _ in range(n)]
    for u, v in zip(us, vs):
        indeg[int(v)] += 1
        succ[int(u)].append(int(v))
    freed = {v: -1 for v in range(n) if indeg[v] == 0}
    out = []
    for step in range(n):
        v = min(freed, key=lambda x: (-freed[x], x))
        del freed[v]
        out.append(v)
        for s in succ[v]:
            indeg[s] -= 1
            if indeg[s] == 0:
                freed[s] = step
    return out


def test_dfs_two_chains_keeps_chains_whole():
    # two chains with interleaved ids: level order alternates between them,
    # DFS-TOPO finishes one chain before starting the other
    wl = from_edges(8, [(0, 2), (2, 4), (4, 6), (1, 3), (3, 5), (5, 7)], [1] * 8, [0] * 8, 2,
                    [10 ** 9] * 2, 1, 0)
    order = list(O.dfs_topo(wl))
    assert order == [0, 2, 4, 6, 1, 3, 5, 7]
    _, kahn, _, _ = O.topo_levels(wl)
    assert list(kahn) == list(range(8))

    def cut(order):  # edges between the two halves of the order
        half = set(order[:4])
        return sum((int(u) in half) != (int(v) in half) for u, v in zip(*wl.edges()))
    assert cut(order) == 0 and cut(list(kahn)) == 2


def test_dfs_matches_freed_step_brute_force():
    for wl in small_dags():
        assert list(O.dfs_topo(wl)) == dfs_by_freed_step(wl)
    rng = np.random.default_rng(5)
    for _ in range(40):
        n = int(rng.integers(1, 60))
        edges = sorted({(int(a), int(b)) for a, b in rng.integers(0, n, (2 * n, 2)) if a < b})
        perm = rng.permutation(n)  # ids not in topological order
        edges = [(int(perm[a]), int(perm[b])) for a, b in edges]
        wl = from_edges(n, edges, [1] * n, [0] * n, 2, [10 ** 9] * 2, 1, 0)
        assert list(O.dfs_topo(wl)) == dfs_by_freed_step(wl)


def test_dfs_forest_is_preorder_and_cpd_with_equal_cpath():
    rng = np.random.default_rng(22)
    for _ in range(20):
        n = 1 + int(rng.integers(1, 200))
        parent = [-1 if (v == 0 or rng.random() < 0.1) else int(rng.integers(0, v))
                  for v in range(n)]
        wl = from_edges(n, [(p, v) for v, p in enumerate(parent) if p >= 0], [1] * n, [0] * n, 2,
                        [10 ** 9] * 2, 1, 0)
        assert list(O.dfs_topo(wl)) == preorder(wl, np.zeros(n, np.int64))
    for cfg in (1, 2):  # CPD-TOPO with every cpath equal is DFS-TOPO
        wl = make_config(cfg, 0)
        z = np.zeros(wl.n, np.int64)
        assert np.array_equal(O.dfs_topo(wl), O.cpd_topo(wl, z, z))


def test_dfs_edge_cases():
    assert len(O.dfs_topo(from_edges(0, [], [], [], 2, [5, 5], 3, 1))) == 0
    wl = from_edges(5, [], [1] * 5, [0] * 5, 2, [5, 5], 1, 0)
    assert list(O.dfs_topo(wl)) == list(range(5))  # isolated nodes by id
    wl = from_edges(3, [(0, 1), (1, 2), (2, 0)], [1] * 3, [0] * 3, 2, [5, 5], 1, 0)
    with pytest.raises(O.OracleError):
        O.dfs_topo(wl)


# ------------------------------------------------------- CCR and Order-Place


def test_hand6_ccr_and_order_place():
    gd = load("hand6.json")
    wl = hand6()
    e = gd["ccr"]
    assert O.comm_sums(wl) == (e["edge_comm"], e["w_sum"])
    cid = np.array(gd["order_place"]["cluster_id"], np.int32)
    assert O.comm_sums(wl, cid) == (e["edge_comm_clustered"], e["w_sum"])
    for caps, key in (((60, 60), "caps_60"), ((30, 30), "caps_30")):
        cdev, ndev, be = O.order_place(hand6(cap=caps), cid, 3)
        assert cdev.tolist() == gd["order_place"][key]["cluster_dev"]
        assert be == gd["order_place"][key]["best_effort"]
        assert ndev.tolist() == [int(cdev[c]) for c in cid]


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_ccr_sums_configs(cfg):
    """Unclustered: sum over nodes of out-degree x c (closed form); clustered by
    the DP: equal to the DP's own cut cost S(n)."""
    wl = make_config(cfg, 0)
    c = np.asarray(O.comm(wl), np.int64)
    outdeg = np.diff(np.asarray(wl.out_ptr)).astype(np.int64)
    assert O.comm_sums(wl) == (int((outdeg * c).sum()), int(np.asarray(wl.w).sum()))
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    cid, C, cut = O.cluster(wl, pr, 200, -1)
    assert O.comm_sums(wl, cid)[0] == cut


def test_order_place_properties():
    rng = np.random.default_rng(8)
    for s in range(40):
        wl = make_random_dag(900 + s, 5 + s * 7, p_edge=0.1, D=1 + s % 6, cap_frac=(1, 1 + s % 4))
        order = O.topo_levels(wl)[1]
        cid, C, _ = O.cluster(wl, order, int(rng.integers(1, 12)), -1, s % 2)
        cdev, ndev, be = O.order_place(wl, cid, C)
        mem = np.zeros(C, np.int64)
        np.add.at(mem, cid, np.asarray(wl.mem, np.int64))
        cap = np.asarray(wl.cap, np.int64)
        assert np.all(np.diff(cdev.astype(int)) >= 0)           # devices in cluster order
        assert np.array_equal(ndev, cdev[cid])
        used = np.zeros(wl.D, np.int64)
        np.add.at(used, cdev.astype(int), mem)
        if be == 0:
            assert np.all(used <= cap)
        for t in range(1, C):                                    # a move only when forced
            if cdev[t] != cdev[t - 1]:
                prev = cdev[t - 1]
                filled = mem[:t][cdev[:t] == prev].sum()
                assert filled + mem[t] > cap[prev]
    wl = make_random_dag(7, 30, p_edge=0.2, D=1)
    cid = np.arange(30, dtype=np.int32)
    cdev, _, _ = O.order_place(wl, cid, 30)
    assert not cdev.any()                                        # one device takes all


# --------------------------------------------- makespan under device models


def _rand_topo(wl, rng):
    """A random topological order (Kahn with a random pick among the ready)."""
    indeg = np.diff(np.asarray(wl.in_ptr)).astype(np.int64)
    ready = [v for v in range(wl.n) if indeg[v] == 0]
    out = []
    while ready:
        v = ready.pop(int(rng.integers(len(ready))))
        out.append(v)
        for e in range(wl.out_ptr[v], wl.out_ptr[v + 1]):
            t = int(wl.out_idx[e])
            indeg[t] -= 1
            if indeg[t] == 0:
                ready.append(t)
    return np.array(out, np.int32)


def _ready_times(wl, dev, fin, c):
    """Contention-free ready time of every node from its predecessors' finish."""
    rdy = np.zeros(wl.n, np.int64)
    for u, v in zip(*wl.edges()):
        r = fin[u] + (c[u] if dev[u] != dev[v] else 0)
        rdy[v] = max(rdy[v], r)
    return rdy


def test_model_hand_fixtures():
    for case in load("model_hand.json")["cases"]:
        wl = from_edges(case["n"], case["edges"], case["w"], case["ob"], case["D"], case["cap"],
                        case["bw"], case["lat"])
        het = dict(tmul=case.get("tmul"), bw=case.get("bw_matrix"), lat=case.get("lat_matrix"))
        for m, e in case["models"].items():
            ms, st, fi = O.makespan_model(wl, np.array(case["order"], np.int32),
                                          np.array(case["dev"], np.uint8), int(m), **het)
            assert st[0].tolist() == e["start"], (case["name"], m)
            assert fi[0].tolist() == e["finish"] and int(ms[0]) == e["makespan"], (case["name"], m)


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_model0_is_fifo_makespan(cfg):
    """Model 0 must give orc_makespan's schedule node by node."""
    wl = make_config(cfg, 0)
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    rng = np.random.default_rng(cfg)
    P = rng.integers(0, wl.D, (3, wl.n)).astype(np.uint8)
    a = O.makespan(wl, pr, P)
    b = O.makespan_model(wl, pr, P, 0)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_model_insert_is_first_fit():
    """Each node with w > 0 starts at the smallest t >= its ready time at which
    [t, t + w) overlaps none of the intervals of the nodes placed before it (in
    the order) on its device -- the definition of first fit, checked by brute
    force over the candidates {ready} and those nodes' finish times.  Also: the
    schedule respects every edge, devices never overlap, and no node starts
    later than under FIFO devices (insertion only ever adds free slots)."""
    rng = np.random.default_rng(31)
    for s in range(40):
        n = 2 + s % 23
        wl = make_random_dag(4000 + s, n, p_edge=0.15 + 0.02 * (s % 5), D=1 + s % 4,
                             multi=(s % 5 == 0), zero_frac=0.25 if s % 3 == 0 else 0.0)
        order = _rand_topo(wl, rng)
        dev = rng.integers(0, wl.D, n).astype(np.uint8)
        _, st, fi = O.makespan_model(wl, order, dev, O.MODEL_INSERT)
        st, fi = st[0], fi[0]
        c = np.asarray(O.comm(wl), np.int64)
        w = np.asarray(wl.w, np.int64)
        assert np.array_equal(fi, st + w)
        rdy = _ready_times(wl, dev, fi, c)
        _, st0, _ = O.makespan(wl, order, dev)
        assert np.all(st <= st0[0]), s
        for i, v in enumerate(order):
            assert st[v] >= rdy[v]
            if w[v] == 0:
                assert st[v] == rdy[v]
                continue
            before = [u for u in order[:i] if dev[u] == dev[v] and w[u] > 0]

            def free(t):
                return all(t + w[v] <= st[u] or t >= fi[u] for u in before)

            cands = sorted({int(rdy[v])} | {int(fi[u]) for u in before if fi[u] >= rdy[v]})
            first = next((t for t in cands if free(t)), None)
            if first is None:  # after everything placed so far
                first = max([int(rdy[v])] + [int(fi[u]) for u in before])
            assert st[v] == first, (s, v)
        for x in range(wl.D):
            iv = sorted((st[v], fi[v]) for v in range(n) if dev[v] == x and w[v] > 0)
            assert all(a[1] <= b[0] for a, b in zip(iv, iv[1:]))


def test_model_comm_tasks_properties():
    """Transfers as tasks: one device (no transfers) gives the model without
    them; a chain alternating two devices has no contention (sum of w and c);
    every node starts no earlier than with contention-free comm; per device,
    FIFO order is kept."""
    rng = np.random.default_rng(5)
    for s in range(30):
        n = 2 + s * 5
        wl = make_random_dag(5000 + s, n, p_edge=min(0.5, 3.0 / n), D=2 + s % 5,
                             multi=(s % 4 == 0), zero_frac=0.2 if s % 3 == 0 else 0.0)
        order = _rand_topo(wl, rng)
        dev = rng.integers(0, wl.D, n).astype(np.uint8)
        _, st2, _ = O.makespan_model(wl, order, dev, O.MODEL_COMM_TASKS)
        _, st0, _ = O.makespan_model(wl, order, dev, 0)
        assert np.all(st2[0] >= st0[0]), s
        pos = np.empty(n, np.int64)
        pos[order] = np.arange(n)
        for x in range(wl.D):
            on = sorted((pos[v], v) for v in range(n) if dev[v] == x)
            assert all(st2[0][a[1]] + wl.w[a[1]] <= st2[0][b[1]] for a, b in zip(on, on[1:]))
        one = np.zeros(n, np.uint8)
        for m in (0, 1):
            a = O.makespan_model(wl, order, one, m)
            b = O.makespan_model(wl, order, one, m | O.MODEL_COMM_TASKS)
            assert all(np.array_equal(x, y) for x, y in zip(a, b))
    n = 9
    wl = from_edges(n, [(i, i + 1) for i in range(n - 1)], list(range(1, n + 1)), [3] * n, 2,
                    [100, 100], 2, 1)
    dev = np.array([i % 2 for i in range(n)], np.uint8)
    ms, _, _ = O.makespan_model(wl, np.arange(n, dtype=np.int32), dev, O.MODEL_COMM_TASKS)
    assert int(ms[0]) == sum(range(1, n + 1)) + (n - 1) * (2 + 1)  # c = ceil(3/2) + 1


def test_model_comm_block_task_dag():
    """Transfers occupying both devices' compute queues: every finish time
    equals the longest path of an explicit task DAG (nodes, one transfer task
    per producer and other consuming device, device queue edges) built in
    tests/brute.py; and, elementwise, finish(model 4) >= finish(model 2) >=
    finish(model 0): the blocking model keeps every constraint of the
    channel model (a device's queue serialises its sends and receives, and
    compute too), which keeps every constraint of contention-free comm."""
    rng = np.random.default_rng(77)
    for s in range(40):
        n = 2 + (s * 7) % 40
        wl = make_random_dag(6000 + s, n, p_edge=min(0.5, 3.0 / n), D=1 + s % 6,
                             multi=(s % 4 == 0), zero_frac=0.2 if s % 3 == 0 else 0.0)
        order = _rand_topo(wl, rng)
        dev = rng.integers(0, wl.D, n).astype(np.uint8)
        ms4, st4, fi4 = O.makespan_model(wl, order, dev, O.MODEL_COMM_BLOCK)
        ref_ms, ref_fi = B.makespan_blocking_transfers(wl, order, dev)
        assert fi4[0].tolist() == ref_fi and int(ms4[0]) == ref_ms, s
        assert np.array_equal(st4[0], fi4[0] - np.asarray(wl.w, np.int64))
        _, _, fi2 = O.makespan_model(wl, order, dev, O.MODEL_COMM_TASKS)
        _, _, fi0 = O.makespan_model(wl, order, dev, 0)
        assert np.all(fi4[0] >= fi2[0]) and np.all(fi2[0] >= fi0[0]), s
        one = np.zeros(n, np.uint8)  # one device: no transfers at all
        a = O.makespan_model(wl, order, one, 0)
        b = O.makespan_model(wl, order, one, O.MODEL_COMM_BLOCK)
        assert all(np.array_equal(x, y) for x, y in zip(a, b))
    # a chain alternating two devices never finds a device busy: sum w + sum c
    n = 9
    wl = from_edges(n, [(i, i + 1) for i in range(n - 1)], list(range(1, n + 1)), [3] * n, 2,
                    [100, 100], 2, 1)
    dev = np.array([i % 2 for i in range(n)], np.uint8)
    ms, _, _ = O.makespan_model(wl, np.arange(n, dtype=np.int32), dev, O.MODEL_COMM_BLOCK)
    assert int(ms[0]) == sum(range(1, n + 1)) + (n - 1) * (2 + 1)


def test_model_rejects_bad_inputs():
    wl = from_edges(3, [(0, 1), (1, 2)], [1, 1, 1], [0, 0, 0], 2, [5, 5], 1, 0)
    dev = np.zeros(3, np.uint8)
    for bad in (5, 6, 7, 8):  # the blocking model combines with no other bit
        with pytest.raises(RuntimeError):
            O.makespan_model(wl, np.array([0, 1, 2], np.int32), dev, bad)
    with pytest.raises(RuntimeError):
        O.makespan_model(wl, np.array([1, 0, 2], np.int32), dev, 1)
    with pytest.raises(RuntimeError):
        O.makespan_model(wl, np.array([0, 1, 2], np.int32), np.array([0, 2, 0], np.uint8), 2)


# ------------------------------------- heterogeneous devices, co-location


def _rand_het(rng, D, wl):
    tmul = rng.integers(256, 4096, D)
    bw = rng.integers(1, 4 * int(wl.bw) + 2, (D, D))
    lat = rng.integers(0, 3 * int(wl.lat) + 5, (D, D))
    return tmul, bw, lat


def test_hetero_uniform_is_homogeneous():
    """A descriptor that repeats the homogeneous values changes nothing."""
    rng = np.random.default_rng(41)
    for s in range(12):
        n = 3 + s * 17
        wl = make_random_dag(6100 + s, n, p_edge=min(0.5, 3.0 / n), D=1 + s % 5,
                             multi=(s % 3 == 0), zero_frac=0.2 if s % 2 else 0.0)
        order = _rand_topo(wl, rng)
        P = rng.integers(0, wl.D, (2, n)).astype(np.uint8)
        D = wl.D
        for m in range(4):
            a = O.makespan_model(wl, order, P, m)
            b = O.makespan_model(wl, order, P, m, tmul=[1024] * D, bw=np.full((D, D), wl.bw),
                                 lat=np.full((D, D), wl.lat))
            assert all(np.array_equal(x, y) for x, y in zip(a, b)), (s, m)


def test_hetero_closed_forms():
    """tmul = 2048 everywhere with no comm doubles every time (same as w x 2); one
    device runs sum of ceil(w tmul / 1024); an alternating chain on two devices
    with asymmetric links takes sum of durations plus the links crossed."""
    rng = np.random.default_rng(42)
    for s in range(10):
        n = 5 + s * 23
        wl = make_random_dag(6200 + s, n, p_edge=min(0.5, 3.0 / n), D=2 + s % 3)
        wl.ob = np.zeros(n, np.int64)
        wl.lat = 0
        order = _rand_topo(wl, rng)
        P = rng.integers(0, wl.D, (2, n)).astype(np.uint8)
        w2 = from_edges(n, list(zip(*wl.edges())), 2 * np.asarray(wl.w), wl.ob, wl.D, wl.cap,
                        wl.bw, 0)
        for m in range(4):
            a = O.makespan_model(wl, order, P, m, tmul=[2048] * wl.D)
            b = O.makespan_model(w2, order, P, m)
            assert all(np.array_equal(x, y) for x, y in zip(a, b)), (s, m)
        t = int(rng.integers(100, 5000))
        one = O.makespan_model(wl, order, np.zeros(n, np.uint8), s % 4, tmul=[t] * wl.D)
        assert int(one[0][0]) == sum(-(-int(x) * t // 1024) for x in wl.w)
    n = 11
    w = list(range(3, 3 + n))
    ob = [7 + i for i in range(n)]
    wl = from_edges(n, [(i, i + 1) for i in range(n - 1)], w, ob, 2, [100, 100], 1, 0)
    tm, bw, lat = [700, 1500], [[1, 3], [2, 1]], [[0, 4], [9, 0]]
    dev = np.array([i % 2 for i in range(n)], np.uint8)
    expect = sum(-(-w[i] * tm[i % 2] // 1024) for i in range(n))
    expect += sum(-(-ob[i] // bw[i % 2][1 - i % 2]) + lat[i % 2][1 - i % 2] for i in range(n - 1))
    for m in range(4):
        ms, _, _ = O.makespan_model(wl, np.arange(n, dtype=np.int32), dev, m, tmul=tm, bw=bw,
                                    lat=lat)
        assert int(ms[0]) == expect


def test_hetero_insert_is_first_fit():
    """The first-fit definition with per-device durations and per-link comm."""
    rng = np.random.default_rng(43)
    for s in range(25):
        n = 2 + s % 19
        wl = make_random_dag(6300 + s, n, p_edge=0.2, D=2 + s % 3, zero_frac=0.2)
        order = _rand_topo(wl, rng)
        dev = rng.integers(0, wl.D, n).astype(np.uint8)
        tm, bw, lat = _rand_het(rng, wl.D, wl)
        _, st, fi = O.makespan_model(wl, order, dev, O.MODEL_INSERT, tmul=tm, bw=bw, lat=lat)
        st, fi = st[0], fi[0]
        dur = np.array([-(-int(wl.w[v]) * int(tm[dev[v]]) // 1024) for v in range(n)])
        assert np.array_equal(fi - st, dur)
        rdy = np.zeros(n, np.int64)
        for u, v in zip(*wl.edges()):
            a, b = dev[u], dev[v]
            c = 0 if a == b else -(-int(wl.ob[u]) // int(bw[a][b])) + int(lat[a][b])
            rdy[v] = max(rdy[v], fi[u] + c)
        for i, v in enumerate(order):
            if dur[v] == 0:
                assert st[v] == rdy[v]
                continue
            before = [u for u in order[:i] if dev[u] == dev[v] and dur[u] > 0]
            cands = sorted({int(rdy[v])} | {int(fi[u]) for u in before if fi[u] >= rdy[v]})
            first = next(t for t in cands
                         if all(t + dur[v] <= st[u] or t >= fi[u] for u in before))
            assert st[v] == first, (s, v)


def test_hetero_rejects_bad_descriptors():
    wl = from_edges(3, [(0, 1), (1, 2)], [1, 1, 1], [1, 1, 1], 2, [5, 5], 1, 0)
    o, dev = np.array([0, 1, 2], np.int32), np.array([0, 1, 0], np.uint8)
    for kw in (dict(tmul=[0, 1024]), dict(tmul=[1024, 70000]), dict(bw=[[1, 0], [1, 1]]),
               dict(lat=[[0, -1], [0, 0]])):
        with pytest.raises(RuntimeError):
            O.makespan_model(wl, o, dev, 0, **kw)


def test_colocate_hand_and_properties():
    case = load("colocate_hand.json")["cases"][0]
    wl = from_edges(case["n"], case["edges"], [1] * case["n"], [0] * case["n"], 4, [9] * 4, 1, 0)
    got = O.colocate(wl, case["order"], case["group"], case["n_groups"],
                     np.array(case["dev_in"], np.uint8))
    assert got.tolist() == case["dev_out"]
    rng = np.random.default_rng(44)
    for s in range(20):
        n = 1 + s * 13
        wl = make_random_dag(6400 + s, n, p_edge=min(0.5, 3.0 / n), D=1 + s % 6)
        order = _rand_topo(wl, rng)
        G = 1 + s % 7
        grp = rng.integers(-1, G, n).astype(np.int32)
        P = rng.integers(0, wl.D, (3, n)).astype(np.uint8)
        out = O.colocate(wl, order, grp, G, P)
        pos = np.empty(n, np.int64)
        pos[order] = np.arange(n)
        for k in range(3):
            assert np.array_equal(out[k][grp < 0], P[k][grp < 0])
            for x in range(G):
                mem = np.nonzero(grp == x)[0]
                if mem.size:
                    lead = mem[np.argmin(pos[mem])]
                    assert np.all(out[k][mem] == P[k][lead])
        assert np.array_equal(O.colocate(wl, order, grp, G, out), out)  # idempotent
        single = np.arange(n, dtype=np.int32)
        assert np.array_equal(O.colocate(wl, order, single, n, P), P)
    wl = from_edges(2, [(0, 1)], [1, 1], [0, 0], 2, [5, 5], 1, 0)
    with pytest.raises(RuntimeError):
        O.colocate(wl, [0, 1], [0, 2], 2, np.zeros(2, np.uint8))
    with pytest.raises(RuntimeError):
        O.colocate(wl, [1, 0], [0, 0], 1, np.zeros(2, np.uint8))


# ------------- Adjusting Placement with heterogeneous devices/links and co-location


@pytest.mark.parametrize("case", load("place_ext_hand.json")["cases"], ids=lambda c: c["name"])
def test_place_ext_hand_cases(case):
    wl = from_edges(case["n"], case["edges"], case["w"], case["ob"], case["D"], case["cap"],
                    case["bw"], case["lat"])
    for v in case["variants"]:
        cdev, ndev, span, be, fin = O.place_ext(
            wl, case["cluster_id"], case["C"], tmul=v.get("tmul"), bw=v.get("bw_matrix"),
            lat=v.get("lat_matrix"), group=v.get("group"), n_groups=v.get("n_groups", 0))
        assert cdev.tolist() == v["cluster_dev"] and ndev.tolist() == v["node_dev"], case["name"]
        assert fin.tolist() == v["fin"] and span == v["span"] and be == v["be"], case["name"]


def _clustered(wl, seed, R=None):
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    R = R if R is not None else 1 + seed % 9
    cid, C, _ = O.cluster(wl, pr, R, -1, seed % 2)
    return pr, cid, C


def test_place_ext_reduces_to_place():
    """No descriptor and no groups: Algorithm 2 as orc_place computes it (a
    separately pinned function); singleton groups change nothing either."""
    for s in range(30):
        n = 3 + (s * 37) % 300
        wl = make_random_dag(8800 + s, n, p_edge=min(0.5, 4.0 / n), D=1 + s % 7,
                             cap_frac=(1, 1 + s % 5), multi=(s % 3 == 0),
                             zero_frac=0.2 if s % 4 == 0 else 0.0)
        _, cid, C = _clustered(wl, s)
        ref = O.place(wl, cid, C, want_fin=True)
        got = O.place_ext(wl, cid, C)
        single = O.place_ext(wl, cid, C, group=np.arange(n, dtype=np.int32), n_groups=n)
        for r in (got, single):
            assert np.array_equal(r[0], ref[0]) and np.array_equal(r[1], ref[1]), s
            assert r[2] == ref[2] and r[3] == ref[3] and np.array_equal(r[4], ref[4]), s


def test_place_ext_uniform_descriptors():
    """Uniform descriptors reduce to the homogeneous placement: tmul = 2048 on
    every device with no comm doubles every time (the same devices as orc_place
    on the graph with w doubled, the same finish times); link tables repeating
    (bw, lat) with every ob a multiple of bw give exactly the summed c[u] of the
    coarse edges (ceil(OB / bw) + N lat = sum of ceil(ob / bw) + lat)."""
    for s in range(20):
        n = 5 + (s * 53) % 250
        D = 2 + s % 5
        wl = make_random_dag(8900 + s, n, p_edge=min(0.5, 4.0 / n), D=D, cap_frac=(1, 2 + s % 3),
                             multi=(s % 2 == 0), bw=3, lat=0)
        wl.ob = np.zeros(n, np.int64)  # no comm: c = 0 everywhere
        _, cid, C = _clustered(wl, s)
        got = O.place_ext(wl, cid, C, tmul=[2048] * D)
        wl2 = make_random_dag(8900 + s, n, p_edge=min(0.5, 4.0 / n), D=D, cap_frac=(1, 2 + s % 3),
                              multi=(s % 2 == 0), bw=3, lat=0)
        wl2.ob = np.zeros(n, np.int64)
        wl2.w = 2 * np.asarray(wl.w, np.int64)
        ref = O.place(wl2, cid, C, want_fin=True)
        assert np.array_equal(got[0], ref[0]) and np.array_equal(got[4], ref[4]), s
        # link tables equal to the homogeneous link, ob multiples of bw
        wl3 = make_random_dag(9000 + s, n, p_edge=min(0.5, 4.0 / n), D=D, cap_frac=(1, 3),
                              multi=(s % 2 == 1), bw=4, lat=3)
        wl3.ob = 4 * (np.asarray(wl3.ob, np.int64) // 4)
        wl3.mem = 2 * wl3.ob
        _, cid3, C3 = _clustered(wl3, s)
        ref3 = O.place(wl3, cid3, C3, want_fin=True)
        got3 = O.place_ext(wl3, cid3, C3, bw=np.full((D, D), 4), lat=np.full((D, D), 3))
        for a, b in zip(got3, (ref3[0], ref3[1], ref3[2], ref3[3], ref3[4])):
            assert np.array_equal(np.asarray(a), np.asarray(b)), s


def test_place_ext_colocation_memory_and_devices():
    """Co-location inside the algorithm, checked from the outputs alone: every
    group member runs on its leading cluster's device (the smallest cluster
    id among the members); replaying Algorithm 2's memory bookkeeping (the
    followers charged to that device when their own cluster is placed, then
    the cluster's other members to its device), a cluster not placed by best
    effort always fitted its device's remaining memory; with best effort 0,
    every device ends within its cap unless followers overfilled it."""
    rng = np.random.default_rng(8)
    for s in range(25):
        n = 10 + (s * 61) % 400
        D = 2 + s % 6
        wl = make_random_dag(9100 + s, n, p_edge=min(0.5, 4.0 / n), D=D, cap_frac=(1, 1 + s % 4),
                             multi=(s % 3 == 0))
        _, cid, C = _clustered(wl, s)
        G = max(1, n // (3 + s % 5))
        grp = rng.integers(-1, G, n).astype(np.int32)
        het = dict(tmul=rng.integers(512, 3000, D)) if s % 2 else {}
        cdev, ndev, span, be, fin = O.place_ext(wl, cid, C, group=grp, n_groups=G, **het)
        lead = np.full(G, C, np.int64)
        np.minimum.at(lead, grp[grp >= 0], cid[grp >= 0])
        member = grp >= 0
        assert np.array_equal(ndev[member], cdev[lead[grp[member]]])
        assert np.array_equal(ndev[~member], cdev[cid[~member]])
        follower = member & (lead[np.where(member, grp, 0)] < cid)
        mem = np.asarray(wl.mem, np.int64)
        ava = np.asarray(wl.cap, np.int64).copy()
        over = False
        n_be = 0
        for t in range(C):
            for v in np.nonzero(follower & (cid == t))[0]:
                ava[cdev[lead[grp[v]]]] -= mem[v]
            over |= bool((ava < 0).any())
            own = mem[(cid == t) & ~follower].sum()
            if (ava >= own).any():        # some device fits: the pick must fit
                assert ava[cdev[t]] >= own, (s, t)
            else:
                n_be += 1
            ava[cdev[t]] -= own
        assert n_be == be
        if be == 0 and not over:
            assert (ava >= 0).all()


def test_place_ext_rejects_bad_inputs():
    wl = from_edges(3, [(0, 1), (1, 2)], [1, 1, 1], [0, 0, 0], 2, [5, 5], 1, 0)
    with pytest.raises(RuntimeError):  # group id out of range
        O.place_ext(wl, [0, 1, 2], 3, group=[0, 1, 2], n_groups=2)
    with pytest.raises(RuntimeError):  # bad time multiplier
        O.place_ext(wl, [0, 1, 2], 3, tmul=[0, 1024])
    with pytest.raises(RuntimeError):  # clusters against the edges
        O.place_ext(wl, [2, 1, 0], 3)
