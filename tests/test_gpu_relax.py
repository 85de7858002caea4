"""GPU parity of the single-placement makespan by relaxation over the edges
between devices (cel_makespan, K = 1), against the CPU oracle, tolerance 0.

The relaxation's round count is pinned by a property of the schedule: a
round settles every node whose finish is decided by a path with one more
device change, so at most (the longest run of device changes along any
path) + 2 rounds run, the last changing nothing."""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU, skipped there
    pytest.skip("needs a ROCm GPU", allow_module_level=True)

import paper_2208_00184_amd as cel  # noqa: E402
from oracle import oracle as O  # noqa: E402
from workloads import from_edges, make_config  # noqa: E402

DEV = "cuda:0"


def np_(t):
    return t.detach().cpu().numpy()


def tt(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(DEV)


def device_changes(wl, order, dev):
    """Longest run of device changes along a path of the DAG, the device's
    own chain (its nodes in `order`) counting as a path without a change."""
    hop = np.zeros(wl.n, np.int64)
    last = {}
    ip, ix = wl.in_ptr, wl.in_idx
    for v in order:
        d = int(dev[v])
        h = last.get(d, 0)
        for e in range(ip[v], ip[v + 1]):
            u = ix[e]
            if dev[u] != d and hop[u] + 1 > h:
                h = hop[u] + 1
        hop[v] = h
        last[d] = h
    return int(hop.max()) if wl.n else 0


def run_one(wl, order, lev, lp, L, dev, mode=1, want_times=True):
    g, d = cel.Graph.from_arrays(wl, DEV), cel.Devices.from_arrays(wl)
    was = cel.makespan_relax(mode)
    try:
        ms, st, fi = cel.makespan(g, d, tt(order, np.int32), tt(lev, np.int32), tt(lp, np.int32),
                                  L, tt(dev, np.uint8), want_times=want_times)
        info = cel.makespan_info()
    finally:
        cel.makespan_relax(was)
    return ms, st, fi, info


def check(wl, order, dev, got):
    ms, st, fi, _ = got
    ref_ms, ref_st, ref_fi = O.makespan(wl, order, dev[None, :])
    assert np_(ms)[0] == ref_ms[0]
    if fi is not None:
        assert np.array_equal(np_(fi)[0], ref_fi[0]) and np.array_equal(np_(st)[0], ref_st[0])


@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
def test_relax_adjusting_placement(cfg):
    """Adjusting Placement's devices: the relaxation converges, within the
    bound of the longest run of device changes, to the oracle's schedule."""
    wl = make_config(cfg, 0)
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    cid, C, _ = O.cluster(wl, pr, 200, -1)
    _, ndev, _, _ = O.place(wl, cid, C)
    got = run_one(wl, pr, lev, lp, L, ndev)
    check(wl, pr, ndev, got)
    path, rounds = got[3]
    assert path == 0
    assert 2 <= rounds <= device_changes(wl, pr, ndev) + 2
    # the makespan alone (no start / finish arrays)
    got2 = run_one(wl, pr, lev, lp, L, ndev, want_times=False)
    assert np_(got2[0])[0] == np_(got[0])[0] and got2[3] == got[3]


def test_relax_gives_up_on_alternating_chain():
    """A chain whose every edge changes device needs a round per node: the
    relaxation stops at its budget and the level sweep gives the schedule."""
    n = 600
    rng = np.random.default_rng(3)
    edges = [(i, i + 1) for i in range(n - 1)]
    wl = from_edges(n, edges, rng.integers(1, 100, n), rng.integers(0, 5000, n), 2,
                    [10 ** 12] * 2, 5, 40)
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    dev = (np.arange(n) % 2).astype(np.uint8)
    got = run_one(wl, pr, lev, lp, L, dev)
    check(wl, pr, dev, got)
    path, rounds = got[3]
    assert path == 1 and 0 < rounds < n


def blocked_graph(seed):
    """5,000 nodes in 100 levels of 50; devices by ranges of the priority
    order, so the chains start at slots 0, 256, 257, 512, 1536, 2559, 3584
    and 3884 (a workgroup's first slot, mid-tile, the next slot); a few
    nodes have 3-8 or 20 predecessors on other devices."""
    rng = np.random.default_rng(seed)
    W, Lv = 50, 100
    n = W * Lv
    edges = set()
    for l in range(1, Lv):
        for j in range(W):
            v = l * W + j
            for u in rng.integers(max(0, l - 3) * W, l * W, int(rng.integers(1, 4))):
                edges.add((int(u), v))
    for v in rng.choice(np.arange(10 * W, n), 12, replace=False):  # wide fan-in nodes
        k = 20 if v % 2 else int(rng.integers(3, 9))
        for u in rng.choice(np.arange(0, (int(v) // W) * W), k, replace=False):
            edges.add((int(u), int(v)))
    D = 8
    wl = from_edges(n, sorted(edges), rng.integers(1, 3000, n), rng.integers(0, 1 << 20, n), D,
                    [10 ** 12] * D, 9, 700)
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    counts = [256, 1, 255, 1024, 1023, 1025, 300, 1116]  # nodes of device 0, 1, ...
    dev = np.empty(n, np.uint8)
    dev[pr] = np.repeat(np.arange(D), counts)  # by position in the priority order
    # swaps of two nodes' devices (the counts stay): more edges between devices
    for a, b in rng.choice(n, (8, 2), replace=False):
        dev[a], dev[b] = dev[b], dev[a]
    return wl, pr, lev, lp, L, dev


@pytest.mark.parametrize("mode", [1, 2, 3, 5, 20])
def test_relax_workgroup_and_tile_boundaries(mode):
    """The same schedule with the slots spread over 20 workgroups of one tile
    (mode 1) or packed into 2, 3 and 5 workgroups of up to 16 tiles: chain
    starts on workgroup, tile and wave boundaries, carries across tiles and
    workgroups."""
    wl, pr, lev, lp, L, dev = blocked_graph(11)
    got = run_one(wl, pr, lev, lp, L, dev, mode=mode)
    check(wl, pr, dev, got)
    path, rounds = got[3]
    assert path == 0 and 2 <= rounds <= device_changes(wl, pr, dev) + 2


def test_relax_one_device_and_tiny():
    """No edge between devices: two rounds; one node; two nodes on two devices."""
    wl, pr, lev, lp, L, _ = blocked_graph(12)
    dev = np.full(wl.n, 5, np.uint8)
    got = run_one(wl, pr, lev, lp, L, dev)
    check(wl, pr, dev, got)
    assert got[3] == (0, 2)
    for n, edges, dev in [(1, [], [1]), (2, [(0, 1)], [1, 0]), (3, [], [2, 0, 2])]:
        wl = from_edges(n, edges, [7, 3, 4][:n], [100, 0, 9][:n], 3, [10 ** 9] * 3, 3, 1)
        lev, oid, lp, L = O.topo_levels(wl)
        _, _, pr, _ = O.blevel(wl, lev, oid)
        dev = np.asarray(dev, np.uint8)
        got = run_one(wl, pr, lev, lp, L, dev)
        check(wl, pr, dev, got)
        assert got[3][0] == 0


def test_relax_sink_with_huge_comm():
    """A sink's output tensor may exceed what the overflow bound covers (it
    is never sent): the relaxation must not form fin + c for it."""
    n = 4
    edges = [(0, 1), (1, 2), (0, 3)]
    wl = from_edges(n, edges, [5, 6, 7, 8], [10, 20, 2 ** 62, 2 ** 62], 2, [10 ** 12] * 2, 1, 3,
                    mem=[1, 1, 1, 1])
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid, comm_off=True)
    dev = np.array([0, 1, 0, 1], np.uint8)
    got = run_one(wl, pr, lev, lp, L, dev)
    check(wl, pr, dev, got)
    assert got[3][0] == 0
