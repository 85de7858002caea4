"""GPU parity of the longest paths (levels, b-level eq. 3, t-level eq. 2) and
of the clustering DP (eq. 4-6) by policy iteration, against the CPU oracle,
tolerance 0, with the path each call took (cel_blevel_info, cel_topo_levels_info,
cel_cluster_info); every test in both evaluation modes."""
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


@pytest.fixture(autouse=True, params=[1, 2], ids=["packed", "rounds"])
def pi_mode(request):
    """Every test twice: packed entries with asynchronous pointer jumping
    (where the values fit), and 16-byte entries with synchronous rounds."""
    was = cel.policy_iteration(request.param)
    yield request.param
    cel.policy_iteration(was)


def np_(t):
    return t.detach().cpu().numpy()


def tt(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(DEV)


def run(wl, comm_off=False):
    lev, oid, lp, L = O.topo_levels(wl)
    ref = O.blevel(wl, lev, oid, comm_off=comm_off)
    g, d = cel.Graph.from_arrays(wl, DEV), cel.Devices.from_arrays(wl)
    bl, tl, pr, cp = cel.blevel(g, d, tt(lev, np.int32), tt(lp, np.int32), tt(oid, np.int32), L,
                                comm_off=comm_off, want_tlevel=True)
    info = cel.blevel_info()
    assert cp == ref[3]
    assert np.array_equal(np_(bl), ref[0]) and np.array_equal(np_(tl), ref[1])
    assert np.array_equal(np_(pr), ref[2])
    return L, info


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_policy_converges_on_configs(cfg):
    """Both longest paths by policy iteration, exact; a node h hops from the
    end of its paths is exact after h + 1 iterations, so at most L + 1 run."""
    L, info = run(make_config(cfg, 0))
    for path, iters in info:
        assert path == 0 and 1 <= iters <= L + 1


def test_policy_budget_then_sweep():
    """Layered-200k (196 levels, parents from up to 8 levels back) needs more
    iterations than its budget: the level sweeps give the exact values."""
    L, info = run(make_config(5, 0))
    for path, iters in info:
        assert path in (0, 1) and iters >= 1


def test_policy_ties_and_zero_costs():
    """Many equal values: zero compute and comm everywhere but a few nodes,
    a diamond lattice of equal-length paths (values spread one level per
    iteration here, so the budget may run out before the sweep's cost: either
    path, exact)."""
    n, W = 4000, 40
    edges = []
    for v in range(W, n):
        lvl, j = divmod(v, W)
        edges.append(((lvl - 1) * W + j, v))
        edges.append(((lvl - 1) * W + (j + 1) % W, v))
    rng = np.random.default_rng(4)
    w = np.zeros(n, np.int64)
    w[rng.choice(n, 10, replace=False)] = 5
    wl = from_edges(n, edges, w, np.zeros(n, np.int64), 2, [10 ** 9] * 2, 1, 0)
    L, info = run(wl)
    for path, iters in info:
        assert path in (0, 1) and 1 <= iters <= L + 1
    run(wl, comm_off=True)


def test_policy_long_lists_both_ways():
    """A source with 20,000 successors (five chunks of the b-level's long-list
    path) and a sink with 12,000 predecessors (the t-level's), between chains."""
    rng = np.random.default_rng(8)
    n = 33000
    edges = [(0, j) for j in range(1, 20001)]
    edges += [(j, 32999) for j in range(20001, 32999)]
    edges += [(j, 20001 + int(rng.integers(0, 12998))) for j in range(1, 20001)]
    edges += [(j, j + 1) for j in range(20001, 32998, 7)]
    edges = sorted(set((u, v) for u, v in edges if u < v))
    wl = from_edges(n, edges, rng.integers(1, 90, n), rng.integers(0, 3000, n), 4,
                    [10 ** 12] * 4, 5, 3)
    L, info = run(wl)
    for path, iters in info:
        assert path == 0 and iters <= L + 1


@pytest.mark.parametrize("cfg", [2, 3, 5])
def test_levels_by_policy_iteration(cfg):
    """Kahn's levels as longest paths over the predecessors: the level of
    every node, the level-sorted order (ids ascending within a level) and the
    level starts equal the oracle's; layered-200k may exceed the budget of
    12 iterations and take Kahn's kernel."""
    wl = make_config(cfg, 0)
    ref = O.topo_levels(wl)
    g = cel.Graph.from_arrays(wl, DEV)
    lev, oid, lp, L = cel.topo_levels(g)
    path, iters = cel.topo_levels_info()
    assert L == ref[3]
    assert np.array_equal(np_(lev), ref[0]) and np.array_equal(np_(oid), ref[1])
    assert np.array_equal(np_(lp), ref[2])
    assert (path, iters > 0) in ((0, True), (1, True))
    if cfg in (2, 3):
        assert path == 0 and iters <= 12


def test_levels_policy_cycle_detected():
    """A cycle in a graph large enough for policy iteration is reported as
    such (by a pointer cycle, or by Kahn's kernel after the budget)."""
    n = 20000
    edges = [(i, i + 1) for i in range(n - 1)] + [(n - 1, n // 2)]
    wl = from_edges(n, edges, [1] * n, [1] * n, 1, [1], 1, 0)
    g = cel.Graph.from_arrays(wl, DEV)
    with pytest.raises(cel.CelError) as ei:
        cel.topo_levels(g)
    assert ei.value.code == -2


def gpu_cluster(wl, order, R, M):
    g, d = cel.Graph.from_arrays(wl, DEV), cel.Devices.from_arrays(wl)
    cid, C, cut = cel.cluster(g, d, tt(order, np.int32), R, M, cel.CLUSTER_DP)
    return np_(cid), C, cut, cel.cluster_info()


@pytest.mark.parametrize("cfg", [2, 3, 5])
def test_cluster_dp_by_policy_iteration(cfg):
    """The DP of eq. 4-6 as a shortest path over breakpoints, by policy
    iteration: clusters, their number and the cut cost equal the oracle's
    sequential DP (ties to the smallest start) for several windows and caps."""
    wl = make_config(cfg, 0)
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    avg = int(wl.mem.sum()) // wl.n
    for R, M in ((200, -1), (37, -1), (1, -1), (1000, avg * 40)):
        ref = O.cluster(wl, pr, R, M)
        cid, C, cut, (path, iters) = gpu_cluster(wl, pr, R, M)
        assert C == ref[1] and cut == ref[2] and np.array_equal(cid, ref[0]), (R, M)
        assert path in (0, 1) and iters >= 1, (R, M)
        if cfg in (2, 3) and R == 200:
            assert path == 0, (R, M)


def test_cluster_dp_policy_random_orders():
    """Random DAGs of 20,000-30,000 nodes (1-3 parents among the previous 500
    ids, some edges doubled, some costs zero), clustered on random
    topological orders (not level-monotone)."""
    import heapq
    for s in range(3):
        n = 20000 + 5000 * s
        rng = np.random.default_rng(900 + s)
        k = rng.integers(1, 4, n)
        k[0] = 0
        dst = np.repeat(np.arange(n), k)
        src = dst - 1 - (rng.random(dst.size) * np.minimum(dst, 500)).astype(np.int64)
        edges = list(zip(src.tolist(), dst.tolist()))
        if s == 1:  # parallel edges
            edges += edges[::7]
        w = rng.integers(1, 60, n)
        ob = rng.integers(0, 300, n)
        if s == 2:
            w[rng.random(n) < 0.2] = 0
            ob[rng.random(n) < 0.2] = 0
        wl = from_edges(n, edges, w, ob, 3, [int(2 * ob.sum() + n)] * 3, 7, 3)
        # a random topological order: Kahn with random priorities
        indeg = np.diff(wl.in_ptr).copy()
        key = rng.random(n)
        heap = [(key[v], v) for v in range(n) if indeg[v] == 0]
        heapq.heapify(heap)
        order = []
        while heap:
            _, u = heapq.heappop(heap)
            order.append(u)
            for e in range(wl.out_ptr[u], wl.out_ptr[u + 1]):
                v = wl.out_idx[e]
                indeg[v] -= 1
                if indeg[v] == 0:
                    heapq.heappush(heap, (key[v], v))
        order = np.array(order, np.int32)
        for R in (64, 300):
            ref = O.cluster(wl, order, R, -1)
            cid, C, cut, (path, iters) = gpu_cluster(wl, order, R, -1)
            assert C == ref[1] and cut == ref[2] and np.array_equal(cid, ref[0]), (s, R)


def test_policy_values_beyond_packed_entries():
    """Transformer-24 with w and output sizes scaled by 2^22: the total of w
    and c (and the DP's largest S) exceeds the 40 bits of a packed entry, so
    even the packed mode takes the 16-byte rounds; exact all the same."""
    import dataclasses
    wl = make_config(2, 0)
    wl = dataclasses.replace(wl, w=wl.w << 22, ob=wl.ob << 22)
    src = np.repeat(np.arange(wl.n), np.diff(wl.out_ptr))
    c = wl.ob // wl.bw + (wl.ob % wl.bw != 0) + wl.lat
    assert int(wl.w.sum()) + int(c[src].sum()) >= 2 ** 40
    L, info = run(wl)
    for path, iters in info:
        assert path == 0 and iters >= 1
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    ref = O.cluster(wl, pr, 200, -1)
    cid, C, cut, (path, iters) = gpu_cluster(wl, pr, 200, -1)
    assert C == ref[1] and cut == ref[2] and np.array_equal(cid, ref[0])
