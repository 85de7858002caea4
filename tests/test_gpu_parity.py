"""GPU parity: the HIP path (through the C ABI) against the CPU oracle,
element by element, tolerance 0 (all arithmetic is int64)."""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU, skipped there
    pytest.skip("needs a ROCm GPU", allow_module_level=True)

import paper_2208_00184_amd as cel  # noqa: E402
from oracle import oracle as O  # noqa: E402
from workloads import from_edges, make_config, make_random_dag, perturb_placements  # noqa: E402

DEV = "cuda:0"


def np_(t):
    return t.detach().cpu().numpy()


def up(wl):
    return cel.Graph.from_arrays(wl, DEV), cel.Devices.from_arrays(wl)


def tt(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(DEV)


_cache = {}


def config(cfg, seed):
    key = (cfg, seed)
    if key not in _cache:
        _cache.clear()
        wl = make_config(cfg, seed)
        lev, oid, lp, L = O.topo_levels(wl)
        bl, tl, pr, cp = O.blevel(wl, lev, oid)
        _cache[key] = (wl, (lev, oid, lp, L), (bl, tl, pr, cp))
    return _cache[key]


def run_topo_blevel(wl, want_tlevel=True):
    g, d = up(wl)
    lev, oid, lp, L = cel.topo_levels(g)
    bl, tl, pr, cp = cel.blevel(g, d, lev, lp, oid, L, want_tlevel=want_tlevel)
    return g, d, (lev, oid, lp, L), (bl, tl, pr, cp)


def assert_topo_blevel(wl, ref_t, ref_b, got_t, got_b):
    lev, oid, lp, L = got_t
    assert L == ref_t[3]
    assert np.array_equal(np_(lev), ref_t[0])
    assert np.array_equal(np_(oid), ref_t[1])
    assert np.array_equal(np_(lp), ref_t[2])
    bl, tl, pr, cp = got_b
    assert cp == ref_b[3]
    assert np.array_equal(np_(bl), ref_b[0])
    if tl is not None:
        assert np.array_equal(np_(tl), ref_b[1])
    assert np.array_equal(np_(pr), ref_b[2])


# ------------------------------------------------------------ configs 1-3, 5


@pytest.fixture(params=[1, 2, 0], ids=["policy", "policy-rounds", "sweep"])
def bl_path(request):
    """b-level and t-level by policy iteration (packed entries and
    asynchronous jumps, or 16-byte entries and synchronous rounds; falling
    back to the level sweeps when it does not converge) or by the level
    sweeps."""
    was = cel.policy_iteration(request.param)
    yield request.param
    cel.policy_iteration(was)


@pytest.mark.parametrize("cfg,seed", [(1, 0), (1, 1), (1, 2), (2, 0), (2, 1), (3, 0), (3, 2),
                                      (5, 0)])
def test_topo_blevel_configs(cfg, seed, bl_path):
    wl, rt, rb = config(cfg, seed)
    _, _, gt, gb = run_topo_blevel(wl)
    assert_topo_blevel(wl, rt, rb, gt, gb)


@pytest.mark.parametrize("cfg", [1, 2, 3])
def test_blevel_comm_off(cfg, bl_path):
    wl, rt, _ = config(cfg, 0)
    lev, oid, lp, L = rt
    ref = O.blevel(wl, lev, oid, comm_off=True)
    g, d = up(wl)
    bl, _, pr, cp = cel.blevel(g, d, tt(lev, np.int32), tt(lp, np.int32), tt(oid, np.int32), L,
                               comm_off=True)
    assert cp == ref[3]
    assert np.array_equal(np_(bl), ref[0]) and np.array_equal(np_(pr), ref[2])


def test_blevel_tlevel_on_caller_streams(bl_path):
    """The t-level sweep runs on a side stream joined back into the caller's
    stream: results must be complete when the call returns, on the default
    stream and on user streams used in turn (the side stream is shared)."""
    outs = []
    for cfg in (1, 3):
        wl, rt, rb = config(cfg, 0)
        lev, oid, lp, L = rt
        g, d = up(wl)
        args = (tt(lev, np.int32), tt(lp, np.int32), tt(oid, np.int32), L)
        torch.cuda.synchronize()
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        for stream in (None, s1, s2, s1):
            if stream is None:
                bl, tl, pr, cp = cel.blevel(g, d, *args, want_tlevel=True)
            else:
                with torch.cuda.stream(stream):
                    bl, tl, pr, cp = cel.blevel(g, d, *args, want_tlevel=True)
                    tl_host = tl.to("cpu", non_blocking=False)  # ordered on `stream`
                assert np.array_equal(tl_host.numpy(), rb[1])
            torch.cuda.synchronize()
            assert cp == rb[3]
            assert np.array_equal(np_(bl), rb[0]) and np.array_equal(np_(tl), rb[1])
            assert np.array_equal(np_(pr), rb[2])
        outs.append(cfg)
    assert outs == [1, 3]


@pytest.fixture(params=[1, 0], ids=["relax", "sweep"])
def ms_path(request):
    """K = 1 makespans by the relaxation over cross-device edges (falling back
    to the level sweep when it does not converge) or by the level sweep."""
    was = cel.makespan_relax(request.param)
    yield request.param
    cel.makespan_relax(was)


def random_placements(wl, K, seed):
    rng = np.random.default_rng([77, seed])
    return rng.integers(0, wl.D, (K, wl.n)).astype(np.uint8)


@pytest.mark.parametrize("cfg,seed", [(1, 0), (2, 0), (3, 1), (5, 0)])
def test_makespan_configs(cfg, seed, ms_path):
    wl, rt, rb = config(cfg, seed)
    lev, oid, lp, L = rt
    pr = rb[2]
    # the oracle's own placement plus random ones
    cid, C, _ = O.cluster(wl, pr, 200, -1)
    _, ndev, _, _ = O.place(wl, cid, C)
    P = np.concatenate([ndev[None, :], random_placements(wl, 5, seed)])
    ref_ms, ref_st, ref_fi = O.makespan(wl, pr, P)
    g, d = up(wl)
    args = (tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L)
    ms, st, fi = cel.makespan(g, d, *args, tt(P, np.uint8), want_times=True)  # batched
    assert np.array_equal(np_(ms), ref_ms)
    assert np.array_equal(np_(st), ref_st) and np.array_equal(np_(fi), ref_fi)
    for k in (0, 3):  # single placement path
        ms1, st1, fi1 = cel.makespan(g, d, *args, tt(P[k], np.uint8), want_times=True)
        assert np_(ms1)[0] == ref_ms[k]
        assert np.array_equal(np_(fi1)[0], ref_fi[k])


def test_makespan_large_batches():
    """Batches larger than the CU count take the small-window kernel: every row
    of a 400-placement batch on config 1, and sampled rows of the 1,024 perturbed
    placements of config 5 (the batched-scoring workload)."""
    wl, rt, rb = config(1, 1)
    lev, oid, lp, L = rt
    pr = rb[2]
    P = random_placements(wl, 400, 7)
    ref_ms, _, ref_fi = O.makespan(wl, pr, P)
    g, d = up(wl)
    args = (tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L)
    ms, st, fi = cel.makespan(g, d, *args, tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), ref_ms) and np.array_equal(np_(fi), ref_fi)

    wl5 = make_config(5, 0)
    lev5, oid5, lp5, L5 = O.topo_levels(wl5)
    _, _, pr5, _ = O.blevel(wl5, lev5, oid5)
    cid5, C5, _ = O.cluster(wl5, pr5, 200, -1)
    cdev5, _, _, _ = O.place(wl5, cid5, C5)
    P5 = perturb_placements(cdev5, wl5.D, 1024, 0)[:, cid5]
    g5, d5 = up(wl5)
    ms5, st5, fi5 = cel.makespan(g5, d5, tt(pr5, np.int32), tt(lev5, np.int32),
                                 tt(lp5, np.int32), L5, tt(P5, np.uint8), want_times=True)
    ms5 = np_(ms5)
    # every one of the 1,024 makespans (the oracle's rows are independent, so
    # slices of them run on host threads: ctypes releases the GIL)
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(8) as ex:
        parts = list(ex.map(lambda a: O.makespan(wl5, pr5, P5[a:a + 64], want_times=False)[0],
                            range(0, 1024, 64)))
    assert np.array_equal(ms5, np.concatenate(parts))
    # full start and finish arrays of rows spread over the batch
    rows = [0, 1, 255, 256, 511, 777, 1022, 1023]
    _, ref_st, ref_fi = O.makespan(wl5, pr5, P5[rows])
    ridx = torch.tensor(rows, device=DEV)
    assert np.array_equal(np_(fi5.index_select(0, ridx)), ref_fi)
    assert np.array_equal(np_(st5.index_select(0, ridx)), ref_st)


def _all_placements(n, D):
    """Every device assignment of n nodes to D devices, [D**n, n] uint8 (row k
    reads k in base D, node 0 the most significant digit)."""
    k = np.arange(D ** n, dtype=np.int64)
    digits = [(k // D ** (n - 1 - i)) % D for i in range(n)]
    return np.stack(digits, axis=1).astype(np.uint8)


@pytest.mark.parametrize("n,D,seed", [(10, 4, 0), (10, 2, 1), (9, 3, 2), (8, 4, 3), (6, 5, 4),
                                      (1, 4, 5)])
def test_makespan_brute_force_batch(n, D, seed):
    """Every one of the D^n placements of a DAG of at most 10 nodes in ONE
    batched call (up to 4^10 = 1,048,576 rows), row by row against the oracle;
    the optimum over all placements lies between the lower bound max(CP0,
    ceil(sum w / D)) and the makespan of Adjusting Placement's placement."""
    wl = make_random_dag(950 + seed, n, p_edge=0.35, D=D, cap_frac=(1, 1),
                         multi=(seed % 2 == 0))
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
    P = _all_placements(n, D)
    K = P.shape[0]
    ref, _, _ = O.makespan(wl, pr, P, want_times=False)
    g, d = up(wl)
    ms, _, fi = cel.makespan(g, d, tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                             tt(P, np.uint8), want_times=(K <= 4096))
    got = np_(ms)
    assert got.shape == (K,) and np.array_equal(got, ref)
    if fi is not None:
        assert np.array_equal(np_(fi), O.makespan(wl, pr, P)[2])
    opt = int(got.min())
    _, _, _, cp0 = O.blevel(wl, lev, oid, comm_off=True, want_tlevel=False)
    assert opt >= max(int(cp0), -(-int(wl.w.sum()) // D))
    cid = np.empty(n, np.int32)
    cid[pr] = np.arange(n)  # every node its own cluster, in priority order
    _, ndev, _, _ = cel.place(g, d, tt(cid, np.int32), n)
    ms_p, _, _ = cel.makespan(g, d, tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L, ndev)
    assert opt <= int(np_(ms_p)[0])
    # the row of Adjusting Placement's devices is that same value
    row = int(sum(int(x) * D ** (n - 1 - i) for i, x in enumerate(np_(ndev))))
    assert got[row] == int(np_(ms_p)[0])


def _wide_layered(seed, widths, max_fanin, D):
    """Layered DAG with the given level widths; each node draws 1..max_fanin
    parents (with repeats: multi-edges) from the previous level."""
    rng = np.random.default_rng([91, seed])
    starts = np.concatenate([[0], np.cumsum(widths)])
    n = int(starts[-1])
    edges = []
    for li in range(1, len(widths)):
        for v in range(int(starts[li]), int(starts[li + 1])):
            k = int(rng.integers(1, max_fanin + 1))
            for u in rng.integers(starts[li - 1], starts[li], k):
                edges.append((int(u), v))
    w = rng.integers(1, 5000, n)
    ob = rng.integers(0, 1 << 20, n)
    return from_edges(n, edges, w, ob, D, np.full(D, 1 << 40), 7, 300, name="wide-layered")


@pytest.mark.parametrize("widths,fanin,D,K", [
    ([700, 1300, 900], 10, 200, 3),     # passes of 512 nodes, tail in-edges, 8-bit devices
    ([700, 1300, 900], 10, 12, 3),      # the LDS-ring kernel (D <= 16) with in-edges past three
    ([257, 513, 1025, 300], 3, 16, 5),  # ragged chunks
    ([600, 600], 1, 1, 2),              # one device
])
def test_makespan_wide_levels_batch(widths, fanin, D, K):
    """Batches on graphs with wide levels run without LDS windows."""
    wl = _wide_layered(len(widths) * 100 + fanin, widths, fanin, D)
    lev, oid, lp, L = O.topo_levels(wl)
    assert wl.n >= 256 * L  # the window-free kernel's regime
    _, _, pr, _ = O.blevel(wl, lev, oid)
    P = random_placements(wl, K, D)
    ref_ms, ref_st, ref_fi = O.makespan(wl, pr, P)
    g, d = up(wl)
    ms, st, fi = cel.makespan(g, d, tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                              tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), ref_ms)
    assert np.array_equal(np_(st), ref_st) and np.array_equal(np_(fi), ref_fi)


def test_makespan_one_run_boundaries(ms_path):
    """K = 1: the device runs of a level (consecutive slots of the
    device-grouped order) start at lane 0 of a row, inside a row, exactly at
    the second row's lane 0 and in later rows, or a level sits on one device
    and its run spans up to four rows; predecessors are near (the previous
    levels) and far (more than 2,048 slots back)."""
    rng = np.random.default_rng(17)
    # per level, the sizes of its device runs (device ids ascending)
    runs = [[64, 64], [1, 127], [127, 1], [128], [63, 65], [65, 63], [200], [64, 64, 64],
            [30, 34, 64, 2], [256], [17], [64], [129], [1, 1, 1, 61, 64], [192, 64]]
    runs = runs * 6
    widths = [sum(r) for r in runs]
    starts = np.concatenate([[0], np.cumsum(widths)])
    n = int(starts[-1])
    D = 6
    dev = np.zeros(n, np.int64)
    edges = []
    for li, rs in enumerate(runs):
        devs = np.sort(rng.choice(D, len(rs), replace=False))
        s0 = int(starts[li])
        for d_, k in zip(devs, rs):
            dev[s0:s0 + k] = d_
            s0 += k
        if li == 0:
            continue
        for v in range(int(starts[li]), int(starts[li + 1])):
            edges.append((int(rng.integers(starts[li - 1], starts[li])), v))
            for u in rng.integers(0, starts[li], int(rng.integers(0, 4))):
                edges.append((int(u), v))
    edges = sorted(set(edges))
    wl = from_edges(n, edges, rng.integers(1, 5000, n), rng.integers(0, 1 << 20, n), D,
                    np.full(D, 1 << 40), 7, 300, name="run-boundaries")
    lev, oid, lp, L = O.topo_levels(wl)
    assert L == len(runs)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    # the placement puts each level's runs where the sizes say, whatever the
    # priority order inside the level
    P = np.zeros((1, n), np.uint8)
    for li in range(L):
        nodes = np.asarray(pr[lp[li]:lp[li + 1]])
        P[0, nodes] = np.sort(dev[starts[li]:starts[li + 1]])
    ref_ms, ref_st, ref_fi = O.makespan(wl, pr, P)
    g, d = up(wl)
    ms, st, fi = cel.makespan(g, d, tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                              tt(P[0], np.uint8), want_times=True)
    assert np_(ms)[0] == ref_ms[0]
    assert np.array_equal(np_(st)[0], ref_st[0]) and np.array_equal(np_(fi)[0], ref_fi[0])


def test_makespan_batch_level_paths():
    """K > 1 over the priority order: the run-boundary DAG under four
    placements at once: the levels' device runs as sized (several devices per
    row), everything on one device (one-device levels of up to four rows),
    one device per level (chains continue through free times across
    levels), and uniform random devices."""
    rng = np.random.default_rng(23)
    runs = [[64, 64], [1, 127], [127, 1], [128], [63, 65], [65, 63], [200], [64, 64, 64],
            [30, 34, 64, 2], [256], [17], [64], [129], [1, 1, 1, 61, 64], [192, 64]] * 4
    widths = [sum(r) for r in runs]
    starts = np.concatenate([[0], np.cumsum(widths)])
    n = int(starts[-1])
    D = 6
    edges = []
    for li in range(1, len(runs)):
        for v in range(int(starts[li]), int(starts[li + 1])):
            edges.append((int(rng.integers(starts[li - 1], starts[li])), v))
            for u in rng.integers(0, starts[li], int(rng.integers(0, 4))):
                edges.append((int(u), v))
    edges = sorted(set(edges))
    wl = from_edges(n, edges, rng.integers(1, 5000, n), rng.integers(0, 1 << 20, n), D,
                    np.full(D, 1 << 40), 7, 300, name="batch-paths")
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    P = np.zeros((4, n), np.uint8)
    for li in range(L):
        nodes = np.asarray(pr[lp[li]:lp[li + 1]])
        devs = np.sort(rng.choice(D, len(runs[li]), replace=False))
        P[0, nodes] = np.repeat(devs, runs[li])  # sized runs, in priority order
        P[2, nodes] = li % D
    P[1, :] = 3
    P[3] = rng.integers(0, D, n)
    ref_ms, ref_st, ref_fi = O.makespan(wl, pr, P)
    g, d = up(wl)
    ms, st, fi = cel.makespan(g, d, tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                              tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), ref_ms)
    assert np.array_equal(np_(st), ref_st) and np.array_equal(np_(fi), ref_fi)


def test_makespan_wide_far_predecessors_batch():
    """Wide levels whose nodes take up to 7 parents from the previous four
    levels of 3,000: predecessors more than 8,192 positions back (read from the
    placement's finish times in global memory, ahead or one by one past the
    third in-edge) beside near ones (from the LDS ring), D = 9, 70 placements
    (the LDS-staged device gather as well)."""
    rng = np.random.default_rng(44)
    widths = [3000] * 7
    starts = np.concatenate([[0], np.cumsum(widths)])
    n = int(starts[-1])
    edges = []
    for li in range(1, len(widths)):
        lo = int(starts[max(0, li - 4)])
        for v in range(int(starts[li]), int(starts[li + 1])):
            k = int(rng.integers(1, 8))
            ps = {int(rng.integers(starts[li - 1], starts[li]))}  # one parent in the level below
            ps.update(int(u) for u in rng.integers(lo, starts[li], k - 1))
            edges += [(u, v) for u in sorted(ps)]
    wl = from_edges(n, edges, rng.integers(1, 5000, n), rng.integers(0, 1 << 20, n), 9,
                    np.full(9, 1 << 40), 7, 300, name="wide-far")
    lev, oid, lp, L = O.topo_levels(wl)
    assert wl.n >= 256 * L
    _, _, pr, _ = O.blevel(wl, lev, oid)
    P = random_placements(wl, 70, 9)
    ref_ms, ref_st, ref_fi = O.makespan(wl, pr, P)
    g, d = up(wl)
    ms, st, fi = cel.makespan(g, d, tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                              tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), ref_ms)
    assert np.array_equal(np_(st), ref_st) and np.array_equal(np_(fi), ref_fi)


def test_makespan_wide_no_edges_batch():
    """Sources only: one level of 3,000 isolated nodes, 4 placements."""
    n, D = 3000, 5
    rng = np.random.default_rng(5)
    wl = from_edges(n, [], rng.integers(1, 100, n), rng.integers(0, 1000, n), D,
                    np.full(D, 1 << 40), 3, 10)
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    P = random_placements(wl, 4, 1)
    ref_ms, _, ref_fi = O.makespan(wl, pr, P)
    g, d = up(wl)
    ms, _, fi = cel.makespan(g, d, tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                             tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), ref_ms) and np.array_equal(np_(fi), ref_fi)
    P[2, 1234] = D  # a device id out of range is rejected on this path too
    with pytest.raises(cel.CelError):
        cel.makespan(g, d, tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                     tt(P, np.uint8))


def test_makespan_batch_rows_gather():
    """Batches of 64 and more placements stage each placement's devices in LDS
    before ordering them by position: 80 rows of a 3,000-node DAG (more nodes
    than one staging pass on a second graph of 140,000 isolated nodes; node
    counts that are and are not multiples of 4), and a device id out of range
    is rejected there too."""
    wl = make_random_dag(77, 3001, p_edge=0.002, D=6)
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    P = random_placements(wl, 80, 3)
    ref_ms, _, ref_fi = O.makespan(wl, pr, P)
    g, d = up(wl)
    args = (tt(pr, np.int32), tt(lev, np.int32), tt(lp, np.int32), L)
    ms, _, fi = cel.makespan(g, d, *args, tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), ref_ms) and np.array_equal(np_(fi), ref_fi)
    P[77, 2999] = 6
    with pytest.raises(cel.CelError):
        cel.makespan(g, d, *args, tt(P, np.uint8))
    n, D = 140000, 3
    rng = np.random.default_rng(8)
    wl2 = from_edges(n, [], rng.integers(1, 100, n), rng.integers(0, 1000, n), D,
                     np.full(D, 1 << 40), 3, 10)
    lev2, oid2, lp2, L2 = O.topo_levels(wl2)
    _, _, pr2, _ = O.blevel(wl2, lev2, oid2)
    P2 = random_placements(wl2, 64, 4)
    ref2, _, _ = O.makespan(wl2, pr2, P2, want_times=False)
    g2, d2 = up(wl2)
    ms2, _, _ = cel.makespan(g2, d2, tt(pr2, np.int32), tt(lev2, np.int32), tt(lp2, np.int32),
                             L2, tt(P2, np.uint8))
    assert np.array_equal(np_(ms2), ref2)
    P2[63, 139999] = 200
    with pytest.raises(cel.CelError):
        cel.makespan(g2, d2, tt(pr2, np.int32), tt(lev2, np.int32), tt(lp2, np.int32), L2,
                     tt(P2, np.uint8))


# ---------------------------------------------------------- random small DAGs


def test_random_dags(ms_path, bl_path):
    for s in range(40):
        n = 1 + (s * 37) % 300
        wl = make_random_dag(1000 + s, n, p_edge=min(0.5, 4.0 / max(n, 1)), D=1 + s % 7,
                             multi=(s % 3 == 0), zero_frac=0.2 if s % 5 == 0 else 0.0)
        rt = O.topo_levels(wl)
        rb = O.blevel(wl, rt[0], rt[1])
        g, d, gt, gb = run_topo_blevel(wl)
        assert_topo_blevel(wl, rt, rb, gt, gb)
        P = random_placements(wl, 3, s)
        ref = O.makespan(wl, rb[2], P)
        ms, st, fi = cel.makespan(g, d, gb[2], gt[0], gt[2], gt[3], tt(P, np.uint8),
                                  want_times=True)
        assert np.array_equal(np_(ms), ref[0]) and np.array_equal(np_(fi), ref[2])
        ms1, st1, fi1 = cel.makespan(g, d, gb[2], gt[0], gt[2], gt[3], tt(P[s % 3], np.uint8),
                                     want_times=True)
        assert np_(ms1)[0] == ref[0][s % 3]
        assert np.array_equal(np_(fi1)[0], ref[2][s % 3])
        assert np.array_equal(np_(st1)[0], ref[1][s % 3])


def test_wide_levels_and_many_devices(ms_path):
    """Levels wider than a workgroup (ragged chunks) and D = 255."""
    rng = np.random.default_rng(5)
    n0, n1 = 3000, 2500
    edges = [(int(rng.integers(0, n0)), n0 + j) for j in range(n1)]
    edges += [(int(rng.integers(0, n0)), n0 + j) for j in range(0, n1, 3)]
    n = n0 + n1
    wl = from_edges(n, edges, rng.integers(0, 100, n), rng.integers(0, 5000, n), 255,
                    [10 ** 12] * 255, 3, 7)
    rt = O.topo_levels(wl)
    rb = O.blevel(wl, rt[0], rt[1])
    g, d, gt, gb = run_topo_blevel(wl)
    assert_topo_blevel(wl, rt, rb, gt, gb)
    P = rng.integers(0, 255, (2, n)).astype(np.uint8)
    ref = O.makespan(wl, rb[2], P)
    ms, _, fi = cel.makespan(g, d, gb[2], gt[0], gt[2], gt[3], tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), ref[0]) and np.array_equal(np_(fi), ref[2])
    ms1, _, fi1 = cel.makespan(g, d, gb[2], gt[0], gt[2], gt[3], tt(P[1], np.uint8),
                               want_times=True)
    assert np_(ms1)[0] == ref[0][1] and np.array_equal(np_(fi1)[0], ref[2][1])


def test_heavy_fanout_node():
    """One node with thousands of successors and one with thousands of predecessors."""
    n = 6000
    edges = [(0, j) for j in range(1, 4000)] + [(j, 5999) for j in range(4000, 5999)]
    edges += [(j, 4000 + (j % 1999)) for j in range(1, 4000)]
    rng = np.random.default_rng(9)
    wl = from_edges(n, edges, rng.integers(1, 50, n), rng.integers(0, 900, n), 3,
                    [10 ** 12] * 3, 4, 2)
    rt = O.topo_levels(wl)
    rb = O.blevel(wl, rt[0], rt[1])
    g, d, gt, gb = run_topo_blevel(wl)
    assert_topo_blevel(wl, rt, rb, gt, gb)


def test_heavy_window_nodes(ms_path, bl_path):
    """Nodes with more neighbours than a sweep window holds edges: a source with
    9,999 successors (b-level), a sink with 10,000 predecessors (t-level and
    makespan), both between ordinary levels, for every sweep and both
    makespan paths."""
    n = 24000
    rng = np.random.default_rng(13)
    edges = [(0, j) for j in range(1, 10000)]
    edges += [(j, 23999) for j in range(10000, 20000)]
    edges += [(j, 10000 + int(rng.integers(0, 10000))) for j in range(1, 10000)]
    edges += [(20000 + (j % 3999), 20001 + (j % 3998)) for j in range(0, 3998)]
    edges += [(j, 20000 + int(rng.integers(0, 3999))) for j in range(10000, 20000, 7)]
    edges = sorted(set((u, v) for u, v in edges if u < v))
    wl = from_edges(n, edges, rng.integers(1, 50, n), rng.integers(0, 900, n), 5,
                    [10 ** 12] * 5, 4, 2)
    rt = O.topo_levels(wl)
    rb = O.blevel(wl, rt[0], rt[1])
    g, d, gt, gb = run_topo_blevel(wl)
    assert_topo_blevel(wl, rt, rb, gt, gb)
    lev, oid, lp, L = rt
    P = random_placements(wl, 3, 5)
    ref_ms, _, ref_fi = O.makespan(wl, rb[2], P)
    args = (tt(rb[2], np.int32), tt(lev, np.int32), tt(lp, np.int32), L)
    ms, _, fi = cel.makespan(g, d, *args, tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), ref_ms) and np.array_equal(np_(fi), ref_fi)
    ms1, _, fi1 = cel.makespan(g, d, *args, tt(P[1], np.uint8), want_times=True)
    assert np_(ms1)[0] == ref_ms[1] and np.array_equal(np_(fi1)[0], ref_fi[1])


def test_sweep_many_near_neighbours(bl_path):
    """Narrow levels (1..150 nodes) where about one node in 20 has 9..300
    successors or predecessors within the next few levels: the b-level and
    t-level sweeps gather those along slot lists instead of pull records, and
    rows mixing such nodes with ordinary ones, or ending mid-row, take every
    gather width."""
    rng = np.random.default_rng(21)
    widths = [int(x) for x in rng.integers(1, 151, 120)]
    starts = np.concatenate([[0], np.cumsum(widths)])
    n = int(starts[-1])
    edges = set()
    for li in range(len(widths) - 1):
        for v in range(int(starts[li]), int(starts[li + 1])):
            hi = int(starts[min(li + 4, len(widths))])
            lo = int(starts[li + 1])
            k = int(rng.integers(1, 4))
            if rng.random() < 0.05:
                k = int(rng.integers(9, 301))
            for u in rng.integers(lo, hi, k):
                edges.add((v, int(u)))
        # a node of the next level with many predecessors
        if rng.random() < 0.3:
            t = int(rng.integers(starts[li + 1], starts[li + 2]))
            lo = int(starts[max(0, li - 3)])
            for u in rng.integers(lo, int(starts[li + 1]), int(rng.integers(9, 301))):
                edges.add((int(u), t))
    # every node but the first level's keeps its level: one edge from the level below
    for li in range(1, len(widths)):
        for v in range(int(starts[li]), int(starts[li + 1])):
            edges.add((int(rng.integers(starts[li - 1], starts[li])), v))
    edges = sorted(edges)
    wl = from_edges(n, edges, rng.integers(1, 50, n), rng.integers(0, 900, n), 4,
                    [10 ** 12] * 4, 4, 2)
    rt = O.topo_levels(wl)
    assert rt[3] == len(widths)
    rb = O.blevel(wl, rt[0], rt[1])
    g, d, gt, gb = run_topo_blevel(wl)
    assert_topo_blevel(wl, rt, rb, gt, gb)


def _grid_level_dag(seed):
    """Levels of widths 20000 (sources), 50, 30, 40, 10 (hubs), 60, 12000, 80,
    2000, 5 (collectors), 70, 30, 20000: one source has 24,375 successors (every
    node of the levels between and half the sinks), each hub 3,000..9,000
    successors in the next four levels, each collector 5,000 predecessors
    below it."""
    rng = np.random.default_rng(seed)
    widths = [20000, 50, 30, 40, 10, 60, 12000, 80, 2000, 5, 70, 30, 20000]
    starts = np.concatenate([[0], np.cumsum(widths)]).astype(np.int64)
    n = int(starts[-1])
    nl = len(widths)
    src, dst = [], []

    def add(u, v):
        src.append(np.asarray(u, np.int64).ravel())
        dst.append(np.asarray(v, np.int64).ravel())

    for li in range(1, nl):
        v = np.arange(starts[li], starts[li + 1])
        add(rng.integers(starts[li - 1], starts[li], v.size), v)
    for li in range(nl - 1):
        u = np.arange(starts[li], starts[li + 1])
        k = rng.integers(1, 4, u.size)
        uu = np.repeat(u, k)
        add(uu, rng.integers(starts[li + 1], starts[min(li + 4, nl)], uu.size))
    add(np.zeros(n - widths[0] - widths[-1] + widths[-1] // 2, np.int64),
        np.concatenate([np.arange(starts[1], starts[nl - 1]),
                        np.arange(starts[nl - 1], starts[nl - 1] + widths[-1] // 2)]))
    for h in range(starts[4], starts[5]):
        t = rng.choice(np.arange(starts[5], starts[9]), int(rng.integers(3000, 9001)), replace=False)
        add(np.full(t.size, h), t)
    for c in range(starts[9], starts[10]):
        u = rng.choice(np.arange(0, starts[9]), 5000, replace=False)
        add(u, np.full(u.size, c))
    e = np.unique(np.stack([np.concatenate(src), np.concatenate(dst)], 1), axis=0)
    edges = [(int(a), int(b)) for a, b in e]
    wl = from_edges(n, edges, rng.integers(1, 50, n), rng.integers(0, 900, n), 4,
                    [10 ** 12] * 4, 4, 2)
    return wl, nl


def test_sweep_grid_levels(bl_path):
    """Levels of at least 16,384 nodes or edges run on the whole GPU between
    single-workgroup segments, in both sweep directions; rows of more than 64
    neighbours there are split over workgroups (the 24,375-successor source in
    6 chunks of 4,096 edges)."""
    wl, nl = _grid_level_dag(31)
    rt = O.topo_levels(wl)
    assert rt[3] == nl
    rb = O.blevel(wl, rt[0], rt[1])
    g, d, gt, gb = run_topo_blevel(wl)
    assert_topo_blevel(wl, rt, rb, gt, gb)
    # again without the t-level (the b-level alone on the caller's stream)
    bl, tl, pr, cp = cel.blevel(g, d, gt[0], gt[2], gt[1], gt[3], want_tlevel=False)
    assert tl is None and cp == rb[3] and np.array_equal(np_(bl), rb[0])


# -------------------------------------------------------------- edge cases


def test_empty_and_single(ms_path):
    wl = from_edges(0, [], [], [], 2, [5, 5], 3, 1)
    g, d = up(wl)
    lev, oid, lp, L = cel.topo_levels(g)
    assert L == 0 and np_(lp).tolist() == [0]
    bl, _, pr, cp = cel.blevel(g, d, lev, lp, oid, L)
    assert cp == 0
    ms, _, _ = cel.makespan(g, d, pr, lev, lp, L, torch.zeros((3, 0), dtype=torch.uint8,
                                                                 device=DEV))
    assert np_(ms).tolist() == [0, 0, 0]
    wl = from_edges(1, [], [7], [100], 2, [5, 5], 3, 1)
    g, d = up(wl)
    lev, oid, lp, L = cel.topo_levels(g)
    bl, tl, pr, cp = cel.blevel(g, d, lev, lp, oid, L, want_tlevel=True)
    assert L == 1 and cp == 7 and np_(tl).tolist() == [0]
    ms, st, fi = cel.makespan(g, d, pr, lev, lp, L, torch.ones(1, dtype=torch.uint8, device=DEV),
                              want_times=True)
    assert np_(ms).tolist() == [7] and np_(fi).tolist() == [[7]]


@pytest.mark.parametrize("edges", [[(0, 0)], [(0, 1), (1, 2), (2, 0)], [(0, 1), (1, 2), (2, 1), (0, 3)]])
def test_cycle_detected(edges):
    n = 1 + max(max(e) for e in edges)
    wl = from_edges(n, edges, [1] * n, [1] * n, 1, [1], 1, 0)
    g, _ = up(wl)
    with pytest.raises(cel.CelError) as ei:
        cel.topo_levels(g)
    assert ei.value.code == -2


def test_bad_inputs_rejected():
    wl, rt, rb = config(1, 0)
    lev, oid, lp, L = rt
    g, d = up(wl)
    bad = oid.copy(); bad[[3, 700]] = bad[[700, 3]]  # breaks level-monotonicity
    with pytest.raises(cel.CelError) as ei:
        cel.blevel(g, d, tt(lev, np.int32), tt(lp, np.int32), tt(bad, np.int32), L)
    assert ei.value.code == -6
    dup = rb[2].copy(); dup[5] = dup[6]
    with pytest.raises(cel.CelError) as ei:
        cel.makespan(g, d, tt(dup, np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                     torch.zeros(wl.n, dtype=torch.uint8, device=DEV))
    assert ei.value.code == -6
    with pytest.raises(cel.CelError) as ei:  # device id >= D
        cel.makespan(g, d, tt(rb[2], np.int32), tt(lev, np.int32), tt(lp, np.int32), L,
                     torch.full((wl.n,), wl.D, dtype=torch.uint8, device=DEV))
    assert ei.value.code == -1
    wl2 = from_edges(2, [(0, 1)], [5, 6], [2 ** 62 - 10, 0], 1, [1], 1, 0, mem=[1, 1])
    g2, d2 = up(wl2)
    lev2, oid2, lp2, L2 = cel.topo_levels(g2)
    with pytest.raises(cel.CelError) as ei:
        cel.blevel(g2, d2, lev2, lp2, oid2, L2)
    assert ei.value.code == -3
    wl3 = from_edges(3, [(0, 1), (1, 2)], [1, 1, 1], [1, 1, 1], 1, [1], 1, 0)
    wl3.in_idx = wl3.in_idx.copy(); wl3.in_idx[0] = 2  # CSC disagrees with CSR
    g3, _ = up(wl3)
    with pytest.raises(cel.CelError):
        cel.topo_levels(g3)


def test_deterministic_repeat():
    wl, rt, rb = config(3, 0)
    g, d, gt1, gb1 = run_topo_blevel(wl)
    _, _, gt2, gb2 = run_topo_blevel(wl)
    for a, b in zip(gt1[:3] + gb1[:3], gt2[:3] + gb2[:3]):
        assert torch.equal(a, b)


# ------------------------------------------------------------ clustering


def gpu_cluster(wl, order, R, M, mode):
    g, d = up(wl)
    cid, C, cut = cel.cluster(g, d, tt(order, np.int32), R, M, mode)
    return np_(cid), C, cut


@pytest.mark.parametrize("cfg,seed", [(1, 0), (2, 0), (3, 0), (5, 1)])
@pytest.mark.parametrize("mode", [0, 1])
def test_cluster_configs(cfg, seed, mode, bl_path):
    wl, rt, rb = config(cfg, seed)
    pr = rb[2]
    for R, M in ((200, -1), (37, -1), (300, int(wl.cap.min()) // 9)):
        ref = O.cluster(wl, pr, R, M, mode)
        cid, C, cut = gpu_cluster(wl, pr, R, M, mode)
        assert C == ref[1] and cut == ref[2], (R, M)
        assert np.array_equal(cid, ref[0]), (R, M)


def test_cluster_window_sizes_and_orders():
    rng = np.random.default_rng(21)
    for s in range(24):
        n = 2 + (s * 53) % 700
        wl = make_random_dag(2000 + s, n, p_edge=min(0.6, 5.0 / n), D=3, multi=(s % 4 == 1),
                             zero_frac=0.15 if s % 3 == 0 else 0.0)
        lev, oid, _, _ = O.topo_levels(wl)
        # a random topological order (not level-monotone): random priorities + Kahn
        order = random_topo_order(wl, rng)
        R = [1, 2, 63, 64, 65, 129, 200, 257, 700, 1500, 4096][s % 11]
        M = [-1, 0, int(wl.mem.sum()) // 5, 10 ** 15][s % 4]
        for mode in (0, 1):
            ref = O.cluster(wl, order, R, M, mode)
            got = gpu_cluster(wl, order, R, M, mode)
            assert got[1] == ref[1] and got[2] == ref[2] and np.array_equal(got[0], ref[0]), \
                (s, R, M, mode)


def _cluster_with_kernels(wl, order, R, M):
    """GPU clustering plus the names of the DP kernels it launched."""
    cel.timing(True)
    cel.kernel_stats(reset=True)
    try:
        got = gpu_cluster(wl, order, R, M, 0)
        ks = cel.kernel_stats(reset=True)
    finally:
        cel.timing(False)
    return got, {k for k in ks if k.startswith("k_cluster_dp")}


# (seed, n, p_edge, max fan-in, R, M, DP kernel): dense local structure on both
# sides of the blocked kernel's staging size (1024 window edges per block of 64
# targets): many edges per candidate and inside one block, several edge
# batches, the prefetch remainder (R <= 64: one candidate wave), and blocks too
# dense for staging (taken target by target inside the blocked kernel).
DENSE_CASES = [
    (4, 600, 0.12, 20, 130, -1, "k_cluster_dp"),
    (6, 2000, 0.02, 30, 1000, -1, "k_cluster_dp"),
    (7, 800, 0.1, 12, 60, -1, "k_cluster_dp"),
    (6, 2000, 0.02, 30, 1000, 10 ** 15, "k_cluster_dp"),
    (1, 400, 0.5, 400, 200, -1, "k_cluster_dp"),
    (8, 800, 0.2, 16, 40, -1, "k_cluster_dp"),
    (10, 1000, 0.3, 10, 30, -1, "k_cluster_dp"),
]


@pytest.mark.parametrize("case", DENSE_CASES, ids=[f"s{c[0]}-R{c[4]}-{c[6]}" for c in DENSE_CASES])
def test_cluster_dense_blocks(case):
    seed, n, p, fan, R, M, kern = case
    wl = make_random_dag(seed, n, p, D=3, max_fanin=fan)
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    for k, order in enumerate((pr, random_topo_order(wl, np.random.default_rng(seed)))):
        ref = O.cluster(wl, order, R, M)
        got, used = _cluster_with_kernels(wl, order, R, M)
        assert got[1] == ref[1] and got[2] == ref[2] and np.array_equal(got[0], ref[0]), k
        if k == 0:  # the priority order is the one the case was sized on
            assert used == {kern}


@pytest.mark.parametrize("seed", range(6))
def test_cluster_memory_bound_windows(seed):
    """Memory caps that end windows inside a block of 64 targets: targets of one
    block see different first candidates (some none below the block)."""
    n = 400 + 230 * seed
    wl = make_random_dag(4000 + seed, n, min(0.5, 5.0 / n), D=3, multi=seed % 2 == 1)
    lev, oid, _, _ = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    avg = int(wl.mem.sum()) // n
    for width in (20, 45, 70, 120):
        for R in (64, 200):
            M = avg * width
            ref = O.cluster(wl, pr, R, M)
            got, used = _cluster_with_kernels(wl, pr, R, M)
            assert got[1] == ref[1] and got[2] == ref[2] and np.array_equal(got[0], ref[0]), \
                (width, R)
            assert used == {"k_cluster_dp"}


def test_cluster_huge_comm_takes_step_kernel():
    """Total comm at or above 2^46 ns: the step-wise kernel, same results."""
    for seed, n in ((11, 300), (12, 90)):
        wl = make_random_dag(seed, n, min(0.5, 6.0 / n), D=3, ob_max=1 << 45, bw=1, lat=5)
        lev, oid, _, _ = O.topo_levels(wl)
        _, _, pr, _ = O.blevel(wl, lev, oid)
        for R in (200, 17):
            ref = O.cluster(wl, pr, R, -1)
            got, used = _cluster_with_kernels(wl, pr, R, -1)
            assert got[1] == ref[1] and got[2] == ref[2] and np.array_equal(got[0], ref[0])
            assert used == {"k_cluster_dp_step"}


def random_topo_order(wl, rng):
    import heapq
    indeg = np.diff(wl.in_ptr).copy()
    key = rng.random(wl.n)
    heap = [(key[v], v) for v in range(wl.n) if indeg[v] == 0]
    heapq.heapify(heap)
    out = []
    while heap:
        _, u = heapq.heappop(heap)
        out.append(u)
        for v in wl.out_idx[wl.out_ptr[u]:wl.out_ptr[u + 1]]:
            indeg[v] -= 1
            if indeg[v] == 0:
                heapq.heappush(heap, (key[v], v))
    return np.array(out, np.int32)


def test_cluster_rejects_non_topological_order():
    wl, rt, rb = config(1, 0)
    bad = rb[2][::-1].copy()
    g, d = up(wl)
    with pytest.raises(cel.CelError) as ei:
        cel.cluster(g, d, tt(bad, np.int32), 200, -1)
    assert ei.value.code == -6
    with pytest.raises(cel.CelError) as ei:
        cel.cluster(g, d, tt(rb[2], np.int32), 0, -1)
    assert ei.value.code == -1


# ------------------------------------------------------------- placement


def check_place(wl, cid, C):
    ref = O.place(wl, cid, C, want_fin=True)
    g, d = up(wl)
    cdev, ndev, span, be, fin = cel.place(g, d, tt(cid, np.int32), C, want_fin=True)
    assert span == ref[2] and be == ref[3]
    assert np.array_equal(np_(cdev), ref[0])
    assert np.array_equal(np_(ndev), ref[1])
    assert np.array_equal(np_(fin), ref[4])


@pytest.mark.parametrize("cfg,seed", [(1, 0), (1, 1), (2, 0), (3, 0), (5, 0)])
def test_place_configs(cfg, seed):
    wl, rt, rb = config(cfg, seed)
    cid, C, _ = O.cluster(wl, rb[2], 200, -1)
    check_place(wl, cid, C)
    cid, C, _ = O.cluster(wl, rb[2], 40, -1, O.GREEDY)
    check_place(wl, cid, C)


def test_place_hand_fixtures():
    import json
    import os
    gold = os.path.join(os.path.dirname(__file__), "golden", "place_hand.json")
    for case in json.load(open(gold))["cases"]:
        n = case["n"]
        wl = from_edges(n, case["edges"], case["w"], case["ob"], case["D"], case["cap"],
                        case["bw"], case["lat"], mem=case["mem"])
        cid = np.array(case.get("cluster_id", range(n)), np.int32)
        g, d = up(wl)
        cdev, _, span, be, fin = cel.place(g, d, tt(cid, np.int32), int(cid.max()) + 1,
                                           want_fin=True)
        assert np_(cdev).tolist() == case["cluster_dev"], case["name"]
        assert np_(fin).tolist() == case["cluster_fin"] and span == case["coarse_makespan"]
        assert be == case["best_effort_count"]


def test_place_random():
    rng = np.random.default_rng(4)
    for s in range(30):
        n = 3 + (s * 41) % 400
        wl = make_random_dag(3000 + s, n, p_edge=min(0.5, 4.0 / n), D=1 + s % 9,
                             cap_frac=(1, 1 + s % 6), multi=(s % 3 == 0),
                             zero_frac=0.2 if s % 4 == 0 else 0.0)
        order = random_topo_order(wl, rng)
        R = int(rng.integers(1, 60))
        cid, C, _ = O.cluster(wl, order, R, -1, s % 2)
        check_place(wl, cid, C)


def test_place_many_clusters_and_devices():
    """More clusters than the placement keeps in LDS (config 3, R = 4: 14,429
    clusters), and 80 or 200 devices, where the busy lists outgrow their LDS
    share and the device choice takes the wave reductions."""
    wl, rt, rb = config(3, 0)
    cid, C, _ = O.cluster(wl, rb[2], 4, -1)
    assert C > 8192
    check_place(wl, cid, C)
    for D in (80, 200):
        wl2 = make_random_dag(77 + D, 3000, p_edge=4.0 / 3000, D=D, cap_frac=(1, 3))
        lev2, oid2, lp2, L2 = O.topo_levels(wl2)
        _, _, pr2, _ = O.blevel(wl2, lev2, oid2)
        cid2, C2, _ = O.cluster(wl2, pr2, 2, -1)
        check_place(wl2, cid2, C2)


def test_place_wide_fan_in():
    """Clusters with more than 64 and more than 128 coarse preds (the two-pass
    pred path), on several devices, with ties of Fin + cc across devices."""
    rng = np.random.default_rng(21)
    for s, (k, D) in enumerate(((70, 3), (150, 7), (300, 16), (129, 64))):
        n = k + 40
        edges = [(u, k) for u in range(k)]                    # node k: k preds
        edges += [(u, k + 1 + (u % 5)) for u in range(0, k, 2)]  # 5 nodes, k / 10 preds each
        edges += [(k + j, k + j + 1) for j in range(39)]
        w = rng.integers(0, 50, n)
        ob = rng.integers(0, 3, n) * 1000 if s % 2 else rng.integers(0, 5000, n)
        wl = from_edges(n, sorted(set(edges)), w, ob, D, [int(rng.integers(5, 20)) * 10 ** 4] * D,
                        7, 2, mem=rng.integers(1, 10 ** 4, n))
        cid = np.arange(n, dtype=np.int32)  # every node its own cluster
        check_place(wl, cid, n)


def test_place_cpd_transformer96():
    """Full size: the CPD-TOPO clustering of transformer-96 (6,284 clusters), the
    largest cluster counts whose finish times and devices stay in LDS."""
    wl = make_config(4, 0)
    cid, C, _ = O.cluster(wl, oracle_cpd(wl), 200, -1)
    assert 6144 < C <= 8192
    check_place(wl, cid, C)


def test_place_rejects_bad_clusters():
    wl, rt, rb = config(1, 0)
    cid, C, _ = O.cluster(wl, rb[2], 200, -1)
    g, d = up(wl)
    with pytest.raises(cel.CelError) as ei:  # id out of range
        cel.place(g, d, tt(np.full(wl.n, C, np.int32), np.int32), C)
    assert ei.value.code == -1
    rev = (C - 1 - cid).astype(np.int32)  # clusters in reverse topological order
    with pytest.raises(cel.CelError) as ei:
        cel.place(g, d, tt(rev, np.int32), C)
    assert ei.value.code == -6


# ----------------------------------------------- whole path at full size


@pytest.mark.parametrize("cfg", [4])
def test_full_path_large(cfg):
    """Every output of the whole path on the 1.07M-node transformer graph."""
    wl = make_config(cfg, 0)
    rt = O.topo_levels(wl)
    rb = O.blevel(wl, rt[0], rt[1])
    g, d, gt, gb = run_topo_blevel(wl)
    assert_topo_blevel(wl, rt, rb, gt, gb)
    assert [p for p, _ in cel.blevel_info()] == [0, 0]  # both by policy iteration
    assert cel.topo_levels_info()[0] == 0                # the levels too
    was = cel.policy_iteration(0)  # and by Kahn's kernel and the level sweeps
    try:
        gt0 = cel.topo_levels(g)
        assert cel.topo_levels_info() == (1, 0)
        gb0 = cel.blevel(g, d, gt0[0], gt0[2], gt0[1], gt0[3], want_tlevel=True)
        assert cel.blevel_info() == ((1, 0), (1, 0))
    finally:
        cel.policy_iteration(was)
    assert_topo_blevel(wl, rt, rb, gt0, gb0)
    rc = O.cluster(wl, rb[2], 200, -1)
    cid, C, cut = cel.cluster(g, d, gb[2], 200, -1)
    assert C == rc[1] and cut == rc[2] and np.array_equal(np_(cid), rc[0])
    rp = O.place(wl, rc[0], rc[1])
    cdev, ndev, span, be = cel.place(g, d, cid, C)
    assert span == rp[2] and be == rp[3] and np.array_equal(np_(ndev), rp[1])
    P = np.concatenate([rp[1][None, :], random_placements(wl, 3, 4)])
    rm = O.makespan(wl, rb[2], P)
    ms, st, fi = cel.makespan(g, d, gb[2], gt[0], gt[2], gt[3], tt(P, np.uint8), want_times=True)
    assert np.array_equal(np_(ms), rm[0]) and np.array_equal(np_(fi), rm[2])
    # the single-placement paths on Adjusting Placement's devices: every start
    # and finish time of the 1.07M nodes, element by element, by the
    # relaxation (which converges in a few rounds here) and by the level sweep
    for mode in (1, 0):
        was = cel.makespan_relax(mode)
        try:
            ms1, st1, fi1 = cel.makespan(g, d, gb[2], gt[0], gt[2], gt[3], ndev, want_times=True)
            path, rounds = cel.makespan_info()
        finally:
            cel.makespan_relax(was)
        assert (path, rounds > 0) == ((0, True) if mode else (1, False))
        assert np_(ms1)[0] == rm[0][0]
        assert np.array_equal(np_(fi1)[0], rm[2][0]) and np.array_equal(np_(st1)[0], rm[1][0])
    for k in (1, 3):  # random placements (the relaxation gives up on them: the sweep)
        msk, stk, fik = cel.makespan(g, d, gb[2], gt[0], gt[2], gt[3], tt(P[k], np.uint8),
                                     want_times=True)
        assert np_(msk)[0] == rm[0][k]
        assert np.array_equal(np_(fik)[0], rm[2][k]) and np.array_equal(np_(stk)[0], rm[1][k])


# ------------------------------------------------------------- CPD-TOPO order


def gpu_cpd(g, d, comm_off=False):
    lev, oid, lp, L = cel.topo_levels(g)
    bl, tl, _, _ = cel.blevel(g, d, lev, lp, oid, L, comm_off=comm_off, want_tlevel=True,
                              want_prio=False)
    return cel.cpd_order(g, bl, tl)


def oracle_cpd(wl, comm_off=False):
    lev, oid, lp, L = O.topo_levels(wl)
    bl, tl, _, _ = O.blevel(wl, lev, oid, comm_off=comm_off, want_prio=False)
    return O.cpd_topo(wl, bl, tl)


@pytest.mark.parametrize("cfg,comm_off", [(1, False), (1, True), (2, False), (3, False),
                                          (5, False)])
def test_cpd_order_configs(cfg, comm_off):
    wl, _, _ = config(cfg, 0)
    g, d = up(wl)
    got = np_(gpu_cpd(g, d, comm_off))
    assert np.array_equal(got, oracle_cpd(wl, comm_off))


def test_cpd_order_transformer96():
    wl = make_config(4, 0)
    g, d = up(wl)
    assert np.array_equal(np_(gpu_cpd(g, d)), oracle_cpd(wl))


def test_cpd_order_random_and_edge_cases():
    for s in range(12):
        wl = make_random_dag(500 + s, 20 + 37 * s, p_edge=min(0.5, 3.0 / (20 + 37 * s)),
                             D=2 + s % 4, multi=(s % 2 == 0), zero_frac=0.2 if s % 3 == 0 else 0)
        g, d = up(wl)
        assert np.array_equal(np_(gpu_cpd(g, d)), oracle_cpd(wl)), s
    wl = from_edges(0, [], [], [], 2, [5, 5], 3, 1)
    g, d = up(wl)
    assert np_(gpu_cpd(g, d)).size == 0
    wl = from_edges(1, [], [7], [100], 2, [5, 5], 3, 1)
    g, d = up(wl)
    assert np_(gpu_cpd(g, d)).tolist() == [0]
    wl = from_edges(3, [(0, 1), (1, 2), (2, 0)], [1] * 3, [0] * 3, 2, [5, 5], 1, 0)
    g, d = up(wl)
    z = torch.zeros(3, dtype=torch.int64, device=DEV)
    with pytest.raises(cel.CelError) as ei:
        cel.cpd_order(g, z, z)
    assert ei.value.code == -2


@pytest.mark.parametrize("cfg", [1, 3])
def test_cluster_on_cpd_order(cfg):
    wl, _, _ = config(cfg, 0)
    g, d = up(wl)
    order = gpu_cpd(g, d)
    ref = O.cluster(wl, oracle_cpd(wl), 200, -1)
    cid, C, cut = cel.cluster(g, d, order, 200, -1)
    assert C == ref[1] and cut == ref[2]
    assert np.array_equal(np_(cid), ref[0])


# ------------------------------------------------------------- DFS-TOPO order


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_dfs_order_configs(cfg):
    wl = make_config(cfg, 0) if cfg == 4 else config(cfg, 0)[0]
    g, _ = up(wl)
    assert np.array_equal(np_(cel.dfs_order(g)), O.dfs_topo(wl))


def test_dfs_order_random_and_edge_cases():
    for s in range(12):
        wl = make_random_dag(700 + s, 20 + 41 * s, p_edge=min(0.5, 3.0 / (20 + 41 * s)),
                             D=2 + s % 4, multi=(s % 2 == 0), zero_frac=0.2 if s % 3 == 0 else 0)
        g, _ = up(wl)
        assert np.array_equal(np_(cel.dfs_order(g)), O.dfs_topo(wl)), s
    g, _ = up(from_edges(0, [], [], [], 2, [5, 5], 3, 1))
    assert np_(cel.dfs_order(g)).size == 0
    g, _ = up(from_edges(8, [(0, 2), (2, 4), (4, 6), (1, 3), (3, 5), (5, 7)], [1] * 8, [0] * 8, 2,
                         [10 ** 9] * 2, 1, 0))
    assert np_(cel.dfs_order(g)).tolist() == [0, 2, 4, 6, 1, 3, 5, 7]
    g, _ = up(from_edges(3, [(0, 1), (1, 2), (2, 0)], [1] * 3, [0] * 3, 2, [5, 5], 1, 0))
    with pytest.raises(cel.CelError) as ei:
        cel.dfs_order(g)
    assert ei.value.code == -2


def test_cluster_and_place_on_dfs_order():
    wl, _, _ = config(3, 0)
    g, d = up(wl)
    order = cel.dfs_order(g)
    ref = O.cluster(wl, O.dfs_topo(wl), 200, -1)
    cid, C, cut = cel.cluster(g, d, order, 200, -1)
    assert C == ref[1] and cut == ref[2]
    assert np.array_equal(np_(cid), ref[0])


# ----------------------------------------- Order-Place and the CCR parts


def check_order_place(wl, cid, C):
    ref = O.order_place(wl, cid, C)
    g, d = up(wl)
    cdev, ndev, be = cel.order_place(g, d, tt(cid, np.int32), C)
    assert be == ref[2]
    assert np.array_equal(np_(cdev), ref[0])
    assert np.array_equal(np_(ndev), ref[1])
    return ref


def check_comm_sums(wl, cid=None):
    ref = O.comm_sums(wl, cid)
    g, d = up(wl)
    got = cel.comm_sums(g, d, None if cid is None else tt(cid, np.int32))
    assert got == ref
    return ref


def test_order_place_and_ccr_hand6():
    import json
    import os
    gd = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand6.json")))
    g6 = gd["graph"]
    cid = np.array(gd["order_place"]["cluster_id"], np.int32)
    for caps, key in (((60, 60), "caps_60"), ((30, 30), "caps_30")):
        wl = from_edges(g6["n"], g6["edges"], g6["w"], g6["ob"], 2, caps, g6["bw"], g6["lat"],
                        mem=g6["mem"])
        g, d = up(wl)
        cdev, ndev, be = cel.order_place(g, d, tt(cid, np.int32), 3)
        assert np_(cdev).tolist() == gd["order_place"][key]["cluster_dev"]
        assert be == gd["order_place"][key]["best_effort"]
        assert np_(ndev).tolist() == [np_(cdev)[c] for c in cid]
    assert cel.comm_sums(g, d) == (gd["ccr"]["edge_comm"], gd["ccr"]["w_sum"])
    assert cel.comm_sums(g, d, tt(cid, np.int32))[0] == gd["ccr"]["edge_comm_clustered"]


@pytest.mark.parametrize("cfg,seed", [(1, 0), (2, 0), (3, 0), (5, 0)])
def test_order_place_and_ccr_configs(cfg, seed):
    """The priority- and CPD-order clusterings of each config, at its own caps and
    at caps tight enough to move across devices and end in best effort."""
    import dataclasses
    wl, rt, rb = config(cfg, seed)
    check_comm_sums(wl)
    for order in (rb[2], oracle_cpd(wl)):
        for R, mode in ((200, O.DP), (40, O.GREEDY)):
            cid, C, cut = O.cluster(wl, order, R, -1, mode)
            ec, ws = check_comm_sums(wl, cid)
            assert ec == cut
            for frac in (None, 8, 64):
                w2 = wl if frac is None else dataclasses.replace(
                    wl, cap=np.full(wl.D, int(wl.mem.sum()) // frac, np.int64))
                check_order_place(w2, cid, C)


def test_order_place_random_and_edge_cases():
    import dataclasses
    rng = np.random.default_rng(9)
    for s in range(24):
        n = 2 + (s * 53) % 700
        wl = make_random_dag(900 + s, n, p_edge=min(0.5, 4.0 / n), D=1 + s % 7,
                             cap_frac=(1, 1 + s % 9), multi=(s % 3 == 0),
                             zero_frac=0.2 if s % 4 == 0 else 0.0)
        check_comm_sums(wl)
        order = random_topo_order(wl, rng)
        cid, C, _ = O.cluster(wl, order, int(rng.integers(1, 30)), -1, s % 2)
        check_comm_sums(wl, cid)
        check_order_place(wl, cid, C)
        # caps that differ per device (some zero), and empty clusters past the used ids
        w2 = dataclasses.replace(wl, cap=rng.integers(0, max(2, int(wl.mem.sum()) // 2),
                                                      wl.D).astype(np.int64))
        check_order_place(w2, cid, C + 1 + s % 70)
    wl = from_edges(0, [], [], [], 2, [5, 5], 3, 1)
    g, d = up(wl)
    assert cel.comm_sums(g, d) == (0, 0)
    z = torch.zeros(0, dtype=torch.int32, device=DEV)
    cdev, ndev, be = cel.order_place(g, d, z, 0)
    assert np_(cdev).size == 0 and np_(ndev).size == 0 and be == 0
    check_order_place(wl, np.zeros(0, np.int32), 3)
    wl = from_edges(3, [(0, 1), (1, 2)], [1, 2, 3], [4, 5, 6], 3, [10, 0, 3], 2, 1)
    check_order_place(wl, np.array([0, 1, 2], np.int32), 3)  # mem 8, 10, 12
    check_order_place(wl, np.array([0, 0, 0], np.int32), 1)
    g, d = up(wl)
    with pytest.raises(cel.CelError) as ei:  # id out of range
        cel.order_place(g, d, tt(np.array([0, 1, 3], np.int32), np.int32), 3)
    assert ei.value.code == -1
    with pytest.raises(cel.CelError) as ei:  # no clusters for three nodes
        cel.order_place(g, d, tt(np.zeros(3, np.int32), np.int32), 0)
    assert ei.value.code == -1
    wl = from_edges(2, [(0, 1)], [1, 1], [2 ** 62, 0], 2, [5, 5], 1, 0, mem=[0, 0])
    g, d = up(wl)
    with pytest.raises(cel.CelError) as ei:
        cel.comm_sums(g, d)
    assert ei.value.code == -3


def test_order_place_and_ccr_transformer96():
    """Full size: 1.07M nodes, the CPD-order clustering of Section 5.1.3."""
    wl = make_config(4, 0)
    g, d = up(wl)
    ocpd = oracle_cpd(wl)
    cid, C, cut = O.cluster(wl, ocpd, 200, -1)
    assert check_comm_sums(wl, cid)[0] == cut
    check_comm_sums(wl)
    check_order_place(wl, cid, C)


# ------------------------------------ makespan under device models (insertion, transfers)

MODELS = (0, cel.MODEL_INSERT, cel.MODEL_COMM_TASKS, cel.MODEL_INSERT | cel.MODEL_COMM_TASKS,
          cel.MODEL_COMM_BLOCK)


def check_model(wl, order, P, models=MODELS, **het):
    g, d = up(wl)
    o = tt(order, np.int32)
    Pt = tt(P, np.uint8)
    for m in models:
        ref = O.makespan_model(wl, order, P, m, **het)
        print(f"[model] n={wl.n} D={wl.D} K={1 if P.ndim == 1 else P.shape[0]} model={m} "
              f"het={sorted(k for k, v in het.items() if v is not None)}", flush=True)
        ms, st, fi = cel.makespan_model(g, d, o, Pt, m, want_times=True, **het)
        assert np.array_equal(np_(ms), ref[0]), m
        assert np.array_equal(np_(fi), ref[2]), m
        assert np.array_equal(np_(st), ref[1]), m


def test_model_hand_fixtures():
    import json
    import os
    gold = os.path.join(os.path.dirname(__file__), "golden", "model_hand.json")
    for case in json.load(open(gold))["cases"]:
        wl = from_edges(case["n"], case["edges"], case["w"], case["ob"], case["D"], case["cap"],
                        case["bw"], case["lat"])
        g, d = up(wl)
        het = dict(tmul=case.get("tmul"), bw=case.get("bw_matrix"), lat=case.get("lat_matrix"))
        for m, e in case["models"].items():
            ms, st, fi = cel.makespan_model(g, d, tt(case["order"], np.int32),
                                            tt(case["dev"], np.uint8), int(m), want_times=True,
                                            **het)
            assert np_(st)[0].tolist() == e["start"], (case["name"], m)
            assert np_(fi)[0].tolist() == e["finish"] and int(np_(ms)[0]) == e["makespan"]


@pytest.mark.parametrize("cfg,seed", [(1, 0), (2, 0), (3, 0), (5, 0)])
def test_model_configs(cfg, seed):
    """Priority and CPD-TOPO orders; random placements and Adjusting Placement's."""
    wl, rt, rb = config(cfg, seed)
    P = random_placements(wl, 2, 9 + cfg)
    cid, C, _ = O.cluster(wl, rb[2], 200, -1)
    P = np.concatenate([O.place(wl, cid, C)[1][None, :], P])
    check_model(wl, rb[2], P)
    check_model(wl, oracle_cpd(wl), P[:1])
    # model 0 is cel_makespan's schedule
    g, d = up(wl)
    ms0, _, _ = cel.makespan_model(g, d, tt(rb[2], np.int32), tt(P, np.uint8), 0)
    ms1, _, _ = cel.makespan(g, d, tt(rb[2], np.int32), tt(rt[0], np.int32), tt(rt[2], np.int32),
                             rt[3], tt(P, np.uint8))
    assert np.array_equal(np_(ms0), np_(ms1))


def test_model_random_dags():
    """Random topological orders (not level-monotone), multi-edges, zero w,
    1..64 devices, rows of many inputs (folded by the whole wave)."""
    rng = np.random.default_rng(12)
    for s in range(16):
        n = 5 + (s * 131) % 1500
        D = [1, 2, 3, 5, 8, 17, 64, 40][s % 8]
        wl = make_random_dag(7000 + s, n, p_edge=min(0.6, (2.0 + 30.0 * (s % 3 == 0)) / n), D=D,
                             multi=(s % 3 == 0), zero_frac=0.25 if s % 4 == 0 else 0.0)
        order = random_topo_order(wl, rng)
        P = rng.integers(0, D, (2, n)).astype(np.uint8)
        check_model(wl, order, P)


def test_model_heavy_rows():
    """Rows with more inputs than one lane folds (16): a sink fed by every node,
    a node fed by the 100 positions just before it (inputs inside and before
    its window), and a source feeding everything (transfers to every device)."""
    rng = np.random.default_rng(21)
    n = 3000
    edges = [(0, v) for v in range(1, n)]
    edges += [(u, n - 1) for u in range(1, n - 1)]
    edges += [(u, 1530) for u in range(1430, 1530)]
    wl = from_edges(n, edges, rng.integers(0, 50, n), rng.integers(0, 200, n), 7,
                    [10 ** 9] * 7, 3, 2)
    order = np.arange(n, dtype=np.int32)
    check_model(wl, order, rng.integers(0, 7, (2, n)).astype(np.uint8))


def test_model_many_gaps():
    """Hundreds of idle gaps on one device, filled late: chunked walk back over
    the gap list, splits that shift the gaps above, exact fills."""
    rng = np.random.default_rng(3)
    A, edges, w, ob, dev = 300, [], [], [], []
    for i in range(A):  # a_i (dev0, w 10) -> b_i (dev1, w 1), c = 5
        edges.append((2 * i, 2 * i + 1))
        if i:
            edges.append((2 * i - 2, 2 * i))
        w += [10, 1]
        ob += [5, 0]
        dev += [0, 1]
    base = 2 * A
    late = 400
    for j in range(late):  # late nodes on dev1: no inputs, or an input from some a_i
        w.append(int(rng.integers(1, 9)))
        ob.append(0)
        dev.append(1)
        if j % 3 == 0:
            edges.append((2 * int(rng.integers(0, A)), base + j))
    n = base + late
    wl = from_edges(n, edges, w, ob, 2, [10 ** 9, 10 ** 9], 1, 0)
    order = np.arange(n, dtype=np.int32)
    check_model(wl, order, np.array(dev, np.uint8))


def test_model_edge_cases_and_errors():
    wl = from_edges(0, [], [], [], 2, [5, 5], 3, 1)
    g, d = up(wl)
    z = torch.zeros((3, 0), dtype=torch.uint8, device=DEV)
    ms, _, _ = cel.makespan_model(g, d, torch.zeros(0, dtype=torch.int32, device=DEV), z, 3)
    assert np_(ms).tolist() == [0, 0, 0]
    wl = from_edges(1, [], [7], [100], 3, [5, 5, 5], 3, 1)
    check_model(wl, np.array([0], np.int32), np.array([2], np.uint8))
    wl = from_edges(3, [(0, 1), (1, 2)], [1, 2, 3], [4, 5, 6], 2, [10, 10], 2, 1)
    g, d = up(wl)
    o = tt([0, 1, 2], np.int32)
    for bad in (8, 5, 6, 7):  # an unknown bit; the blocking model combined with another
        with pytest.raises(cel.CelError) as ei:
            cel.makespan_model(g, d, o, tt([0, 1, 0], np.uint8), bad)
        assert ei.value.code == -1
    with pytest.raises(cel.CelError) as ei:  # device out of range
        cel.makespan_model(g, d, o, tt([0, 2, 0], np.uint8), 2)
    assert ei.value.code == -1
    with pytest.raises(cel.CelError) as ei:  # not topological
        cel.makespan_model(g, d, tt([1, 0, 2], np.int32), tt([0, 1, 0], np.uint8), 1)
    assert ei.value.code == -6
    wl = make_random_dag(3, 50, p_edge=0.1, D=65)
    g, d = up(wl)
    with pytest.raises(cel.CelError) as ei:  # more than 64 devices
        cel.makespan_model(g, d, tt(O.topo_levels(wl)[1], np.int32),
                           torch.zeros(50, dtype=torch.uint8, device=DEV), 1)
    assert ei.value.code == -1


def test_model_transformer96():
    """Full size (1.07M nodes): every model on Adjusting Placement's placement
    of the CPD-TOPO clustering and on a random placement."""
    wl = make_config(4, 0)
    ocpd = oracle_cpd(wl)
    cid, C, _ = O.cluster(wl, ocpd, 200, -1)
    P = np.stack([O.place(wl, cid, C)[1], random_placements(wl, 1, 5)[0]])
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    check_model(wl, pr, P)



# ------------------------------------------- heterogeneous devices, co-location


def rand_het(rng, wl, parts=("tmul", "bw", "lat")):
    D = wl.D
    het = dict(tmul=None, bw=None, lat=None)
    if "tmul" in parts:
        het["tmul"] = rng.integers(200, 5000, D)
    if "bw" in parts:
        het["bw"] = rng.integers(1, 4 * int(wl.bw) + 2, (D, D))
    if "lat" in parts:
        het["lat"] = rng.integers(0, 3 * int(wl.lat) + 5, (D, D))
    return het


def test_hetero_random_dags():
    rng = np.random.default_rng(51)
    parts = [("tmul", "bw", "lat"), ("tmul",), ("bw",), ("lat", "bw")]
    for s in range(12):
        n = 5 + (s * 151) % 1200
        D = [2, 3, 8, 64, 5, 17][s % 6]
        wl = make_random_dag(8100 + s, n, p_edge=min(0.6, (2.0 + 20.0 * (s % 4 == 0)) / n), D=D,
                             multi=(s % 3 == 0), zero_frac=0.2 if s % 2 else 0.0)
        order = random_topo_order(wl, rng)
        P = rng.integers(0, D, (2, n)).astype(np.uint8)
        check_model(wl, order, P, **rand_het(rng, wl, parts[s % 4]))


def test_hetero_configs_and_overflow():
    wl, rt, rb = config(3, 0)
    rng = np.random.default_rng(52)
    cid, C, _ = O.cluster(wl, rb[2], 200, -1)
    P = np.concatenate([O.place(wl, cid, C)[1][None, :], random_placements(wl, 1, 3)])
    check_model(wl, rb[2], P, **rand_het(rng, wl))
    big = from_edges(2, [(0, 1)], [2 ** 50, 1], [0, 0], 2, [5, 5], 1, 0)
    g, d = up(big)
    o, dv = tt([0, 1], np.int32), tt([0, 1], np.uint8)
    with pytest.raises(cel.CelError) as ei:  # link latencies must stay below 2^31
        cel.makespan_model(g, d, o, dv, 0, tmul=[65536, 1024], bw=[[1, 1], [1, 1]],
                           lat=[[0, 2 ** 31], [0, 0]])
    assert ei.value.code == -1
    ms, _, _ = cel.makespan_model(g, d, o, dv, 0, tmul=[65536, 1024])  # 2^50 x 64 = 2^56 fits
    assert int(np_(ms)[0]) == int(O.makespan_model(big, [0, 1], [0, 1], 0, tmul=[65536, 1024])[0][0])
    huge = from_edges(2, [(0, 1)], [2 ** 57, 1], [0, 0], 2, [5, 5], 1, 0)
    g, d = up(huge)
    with pytest.raises(cel.CelError) as ei:  # 2^57 x 64 = 2^63: rejected like the oracle
        cel.makespan_model(g, d, o, dv, 1, tmul=[65536, 1024])
    assert ei.value.code == -3
    with pytest.raises(O.OracleError):
        O.makespan_model(huge, [0, 1], [0, 1], 1, tmul=[65536, 1024])


def test_hetero_transformer96():
    """Full size: two device speeds, faster links inside pairs of devices."""
    wl = make_config(4, 0)
    D = wl.D
    tmul = [1024 if x < D // 2 else 2048 for x in range(D)]
    bw = [[2 * wl.bw if x // 2 == y // 2 else wl.bw for y in range(D)] for x in range(D)]
    lat = [[wl.lat // 2 if x // 2 == y // 2 else wl.lat for y in range(D)] for x in range(D)]
    ocpd = oracle_cpd(wl)
    cid, C, _ = O.cluster(wl, ocpd, 200, -1)
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid)
    check_model(wl, pr, O.place(wl, cid, C)[1], tmul=tmul, bw=bw, lat=lat)


def check_colocate(wl, order, grp, G, P):
    ref = O.colocate(wl, order, grp, G, P)
    g, _ = up(wl)
    got = tt(P, np.uint8)
    cel.colocate(g, tt(order, np.int32), tt(grp, np.int32), G, got)
    assert np.array_equal(np_(got), ref)


def test_colocate():
    import json
    import os
    case = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                       "colocate_hand.json")))["cases"][0]
    wl = from_edges(case["n"], case["edges"], [1] * case["n"], [0] * case["n"], 4, [9] * 4, 1, 0)
    g, _ = up(wl)
    nd = tt(case["dev_in"], np.uint8)
    cel.colocate(g, tt(case["order"], np.int32), tt(case["group"], np.int32), case["n_groups"], nd)
    assert np_(nd).tolist() == case["dev_out"]
    rng = np.random.default_rng(53)
    for cfg in (1, 3):
        wl, rt, rb = config(cfg, 0)
        for G in (1, 37, wl.n // 3):
            grp = rng.integers(-1, G, wl.n).astype(np.int32)
            check_colocate(wl, rb[2], grp, G, random_placements(wl, 3, G))
    check_colocate(wl, rb[2], np.full(wl.n, -1, np.int32), 0, random_placements(wl, 1, 1))
    g, _ = up(wl)
    with pytest.raises(cel.CelError) as ei:
        cel.colocate(g, tt(rb[2], np.int32), tt(np.full(wl.n, 5, np.int32), np.int32), 5,
                     tt(random_placements(wl, 1, 1), np.uint8))
    assert ei.value.code == -1


def test_model_many_placements():
    """More placements than compute units in one call (K = 300, one wave each),
    64 devices, every model; and K = 257 on config 1."""
    rng = np.random.default_rng(61)
    wl = make_random_dag(9100, 1500, p_edge=3.0 / 1500, D=64, multi=True, zero_frac=0.1)
    order = random_topo_order(wl, rng)
    P = rng.integers(0, 64, (300, wl.n)).astype(np.uint8)
    check_model(wl, order, P)
    wl, rt, rb = config(1, 0)
    check_model(wl, rb[2], random_placements(wl, 257, 8), models=(cel.MODEL_INSERT,
                                                                  cel.MODEL_COMM_TASKS,
                                                                  cel.MODEL_COMM_BLOCK))


# ------------------------------------------------------------ diagnostics


def test_step_latency_probe():
    """The dependent-step probe behind the bench's depth ceiling returns a
    plausible time per step for each variant (a few ns to a few us)."""
    for v in (0, 1, 2):
        ns = cel.step_latency(v, 20000)
        assert 5.0 < ns < 5000.0, (v, ns)
    with pytest.raises(cel.CelError):
        cel.step_latency(3, 100)


# ------------- Adjusting Placement with heterogeneous devices/links and co-location


def check_place_ext(wl, cid, C, het=None, grp=None, G=0):
    het = het or {}
    ref = O.place_ext(wl, cid, C, group=grp, n_groups=G, **het)
    g, d = up(wl)
    print(f"[place_ext] n={wl.n} C={C} D={wl.D} het={sorted(het)} groups={G}", flush=True)
    got = cel.place_ext(g, d, tt(cid, np.int32), C, group=None if grp is None else tt(grp, np.int32),
                        n_groups=G, **het)
    assert np.array_equal(np_(got[0]), ref[0]) and np.array_equal(np_(got[1]), ref[1])
    assert got[2] == ref[2] and got[3] == ref[3] and np.array_equal(np_(got[4]), ref[4])
    return ref


def test_place_ext_hand_fixtures():
    import json
    import os
    gold = os.path.join(os.path.dirname(__file__), "golden", "place_ext_hand.json")
    for case in json.load(open(gold))["cases"]:
        wl = from_edges(case["n"], case["edges"], case["w"], case["ob"], case["D"], case["cap"],
                        case["bw"], case["lat"])
        g, d = up(wl)
        for v in case["variants"]:
            grp = v.get("group")
            cdev, ndev, span, be, fin = cel.place_ext(
                g, d, tt(case["cluster_id"], np.int32), case["C"], tmul=v.get("tmul"),
                bw=v.get("bw_matrix"), lat=v.get("lat_matrix"),
                group=None if grp is None else tt(grp, np.int32), n_groups=v.get("n_groups", 0))
            assert np_(cdev).tolist() == v["cluster_dev"] and np_(ndev).tolist() == v["node_dev"]
            assert np_(fin).tolist() == v["fin"] and span == v["span"] and be == v["be"]


def test_place_ext_without_extras_is_place():
    for cfg in (1, 3):
        wl, rt, rb = config(cfg, 0)
        cid, C, _ = O.cluster(wl, rb[2], 200, -1)
        ref = check_place_ext(wl, cid, C)
        g, d = up(wl)
        cdev, ndev, span, be = cel.place(g, d, tt(cid, np.int32), C)
        assert np.array_equal(np_(cdev), ref[0]) and span == ref[2] and be == ref[3]


def test_place_ext_random():
    rng = np.random.default_rng(71)
    for s in range(24):
        n = 5 + (s * 97) % 700
        D = [1, 2, 3, 5, 8, 16, 64, 33][s % 8]
        wl = make_random_dag(9300 + s, n, p_edge=min(0.5, 4.0 / n), D=D,
                             cap_frac=(1, 1 + s % 5), multi=(s % 3 == 0),
                             zero_frac=0.2 if s % 4 == 0 else 0.0)
        order = random_topo_order(wl, rng)
        cid, C, _ = O.cluster(wl, order, int(rng.integers(1, 40)), -1, s % 2)
        parts = [("tmul", "bw", "lat"), ("tmul",), ("bw",), ("lat",), ()][s % 5]
        het = {k: v for k, v in rand_het(rng, wl, parts).items() if v is not None}
        G = 0 if s % 3 == 0 else max(1, n // (2 + s % 7))
        grp = rng.integers(-1, G, n).astype(np.int32) if G else None
        check_place_ext(wl, cid, C, het, grp, G)


@pytest.mark.parametrize("cfg", [1, 2, 3, 5])
def test_place_ext_configs(cfg):
    wl, rt, rb = config(cfg, 0)
    rng = np.random.default_rng(72 + cfg)
    cid, C, _ = O.cluster(wl, rb[2], 200, -1)
    G = wl.n // 40
    grp = np.full(wl.n, -1, np.int32)
    pick = rng.permutation(wl.n)[:4 * G]
    grp[pick] = np.repeat(np.arange(G, dtype=np.int32), 4)
    check_place_ext(wl, cid, C, {k: v for k, v in rand_het(rng, wl).items()}, grp, G)
    check_place_ext(wl, cid, C, {"tmul": rand_het(rng, wl, ("tmul",))["tmul"]})


def test_place_ext_many_clusters():
    """More clusters than the placement keeps in LDS (config 3, R = 4)."""
    wl, rt, rb = config(3, 0)
    rng = np.random.default_rng(74)
    cid, C, _ = O.cluster(wl, rb[2], 4, -1)
    assert C > 8192
    grp = rng.integers(-1, 500, wl.n).astype(np.int32)
    check_place_ext(wl, cid, C, {k: v for k, v in rand_het(rng, wl).items()}, grp, 500)


def test_place_ext_transformer96():
    """Full size: the CPD-TOPO clustering of transformer-96 (6,284 clusters, 16
    devices) with two device speeds, faster links inside device pairs and
    26,765 co-location groups of 4 nodes."""
    wl = make_config(4, 0)
    D = wl.D
    het = dict(tmul=[1024 if x < D // 2 else 2048 for x in range(D)],
               bw=[[2 * wl.bw if x // 2 == y // 2 else wl.bw for y in range(D)] for x in range(D)],
               lat=[[wl.lat // 2 if x // 2 == y // 2 else wl.lat for y in range(D)]
                    for x in range(D)])
    rng = np.random.default_rng(75)
    G = wl.n // 40
    grp = np.full(wl.n, -1, np.int32)
    grp[rng.permutation(wl.n)[:4 * G]] = np.repeat(np.arange(G, dtype=np.int32), 4)
    cid, C, _ = O.cluster(wl, oracle_cpd(wl), 200, -1)
    check_place_ext(wl, cid, C, het, grp, G)


def test_place_ext_errors():
    wl, rt, rb = config(1, 0)
    cid, C, _ = O.cluster(wl, rb[2], 200, -1)
    g, d = up(wl)
    c = tt(cid, np.int32)
    with pytest.raises(cel.CelError) as ei:  # group id beyond n_groups
        cel.place_ext(g, d, c, C, group=tt(np.full(wl.n, 3, np.int32), np.int32), n_groups=3)
    assert ei.value.code == -1
    with pytest.raises(cel.CelError) as ei:  # a time multiplier out of range
        cel.place_ext(g, d, c, C, tmul=[0] * wl.D)
    assert ei.value.code == -1
    wl2 = make_random_dag(5, 80, p_edge=0.05, D=65)
    g2, d2 = up(wl2)
    with pytest.raises(cel.CelError) as ei:  # more than 64 devices
        cel.place_ext(g2, d2, tt(np.zeros(80, np.int32), np.int32), 1)
    assert ei.value.code == -1
