"""cel_makespan_noalloc (scratch in a fixed device array, no allocation)
against cel_makespan, bit for bit, on consecutive calls of shrinking size."""
from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on CPU, skipped there
    pytest.skip("needs a ROCm GPU", allow_module_level=True)

import paper_2208_00184_amd as cel  # noqa: E402
from oracle import oracle as O  # noqa: E402
from workloads import make_config, make_random_dag  # noqa: E402

DEV = "cuda:0"


def np_(t):
    return t.detach().cpu().numpy()


def prepared(wl, K, seed):
    """Graph on the GPU, the oracle's level-monotone priority order and K
    random placements (row 0: the oracle's Adjusting Placement)."""
    lev, oid, lp, L = O.topo_levels(wl)
    _, _, pr, _ = O.blevel(wl, lev, oid, want_tlevel=False)
    cid, C, _ = O.cluster(wl, pr, 200, -1)
    _, ndev, _, _ = O.place(wl, cid, C)
    rng = np.random.default_rng([31, seed])
    P = rng.integers(0, wl.D, (K, wl.n)).astype(np.uint8)
    P[0] = ndev
    g = cel.Graph.from_arrays(wl, DEV)
    d = cel.Devices.from_arrays(wl)
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(DEV)  # noqa: E731
    args = (t(pr, np.int32), t(lev, np.int32), t(lp, np.int32), L)
    return g, d, args, t(P if K > 1 else P[0], np.uint8), (wl, pr, P)


def both(g, d, args, P):
    a = cel.makespan(g, d, *args, P, want_times=True)
    b = cel.makespan(g, d, *args, P, want_times=True, noalloc=True)
    torch.cuda.synchronize()
    return [np_(x) for x in a], [np_(x) for x in b]


@pytest.mark.parametrize("cases", [
    [(5, 1), (1, 1)],          # 200k nodes, then 2k nodes (single-placement path)
    [(1, 24), (0, 3)],         # a batch, then a small random DAG's batch
    [(3, 1), (2, 6), (1, 1)],  # 55k, 20k with a batch, 2k
])
def test_noalloc_matches_makespan_on_shrinking_calls(cases):
    for i, (cfg, K) in enumerate(cases):
        wl = make_config(cfg, 0) if cfg else make_random_dag(4242, 37, p_edge=0.2, D=3)
        g, d, args, P, ref_in = prepared(wl, K, i)
        (ma, sa, fa), (mb, sb, fb) = both(g, d, args, P)
        assert np.array_equal(ma, mb) and np.array_equal(fa, fb) and np.array_equal(sa, sb), (cfg, K)
        wl_, pr, Ph = ref_in
        rm, _, rf = O.makespan(wl_, pr, Ph)
        assert np.array_equal(mb, rm) and np.array_equal(fb, rf), (cfg, K)


def test_noalloc_rejects_inputs_above_its_scratch():
    wl = make_config(1, 0)
    g, d, args, _, _ = prepared(wl, 1, 0)
    K = 8000  # bound 65536 + 200 (n + 1) + 16 m + 21 K n > 128 MiB at n = 2048
    P = torch.zeros((K, wl.n), dtype=torch.uint8, device=DEV)
    with pytest.raises(cel.CelError) as ei:
        cel.makespan(g, d, *args, P, noalloc=True)
    assert ei.value.code == -1 and "fixed" in str(ei.value)
    # the same batch through cel_makespan works, and a fitting call still does
    ms, _, _ = cel.makespan(g, d, *args, P)
    assert ms.shape[0] == K
    g2, d2, args2, P2, _ = prepared(wl, 4, 1)
    (ma, _, fa), (mb, _, fb) = both(g2, d2, args2, P2)
    assert np.array_equal(ma, mb) and np.array_equal(fa, fb)
