"""Benchmark of the placement hot path on one MI355X.

A step is one pass of the whole path over the 1.07M-node transformer training
graph (96 blocks, hidden 8192, micro-op granularity): Kahn levels -> b-level
and priority order -> DP clustering (R = 200) -> Adjusting Placement ->
makespan of the resulting placement -> makespan of a batch of 64 perturbed
placements (5% of the clusters moved to a random device).  Inputs are
device-resident before timing starts.

Headline: DAG edges/s of the b-level + makespan evaluation (m divided by the
time of the b-level call plus the single-placement makespan call).  Also
reported: placement-generation ms (levels + b-level + clustering +
placement), per-stage and per-kernel times with algorithmic-byte rooflines,
the per-level latency of the level sweeps (a single placement of a graph
10^4 levels deep is bound by it, not by HBM), the t-level pass (an optional
output, timed apart), batched scoring of 1,024 perturbed placements of the
200k-node layered DAG in one call (the bandwidth-bound regime), and the CPU
oracle (one pinned core, every stage) on the same 1.07M-node graph.  Further
rows: the CPD-TOPO order against the priority and DFS-TOPO orders, the CCR before and
after fusion, Order-Place against Adjusting Placement, and the makespan under
the device models (first-fit insertion, transfers as tasks, heterogeneous
devices, co-location).

Usage: python bench.py [--gpus 1] [--steps 5] [--warmup 2] [--no-cpu] [--no-batch]
                       [--no-models]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "DAG edges/sec for b-level+makespan eval (1M-node graph); placement-gen ms"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s
VALU_I32_PEAK = 256 * 4 * 16 * 2.4e9  # lane-ops/s: 256 CUs x 4 SIMD16 x 2.4 GHz
BATCH = 64
BATCH5 = 1024  # candidates of the 200k-node batched-scoring row


def algorithmic_bytes(kernel: str, n: int, m: int, K: int) -> float | None:
    """Bytes each kernel must move per launch (int32 indices, int64 times, u8
    devices): what one pass of the operation needs, whatever the kernel's
    method (policy iteration and relaxation rounds re-read more)."""
    if kernel in ("k_blevel_sweep", "k_blevel_policy"):  # per node: order 4, ptr 4, w 8, c 8, write 8; per edge: idx 4, gather 8
        return 32.0 * n + 12.0 * m
    if kernel in ("k_tlevel_sweep", "k_tlevel_policy"):
        return 32.0 * n + 12.0 * m
    if kernel == "k_makespan_one":    # per node: order 4, ptr 4, w 8, c 8, dev 1, fin 8; per edge: idx 4, fin 8, dev 1, c 8
        return 33.0 * n + 21.0 * m
    if kernel == "k_makespan_batch":    # shared structure once + per placement dev, fin write, dev/fin gathers
        return 24.0 * n + 12.0 * m + K * (9.0 * n + 9.0 * m)
    return None


# rocprofv3 --pmc summaries (see --pmc-summary): one bench step on the
# transformer graph, and the 1,024-placement scoring row
TRAFFIC_FILES = [os.path.join(ROOT, "profiles", f) for f in
                 ("pmc_transformer96_step.md", "pmc_layered200k_batch1024.md")]
CSRC = os.path.join(ROOT, "paper_2208_00184_amd", "csrc")
# kernels the bench names, their symbols in rocprofv3 output and their sources
PMC_KERNELS = {
    "k_makespan_one": ("cel::k_rx_relax<", ["ms_relax.hip", "cel_internal.h"]),
    "k_makespan_sweep_one": ("cel::k_ms_ring(", ["ms_ring.hip", "cel_internal.h"]),
    "k_blevel_policy": ("cel::k_lp_policy<0>", ["lp_policy.hip", "cel_internal.h"]),
    "k_tlevel_policy": ("cel::k_lp_policy<1>", ["lp_policy.hip", "cel_internal.h"]),
    "k_levels_policy": ("cel::k_lp_policy<2>", ["lp_policy.hip", "cel_internal.h"]),
    "k_blevel_sweep": ("cel::k_ring_sweep<true>", ["sweep.hip", "cel_internal.h"]),
    "k_tlevel_sweep": ("cel::k_ring_sweep<false>", ["sweep.hip", "cel_internal.h"]),
    "k_makespan_batch": ("cel::k_mb_ring(", ["ms_batch.hip", "cel_internal.h"]),
    "k_makespan_batch_wide": ("cel::(anonymous namespace)::k_mw_batch(", ["ms_wide.hip", "cel_internal.h"]),
    "k_kahn": ("cel::k_kahn(", ["topo.hip", "cel_internal.h"]),
    "k_cluster_dp": ("cel::k_cluster_dp<true>(", ["cluster.hip", "cel_internal.h"]),
    "k_cluster_policy": ("cel::k_dp_policy(", ["dp_policy.hip", "cel_internal.h"]),
    "k_place": ("cel::k_place<", ["place.hip", "cel_internal.h"]),
}


def source_hash(files) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def pmc_summary(fetch_csv: str, write_csv: str, calib_mib: int, extra_csvs=(), only=None) -> str:
    """Markdown summary of rocprofv3 counter CSVs: per kernel, the counters of
    its first dispatch (in a run with --warmup 0 --steps 1 that is the timed
    step's; later dispatches of the same kernel belong to other rows, on other
    graphs or placements), FETCH_SIZE / WRITE_SIZE scaled by what they read
    for a plain copy of calib_mib MiB (the largest __amd_rocclr_copyBuffer
    dispatch)."""
    import csv
    from collections import defaultdict

    # kernel -> counter -> {dispatch id: value}
    vals = defaultdict(lambda: defaultdict(dict))
    for path in (fetch_csv, write_csv, *extra_csvs):
        with open(path) as fh:
            for r in csv.DictReader(fh):
                vals[r["Kernel_Name"]][r["Counter_Name"]][int(r["Dispatch_Id"])] = \
                    float(r["Counter_Value"])
    copy = [v for k, v in vals.items() if k.startswith("__amd_rocclr_copyBuffer")]
    cf = max(x for v in copy for x in v.get("FETCH_SIZE", {0: 0}).values())
    cw = max(x for v in copy for x in v.get("WRITE_SIZE", {0: 0}).values())
    kib = calib_mib * 1024.0
    ff, fw = kib / cf, kib / cw
    lines = [f"copy calibration: {calib_mib} MiB copied; FETCH_SIZE read {cf:.1f} KiB, "
             f"WRITE_SIZE {cw:.1f} KiB; factors fetch {ff:.4f} write {fw:.4f}", "",
             "| kernel | source | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | HBM bytes (scaled) |"
             " other counters (first dispatch) |",
             "|---|---|---:|---:|---:|---:|---|"]

    def first(d):
        return d[min(d)]

    for name, (sym, files) in PMC_KERNELS.items():
        if only and name not in only:
            continue
        hits = [v for k, v in vals.items() if k.removeprefix("void ").startswith(sym)]
        if not hits:
            continue
        v = hits[0]
        f, w = first(v["FETCH_SIZE"]), first(v["WRITE_SIZE"])
        other = ", ".join(f"{c} {first(x):.0f}" for c, x in sorted(v.items())
                          if c not in ("FETCH_SIZE", "WRITE_SIZE"))
        lines.append(f"| {name} | {source_hash(files)} | {len(v['FETCH_SIZE'])} | {f:.1f} | "
                     f"{w:.1f} | {(f * ff + w * fw) * 1024:.0f} | {other} |")
    return "\n".join(lines)


def stats_summary(stats_csv: str, top: int = 40) -> str:
    """Markdown table of a rocprofv3 --stats kernel_stats CSV (largest total first)."""
    import csv
    rows = []
    with open(stats_csv) as fh:
        for r in csv.DictReader(fh):
            rows.append((r["Name"].split("(")[0][:70], int(r["Calls"]),
                         float(r["TotalDurationNs"]) / 1e6, float(r["AverageNs"]) / 1e3))
    rows.sort(key=lambda x: -x[2])
    out = ["| kernel | calls | total ms | avg us |", "|---|---:|---:|---:|"]
    out += [f"| {n} | {c} | {t:.3f} | {a:.1f} |" for n, c, t, a in rows[:top]]
    return "\n".join(out)


def trace_kernel(trace_csv: str, name: str, top: int = 12) -> str:
    """Dispatch durations of one kernel from a rocprofv3 kernel_trace CSV,
    largest first (a run mixes graphs of several sizes; the largest
    dispatches are the transformer-96 ones)."""
    import csv
    durs = []
    with open(trace_csv) as fh:
        for r in csv.DictReader(fh):
            if r["Kernel_Name"].removeprefix("void ").startswith(name):
                durs.append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e6)
    durs.sort(reverse=True)
    head = durs[:top]
    out = [f"{name}: {len(durs)} dispatches; the {len(head)} largest (ms): " +
           ", ".join(f"{d:.3f}" for d in head)]
    return "\n".join(out)


def load_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from the committed counter summary, or
    None when the summary is missing or the kernel's sources changed since."""
    if kernel not in PMC_KERNELS:
        return None
    want = source_hash(PMC_KERNELS[kernel][1])
    for path in TRAFFIC_FILES:
        if not os.path.exists(path):
            continue
        with open(path) as fh:
            for line in fh:
                cells = [c.strip() for c in line.strip().strip("|").split("|")]
                if len(cells) >= 6 and cells[0] == kernel:
                    return float(cells[5]) if cells[1] == want else None
    return None


def batched_row(cel, torch, dev, args):
    """1,024 perturbed placements of the 200k-node layered DAG scored in one call."""
    from workloads import make_config, perturb_placements
    wl = make_config(5, args.seed)
    g = cel.Graph.from_arrays(wl, dev)
    d = cel.Devices.from_arrays(wl)
    lev, oid, lp, L = cel.topo_levels(g)
    _, _, pr, _ = cel.blevel(g, d, lev, lp, oid, L)
    cid, C, _ = cel.cluster(g, d, pr, 200, -1)
    cdev, ndev, _, _ = cel.place(g, d, cid, C)
    cand = perturb_placements(cdev.cpu().numpy(), wl.D, BATCH5, args.seed)
    nd = torch.gather(torch.from_numpy(cand).to(dev), 1,
                      cid.long().unsqueeze(0).expand(BATCH5, -1)).contiguous()
    del cand
    stream = torch.cuda.current_stream()
    cel.makespan(g, d, pr, lev, lp, L, nd)  # warm-up
    torch.cuda.synchronize()
    cel.kernel_stats(reset=True)
    cel.timing(True)
    times = []
    for _ in range(max(1, args.steps)):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        ms, _, _ = cel.makespan(g, d, pr, lev, lp, L, nd)
        e1.record(stream)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    cel.timing(False)
    ks = cel.kernel_stats(reset=True)
    c_, t_ = ks["k_makespan_batch"]
    kms = t_ / c_
    B = algorithmic_bytes("k_makespan_batch", wl.n, wl.m, BATCH5)
    call_ms = float(np.mean(times))
    print(f"[bench] 200k-node scoring of {BATCH5} placements: {call_ms:.2f} ms per call",
          file=sys.stderr, flush=True)
    parity = None
    if not args.no_cpu:
        # 16 rows spread over the batch against the oracle, whose inputs (order,
        # clustering, placement, perturbation) it derives on its own
        from oracle import oracle as O
        lev_o, oid_o, _, _ = O.topo_levels(wl)
        _, _, pr_o, _ = O.blevel(wl, lev_o, oid_o)
        cid_o, C_o, _ = O.cluster(wl, pr_o, 200, -1)
        cdev_o, _, _, _ = O.place(wl, cid_o, C_o)
        rows = np.linspace(0, BATCH5 - 1, 16).astype(np.int64)
        cand_o = perturb_placements(cdev_o, wl.D, BATCH5, args.seed)[rows][:, cid_o]
        ref, _, _ = O.makespan(wl, pr_o, cand_o, want_times=False)
        parity = {"makespan_rows": bool(np.array_equal(ms.cpu().numpy()[rows], ref))}
    return {"workload": f"layered-200k: 400 x 500 layered DAG, {BATCH5} placements (5% of the "
                        f"clusters of the Adjusting Placement moved at random)",
            "n": wl.n, "m": wl.m, "levels": L, "K": BATCH5, "call_ms": call_ms,
            "edges_per_s": BATCH5 * wl.m / (call_ms * 1e-3), "kernel_ms": kms,
            "algorithmic_bytes": B, "achieved_GBs": round(B / (kms * 1e-3) / 1e9, 2),
            "frac": round(B / (kms * 1e-3) / 1e9 / HBM_PEAK_GBS, 5),
            "traffic": load_traffic("k_makespan_batch_wide"),
            "makespan_min_ns": int(ms.min().item()), "makespan_max_ns": int(ms.max().item()),
            "parity": parity}


def _timed(torch, f, reps=3):
    ts, out = [], None
    for _ in range(reps):
        torch.cuda.synchronize()
        a = time.perf_counter()
        out = f()
        torch.cuda.synchronize()
        ts.append((time.perf_counter() - a) * 1e3)
    return out, float(np.median(ts))


def cpd_compare(cel, torch, g, d, bl, tl, prio, lev, lp, L):
    """CPD-TOPO order (host walk over GPU b-/t-levels) and what it changes
    downstream: DP clustering (R = 200) on it against the level-monotone
    priority order and the DFS-TOPO order; for each, the CCR before and after
    fusion (eq. 1, as in the paper's CCR table) and the makespan of Order-Place
    against Adjusting Placement on the same clusters (as in its placement
    comparison)."""
    cpd, cpd_ms = _timed(torch, lambda: cel.cpd_order(g, bl, tl))
    dfs, dfs_ms = _timed(torch, lambda: cel.dfs_order(g))
    (ec0, ws), ccr_ms = _timed(torch, lambda: cel.comm_sums(g, d))
    row = {"cpd_order_ms": cpd_ms, "dfs_order_ms": dfs_ms, "comm_sums_ms": ccr_ms, "n": g.n,
           "ccr": ec0 / ws}
    for name, order in (("priority", prio), ("dfs", dfs), ("cpd", cpd)):
        cid, C, cut = cel.cluster(g, d, order, 200, -1)
        ec, _ = cel.comm_sums(g, d, cid)
        _, ndev, cms, be = cel.place(g, d, cid, C)
        ms, _, _ = cel.makespan(g, d, prio, lev, lp, L, ndev)
        (_, ndev_o, be_o), op_ms = _timed(torch, lambda: cel.order_place(g, d, cid, C))
        ms_o, _, _ = cel.makespan(g, d, prio, lev, lp, L, ndev_o)
        row[name] = {"clusters": C, "cut_cost_ns": cut, "ccr_fused": ec / ws,
                     "coarse_makespan_ns": cms, "best_effort": be, "makespan_ns": int(ms[0].item()),
                     "order_place": {"makespan_ns": int(ms_o[0].item()), "best_effort": be_o,
                                     "ms": op_ms}}
    return row, ndev, cid, C


def check_parity(pairs: dict) -> dict:
    """{name: (gpu, oracle)} -> {name: equal}; arrays compare element by element."""
    return {k: bool(np.array_equal(np.asarray(a), np.asarray(b))) for k, (a, b) in pairs.items()}


def config_rows(cel, torch, dev, args):
    """The smaller graphs, stage by stage: Kahn levels, b-level with the
    priority order, DP clustering (R = 200), Adjusting Placement and the
    makespan of the placement, each timed with HIP events (median of 5 after 2
    warm-ups), beside the oracle's time per stage on one core (median of 3) and
    a check of every result against the oracle's."""
    from workloads import make_config
    rows = {}
    for cfg in (1, 2, 3):
        wl = make_config(cfg, args.seed)
        g = cel.Graph.from_arrays(wl, dev)
        d = cel.Devices.from_arrays(wl)
        stream = torch.cuda.current_stream()
        names = ["topo_levels", "blevel", "cluster", "place", "makespan"]
        rec = {k: [] for k in names}
        out = None
        for it in range(7):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
            ev[0].record(stream)
            lev, oid, lp, L = cel.topo_levels(g)
            ev[1].record(stream)
            bl, _, pr, cp = cel.blevel(g, d, lev, lp, oid, L)
            ev[2].record(stream)
            cid, C, cut = cel.cluster(g, d, pr, 200, -1)
            ev[3].record(stream)
            cdev, ndev, cms, be = cel.place(g, d, cid, C)
            ev[4].record(stream)
            ms, st, fi = cel.makespan(g, d, pr, lev, lp, L, ndev, want_times=True)
            ev[5].record(stream)
            torch.cuda.synchronize()
            if it >= 2:
                for i, k in enumerate(names):
                    rec[k].append(ev[i].elapsed_time(ev[i + 1]))
            out = (lev, oid, lp, L, bl, pr, cp, cid, C, cut, ndev, cms, be, ms, fi)
        stages = {k: round(float(np.median(v)), 3) for k, v in rec.items()}
        lev, oid, lp, L, bl, pr, cp, cid, C, cut, ndev, cms, be, ms, fi = out
        row = {"workload": wl.name, "n": wl.n, "m": wl.m, "levels": L, "D": wl.D,
               "stages_ms": stages,
               "placement_gen_ms": round(sum(stages[k] for k in names[:4]), 3),
               "edges_per_s": wl.m / ((stages["blevel"] + stages["makespan"]) * 1e-3)}
        if not args.no_cpu:
            from oracle import oracle as O
            import statistics
            st_cpu = {}

            def tm(name, f, reps=3):
                ts, r = [], None
                for _ in range(reps):
                    a = time.perf_counter()
                    r = f()
                    ts.append(time.perf_counter() - a)
                st_cpu[name] = round(statistics.median(ts) * 1e3, 3)
                return r

            aff = os.sched_getaffinity(0)
            os.sched_setaffinity(0, {min(aff)})
            try:
                r_lev, r_oid, r_lp, r_L = tm("topo_levels", lambda: O.topo_levels(wl))
                r_bl, _, r_pr, r_cp = tm("blevel", lambda: O.blevel(wl, r_lev, r_oid))
                r_cid, r_C, r_cut = tm("cluster", lambda: O.cluster(wl, r_pr, 200, -1))
                r_pl = tm("place", lambda: O.place(wl, r_cid, r_C))
                r_ms, _, r_fi = tm("makespan", lambda: O.makespan(wl, r_pr, r_pl[1]))
            finally:
                os.sched_setaffinity(0, aff)
            row["oracle_stages_ms"] = st_cpu
            row["oracle_edges_per_s"] = wl.m / ((st_cpu["blevel"] + st_cpu["makespan"]) * 1e-3)
            row["parity"] = check_parity({
                "level": (lev.cpu().numpy(), r_lev), "order_id": (oid.cpu().numpy(), r_oid),
                "level_ptr": (lp.cpu().numpy(), r_lp), "blevel": (bl.cpu().numpy(), r_bl),
                "prio_order": (pr.cpu().numpy(), r_pr), "critical_path_ns": (cp, int(r_cp)),
                "cluster_id": (cid.cpu().numpy(), r_cid), "cut_cost_ns": (cut, int(r_cut)),
                "node_dev": (ndev.cpu().numpy(), r_pl[1]), "coarse_makespan_ns": (cms, int(r_pl[2])),
                "best_effort": (be, int(r_pl[3])), "finish": (fi.cpu().numpy(), r_fi),
                "makespan_ns": (ms.cpu().numpy(), r_ms)})
        rows[f"config{cfg}"] = row
        print(f"[bench] {wl.name}: placement-gen {row['placement_gen_ms']:.2f} ms", file=sys.stderr,
              flush=True)
    return rows


MODEL_NAMES = {0: "fifo", 1: "insert", 2: "comm_tasks", 3: "insert+comm_tasks", 4: "comm_block"}


def models_row(cel, torch, g, d, prio, ndev, seed, K=64, cid=None, C=0):
    """The makespan under each device model (first-fit insertion, transfers as
    tasks) of Adjusting Placement's placement (K = 1) and of K placements in one
    call (that one first, the rest random), on the priority order."""
    n, m = g.n, g.m
    rng = np.random.default_rng([seed, 17])
    PK = torch.from_numpy(rng.integers(0, d.D, (K, n)).astype(np.uint8)).to(ndev.device)
    PK[0] = ndev
    row = {}
    for model, name in MODEL_NAMES.items():
        r = {}
        for k, P in ((1, ndev), (K, PK)):
            cel.kernel_stats(reset=True)
            cel.timing(True)
            (ms, _, _), call_ms = _timed(torch, lambda: cel.makespan_model(g, d, prio, P, model),
                                         reps=2)
            cel.timing(False)
            c_, t_ = cel.kernel_stats(reset=True).get("k_makespan_model", (1, float("nan")))
            kms = t_ / c_
            B = k * (29.0 * n + 21.0 * m)  # per placement: dev, w, c, ptr, fin write; per edge: idx, dev, c, fin
            r[f"K{k}"] = {"call_ms": round(call_ms, 2), "kernel_ms": round(kms, 2),
                          "edges_per_s": k * m / (call_ms * 1e-3),
                          "achieved_GBs": round(B / (kms * 1e-3) / 1e9, 3),
                          "makespan_ns": int(ms[0].item())}
        row[name] = r
    # heterogeneous devices: the upper half of the devices twice as slow, links
    # inside a pair of devices twice as fast with half the latency
    D = d.D
    het = dict(tmul=[1024 if x < D // 2 else 2048 for x in range(D)],
               bw=[[2 * d.bw if x // 2 == y // 2 else d.bw for y in range(D)] for x in range(D)],
               lat=[[d.lat // 2 if x // 2 == y // 2 else d.lat for y in range(D)] for x in range(D)])
    row["hetero"] = {"devices": "tmul 1024 on devices 0..D/2-1, 2048 above; pairs (2i, 2i+1) "
                                "linked at 2 x bw, lat / 2"}
    for model, name in MODEL_NAMES.items():
        (ms, _, _), call_ms = _timed(torch, lambda: cel.makespan_model(g, d, prio, ndev, model,
                                                                        **het), reps=2)
        row["hetero"][name] = {"call_ms": round(call_ms, 2), "makespan_ns": int(ms[0].item())}
    # co-location: seeded groups of 4 over a tenth of the nodes, K placements
    G = n // 40
    grp = np.full(n, -1, np.int32)
    pick = rng.permutation(n)[:4 * G]
    grp[pick] = np.repeat(np.arange(G, dtype=np.int32), 4)
    grp_t = torch.from_numpy(grp).to(ndev.device)
    PK2 = PK.clone()
    _, colo_ms = _timed(torch, lambda: cel.colocate(g, prio, grp_t, G, PK2), reps=3)
    nd1 = ndev.clone()
    cel.colocate(g, prio, grp_t, G, nd1)
    (ms_c, _, _), _ = _timed(torch, lambda: cel.makespan_model(g, d, prio, nd1, 0), reps=1)
    row["colocate"] = {"groups": G, "group_size": 4, "K": K, "call_ms": round(colo_ms, 2),
                       "makespan_ns_after": int(ms_c[0].item()),
                       "makespan_ns_before": row["fifo"]["K1"]["makespan_ns"]}
    # the optimiser itself under the same devices and groups: Adjusting
    # Placement with per-device durations, per-link costs and co-location
    # inside the algorithm, against the homogeneous placement made
    # co-located afterwards, both scored under the heterogeneous model
    if cid is not None:
        (cd_x, nd_x, cms_x, be_x, _), px_ms = _timed(
            torch, lambda: cel.place_ext(g, d, cid, C, group=grp_t, n_groups=G, **het), reps=3)
        cel.kernel_stats(reset=True)
        cel.timing(True)
        cel.place_ext(g, d, cid, C, group=grp_t, n_groups=G, **het)
        cel.timing(False)
        kx = cel.kernel_stats(reset=True).get("k_place_ext", (1, float("nan")))
        (ms_x, _, _), _ = _timed(torch, lambda: cel.makespan_model(g, d, prio, nd_x, 0, **het),
                                 reps=1)
        nd_h = ndev.clone()
        cel.colocate(g, prio, grp_t, G, nd_h)
        (ms_h, _, _), _ = _timed(torch, lambda: cel.makespan_model(g, d, prio, nd_h, 0, **het),
                                 reps=1)
        row["place_ext"] = {"clusters": C, "groups": G, "call_ms": round(px_ms, 2),
                            "k_place_ext_ms": round(kx[1] / kx[0], 2),
                            "coarse_makespan_ns": cms_x, "best_effort": be_x,
                            "makespan_ns_hetero_model": int(ms_x[0].item()),
                            "homogeneous_place_then_colocate_ns": int(ms_h[0].item())}
    return row


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-models", action="store_true",
                    help="skip the device-model rows (insertion, transfers as tasks, "
                         "heterogeneous devices, co-location)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-stage rows of the 2k-, 20k- and 55k-node graphs")
    ap.add_argument("--no-batch", action="store_true",
                    help="skip the 1,024-candidate scoring row on the 200k-node DAG")
    ap.add_argument("--calib-copy", type=int, default=0, metavar="MIB",
                    help="first copy MIB MiB device-to-device once: the reference dispatch "
                         "that scales rocprofv3 FETCH_SIZE / WRITE_SIZE into bytes")
    ap.add_argument("--pmc-summary", nargs="+", metavar="CSV",
                    help="print the counter summary of rocprofv3 counter_collection CSVs "
                         "(FETCH_SIZE run, WRITE_SIZE run, then any others) and exit; "
                         "--calib-copy gives the copy size of those runs")
    ap.add_argument("--pmc-kernels", nargs="+", metavar="NAME",
                    help="restrict --pmc-summary to these kernels")
    ap.add_argument("--stats-summary", metavar="CSV",
                    help="print a rocprofv3 --stats kernel_stats CSV as a table and exit")
    ap.add_argument("--trace-kernel", nargs=3, metavar=("CSV", "NAME", "TOP"),
                    help="print the TOP largest dispatch durations of kernel NAME from a "
                         "rocprofv3 kernel_trace CSV and exit")
    args = ap.parse_args()
    if args.stats_summary:
        print(stats_summary(args.stats_summary))
        return 0
    if args.trace_kernel:
        print(trace_kernel(args.trace_kernel[0], args.trace_kernel[1], int(args.trace_kernel[2])))
        return 0
    if args.pmc_summary:
        if len(args.pmc_summary) < 2 or args.calib_copy <= 0:
            print("--pmc-summary needs the FETCH_SIZE and WRITE_SIZE CSVs and --calib-copy",
                  file=sys.stderr)
            return 2
        print(pmc_summary(args.pmc_summary[0], args.pmc_summary[1], args.calib_copy,
                          args.pmc_summary[2:], args.pmc_kernels))
        return 0
    if args.gpus != 1:
        print(f"bench.py: this benchmark runs on one GPU only (got --gpus {args.gpus}); the "
              "placement path has no multi-GPU mode", file=sys.stderr)
        return 2

    import torch

    import paper_2208_00184_amd as cel
    from workloads import make_config, perturb_placements

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.calib_copy > 0:
        nb = args.calib_copy << 20
        src = torch.ones(nb // 8, dtype=torch.int64, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy of {args.calib_copy} MiB done", file=sys.stderr, flush=True)
        del src, dst
    t0 = time.time()
    wl = make_config(4, args.seed)
    print(f"[bench] generated {wl.name}: n={wl.n} m={wl.m} in {time.time() - t0:.1f}s",
          file=sys.stderr, flush=True)
    g = cel.Graph.from_arrays(wl, dev)
    d = cel.Devices.from_arrays(wl)
    n, m = wl.n, wl.m
    stream = torch.cuda.current_stream()

    state = {}

    def step(record=None):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(7)]
        ev[0].record(stream)
        lev, oid, lp, L = cel.topo_levels(g)
        ev[1].record(stream)
        bl, _, pr, cp = cel.blevel(g, d, lev, lp, oid, L)
        ev[2].record(stream)
        cid, C, cut = cel.cluster(g, d, pr, 200, -1)
        ev[3].record(stream)
        cdev, ndev, cms, be = cel.place(g, d, cid, C)
        ev[4].record(stream)
        bl_info = cel.blevel_info()
        ms1, _, _ = cel.makespan(g, d, pr, lev, lp, L, ndev)
        ev[5].record(stream)
        ms_info = cel.makespan_info()
        if "cand" not in state:  # input prep for the batched row (random draws)
            cand = perturb_placements(cdev.cpu().numpy(), wl.D, BATCH, args.seed)
            candt = torch.from_numpy(cand).to(dev)
            state["cand"] = torch.gather(candt, 1, cid.long().unsqueeze(0).expand(BATCH, -1))
            state["cand"] = state["cand"].contiguous()
            torch.cuda.synchronize()
            ev[5].record(stream)
        msK, _, _ = cel.makespan(g, d, pr, lev, lp, L, state["cand"])
        ev[6].record(stream)
        torch.cuda.synchronize()
        if record is not None:
            names = ["topo_levels", "blevel", "cluster", "place", "makespan", "makespan_batch"]
            for i, nm in enumerate(names):
                record.setdefault(nm, []).append(ev[i].elapsed_time(ev[i + 1]))
        paths = ("policy iteration", "level sweep", "none", "batch")
        state["passes"] = {
            "blevel": {"path": paths[bl_info[0][0]], "iterations": bl_info[0][1]},
            "makespan": {"path": "relaxation" if ms_info[0] == 0 else paths[ms_info[0]],
                         "rounds": ms_info[1]}}
        state.update(L=L, C=C, cp=cp, cut=cut, cms=cms, be=be, ms1=int(ms1[0].item()), cdev=cdev.cpu().numpy(),
                     msK=msK.cpu().numpy(), cid=cid, ndev=ndev, pr=pr)

    for _ in range(args.warmup):
        step()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)
    cel.kernel_stats(reset=True)
    cel.timing(True)
    rec: dict = {}
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(rec)
        print(f"[bench] step {i + 1}/{args.steps}: {sum(v[-1] for v in rec.values()):.1f} ms",
              file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    cel.timing(False)
    kstats = cel.kernel_stats(reset=True)

    # t-level (optional output of the b-level call): one warm-up call (it
    # creates the side stream), then the median of 3 timed calls
    lev, oid, lp, L = cel.topo_levels(g)
    bl_t, tl_t, pr_t, _ = cel.blevel(g, d, lev, lp, oid, L, want_tlevel=True)
    torch.cuda.synchronize()
    cel.kernel_stats(reset=True)
    cel.timing(True)
    t_ms = []
    for _ in range(3):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        bl_t, tl_t, pr_t, _ = cel.blevel(g, d, lev, lp, oid, L, want_tlevel=True)
        e1.record(stream)
        torch.cuda.synchronize()
        t_ms.append(e0.elapsed_time(e1))
    cel.timing(False)
    ks_t = cel.kernel_stats(reset=True)
    tk = "k_tlevel_policy" if "k_tlevel_policy" in ks_t else "k_tlevel_sweep"
    launches, tot = ks_t.get(tk, (1, float("nan")))
    (pb_, ib_), (pt_, it_) = cel.blevel_info()
    tlevel_row = {"blevel_with_tlevel_ms": sorted(t_ms)[1], "kernel": tk,
                  "kernel_ms": tot / max(launches, 1),
                  "iterations": {"blevel": ib_ if pb_ == 0 else None, "tlevel": it_ if pt_ == 0 else None}}

    cpd_row, ndev_cpd, cid_cpd, C_cpd = cpd_compare(cel, torch, g, d, bl_t, tl_t, pr_t, lev, lp, L)
    model_row = None
    if not args.no_models:
        print("[bench] device models", file=sys.stderr, flush=True)
        model_row = models_row(cel, torch, g, d, pr_t, ndev_cpd, args.seed, cid=cid_cpd, C=C_cpd)

    batch5 = None if args.no_batch else batched_row(cel, torch, dev, args)

    stages = {k: float(np.mean(v)) for k, v in rec.items()}
    eval_ms = stages["blevel"] + stages["makespan"]
    value = m / (eval_ms * 1e-3)
    placement_gen_ms = stages["topo_levels"] + stages["blevel"] + stages["cluster"] + stages["place"]
    ms_per_step = wall * 1e3 / args.steps
    kernels = {k: {"launches_per_step": c / args.steps, "avg_ms": t / c} for k, (c, t) in
               kstats.items()}

    # roofline of the dominant kernel of the measured (b-level + makespan) pass
    dom = max((k for k in ("k_blevel_policy", "k_blevel_sweep", "k_makespan_one") if k in kernels),
              key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches_per_step"])
    B = algorithmic_bytes(dom, n, m, 1)
    t_dom = kernels[dom]["avg_ms"] * 1e-3
    achieved = B / t_dom / 1e9
    L = state["L"]
    roofline = {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 3),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 6),
                "traffic": load_traffic(dom), "algorithmic_bytes": B,
                "launch_ms": round(t_dom * 1e3, 4)}
    # how the pass ran: policy iterations of the b-level, relaxation rounds of
    # the makespan (each a few whole-GPU passes), against the floor of any
    # level-synchronous method: b-level and makespan as chains of L dependent
    # levels each, a level no faster than the dependent step the library's
    # probe measures on this GPU right now (one wave: LDS gather -> 64-bit
    # segmented max-plus DPP scan -> LDS write)
    roofline["passes"] = state.get("passes")
    probe = {name: round(cel.step_latency(v, 200000), 1)
             for v, name in ((0, "wave_lds_ns"), (1, "block_barrier_ns"), (2, "wave_l2_ns"))}
    t_level_ns = probe["wave_lds_ns"]
    B_pass = algorithmic_bytes("k_blevel_sweep", n, m, 1) + algorithmic_bytes("k_makespan_one",
                                                                              n, m, 1)
    floor_s = 2 * L * t_level_ns * 1e-9
    roofline["level_sync_floor"] = {
        "t_level_ns": t_level_ns, "probe": probe, "levels": L,
        "pass_floor_ms": round(floor_s * 1e3, 3),
        "frac_ceiling": round(B_pass / floor_s / 1e9 / HBM_PEAK_GBS, 5),
        "eval_ms": round(eval_ms, 3),
        "frac_pass": round(B_pass / (eval_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 6)}
    # the level sweeps are chains of L dependent levels: per-level latency
    per_level = {k: round(kernels[k]["avg_ms"] * 1e6 / L, 1)
                 for k in ("k_kahn", "k_blevel_sweep", "k_makespan_batch") if k in kernels}
    for k, v in kernels.items():
        b_ = algorithmic_bytes(k, n, m, BATCH if k == "k_makespan_batch" else 1)
        if b_ is not None:
            v["achieved_GBs"] = round(b_ / (v["avg_ms"] * 1e-3) / 1e9, 3)
            v["hbm_frac"] = round(b_ / (v["avg_ms"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 6)
    Bk = algorithmic_bytes("k_makespan_batch", n, m, BATCH)
    tk = kernels["k_makespan_batch"]["avg_ms"] * 1e-3
    batched = {"K": BATCH, "edges_per_s": BATCH * m / (stages["makespan_batch"] * 1e-3),
               "kernel_ms": kernels["k_makespan_batch"]["avg_ms"],
               "achieved_GBs": round(Bk / tk / 1e9, 2), "frac": round(Bk / tk / 1e9 / HBM_PEAK_GBS, 5)}
    if not args.no_batch:
        # 256 perturbed placements in one call: one workgroup per CU
        K2 = 256
        cand2 = perturb_placements(state["cdev"], wl.D, K2, args.seed + 1)
        cand2 = torch.from_numpy(cand2).to(dev)
        cand2 = torch.gather(cand2, 1, state["cid"].long().unsqueeze(0).expand(K2, -1)).contiguous()
        cel.makespan(g, d, state["pr"], lev, lp, L, cand2)  # warm-up
        cel.kernel_stats(reset=True)
        cel.timing(True)
        t2 = []
        for _ in range(3):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            cel.makespan(g, d, state["pr"], lev, lp, L, cand2)
            torch.cuda.synchronize()
            t2.append((time.perf_counter() - t0) * 1e3)
        cel.timing(False)
        cnt2, tot2 = cel.kernel_stats(reset=True)["k_makespan_batch"]
        k2 = tot2 / cnt2
        B2 = algorithmic_bytes("k_makespan_batch", n, m, K2)
        batched["K256"] = {"K": K2, "call_ms": round(sorted(t2)[1], 3), "kernel_ms": round(k2, 3),
                           "edges_per_s": K2 * m / (sorted(t2)[1] * 1e-3),
                           "achieved_GBs": round(B2 / (k2 * 1e-3) / 1e9, 2),
                           "frac": round(B2 / (k2 * 1e-3) / 1e9 / HBM_PEAK_GBS, 5)}
        del cand2

    cpu = None
    parity = None
    cfg_rows = None if args.no_configs else config_rows(cel, torch, dev, args)
    if not args.no_cpu:
        # the oracle as it stands, one thread pinned to one core, every stage of
        # the path on the same graph (median of 3)
        from oracle import oracle as O
        import statistics
        aff = os.sched_getaffinity(0)
        os.sched_setaffinity(0, {min(aff)})
        st_cpu = {}

        def tm(name, f, reps=3):
            ts, r = [], None
            for _ in range(reps):
                a = time.perf_counter()
                r = f()
                ts.append(time.perf_counter() - a)
            st_cpu[name] = round(statistics.median(ts) * 1e3, 1)
            return r

        try:
            lev_o, oid_o, _, _ = tm("topo_levels", lambda: O.topo_levels(wl))
            _, _, pr_o, cp_o = tm("blevel", lambda: O.blevel(wl, lev_o, oid_o))
            cid_o, C_o, cut_o = tm("cluster", lambda: O.cluster(wl, pr_o, 200, -1))
            pl_o = tm("place", lambda: O.place(wl, cid_o, C_o))
            ms_o = tm("makespan", lambda: O.makespan(wl, pr_o, pl_o[1], want_times=False))
        finally:
            os.sched_setaffinity(0, aff)
        # self-check: the timed GPU results against the oracle's on the same graph
        parity = check_parity({
            "critical_path_ns": (state["cp"], int(cp_o)), "clusters": (state["C"], int(C_o)),
            "cut_cost_ns": (state["cut"], int(cut_o)),
            "coarse_makespan_ns": (state["cms"], int(pl_o[2])),
            "best_effort": (state["be"], int(pl_o[3])), "makespan_ns": (state["ms1"], int(ms_o[0][0])),
            "prio_order": (state["pr"].cpu().numpy(), pr_o),
            "cluster_id": (state["cid"].cpu().numpy(), cid_o),
            "node_dev": (state["ndev"].cpu().numpy(), pl_o[1])})
        t_pass = (st_cpu["blevel"] + st_cpu["makespan"]) * 1e-3
        model = ""
        try:
            with open("/proc/cpuinfo") as fh:
                model = next(line.split(":", 1)[1].strip() for line in fh
                             if line.startswith("model name"))
        except (OSError, StopIteration):
            pass
        cpu = {"value": m / t_pass, "unit": "edges/s", "cores": 1, "kind": "oracle",
               "sample": f"b-level (with priority order) + makespan of the Adjusting Placement on "
                         f"the full {n}-node graph, median of 3, single-threaded C pinned to one "
                         f"core",
               "stages_ms": st_cpu,
               "placement_gen_ms": round(sum(st_cpu[k] for k in ("topo_levels", "blevel",
                                                                  "cluster", "place")), 1),
               "host": {"nproc": os.cpu_count(), "cpu_model": model,
                        "oracle_cores": f"1 of {len(aff)}"}}
        print(f"[bench] cpu oracle {t_pass * 1e3:.0f} ms per pass", file=sys.stderr, flush=True)

    props = torch.cuda.get_device_properties(0)
    device = {"name": props.name, "arch": getattr(props, "gcnArchName", ""),
              "compute_units": props.multi_processor_count,
              "memory_GB": round(props.total_memory / 1e9, 1), "hbm_peak_GBs": HBM_PEAK_GBS}

    out = {
        "metric": METRIC, "value": value, "unit": "edges/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": "transformer-96: 96-block fwd+bwd+Adam micro-op graph, hidden "
                               "8192, 64 heads, 32 column tiles", "n": n, "m": m,
                   "levels": L, "D": wl.D, "R": 200, "batch_K": BATCH, "seed": args.seed},
        "placement_gen_ms": placement_gen_ms,
        "eval_ms": eval_ms,
        "stages_ms": stages,
        "kernels": kernels,
        "roofline": roofline,
        "device": device,
        "ns_per_level": per_level,
        "tlevel": tlevel_row,
        "cpd_topo": cpd_row,
        "device_models": model_row,
        "batched_makespan": batched,
        "batched_scoring_200k": batch5,
        "cpu_baseline": cpu,
        "parity": parity,
        "configs": cfg_rows,
        "results": {"critical_path_ns": state["cp"], "clusters": state["C"],
                    "cut_cost_ns": state["cut"], "coarse_makespan_ns": state["cms"],
                    "best_effort": state["be"], "makespan_ns": state["ms1"],
                    "batch_makespan_min_ns": int(state["msK"].min())},
    }
    print(json.dumps(out))
    bad = [k for r in [parity] + [(c or {}).get("parity") for c in (cfg_rows or {}).values()] +
           [(batch5 or {}).get("parity")] if r for k, v in r.items() if v is False]
    if bad:
        print(f"[bench] PARITY MISMATCH against the oracle: {bad}", file=sys.stderr, flush=True)
        return 1
    return 0


if __name__ == "__main__":
    sys.exit(main())
