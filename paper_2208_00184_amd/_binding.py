"""Thin ctypes binding over libcel.so (the C ABI in include/cel.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  Arrays are torch tensors on a ROCm device; outputs are allocated
with torch on the same device and work is enqueued on the current torch
stream.  There is no CPU fallback: a missing library or a failed call raises.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcel.so")

OK, E_ARG, E_CYCLE, E_OVERFLOW, E_HIP, E_NOMEM, E_ORDER = 0, -1, -2, -3, -4, -5, -6
COMM_OFF = 1
CLUSTER_DP, CLUSTER_GREEDY = 0, 1

EXPORTS = ("cel_topo_levels", "cel_blevel", "cel_cpd_order", "cel_dfs_order", "cel_cluster", "cel_place", "cel_place_ext", "cel_makespan", "cel_makespan_noalloc",
           "cel_makespan_info", "cel_makespan_relax", "cel_blevel_info", "cel_policy_iteration",
           "cel_topo_levels_info", "cel_cluster_info",
           "cel_order_place", "cel_comm_sums", "cel_makespan_model", "cel_colocate", "cel_step_latency", "cel_timing", "cel_kernel_stats", "cel_last_error", "cel_version")


class CelError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libcel error {code}: {msg}")
        self.code = code


class _Graph(C.Structure):
    _fields_ = [("n", C.c_int32), ("m", C.c_int32),
                ("out_ptr", C.c_void_p), ("out_idx", C.c_void_p),
                ("in_ptr", C.c_void_p), ("in_idx", C.c_void_p),
                ("w", C.c_void_p), ("mem", C.c_void_p), ("ob", C.c_void_p)]


class _Hetero(C.Structure):
    _fields_ = [("tmul", C.POINTER(C.c_int64)), ("bw", C.POINTER(C.c_int64)),
                ("lat", C.POINTER(C.c_int64))]


class _Devices(C.Structure):
    _fields_ = [("D", C.c_int32), ("cap", C.POINTER(C.c_int64)),
                ("bw", C.c_int64), ("lat", C.c_int64)]


_lib = None


def lib() -> C.CDLL:
    """Load libcel.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run __graft_entry__.build() "
                               "(or python -m paper_2208_00184_amd.build) first")
        L = C.CDLL(LIB_PATH)
        vp, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
        G, Dv = C.POINTER(_Graph), C.POINTER(_Devices)
        L.cel_topo_levels.argtypes = [G, vp, vp, vp, C.POINTER(i32), vp]
        L.cel_blevel.argtypes = [G, Dv, vp, vp, vp, i32, i32, vp, vp, vp, C.POINTER(i64), vp]
        L.cel_cluster.argtypes = [G, Dv, vp, i32, i64, i32, vp, C.POINTER(i32), C.POINTER(i64), vp]
        L.cel_place.argtypes = [G, Dv, vp, i32, vp, vp, vp, C.POINTER(i64), C.POINTER(i32), vp]
        L.cel_place_ext.argtypes = [G, Dv, C.POINTER(_Hetero), vp, i32, vp, i32, vp, vp, vp,
                                    C.POINTER(i64), C.POINTER(i32), vp]
        L.cel_makespan.argtypes = [G, Dv, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp]
        L.cel_makespan_noalloc.argtypes = [G, Dv, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp]
        L.cel_cpd_order.argtypes = [G, vp, vp, vp, vp]
        L.cel_dfs_order.argtypes = [G, vp, vp]
        L.cel_order_place.argtypes = [G, Dv, vp, i32, vp, vp, C.POINTER(i32), vp]
        L.cel_comm_sums.argtypes = [G, Dv, vp, C.POINTER(i64), C.POINTER(i64), vp]
        L.cel_makespan_model.argtypes = [G, Dv, C.POINTER(_Hetero), vp, i32, vp, i32, vp, vp, vp, vp]
        L.cel_colocate.argtypes = [G, vp, vp, i32, i32, vp, vp]
        for f in ("cel_topo_levels", "cel_blevel", "cel_cluster", "cel_place", "cel_place_ext",
                  "cel_makespan",
                  "cel_makespan_noalloc",
                  "cel_cpd_order", "cel_dfs_order", "cel_order_place", "cel_comm_sums", "cel_makespan_model",
                  "cel_colocate", "cel_version"):
            getattr(L, f).restype = C.c_int
        L.cel_last_error.argtypes = []
        L.cel_last_error.restype = C.c_char_p
        L.cel_step_latency.argtypes = [i32, i32, C.POINTER(C.c_double), vp]
        L.cel_step_latency.restype = C.c_int
        L.cel_timing.argtypes = [C.c_int]
        L.cel_timing.restype = C.c_int
        L.cel_kernel_stats.argtypes = [C.c_char_p, C.c_int, C.c_int]
        L.cel_kernel_stats.restype = C.c_int
        L.cel_makespan_info.argtypes = [C.POINTER(i32), C.POINTER(i32)]
        L.cel_makespan_info.restype = C.c_int
        L.cel_makespan_relax.argtypes = [C.c_int]
        L.cel_makespan_relax.restype = C.c_int
        L.cel_blevel_info.argtypes = [C.POINTER(i32)]
        L.cel_blevel_info.restype = C.c_int
        L.cel_policy_iteration.argtypes = [C.c_int]
        L.cel_policy_iteration.restype = C.c_int
        L.cel_topo_levels_info.argtypes = [C.POINTER(i32)]
        L.cel_topo_levels_info.restype = C.c_int
        L.cel_cluster_info.argtypes = [C.POINTER(i32)]
        L.cel_cluster_info.restype = C.c_int
        _lib = L
    return _lib


def version() -> int:
    return lib().cel_version()


def step_latency(variant: int = 0, steps: int = 200000) -> float:
    """ns per dependent gather -> wave scan -> write step (variant 0: one wave
    over LDS; 1: 1024 threads with a barrier; 2: one wave gathering from L2)."""
    ns = C.c_double(0.0)
    _check(lib().cel_step_latency(int(variant), int(steps), C.byref(ns), _stream()))
    return ns.value


MS_PATH_RELAX, MS_PATH_SWEEP, MS_PATH_BATCH = 0, 1, 2


def makespan_info() -> tuple:
    """(path, rounds) of the calling thread's last makespan call: path 0 =
    relaxation over cross-device edges (exact after `rounds` rounds), 1 = the
    level sweep (after `rounds` relaxation rounds that did not converge), 2 =
    a batch (K > 1)."""
    path, rounds = C.c_int32(0), C.c_int32(0)
    _check(lib().cel_makespan_info(C.byref(path), C.byref(rounds)))
    return path.value, rounds.value


def makespan_relax(mode: int) -> int:
    """K = 1 makespan path of the calling thread: 0 = the level sweep, 1 = the
    relaxation first (default), m >= 2 = the relaxation on at most m
    workgroups; returns the previous mode."""
    r = lib().cel_makespan_relax(int(mode))
    if r < 0:
        _check(r)
    return r


LP_POLICY, LP_SWEEP, LP_NONE = 0, 1, 2


def blevel_info() -> tuple:
    """((path, iterations) of the b-level, (path, iterations) of the t-level)
    of the calling thread's last blevel call: path 0 = policy iteration, 1 =
    the level sweep, 2 = not requested."""
    info = (C.c_int32 * 4)()
    _check(lib().cel_blevel_info(info))
    return (info[0], info[1]), (info[2], info[3])


def topo_levels_info() -> tuple:
    """(path, iterations) of the calling thread's last topo_levels call: path
    0 = policy iteration, 1 = Kahn's level-synchronous kernel."""
    info = (C.c_int32 * 2)()
    _check(lib().cel_topo_levels_info(info))
    return info[0], info[1]


def cluster_info() -> tuple:
    """(path, iterations) of the calling thread's last cluster call (DP mode):
    path 0 = policy iteration, 1 = the blocked DP."""
    info = (C.c_int32 * 2)()
    _check(lib().cel_cluster_info(info))
    return info[0], info[1]


def policy_iteration(mode: int) -> int:
    """Levels, b-level, t-level and clustering-DP path of the calling thread:
    0 = Kahn's kernel, the level sweeps and the blocked DP, 1 = policy
    iteration first (default; packed entries and asynchronous pointer jumping
    where the values fit), 2 = policy iteration first with 16-byte entries and
    synchronous rounds; returns the previous mode."""
    r = lib().cel_policy_iteration(int(mode))
    if r < 0:
        _check(r)
    return r


def timing(enable: bool) -> bool:
    """Turn per-kernel event timing on/off; returns the previous setting."""
    return bool(lib().cel_timing(1 if enable else 0))


def kernel_stats(reset: bool = False) -> dict:
    """{kernel name: (launches, total_ms)} accumulated since the last reset."""
    buf = C.create_string_buffer(1 << 16)
    lib().cel_kernel_stats(buf, len(buf), 1 if reset else 0)
    out = {}
    for line in buf.value.decode().splitlines():
        name, cnt, ms = line.split()
        out[name] = (int(cnt), float(ms))
    return out


def _check(rc: int):
    if rc != OK:
        raise CelError(rc, lib().cel_last_error().decode(errors="replace"))


def _p(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


@dataclass
class Graph:
    """Device-resident operator DAG (int32 CSR/CSC, int64 w/mem/ob)."""
    n: int
    m: int
    out_ptr: torch.Tensor
    out_idx: torch.Tensor
    in_ptr: torch.Tensor
    in_idx: torch.Tensor
    w: torch.Tensor
    mem: torch.Tensor
    ob: torch.Tensor

    @staticmethod
    def from_arrays(wl, device="cuda") -> "Graph":
        """From any object with numpy fields n, m, out_ptr, ... (e.g. a Workload)."""
        def t(a, dt):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=dt)).to(device)
        return Graph(int(wl.n), int(wl.m), t(wl.out_ptr, np.int32), t(wl.out_idx, np.int32),
                     t(wl.in_ptr, np.int32), t(wl.in_idx, np.int32), t(wl.w, np.int64),
                     t(wl.mem, np.int64), t(wl.ob, np.int64))

    @property
    def device(self):
        return self.out_ptr.device

    def _c(self) -> _Graph:
        return _Graph(self.n, self.m, self.out_ptr.data_ptr(), self.out_idx.data_ptr(),
                      self.in_ptr.data_ptr(), self.in_idx.data_ptr(), self.w.data_ptr(),
                      self.mem.data_ptr(), self.ob.data_ptr())


@dataclass
class Devices:
    """Modelled target devices: count, host memory caps, link bw (B/ns) and latency (ns)."""
    D: int
    cap: np.ndarray
    bw: int
    lat: int

    @staticmethod
    def from_arrays(wl) -> "Devices":
        return Devices(int(wl.D), np.ascontiguousarray(wl.cap, np.int64), int(wl.bw), int(wl.lat))

    def _c(self) -> _Devices:
        self._cap = np.ascontiguousarray(self.cap, np.int64)  # keep alive during the call
        return _Devices(int(self.D), self._cap.ctypes.data_as(C.POINTER(C.c_int64)),
                        int(self.bw), int(self.lat))


def _empty(n, dtype, device):
    return torch.empty(max(int(n), 1), dtype=dtype, device=device)


def topo_levels(g: Graph):
    """-> (level int32[n], order_id int32[n], level_ptr int32[L+1], L)"""
    n = g.n
    level = _empty(n, torch.int32, g.device)
    order = _empty(n, torch.int32, g.device)
    lptr = torch.empty(n + 1, dtype=torch.int32, device=g.device)
    L = C.c_int32(0)
    gc = g._c()
    _check(lib().cel_topo_levels(C.byref(gc), _p(level), _p(order), _p(lptr), C.byref(L),
                                 _stream()))
    return level[:n], order[:n], lptr[:L.value + 1], L.value


def blevel(g: Graph, d: Devices, level, level_ptr, order_id, n_levels, comm_off=False,
           want_tlevel=False, want_prio=True):
    """-> (blevel int64[n], tlevel int64[n] | None, prio_order int32[n] | None, cp)"""
    n = g.n
    bl = _empty(n, torch.int64, g.device)
    tl = _empty(n, torch.int64, g.device) if want_tlevel else None
    pr = _empty(n, torch.int32, g.device) if want_prio else None
    cp = C.c_int64(0)
    gc, dc = g._c(), d._c()
    _check(lib().cel_blevel(C.byref(gc), C.byref(dc), _p(level), _p(level_ptr), _p(order_id),
                            int(n_levels), COMM_OFF if comm_off else 0, _p(bl), _p(tl), _p(pr),
                            C.byref(cp), _stream()))
    return bl[:n], (tl[:n] if tl is not None else None), (pr[:n] if pr is not None else None), \
        cp.value


def cpd_order(g: Graph, blevel_, tlevel_):
    """CPD-TOPO order (Algorithm 1) from b-/t-levels -> int32[n] node ids."""
    n = g.n
    out = _empty(n, torch.int32, g.device)
    gc = g._c()
    _check(lib().cel_cpd_order(C.byref(gc), _p(blevel_), _p(tlevel_), _p(out), _stream()))
    return out[:n]


def dfs_order(g: Graph):
    """DFS-TOPO order (Section 4.2.2) -> int32[n] node ids."""
    n = g.n
    out = _empty(n, torch.int32, g.device)
    gc = g._c()
    _check(lib().cel_dfs_order(C.byref(gc), _p(out), _stream()))
    return out[:n]


def cluster(g: Graph, d: Devices, order, R=200, M=-1, mode=CLUSTER_DP):
    """-> (cluster_id int32[n], n_clusters, cut_cost)"""
    n = g.n
    cid = _empty(n, torch.int32, g.device)
    nc = C.c_int32(0)
    cut = C.c_int64(0)
    gc, dc = g._c(), d._c()
    _check(lib().cel_cluster(C.byref(gc), C.byref(dc), _p(order), int(R), int(M), int(mode),
                             _p(cid), C.byref(nc), C.byref(cut), _stream()))
    return cid[:n], nc.value, cut.value


def place(g: Graph, d: Devices, cluster_id, n_clusters, want_fin=False):
    """-> (cluster_dev uint8[C], node_dev uint8[n], coarse_makespan, best_effort_count)
    plus cluster_fin int64[C] when ``want_fin``."""
    n = g.n
    cdev = _empty(n_clusters, torch.uint8, g.device)
    ndev = _empty(n, torch.uint8, g.device)
    fin = _empty(n_clusters, torch.int64, g.device) if want_fin else None
    span = C.c_int64(0)
    be = C.c_int32(0)
    gc, dc = g._c(), d._c()
    _check(lib().cel_place(C.byref(gc), C.byref(dc), _p(cluster_id), int(n_clusters), _p(cdev),
                           _p(ndev), _p(fin), C.byref(span), C.byref(be), _stream()))
    out = (cdev[:n_clusters], ndev[:n], span.value, be.value)
    return out + (fin[:n_clusters],) if want_fin else out


def order_place(g: Graph, d: Devices, cluster_id, n_clusters):
    """Order-Place -> (cluster_dev uint8[C], node_dev uint8[n], best_effort_count)"""
    n = g.n
    cdev = _empty(n_clusters, torch.uint8, g.device)
    ndev = _empty(n, torch.uint8, g.device)
    be = C.c_int32(0)
    gc, dc = g._c(), d._c()
    _check(lib().cel_order_place(C.byref(gc), C.byref(dc), _p(cluster_id), int(n_clusters), _p(cdev),
                                 _p(ndev), C.byref(be), _stream()))
    return cdev[:n_clusters], ndev[:n], be.value


MODEL_INSERT, MODEL_COMM_TASKS, MODEL_COMM_BLOCK = 1, 2, 4


def _hetero(tmul, bw, lat, keep):
    """cel_hetero over host copies (kept alive in `keep`), or None."""
    if tmul is None and bw is None and lat is None:
        return None
    ptrs = []
    for a in (tmul, bw, lat):
        if a is None:
            ptrs.append(None)
            continue
        arr = (C.c_int64 * int(np.asarray(a).size))(*[int(x) for x in np.asarray(a).reshape(-1)])
        keep.append(arr)
        ptrs.append(C.cast(arr, C.POINTER(C.c_int64)))
    return _Hetero(*ptrs)


def place_ext(g: Graph, d: Devices, cluster_id, n_clusters, tmul=None, bw=None, lat=None,
              group=None, n_groups=0):
    """Adjusting Placement with heterogeneous devices/links (host tmul [D], bw / lat
    [D, D]) and co-location groups (device int32 [n] in [-1, n_groups)) inside the
    algorithm -> (cluster_dev, node_dev, coarse_makespan, best_effort_count, cluster_fin)."""
    keep = []
    het = _hetero(tmul, bw, lat, keep)
    n = g.n
    cdev = _empty(n_clusters, torch.uint8, g.device)
    ndev = _empty(n, torch.uint8, g.device)
    fin = _empty(n_clusters, torch.int64, g.device)
    span = C.c_int64(0)
    be = C.c_int32(0)
    gc, dc = g._c(), d._c()
    _check(lib().cel_place_ext(C.byref(gc), C.byref(dc), None if het is None else C.byref(het),
                               _p(group), int(n_groups), _p(cluster_id), int(n_clusters), _p(cdev),
                               _p(ndev), _p(fin), C.byref(span), C.byref(be), _stream()))
    return cdev[:n_clusters], ndev[:n], span.value, be.value, fin[:n_clusters]


def makespan_model(g: Graph, d: Devices, order, node_dev, model, want_times=False, tmul=None,
                   bw=None, lat=None):
    """Makespan under the device models (MODEL_* bits; 0 = FIFO devices, contention-free
    comm). node_dev uint8 [n] or [K, n] -> (makespan int64[K], start, finish) ([K, n] or None).
    tmul [D], bw / lat [D, D]: heterogeneous devices (host values, time x tmul / 1024)."""
    keep = []
    het = _hetero(tmul, bw, lat, keep)
    n = g.n
    nd = node_dev.contiguous()
    K = 1 if nd.dim() == 1 else nd.shape[0]
    ms = torch.empty(K, dtype=torch.int64, device=g.device)
    st = torch.empty((K, max(n, 1)), dtype=torch.int64, device=g.device) if want_times else None
    fi = torch.empty((K, max(n, 1)), dtype=torch.int64, device=g.device) if want_times else None
    gc, dc = g._c(), d._c()
    _check(lib().cel_makespan_model(C.byref(gc), C.byref(dc), None if het is None else C.byref(het),
                                    _p(order), int(K), _p(nd), int(model), _p(st), _p(fi), _p(ms),
                                    _stream()))
    if want_times:
        st, fi = st[:, :n], fi[:, :n]
    return ms, st, fi


def colocate(g: Graph, order, group, n_groups, node_dev):
    """Co-location groups: node_dev (uint8 [n] or [K, n], device) rewritten in place so that
    every group follows its first node in `order`; returns node_dev."""
    nd = node_dev
    assert nd.is_contiguous()
    K = 1 if nd.dim() == 1 else nd.shape[0]
    gc = g._c()
    _check(lib().cel_colocate(C.byref(gc), _p(order), _p(group), int(n_groups), int(K), _p(nd),
                              _stream()))
    return nd


def comm_sums(g: Graph, d: Devices, cluster_id=None):
    """CCR parts (eq. 1) -> (edge comm, total w); with cluster_id only edges between clusters."""
    ec = C.c_int64(0)
    ws = C.c_int64(0)
    gc, dc = g._c(), d._c()
    _check(lib().cel_comm_sums(C.byref(gc), C.byref(dc), _p(cluster_id), C.byref(ec), C.byref(ws),
                               _stream()))
    return ec.value, ws.value


def makespan(g: Graph, d: Devices, order, level, level_ptr, n_levels, node_dev, want_times=False,
             noalloc=False):
    """node_dev uint8 [n] or [K, n] -> (makespan int64[K], start, finish) ([K, n] or None).
    noalloc=True calls cel_makespan_noalloc (the library allocates nothing;
    the outputs are still allocated here by torch)."""
    n = g.n
    nd = node_dev.contiguous()
    K = 1 if nd.dim() == 1 else nd.shape[0]
    ms = torch.empty(K, dtype=torch.int64, device=g.device)
    st = torch.empty((K, max(n, 1)), dtype=torch.int64, device=g.device) if want_times else None
    fi = torch.empty((K, max(n, 1)), dtype=torch.int64, device=g.device) if want_times else None
    gc, dc = g._c(), d._c()
    f = lib().cel_makespan_noalloc if noalloc else lib().cel_makespan
    _check(f(C.byref(gc), C.byref(dc), _p(order), _p(level), _p(level_ptr), int(n_levels), int(K),
             _p(nd), _p(st), _p(fi), _p(ms), _stream()))
    if want_times:
        st, fi = st[:, :n], fi[:, :n]
    return ms, st, fi
