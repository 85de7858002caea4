"""ctypes wrapper over the CPU oracle (oracle/libcel_oracle.so).

Test infrastructure only.  Every function takes host numpy arrays (a
``workloads.Workload`` or any object with the same fields) and returns numpy
arrays; a nonzero status from the C code raises :class:`OracleError`.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import build as _build

OK, E_ARG, E_CYCLE, E_OVERFLOW, E_ORDER = 0, -1, -2, -3, -6
COMM_OFF = 1
DP, GREEDY, DP_DIRECT = 0, 1, 2

_P32 = C.POINTER(C.c_int32)
_P64 = C.POINTER(C.c_int64)
_PU8 = C.POINTER(C.c_uint8)


class OracleError(RuntimeError):
    def __init__(self, code, fn):
        super().__init__(f"{fn} returned {code}")
        self.code = code


class _Graph(C.Structure):
    _fields_ = [("n", C.c_int32), ("m", C.c_int32),
                ("out_ptr", _P32), ("out_idx", _P32),
                ("in_ptr", _P32), ("in_idx", _P32),
                ("w", _P64), ("mem", _P64), ("ob", _P64)]


class _Devices(C.Structure):
    _fields_ = [("D", C.c_int32), ("cap", _P64), ("bw", C.c_int64), ("lat", C.c_int64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        L = C.CDLL(_build.LIB)
        L.orc_topo_levels.argtypes = [C.POINTER(_Graph), _P32, _P32, _P32, _P32]
        L.orc_blevel.argtypes = [C.POINTER(_Graph), C.POINTER(_Devices), _P32, _P32, C.c_int32,
                                 _P64, _P64, _P32, _P64]
        L.orc_cluster.argtypes = [C.POINTER(_Graph), C.POINTER(_Devices), _P32, C.c_int32,
                                  C.c_int64, C.c_int32, _P32, _P32, _P64]
        L.orc_place.argtypes = [C.POINTER(_Graph), C.POINTER(_Devices), _P32, C.c_int32,
                                _PU8, _PU8, _P64, _P64, _P32]
        L.orc_makespan.argtypes = [C.POINTER(_Graph), C.POINTER(_Devices), _P32, C.c_int32,
                                   _PU8, _P64, _P64, _P64]
        L.orc_cpd_topo.argtypes = [C.POINTER(_Graph), _P64, _P64, _P32]
        L.orc_dfs_topo.argtypes = [C.POINTER(_Graph), _P32]
        L.orc_comm_sums.argtypes = [C.POINTER(_Graph), C.POINTER(_Devices), _P32,
                                    C.POINTER(C.c_int64), C.POINTER(C.c_int64)]
        L.orc_order_place.argtypes = [C.POINTER(_Graph), C.POINTER(_Devices), _P32, C.c_int32,
                                      _PU8, _PU8, C.POINTER(C.c_int32)]
        L.orc_makespan_model.argtypes = [C.POINTER(_Graph), C.POINTER(_Devices),
                                         C.POINTER(_Hetero), _P32, C.c_int32, _PU8, C.c_int32,
                                         _P64, _P64, _P64]
        L.orc_colocate.argtypes = [C.POINTER(_Graph), _P32, _P32, C.c_int32, C.c_int32, _PU8]
        L.orc_place_ext.argtypes = [C.POINTER(_Graph), C.POINTER(_Devices), C.POINTER(_Hetero),
                                    _P32, C.c_int32, _P32, C.c_int32, _PU8, _PU8, _P64,
                                    C.POINTER(C.c_int64), C.POINTER(C.c_int32)]
        for f in (L.orc_topo_levels, L.orc_blevel, L.orc_cluster, L.orc_place, L.orc_makespan,
                  L.orc_cpd_topo, L.orc_dfs_topo, L.orc_comm_sums, L.orc_order_place, L.orc_makespan_model,
                  L.orc_colocate, L.orc_place_ext):
            f.restype = C.c_int
        _lib = L
    return _lib


def _ptr(a, t):
    if a is None:
        return C.cast(None, t)
    return a.ctypes.data_as(t)


class _Keep:
    """Holds contiguous copies alive while a call is in flight."""

    def __init__(self, wl):
        self.arrs = dict(
            out_ptr=np.ascontiguousarray(wl.out_ptr, np.int32),
            out_idx=np.ascontiguousarray(wl.out_idx, np.int32),
            in_ptr=np.ascontiguousarray(wl.in_ptr, np.int32),
            in_idx=np.ascontiguousarray(wl.in_idx, np.int32),
            w=np.ascontiguousarray(wl.w, np.int64),
            mem=np.ascontiguousarray(wl.mem, np.int64),
            ob=np.ascontiguousarray(wl.ob, np.int64),
            cap=np.ascontiguousarray(wl.cap, np.int64))
        a = self.arrs
        self.g = _Graph(int(wl.n), int(wl.m), _ptr(a["out_ptr"], _P32), _ptr(a["out_idx"], _P32),
                        _ptr(a["in_ptr"], _P32), _ptr(a["in_idx"], _P32),
                        _ptr(a["w"], _P64), _ptr(a["mem"], _P64), _ptr(a["ob"], _P64))
        self.d = _Devices(int(wl.D), _ptr(a["cap"], _P64), int(wl.bw), int(wl.lat))


def _check(rc, fn):
    if rc != OK:
        raise OracleError(rc, fn)


def topo_levels(wl):
    """-> (level int32[n], order_id int32[n], level_ptr int32[L+1], L)"""
    k = _Keep(wl)
    n = int(wl.n)
    level = np.zeros(max(n, 1), np.int32)
    order = np.zeros(max(n, 1), np.int32)
    lptr = np.zeros(n + 1, np.int32)
    L = C.c_int32(0)
    _check(lib().orc_topo_levels(C.byref(k.g), _ptr(level, _P32), _ptr(order, _P32),
                                 _ptr(lptr, _P32), C.byref(L)), "orc_topo_levels")
    return level[:n], order[:n], lptr[:L.value + 1].copy(), L.value


def blevel(wl, level, order_id, comm_off=False, want_tlevel=True, want_prio=True):
    """-> (blevel int64[n], tlevel int64[n] | None, prio int32[n] | None, cp)"""
    k = _Keep(wl)
    n = int(wl.n)
    level = np.ascontiguousarray(level, np.int32)
    order_id = np.ascontiguousarray(order_id, np.int32)
    bl = np.zeros(max(n, 1), np.int64)
    tl = np.zeros(max(n, 1), np.int64) if want_tlevel else None
    pr = np.zeros(max(n, 1), np.int32) if want_prio else None
    cp = C.c_int64(0)
    _check(lib().orc_blevel(C.byref(k.g), C.byref(k.d), _ptr(level, _P32), _ptr(order_id, _P32),
                            COMM_OFF if comm_off else 0, _ptr(bl, _P64), _ptr(tl, _P64),
                            _ptr(pr, _P32), C.byref(cp)), "orc_blevel")
    return (bl[:n], None if tl is None else tl[:n], None if pr is None else pr[:n], cp.value)


def cpd_topo(wl, blevel, tlevel):
    """CPD-TOPO order (Algorithm 1) from the given b-/t-levels -> int32[n] node ids."""
    k = _Keep(wl)
    n = int(wl.n)
    bl = np.ascontiguousarray(blevel, np.int64)
    tl = np.ascontiguousarray(tlevel, np.int64)
    out = np.zeros(max(n, 1), np.int32)
    _check(lib().orc_cpd_topo(C.byref(k.g), _ptr(bl, _P64), _ptr(tl, _P64), _ptr(out, _P32)),
           "orc_cpd_topo")
    return out[:n]


def dfs_topo(wl):
    """DFS-TOPO order (Section 4.2.2) -> int32[n] node ids."""
    k = _Keep(wl)
    n = int(wl.n)
    out = np.zeros(max(n, 1), np.int32)
    _check(lib().orc_dfs_topo(C.byref(k.g), _ptr(out, _P32)), "orc_dfs_topo")
    return out[:n]


def comm_sums(wl, cluster_id=None):
    """CCR parts (eq. 1) -> (edge comm, total w); with cluster_id only edges between clusters."""
    k = _Keep(wl)
    cid = None if cluster_id is None else np.ascontiguousarray(cluster_id, np.int32)
    ec, ws = C.c_int64(0), C.c_int64(0)
    _check(lib().orc_comm_sums(C.byref(k.g), C.byref(k.d), _ptr(cid, _P32), C.byref(ec),
                               C.byref(ws)), "orc_comm_sums")
    return ec.value, ws.value


def order_place(wl, cluster_id, n_clusters):
    """Order-Place -> (cluster_dev uint8[C], node_dev uint8[n], best_effort_count)."""
    k = _Keep(wl)
    n = int(wl.n)
    cid = np.ascontiguousarray(cluster_id, np.int32)
    cdev = np.zeros(max(n_clusters, 1), np.uint8)
    ndev = np.zeros(max(n, 1), np.uint8)
    be = C.c_int32(0)
    _check(lib().orc_order_place(C.byref(k.g), C.byref(k.d), _ptr(cid, _P32), int(n_clusters),
                                 _ptr(cdev, _PU8), _ptr(ndev, _PU8), C.byref(be)), "orc_order_place")
    return cdev[:n_clusters], ndev[:n], be.value


def cluster(wl, order, R=200, M=-1, mode=DP):
    """-> (cluster_id int32[n], C, cut_cost)"""
    k = _Keep(wl)
    n = int(wl.n)
    order = np.ascontiguousarray(order, np.int32)
    cid = np.zeros(max(n, 1), np.int32)
    nc = C.c_int32(0)
    cut = C.c_int64(0)
    _check(lib().orc_cluster(C.byref(k.g), C.byref(k.d), _ptr(order, _P32), int(R), int(M),
                             int(mode), _ptr(cid, _P32), C.byref(nc), C.byref(cut)),
           "orc_cluster")
    return cid[:n], nc.value, cut.value


def place(wl, cluster_id, n_clusters, want_fin=False):
    """-> (cluster_dev uint8[C], node_dev uint8[n], coarse_makespan, best_effort_count)
    plus cluster_fin int64[C] when ``want_fin``."""
    k = _Keep(wl)
    n = int(wl.n)
    cid = np.ascontiguousarray(cluster_id, np.int32)
    cdev = np.zeros(max(n_clusters, 1), np.uint8)
    ndev = np.zeros(max(n, 1), np.uint8)
    fin = np.zeros(max(n_clusters, 1), np.int64) if want_fin else None
    span = C.c_int64(0)
    be = C.c_int32(0)
    _check(lib().orc_place(C.byref(k.g), C.byref(k.d), _ptr(cid, _P32), int(n_clusters),
                           _ptr(cdev, _PU8), _ptr(ndev, _PU8), _ptr(fin, _P64),
                           C.byref(span), C.byref(be)), "orc_place")
    out = (cdev[:n_clusters], ndev[:n], span.value, be.value)
    return out + (fin[:n_clusters],) if want_fin else out


def place_ext(wl, cluster_id, n_clusters, tmul=None, bw=None, lat=None, group=None,
              n_groups=0):
    """Adjusting Placement with heterogeneous devices/links (tmul [D], bw / lat
    [D, D]) and co-location groups (group [n] in [-1, n_groups)) inside the
    algorithm -> (cluster_dev, node_dev, coarse_makespan, best_effort_count,
    cluster_fin)."""
    k = _Keep(wl)
    het = None
    if tmul is not None or bw is not None or lat is not None:
        arrs = [None if a is None else np.ascontiguousarray(a, np.int64).reshape(-1)
                for a in (tmul, bw, lat)]
        k.het_arrays = arrs
        het = _Hetero(*[_ptr(a, _P64) for a in arrs])
    n = int(wl.n)
    cid = np.ascontiguousarray(cluster_id, np.int32)
    grp = None if group is None else np.ascontiguousarray(group, np.int32)
    cdev = np.zeros(max(n_clusters, 1), np.uint8)
    ndev = np.zeros(max(n, 1), np.uint8)
    fin = np.zeros(max(n_clusters, 1), np.int64)
    span = C.c_int64(0)
    be = C.c_int32(0)
    _check(lib().orc_place_ext(C.byref(k.g), C.byref(k.d), None if het is None else C.byref(het),
                               _ptr(grp, _P32), int(n_groups), _ptr(cid, _P32), int(n_clusters),
                               _ptr(cdev, _PU8), _ptr(ndev, _PU8), _ptr(fin, _P64),
                               C.byref(span), C.byref(be)), "orc_place_ext")
    return cdev[:n_clusters], ndev[:n], span.value, be.value, fin[:n_clusters]


def makespan(wl, order, node_dev, want_times=True):
    """node_dev uint8 [n] or [K, n] -> (makespan int64[K], start, finish) ([K, n] or None)"""
    k = _Keep(wl)
    n = int(wl.n)
    nd = np.ascontiguousarray(node_dev, np.uint8)
    K = 1 if nd.ndim == 1 else nd.shape[0]
    nd = nd.reshape(K, n) if n > 0 else np.zeros((K, 1), np.uint8)
    order = np.ascontiguousarray(order, np.int32)
    st = np.zeros((K, max(n, 1)), np.int64) if want_times else None
    fi = np.zeros((K, max(n, 1)), np.int64) if want_times else None
    ms = np.zeros(K, np.int64)
    _check(lib().orc_makespan(C.byref(k.g), C.byref(k.d), _ptr(order, _P32), K, _ptr(nd, _PU8),
                              _ptr(st, _P64), _ptr(fi, _P64), _ptr(ms, _P64)), "orc_makespan")
    if want_times:
        st, fi = st[:, :n], fi[:, :n]
    return ms, st, fi


MODEL_INSERT, MODEL_COMM_TASKS, MODEL_COMM_BLOCK = 1, 2, 4


class _Hetero(C.Structure):
    _fields_ = [("tmul", _P64), ("bw", _P64), ("lat", _P64)]


def makespan_model(wl, order, node_dev, model, want_times=True, tmul=None, bw=None, lat=None):
    """Makespan under the device models (bits MODEL_INSERT, MODEL_COMM_TASKS, or
    MODEL_COMM_BLOCK alone; 0 is makespan()'s schedule) -> (makespan int64[K], start, finish) ([K, n] or None).
    tmul [D] (compute time x tmul / 1024), bw / lat [D, D] (link a -> b): heterogeneous
    devices; all None = homogeneous."""
    k = _Keep(wl)
    het = None
    if tmul is not None or bw is not None or lat is not None:
        arrs = [None if a is None else np.ascontiguousarray(a, np.int64).reshape(-1)
                for a in (tmul, bw, lat)]
        k.het_arrays = arrs
        het = _Hetero(*[_ptr(a, _P64) for a in arrs])
    n = int(wl.n)
    nd = np.ascontiguousarray(node_dev, np.uint8)
    K = 1 if nd.ndim == 1 else nd.shape[0]
    nd = nd.reshape(K, n) if n > 0 else np.zeros((K, 1), np.uint8)
    order = np.ascontiguousarray(order, np.int32)
    st = np.zeros((K, max(n, 1)), np.int64) if want_times else None
    fi = np.zeros((K, max(n, 1)), np.int64) if want_times else None
    ms = np.zeros(K, np.int64)
    _check(lib().orc_makespan_model(C.byref(k.g), C.byref(k.d),
                                    None if het is None else C.byref(het), _ptr(order, _P32), K,
                                    _ptr(nd, _PU8), int(model), _ptr(st, _P64), _ptr(fi, _P64),
                                    _ptr(ms, _P64)), "orc_makespan_model")
    if want_times:
        st, fi = st[:, :n], fi[:, :n]
    return ms, st, fi


def colocate(wl, order, group, n_groups, node_dev):
    """Co-location: returns node_dev ([n] or [K, n], a copy) with every group on its
    first node's (in order) device."""
    k = _Keep(wl)
    n = int(wl.n)
    nd = np.array(node_dev, np.uint8, copy=True)
    shape = nd.shape
    K = 1 if nd.ndim == 1 else nd.shape[0]
    nd = np.ascontiguousarray(nd.reshape(K, n) if n > 0 else np.zeros((K, 1), np.uint8))
    order = np.ascontiguousarray(order, np.int32)
    grp = np.ascontiguousarray(group, np.int32)
    _check(lib().orc_colocate(C.byref(k.g), _ptr(order, _P32), _ptr(grp, _P32), int(n_groups), K,
                              _ptr(nd, _PU8)), "orc_colocate")
    return nd[:, :n].reshape(shape) if n > 0 else nd[:, :0].reshape(shape)


def comm(wl):
    """c[v] = ceil(ob[v]/bw) + lat, int64 (the oracle's own copy of the cost model)."""
    ob = np.asarray(wl.ob, np.int64)
    return -(-ob // int(wl.bw)) + int(wl.lat)
