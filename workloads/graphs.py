"""Seeded synthetic operator DAGs for the five workload configurations.

Every generator returns a :class:`Workload`: CSR (by source) and CSC (by target)
int32 edge arrays over node ids that have been randomly relabelled (so ids are
*not* a topological order), int64 per-op compute time ``w`` (ns), memory ``mem``
(bytes) and output-tensor bytes ``ob``, plus the modelled devices (count ``D``,
int64 memory caps, link bandwidth ``bw`` in bytes/ns and latency ``lat`` in ns).

The graphs stand in for the paper's TensorFlow models (Inception_V3, NMT,
Transformer, Tensor Holography; Section 6.2), which are not available: they
copy the features the paper stresses -- tens of thousands of nodes, a high
communication-to-computation ratio (Section 5.1.1) and many indegree-0
parameter nodes (Section 4.2.2).  Recipes:

1. ``layered``: 64 layers x 32 nodes; each node of layer l >= 1 draws k ~ U{1,2,3}
   distinct parents uniformly from the union of the previous min(4, l) layers.
   w ~ U[1, 1000] ns, ob ~ U[1 KiB, 1 MiB], D = 4, cap = 0.3 x total memory,
   link 12 B/ns + 5000 ns.
2. ``transformer-24``: 24 transformer blocks (hidden 1024, 16 heads, 4096 tokens)
   as a fwd + bwd + Adam training graph at micro-op granularity.  D = 4,
   cap = 0.35 x total, link 25 B/ns + 3000 ns.
3. ``inception-600``: 600 fork/join modules (4-8 branches of 3-12 chained ops,
   one parameter source per op, 1-3 extra same-module inputs per op, concat
   join).  w ~ lognormal(ln 5000, 1), ob ~ lognormal(ln 256 KiB, 1), D = 8,
   cap = 0.2 x total, link 12 B/ns + 5000 ns.
4. ``transformer-96``: the template of (2) at hidden 8192, 64 heads, GEMMs and
   their epilogues split into 32 column tiles; 96 blocks, ~1.1M nodes, max
   fan-in 6.  D = 16, cap = 0.1 x total, link 50 B/ns + 2000 ns.
5. ``layered-200k``: as (1) with 400 layers x 500 nodes and parents from the
   previous 1-8 layers; D = 8, cap = 0.3 x total, link 12 B/ns + 5000 ns.

Cost rounding: GEMM time = ceil(2 M N K / 1e5) ns (100 TFLOP/s), lognormal
draws -> max(1, rint(x)); op memory = 2 x output bytes for every config.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

CONFIG_NAMES = {
    1: "layered-2k",
    2: "transformer-24",
    3: "inception-600",
    4: "transformer-96",
    5: "layered-200k",
}


@dataclass
class Workload:
    name: str
    n: int
    m: int
    out_ptr: np.ndarray  # int32 [n+1]
    out_idx: np.ndarray  # int32 [m]
    in_ptr: np.ndarray   # int32 [n+1]
    in_idx: np.ndarray   # int32 [m]
    w: np.ndarray        # int64 [n]
    mem: np.ndarray      # int64 [n]
    ob: np.ndarray       # int64 [n]
    D: int
    cap: np.ndarray      # int64 [D]
    bw: int
    lat: int
    meta: dict = field(default_factory=dict)

    def edges(self):
        """(src, dst) int64 arrays in CSR order."""
        src = np.repeat(np.arange(self.n, dtype=np.int64),
                        np.diff(self.out_ptr).astype(np.int64))
        return src, self.out_idx.astype(np.int64)


def _assemble(name, src, dst, w, ob, D, cap_num, cap_den, bw, lat, rng,
              relabel=True, meta=None) -> Workload:
    """Relabel node ids at random and build CSR + CSC."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    w = np.asarray(w, dtype=np.int64)
    ob = np.asarray(ob, dtype=np.int64)
    n = int(w.shape[0])
    if relabel and n > 0:
        perm = rng.permutation(n).astype(np.int64)  # old id i -> new id perm[i]
        w2 = np.empty_like(w); w2[perm] = w
        ob2 = np.empty_like(ob); ob2[perm] = ob
        w, ob = w2, ob2
        src, dst = perm[src], perm[dst]
    m = int(src.shape[0])
    order = np.lexsort((dst, src))
    out_idx = dst[order].astype(np.int32)
    out_ptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(src, minlength=n), out=out_ptr[1:])
    order = np.lexsort((src, dst))
    in_idx = src[order].astype(np.int32)
    in_ptr = np.zeros(n + 1, dtype=np.int64)
    np.cumsum(np.bincount(dst, minlength=n), out=in_ptr[1:])
    mem = 2 * ob
    total = int(mem.sum())
    cap = np.full(D, (total * cap_num) // cap_den, dtype=np.int64)
    md = dict(meta or {})
    return Workload(name=name, n=n, m=m,
                    out_ptr=out_ptr.astype(np.int32), out_idx=out_idx,
                    in_ptr=in_ptr.astype(np.int32), in_idx=in_idx,
                    w=w, mem=mem, ob=ob, D=D, cap=cap, bw=int(bw), lat=int(lat),
                    meta=md)


def from_edges(n, edges, w, ob, D, cap, bw, lat, mem=None, name="explicit") -> Workload:
    """A workload with explicit structure and parameters (no relabelling).

    ``edges`` is a sequence of (src, dst) pairs; ``mem`` defaults to 2 x ``ob``.
    """
    e = np.asarray(list(edges), dtype=np.int64).reshape(-1, 2)
    src, dst = e[:, 0], e[:, 1]
    wl = _assemble(name, src, dst, np.asarray(w, np.int64).reshape(n),
                   np.asarray(ob, np.int64).reshape(n), int(D), 1, 1, bw, lat,
                   None, relabel=False)
    if mem is not None:
        wl.mem = np.asarray(mem, np.int64).reshape(n)
    wl.cap = np.asarray(cap, np.int64).reshape(int(D))
    return wl


def _sample_distinct3(rng, P, size):
    """Three distinct uniform draws from [0, P) per row (P >= 3)."""
    r1 = rng.integers(0, P, size)
    r2 = rng.integers(0, P - 1, size)
    r3 = rng.integers(0, P - 2, size)
    x1 = r1
    x2 = r2 + (r2 >= x1)
    lo = np.minimum(x1, x2)
    hi = np.maximum(x1, x2)
    x3 = r3 + (r3 >= lo)
    x3 = x3 + (x3 >= hi)
    return np.stack([x1, x2, x3], axis=1)


def _layered(rng, layers, width, back):
    srcs, dsts = [], []
    for layer in range(1, layers):
        span = min(back, layer)
        base = (layer - span) * width
        P = span * width
        k = rng.integers(1, 4, width)
        picks = _sample_distinct3(rng, P, width) + base
        kids = layer * width + np.arange(width)
        mask = np.arange(3)[None, :] < k[:, None]
        srcs.append(picks[mask])
        dsts.append(np.broadcast_to(kids[:, None], (width, 3))[mask])
    n = layers * width
    src = np.concatenate(srcs) if srcs else np.zeros(0, np.int64)
    dst = np.concatenate(dsts) if dsts else np.zeros(0, np.int64)
    return n, src, dst


def _layered_config(cfg, seed, layers, width, back, D):
    rng = np.random.default_rng([cfg, seed])
    n, src, dst = _layered(rng, layers, width, back)
    w = rng.integers(1, 1001, n)
    ob = rng.integers(1024, 1048577, n)
    return _assemble(CONFIG_NAMES[cfg], src, dst, w, ob, D, 3, 10, 12, 5000, rng,
                     meta=dict(config=cfg, seed=seed, layers=layers, width=width))


def _lognormal_int(rng, mu, sigma, size):
    return np.maximum(1, np.rint(rng.lognormal(mu, sigma, size))).astype(np.int64)


def _inception(cfg, seed, modules=600):
    rng = np.random.default_rng([cfg, seed])
    src, dst = [], []
    n = 1  # node 0: the graph input
    inp = 0
    for _ in range(modules):
        B = int(rng.integers(4, 9))
        by_depth = [[inp]]  # by_depth[t] = ops of this module at branch depth t
        ends = []
        for _b in range(B):
            Lb = int(rng.integers(3, 13))
            prev = inp
            for t in range(1, Lb + 1):
                op = n; param = n + 1; n += 2
                src += [prev, param]; dst += [op, op]
                cand = [x for d in range(t) for x in by_depth[d] if x != prev]
                kx = int(rng.integers(1, 4))
                if cand:
                    sel = rng.choice(len(cand), size=min(kx, len(cand)), replace=False)
                    for s in np.sort(sel):
                        src.append(cand[int(s)]); dst.append(op)
                while len(by_depth) <= t:
                    by_depth.append([])
                by_depth[t].append(op)
                prev = op
            ends.append(prev)
        cat = n; n += 1
        for e in ends:
            src.append(e); dst.append(cat)
        inp = cat
    w = _lognormal_int(rng, math.log(5000.0), 1.0, n)
    ob = _lognormal_int(rng, math.log(262144.0), 1.0, n)
    return _assemble(CONFIG_NAMES[cfg], src, dst, w, ob, 8, 2, 10, 12, 5000, rng,
                     meta=dict(config=cfg, seed=seed, modules=modules))


class _TransformerBuilder:
    """Micro-op fwd + bwd + Adam graph of a stack of transformer blocks.

    Tensors whose last dimension is the hidden size are split into ``T`` column
    tiles; every op on them becomes T nodes.  Reductions and gathers over tiles
    use trees of fan-in at most ``F``.
    """

    EW = -1  # sentinel: elementwise op, cost drawn lognormal at the end

    def __init__(self, rng, h, heads, T, blocks, tokens=4096, batch=4, seq=1024, F=6):
        self.rng = rng
        self.h, self.H, self.T, self.nb = h, heads, T, blocks
        self.M, self.B, self.S, self.F = tokens, batch, seq, F
        self.d = h // heads
        self.tw = h // T  # tile width (columns)
        self.w: list[int] = []
        self.ob: list[int] = []
        self.src: list[int] = []
        self.dst: list[int] = []
        self.step = None    # global step / learning-rate node read by every update
        self.k = {}         # per-block constant nodes (indegree 0)

    # -- primitives -------------------------------------------------------
    def node(self, w, ob, inputs=()):
        v = len(self.w)
        self.w.append(int(w)); self.ob.append(int(ob))
        seen = set()
        for u in inputs:
            if u in seen:
                continue
            seen.add(u)
            self.src.append(u); self.dst.append(v)
        assert len(seen) <= self.F, "fan-in bound"
        return v

    def ew(self, ob, inputs):
        return self.node(self.EW, ob, inputs)

    def gemm_cost(self, M, N, K):
        return -(-(2 * M * N * K) // 100000)

    def tree(self, inputs, ob):
        """Reduce/gather ``inputs`` into one node, fan-in <= F."""
        inputs = list(inputs)
        if len(inputs) == 1:
            return inputs[0]
        while len(inputs) > self.F:
            nxt = []
            for i in range(0, len(inputs), self.F):
                grp = inputs[i:i + self.F]
                nxt.append(grp[0] if len(grp) == 1 else self.ew(ob, grp))
            inputs = nxt
        return self.ew(ob, inputs)

    def act(self, cols):
        return 2 * self.M * cols

    def param(self, nbytes):
        """A parameter with its two Adam moment states (all indegree 0)."""
        return (self.ew(nbytes, ()), self.ew(nbytes, ()), self.ew(nbytes, ()))

    def adam(self, p, grad, nbytes):
        w_, m_, v_ = p
        m2 = self.ew(nbytes, (m_, grad, self.step))
        v2 = self.ew(nbytes, (v_, grad, self.step))
        self.ew(nbytes, (w_, m2, v2, self.step))  # updated weight: a sink

    # -- layer norm -------------------------------------------------------
    def ln_fwd(self, x):
        T, tw = self.T, self.tw
        g = [self.param(2 * tw) for _ in range(T)]
        b = [self.param(2 * tw) for _ in range(T)]
        mean = self.tree(x, 2 * self.M)
        cen = [self.ew(self.act(tw), (x[t], mean)) for t in range(T)]
        sq = [self.ew(self.act(tw), (cen[t],)) for t in range(T)]
        var = self.tree(sq, 2 * self.M)
        eps = self.ew(2 * self.M, (var, self.k["eps"]))
        rstd = self.ew(2 * self.M, (eps,))
        nrm = [self.ew(self.act(tw), (cen[t], rstd)) for t in range(T)]
        sc = [self.ew(self.act(tw), (nrm[t], g[t][0])) for t in range(T)]
        y = [self.ew(self.act(tw), (sc[t], b[t][0])) for t in range(T)]
        return y, dict(g=g, b=b, nrm=nrm, rstd=rstd)

    def ln_bwd(self, dy, s):
        T, tw = self.T, self.tw
        dn = [self.ew(self.act(tw), (dy[t], s["g"][t][0])) for t in range(T)]
        for t in range(T):
            pg = self.ew(self.act(tw), (dy[t], s["nrm"][t]))
            dg = self.ew(2 * tw, (pg,))
            db = self.ew(2 * tw, (dy[t],))
            self.adam(s["g"][t], dg, 2 * tw)
            self.adam(s["b"][t], db, 2 * tw)
        m1 = self.tree(dn, 2 * self.M)
        pr = [self.ew(self.act(tw), (dn[t], s["nrm"][t])) for t in range(T)]
        m2 = self.tree(pr, 2 * self.M)
        a = [self.ew(self.act(tw), (dn[t], m1)) for t in range(T)]
        bb = [self.ew(self.act(tw), (s["nrm"][t], m2)) for t in range(T)]
        dx = [self.ew(self.act(tw), (a[t], bb[t], s["rstd"])) for t in range(T)]
        return dx

    # -- linear layer (column tiles) --------------------------------------
    def lin_fwd(self, xg, K, N):
        """xg: gathered input [M, K]; output N columns in N/tw tiles."""
        nt = N // self.tw
        W = [self.param(2 * K * self.tw) for _ in range(nt)]
        bias = [self.param(2 * self.tw) for _ in range(nt)]
        mm = [self.node(self.gemm_cost(self.M, self.tw, K), self.act(self.tw), (xg, W[j][0]))
              for j in range(nt)]
        y = [self.ew(self.act(self.tw), (mm[j], bias[j][0])) for j in range(nt)]
        return y, dict(W=W, bias=bias, xg=xg, K=K, N=N)

    def lin_bwd(self, dy, s):
        K, N = s["K"], s["N"]
        nt = N // self.tw
        for j in range(nt):
            db = self.ew(2 * self.tw, (dy[j],))
            self.adam(s["bias"][j], db, 2 * self.tw)
        dyg = self.tree(dy, self.act(N))
        Wg = self.tree([p[0] for p in s["W"]], 2 * K * N)
        kt = K // self.tw
        dx = [self.node(self.gemm_cost(self.M, self.tw, N), self.act(self.tw), (dyg, Wg))
              for _ in range(kt)]
        for j in range(nt):
            dW = self.node(self.gemm_cost(K, self.tw, self.M), 2 * K * self.tw, (s["xg"], dy[j]))
            self.adam(s["W"][j], dW, 2 * K * self.tw)
        return dx

    # -- attention ----------------------------------------------------------
    def _tiles_of(self, tiles, col0, ncols):
        a = col0 // self.tw
        b = (col0 + ncols - 1) // self.tw
        return tiles[a:b + 1]

    def attn_fwd(self, qkv):
        h, d, H = self.h, self.d, self.H
        att = self.gemm_cost(self.B * self.S, self.S, d)  # 2 B S S d / 1e5
        big = 2 * self.B * self.S * self.S
        row = 2 * self.B * self.S
        outs, saved = [], []
        for i in range(H):
            q = self.ew(self.act(d), self._tiles_of(qkv, i * d, d))
            k = self.ew(self.act(d), self._tiles_of(qkv, h + i * d, d))
            v = self.ew(self.act(d), self._tiles_of(qkv, 2 * h + i * d, d))
            kt = self.ew(self.act(d), (k,))
            s = self.node(att, big, (q, kt))
            sc = self.ew(big, (s, self.k["scale"]))
            mk = self.ew(big, (sc, self.k["mask"]))
            mx = self.ew(row, (mk,))
            sb = self.ew(big, (mk, mx))
            ex = self.ew(big, (sb,))
            sm = self.ew(row, (ex,))
            p = self.ew(big, (ex, sm))
            rm = self.ew(big, ())  # dropout keep-mask (random source)
            pd = self.ew(big, (p, rm))
            o = self.node(att, self.act(d), (pd, v))
            ro = self.ew(self.act(d), (o,))
            outs.append(ro)
            saved.append(dict(q=q, kt=kt, v=v, p=p, pd=pd, rm=rm))
        per = max(1, H // self.T)
        cat = [self.tree(outs[j * per:(j + 1) * per], self.act(self.tw)) for j in range(self.T)] \
            if self.T <= H else None
        assert cat is not None, "tiles narrower than a head are not modelled"
        return cat, saved

    def attn_bwd(self, dcat, saved):
        h, d, H = self.h, self.d, self.H
        att = self.gemm_cost(self.B * self.S, self.S, d)
        big = 2 * self.B * self.S * self.S
        row = 2 * self.B * self.S
        dq, dk, dv = [], [], []
        for i in range(H):
            sv = saved[i]
            dO = self.ew(self.act(d), self._tiles_of(dcat, i * d, d))
            rO = self.ew(self.act(d), (dO,))
            dpd = self.node(att, big, (rO, sv["v"]))
            dvv = self.node(att, self.act(d), (sv["pd"], rO))
            dp = self.ew(big, (dpd, sv["rm"]))  # dropout bwd
            m1 = self.ew(big, (dp, sv["p"]))
            rs = self.ew(row, (m1,))
            sb = self.ew(big, (dp, rs))
            ds = self.ew(big, (sb, sv["p"]))
            dm = self.ew(big, (ds, self.k["mask"]))
            dsc = self.ew(big, (dm, self.k["scale"]))
            dqq = self.node(att, self.act(d), (dsc, sv["kt"]))
            dkk = self.node(att, self.act(d), (dsc, sv["q"]))
            dq.append(self.ew(self.act(d), (dqq,)))
            dk.append(self.ew(self.act(d), (self.ew(self.act(d), (dkk,)),)))
            dv.append(self.ew(self.act(d), (dvv,)))
        per = H // self.T
        tiles = []
        for grp in (dq, dk, dv):
            tiles += [self.tree(grp[j * per:(j + 1) * per], self.act(self.tw))
                      for j in range(self.T)]
        return tiles

    # -- whole graph ----------------------------------------------------------
    def gelu_fwd(self, u):
        a = self.act(self.tw)
        k = self.k
        c1 = self.ew(a, (u,)); c2 = self.ew(a, (c1, k["g1"])); c3 = self.ew(a, (u, c2))
        c4 = self.ew(a, (c3, k["g2"])); th = self.ew(a, (c4,)); c6 = self.ew(a, (th, k["one"]))
        c7 = self.ew(a, (u, c6)); g = self.ew(a, (c7, k["half"]))
        return g, th

    def gelu_bwd(self, dg, u, th):
        a = self.act(self.tw)
        k = self.k
        e1 = self.ew(a, (th, k["one"])); e2 = self.ew(a, (u, k["g3"])); e3 = self.ew(a, (e1, e2))
        e4 = self.ew(a, (e3, u, k["g4"])); e5 = self.ew(a, (th, k["half"])); e6 = self.ew(a, (e5, e4))
        return self.ew(a, (dg, e6))

    def dropout(self, x, masks=None):
        """Dropout on tiles; fresh random keep-masks unless ``masks`` is given."""
        a = self.act(self.tw)
        if masks is None:
            masks = [self.ew(a, ()) for _ in x]
        return [self.ew(a, (t, mk)) for t, mk in zip(x, masks)], masks

    def build(self):
        T, h = self.T, self.h
        x = [self.ew(self.act(self.tw), ()) for _ in range(T)]  # embedding output
        x0 = x
        self.step = self.ew(8, ())
        saved = []
        for _ in range(self.nb):
            s = {}
            self.k = {nm: self.ew(2, ()) for nm in
                      ("eps", "scale", "mask", "g1", "g2", "g3", "g4", "one", "half")}
            s["k"] = self.k
            y1, s["ln1"] = self.ln_fwd(x)
            xg = self.tree(y1, self.act(h))
            qkv, s["qkv"] = self.lin_fwd(xg, h, 3 * h)
            cat, s["attn"] = self.attn_fwd(qkv)
            cg = self.tree(cat, self.act(h))
            pr, s["proj"] = self.lin_fwd(cg, h, h)
            pr, s["dm1"] = self.dropout(pr)
            r1 = [self.ew(self.act(self.tw), (x[t], pr[t])) for t in range(T)]
            y2, s["ln2"] = self.ln_fwd(r1)
            y2g = self.tree(y2, self.act(h))
            u, s["mlp1"] = self.lin_fwd(y2g, h, 4 * h)
            gl = [self.gelu_fwd(t) for t in u]
            s["u"], s["th"] = u, [g[1] for g in gl]
            gg = self.tree([g[0] for g in gl], self.act(4 * h))
            y3, s["mlp2"] = self.lin_fwd(gg, 4 * h, h)
            y3, s["dm2"] = self.dropout(y3)
            x = [self.ew(self.act(self.tw), (r1[t], y3[t])) for t in range(T)]
            saved.append(s)
        loss = self.tree(x, 2 * self.M)
        dx = [self.ew(self.act(self.tw), (loss, x[t])) for t in range(T)]
        for s in reversed(saved):
            self.k = s["k"]
            d3, _ = self.dropout(dx, s["dm2"])
            dgl = self.lin_bwd(d3, s["mlp2"])
            du = [self.gelu_bwd(dgl[j], s["u"][j], s["th"][j]) for j in range(4 * T)]
            dy2 = self.lin_bwd(du, s["mlp1"])
            dr1 = self.ln_bwd(dy2, s["ln2"])
            dr1 = [self.ew(self.act(self.tw), (dx[t], dr1[t])) for t in range(T)]
            dpr, _ = self.dropout(dr1, s["dm1"])
            dcat = self.lin_bwd(dpr, s["proj"])
            dqkv = self.attn_bwd(dcat, s["attn"])
            dy1 = self.lin_bwd(dqkv, s["qkv"])
            dln = self.ln_bwd(dy1, s["ln1"])
            dx = [self.ew(self.act(self.tw), (dr1[t], dln[t])) for t in range(T)]
        for t in range(T):
            self.ew(self.act(self.tw), (x0[t], dx[t]))  # embedding update: sinks
        w = np.asarray(self.w, dtype=np.int64)
        ew = w == self.EW
        w[ew] = _lognormal_int(self.rng, math.log(2000.0), 0.5, int(ew.sum()))
        return w, np.asarray(self.ob, np.int64), np.asarray(self.src), np.asarray(self.dst)


def _transformer(cfg, seed, h, heads, T, blocks, D, cap_num, cap_den, bw, lat):
    rng = np.random.default_rng([cfg, seed])
    tb = _TransformerBuilder(rng, h, heads, T, blocks)
    w, ob, src, dst = tb.build()
    return _assemble(CONFIG_NAMES[cfg], src, dst, w, ob, D, cap_num, cap_den, bw, lat, rng,
                     meta=dict(config=cfg, seed=seed, hidden=h, heads=heads, tiles=T,
                               blocks=blocks))


def make_config(cfg: int, seed: int = 0) -> Workload:
    """The workload of configuration ``cfg`` (1..5) drawn with ``seed``."""
    if cfg == 1:
        return _layered_config(1, seed, 64, 32, 4, 4)
    if cfg == 2:
        return _transformer(2, seed, 1024, 16, 1, 24, 4, 35, 100, 25, 3000)
    if cfg == 3:
        return _inception(3, seed)
    if cfg == 4:
        return _transformer(4, seed, 8192, 64, 32, 96, 16, 10, 100, 50, 2000)
    if cfg == 5:
        return _layered_config(5, seed, 400, 500, 8, 8)
    raise ValueError(f"unknown config {cfg}")


def make_random_dag(seed: int, n: int, p_edge: float = 0.3, D: int = 3,
                    w_max: int = 50, ob_max: int = 200, bw: int = 7, lat: int = 3,
                    cap_frac=(1, 2), multi: bool = False, zero_frac: float = 0.0,
                    relabel: bool = True, max_fanin: int = 6) -> Workload:
    """Small random DAG for brute-force and property tests.

    Each ordered pair (i < j) of a hidden topological order gets an edge with
    probability ``p_edge`` (fan-in capped at ``max_fanin``); ``multi`` doubles a
    few edges; ``zero_frac`` of the nodes get w = 0 and ob = 0.
    """
    rng = np.random.default_rng([99, seed, n])
    src, dst = [], []
    for j in range(n):
        preds = [i for i in range(j) if rng.random() < p_edge]
        if len(preds) > max_fanin:
            preds = list(rng.choice(preds, size=max_fanin, replace=False))
        for i in sorted(preds):
            src.append(i); dst.append(j)
            if multi and rng.random() < 0.15 and len(preds) < max_fanin:
                src.append(i); dst.append(j)
    w = rng.integers(0 if zero_frac else 1, w_max + 1, n)
    ob = rng.integers(0, ob_max + 1, n)
    if zero_frac:
        z = rng.random(n) < zero_frac
        w[z] = 0; ob[z] = 0
    return _assemble(f"random-{seed}-{n}", src, dst, w, ob, D, cap_frac[0], cap_frac[1],
                     bw, lat, rng, relabel=relabel, meta=dict(seed=seed))


def _splitmix64(x: np.ndarray) -> np.ndarray:
    """SplitMix64 output function (Steele, Lea, Flood 2014) on uint64 arrays."""
    with np.errstate(over="ignore"):
        z = (x + np.uint64(0x9E3779B97F4A7C15)).astype(np.uint64)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


def perturb_placements(cluster_dev: np.ndarray, D: int, K: int, seed: int,
                       frac_num: int = 5, frac_den: int = 100) -> np.ndarray:
    """K candidate cluster->device maps, each the base map with exactly
    round(frac * C) distinct clusters reassigned to a uniform device.

    Clusters are chosen by a partial Fisher-Yates shuffle driven by a SplitMix64
    stream keyed by (seed, k); returns uint8 [K, C].
    """
    base = np.asarray(cluster_dev, dtype=np.uint8)
    C = base.shape[0]
    r = (2 * C * frac_num + frac_den) // (2 * frac_den)  # round half up
    out = np.repeat(base[None, :], K, axis=0)
    for k in range(K):
        state = np.uint64((seed * 0x100000001B3 + k * 0x9E3779B1) & 0xFFFFFFFFFFFFFFFF)
        ctr = np.arange(2 * r, dtype=np.uint64) + state
        rnd = _splitmix64(ctr)
        idx = np.arange(C)
        for t in range(r):
            j = t + int(rnd[t] % np.uint64(C - t))
            idx[t], idx[j] = idx[j], idx[t]
        out[k, idx[:r]] = (rnd[r:2 * r] % np.uint64(D)).astype(np.uint8)
    return out
