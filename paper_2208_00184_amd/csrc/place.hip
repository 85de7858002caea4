// cel_place: coarse graph + Adjusting Placement (Section 5.2, eq. 7-9,
// Algorithm 2).
//
// Coarse graph (data-parallel): cluster sums by atomics; every edge between
// two clusters is bucketed by its target cluster, each bucket sorted by
// (source cluster, edge id) and runs of equal source cluster summed, which
// gives each cluster its list of coarse in-edges (pred, comm) in a fixed order.
//
// Placement (sequential over clusters, as the algorithm is): one workgroup.
// For cluster t, pre_t on device x is max over preds of Fin[p] + I(dev p != x)
// cc; it is evaluated for all devices at once from two block reductions:
// per-device max of Fin over same-device preds, and the largest and
// second-largest (on another device) values of Fin + cc.  Lane x then finds
// the first-fit start on device x in that device's sorted list of busy
// blocks (touching intervals are merged, so the list holds one block per
// idle gap), and a block argmin picks the device.
#include "cel_internal.h"

namespace cel {

__global__ void k_place_nodes(int32_t n, int32_t C, const int32_t *cid, const int64_t *w,
                              const int64_t *mem, uint64_t *W, uint64_t *MEM, Status *st) {
  if (failed(st)) return;
  uint32_t bad = 0;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t c = cid[v];
    if (c < 0 || c >= C) {
      bad |= EB_ARG;
      continue;
    }
    atomicAdd((unsigned long long *)&W[c], (unsigned long long)w[v]);
    atomicAdd((unsigned long long *)&MEM[c], (unsigned long long)mem[v]);
  }
  if (bad) raise_err(st, bad);
}

// Edges between clusters, edge-balanced blocks.  PASS 0
// counts per target cluster (and checks cid[u] <= cid[v]); PASS 1 writes
// (source cluster, edge id) into the target's bucket and the edge's comm.
template <int PASS>
__global__ void k_place_edges(cel_graph g, int64_t bw, int64_t lat, const int32_t *cid,
                              int32_t *cnt, const int32_t *boff, uint64_t *keys, uint32_t *ids,
                              int64_t *ecost, Status *st) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  if (failed(st)) return;
  uint32_t bad = 0;
  for_edges_balanced(g.out_ptr, g.n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    const int32_t a = cid[u], b = cid[g.out_idx[e]];
    if (a == b) return;
    if (a > b) {
      bad |= EB_ORDER;
      return;
    }
    if (PASS == 0) {
      atomicAdd(&cnt[b], 1);
    } else {
      const int32_t slot = boff[b] + atomicAdd(&cnt[b], 1);
      keys[slot] = (uint64_t)a;
      ids[slot] = (uint32_t)e;
      ecost[e] = comm_of(g.ob[u], bw, lat);
    }
  });
  if (bad) raise_err(st, bad);
}

// Per target cluster (one wave each): sum runs of equal source cluster into
// coarse in-edges, written in order at the bucket's front, and raise the
// source's back_cost.  64 bucket entries at a time: run heads from the
// neighbouring key, a segmented sum over the wave, run tails compacted by a
// ballot; a run that reaches the end of a batch carries into the next.
__global__ void k_place_combine(int32_t C, const int32_t *boff, const uint64_t *keys,
                                const uint32_t *ids, const int64_t *ecost, int32_t *ca,
                                int64_t *cc, int32_t *ncp, uint64_t *back, const Status *st) {
  if (failed(st)) return;
  const int lane = threadIdx.x & 63;
  const uint64_t lt = (1ull << lane) - 1ull;
  const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t b = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6; b < C; b += nw) {
    const int32_t k0 = boff[b], k1 = boff[b + 1];
    int32_t out = k0;
    uint64_t ckey = ~0ull;  // run carried from the previous batch (none: ~0)
    int64_t csum = 0;
    for (int32_t base = k0; base < k1; base += 64) {
      const int32_t k = base + lane;
      const bool v = k < k1;
      const uint64_t key = v ? keys[k] : ~0ull;
      const int64_t c = v ? ecost[ids[k]] : 0;
      const uint64_t first = __shfl(key, 0);
      if (ckey != ~0ull && first != ckey) {  // the carried run ended with the last batch
        if (lane == 0) {
          ca[out] = (int32_t)ckey;
          cc[out] = csum;
          atomicMax((unsigned long long *)&back[ckey], (unsigned long long)csum);
        }
        out++;
        ckey = ~0ull;
        csum = 0;
      }
      const uint64_t prev = __shfl_up(key, 1);
      const uint64_t pk = lane == 0 ? ckey : prev;
      const int32_t head = v && key != pk;
      // segmented inclusive sum (segments start at heads)
      int64_t x = c;
      int32_t f = head;
      for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_up(x, d);
        const int32_t g = __shfl_up(f, d);
        if (lane >= d && !f) {
          x += y;
          f = g;
        }
      }
      if (!f) x += csum;  // still in the run carried into this batch
      const uint64_t next = __shfl_down(key, 1);
      const bool last_valid = k1 - base <= 64 ? lane == k1 - base - 1 : lane == 63;
      const bool more = k1 - base > 64;  // the batch's last run may continue
      const bool tail = v && (last_valid ? !more : next != key);
      const uint64_t tm = __ballot(tail);
      if (tail) {
        const int32_t o = out + __popcll(tm & lt);
        ca[o] = (int32_t)key;
        cc[o] = x;
        atomicMax((unsigned long long *)&back[key], (unsigned long long)x);
      }
      out += __popcll(tm);
      // carry: the run open at the end of the batch
      const int src = k1 - base < 64 ? k1 - base - 1 : 63;
      ckey = __shfl(key, src);
      const int64_t xs = __shfl(x, src);
      const bool open = more && !__shfl((int)tail, src);
      csum = open ? xs : 0;
      if (!open) ckey = ~0ull;
    }
    if (lane == 0) ncp[b] = out - k0;
  }
}

constexpr int kPlaceB = 256;

__device__ inline void argmin_i64(int64_t &v, int32_t &i) {  // wave: smallest v, then smallest i
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t ov = __shfl_xor(v, off);
    const int32_t oi = __shfl_xor(i, off);
    if (ov < v || (ov == v && oi < i)) {
      v = ov;
      i = oi;
    }
  }
}

__device__ inline void argmax_i64(int64_t &v, int32_t &i) {  // wave: largest v, then smallest i
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t ov = __shfl_xor(v, off);
    const int32_t oi = __shfl_xor(i, off);
    if (ov > v || (ov == v && oi < i)) {
      v = ov;
      i = oi;
    }
  }
}

__global__ void __launch_bounds__(kPlaceB)
    k_place(int32_t C, int32_t D, const int64_t *cap, const uint64_t *W, const uint64_t *MEM,
            const int32_t *boff, const int32_t *ncp, const int32_t *ca, const int64_t *cc,
            const uint64_t *back, uint8_t *cdev, int64_t *Fin, int64_t *bs, int64_t *bf,
            int32_t bcap, Status *st) {
  __shared__ int64_t s_ava[256], s_devmax[256], s_est[256], s_slot[256], s_last[256];
  __shared__ int32_t s_nb[256];
  __shared__ int64_t s_rv[4];
  __shared__ int32_t s_ri[4];
  __shared__ int64_t s_m1, s_m2;
  __shared__ int32_t s_d1;
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  for (int x = tid; x < 256; x += kPlaceB) {
    s_ava[x] = x < D ? cap[x] : 0;
    s_nb[x] = 0;
    s_last[x] = 0;
  }
  int32_t prev = 0, be = 0;
  int64_t span = 0;
  __syncthreads();
  for (int32_t t = 0; t < C; t++) {
    const int32_t b0 = boff[t], np = ncp[t];
    const int64_t Wt = (int64_t)W[t], Mt = (int64_t)MEM[t], bk = (int64_t)back[t];
    for (int x = tid; x < D; x += kPlaceB) s_devmax[x] = -1;
    __syncthreads();
    // largest Fin + cc over all preds (device of the best, lowest id on ties)
    int64_t v1 = -1;
    int32_t d1 = INT32_MAX;
    for (int32_t k = tid; k < np; k += kPlaceB) {
      const int32_t a = ca[b0 + k];
      const int64_t fa = Fin[a];
      const int32_t da = cdev[a];
      atomicMax((long long *)&s_devmax[da], (long long)fa);
      const int64_t x = fa + cc[b0 + k];
      if (x > v1 || (x == v1 && da < d1)) {
        v1 = x;
        d1 = da;
      }
    }
    argmax_i64(v1, d1);
    if (lane == 0) {
      s_rv[wv] = v1;
      s_ri[wv] = d1;
    }
    __syncthreads();
    if (tid == 0) {
      int64_t bv = s_rv[0];
      int32_t bd = s_ri[0];
      for (int i = 1; i < kPlaceB / 64; i++)
        if (s_rv[i] > bv || (s_rv[i] == bv && s_ri[i] < bd)) {
          bv = s_rv[i];
          bd = s_ri[i];
        }
      s_m1 = bv;
      s_d1 = bd;
    }
    __syncthreads();
    // largest Fin + cc over preds on another device than the best one
    const int32_t D1 = s_d1;
    int64_t v2 = -1;
    int32_t dummy = 0;
    for (int32_t k = tid; k < np; k += kPlaceB) {
      const int32_t a = ca[b0 + k];
      if ((int32_t)cdev[a] == D1) continue;
      const int64_t x = Fin[a] + cc[b0 + k];
      v2 = x > v2 ? x : v2;
    }
    argmax_i64(v2, dummy);
    if (lane == 0) s_rv[wv] = v2;
    __syncthreads();
    if (tid == 0) {
      int64_t bv = s_rv[0];
      for (int i = 1; i < kPlaceB / 64; i++) bv = s_rv[i] > bv ? s_rv[i] : bv;
      s_m2 = bv;
    }
    __syncthreads();
    // lane x: pre_t, first-fit slot and EST on device x  (eq. 7)
    const int64_t M1 = s_m1, M2 = s_m2;
    for (int x = tid; x < D; x += kPlaceB) {
      int64_t pre = 0;
      const int64_t other = (x != D1) ? M1 : M2;
      pre = other > pre ? other : pre;
      pre = s_devmax[x] > pre ? s_devmax[x] : pre;
      int64_t s = pre;
      const int32_t nb = s_nb[x];
      if (Wt > 0 && nb > 0 && s < s_last[x]) {
        const int64_t *xs = bs + (int64_t)x * bcap, *xf = bf + (int64_t)x * bcap;
        int32_t lo = 0, hi = nb;  // first block ending after s
        while (lo < hi) {
          const int32_t mid = (lo + hi) >> 1;
          if (xf[mid] <= s) lo = mid + 1;
          else hi = mid;
        }
        for (int32_t k = lo; k < nb && xs[k] < s + Wt; k++) s = xf[k];
      }
      s_slot[x] = s;
      s_est[x] = s_ava[x] < Mt ? kInf : s;
    }
    __syncthreads();
    // device of smallest EST (lowest id on ties)
    int64_t ev = kInf;
    int32_t ei = INT32_MAX;
    for (int x = tid; x < D; x += kPlaceB)
      if (s_est[x] < ev || (s_est[x] == ev && x < ei)) {
        ev = s_est[x];
        ei = x;
      }
    argmin_i64(ev, ei);
    if (lane == 0) {
      s_rv[wv] = ev;
      s_ri[wv] = ei;
    }
    __syncthreads();
    if (tid == 0) {
      int64_t e1 = s_rv[0];
      int32_t dd = s_ri[0];
      for (int i = 1; i < kPlaceB / 64; i++)
        if (s_rv[i] < e1 || (s_rv[i] == e1 && s_ri[i] < dd)) {
          e1 = s_rv[i];
          dd = s_ri[i];
        }
      const int32_t dk = t == 0 ? 0 : prev;
      int32_t pick;
      if (e1 == kInf) {  // every device full: most remaining memory (best effort)
        pick = 0;
        for (int x = 1; x < D; x++)
          if (s_ava[x] > s_ava[pick]) pick = x;
        be++;
      } else if (s_est[dk] == kInf || s_est[dk] - e1 > bk) {  // eq. 9
        pick = dd;
      } else {
        pick = dk;
      }
      const int64_t s0 = s_slot[pick], f = s0 + Wt;
      cdev[t] = (uint8_t)pick;
      Fin[t] = f;
      span = f > span ? f : span;
      s_ava[pick] -= Mt;
      prev = pick;
      if (Wt > 0) {  // insert [s0, f) into the device's merged busy blocks
        int64_t *xs = bs + (int64_t)pick * bcap, *xf = bf + (int64_t)pick * bcap;
        int32_t nb = s_nb[pick];
        int32_t lo = 0, hi = nb;  // k = number of blocks ending at or before s0
        while (lo < hi) {
          const int32_t mid = (lo + hi) >> 1;
          if (xf[mid] <= s0) lo = mid + 1;
          else hi = mid;
        }
        const int32_t k = lo;
        const bool left = k > 0 && xf[k - 1] == s0;
        const bool right = k < nb && xs[k] == f;
        if (left && right) {
          xf[k - 1] = xf[k];
          for (int32_t q = k; q + 1 < nb; q++) {
            xs[q] = xs[q + 1];
            xf[q] = xf[q + 1];
          }
          nb--;
        } else if (left) {
          xf[k - 1] = f;
        } else if (right) {
          xs[k] = s0;
        } else if (nb < bcap) {
          for (int32_t q = nb; q > k; q--) {
            xs[q] = xs[q - 1];
            xf[q] = xf[q - 1];
          }
          xs[k] = s0;
          xf[k] = f;
          nb++;
        } else {
          raise_err(st, EB_ARG);  // cannot happen: one block per placed cluster at most
        }
        s_nb[pick] = nb;
        s_last[pick] = nb > 0 ? xf[nb - 1] : 0;
      }
    }
    __syncthreads();
  }
  if (tid == 0) {
    st->s0 = span;
    st->i0 = be;
  }
}

__global__ void k_place_out(int32_t n, int32_t C, const int32_t *cid, const uint8_t *cdev,
                            uint8_t *node_dev, const int64_t *Fin, int64_t *fin_out,
                            const Status *st) {
  if (failed(st)) return;
  const int64_t tot = n > C ? n : C;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < tot;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i < n) node_dev[i] = cdev[cid[i]];
    if (fin_out && i < C) fin_out[i] = Fin[i];
  }
}

}  // namespace cel

using namespace cel;

extern "C" int cel_place(const cel_graph *g, const cel_devices *d, const int32_t *cluster_id,
                         int32_t C, uint8_t *cluster_dev, uint8_t *node_dev,
                         int64_t *cluster_fin, int64_t *coarse_makespan,
                         int32_t *best_effort_count, hipStream_t s) {
  const char *fn = "cel_place";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n;
  if (!coarse_makespan || !best_effort_count || (n > 0 && (!cluster_id || !node_dev)) ||
      (C > 0 && !cluster_dev))
    return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  if (C < 0 || (n > 0 && C < 1) || C > (n > 0 ? n : 0))
    return set_error(CEL_E_ARG, "%s: n_clusters = %d out of range", fn, C);
  const int64_t bcap = C;
  if ((int64_t)d->D * bcap > (int64_t)1 << 28)
    return set_error(CEL_E_NOMEM, "%s: D * n_clusters too large for the busy lists", fn);
  Scratch sc(s);
  Status *st;
  int32_t *tmp;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, sc, s));
  if (C == 0) {
    Status h;
    CEL_TRY(read_status(st, &h, s));
    if (h.err) return status_error(h, fn);
    *coarse_makespan = 0;
    *best_effort_count = 0;
    return CEL_OK;
  }
  uint64_t *W, *MEM, *back, *keys;
  int32_t *cnt, *boff, *ca, *ncp;
  int64_t *ecost, *cc, *Fin, *bs, *bf, *dcap;
  uint32_t *ids;
  const int64_t m = g->m;
  CEL_TRY(sc.get(&W, C));
  CEL_TRY(sc.get(&MEM, C));
  CEL_TRY(sc.get(&back, C));
  CEL_TRY(sc.get(&cnt, C));
  CEL_TRY(sc.get(&boff, (int64_t)C + 1));
  CEL_TRY(sc.get(&ncp, C));
  CEL_TRY(sc.get(&Fin, C));
  CEL_TRY(sc.get(&dcap, d->D));
  CEL_TRY(sc.get(&bs, d->D * bcap));
  CEL_TRY(sc.get(&bf, d->D * bcap));
  CEL_HIP(hipMemsetAsync(W, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(MEM, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(back, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(cnt, 0, sizeof(int32_t) * C, s));
  CEL_HIP(hipMemcpyAsync(dcap, d->cap, sizeof(int64_t) * d->D, hipMemcpyHostToDevice, s));
  k_place_nodes<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, C, cluster_id, g->w, g->mem, W, MEM, st);
  const unsigned eb = edge_blocks(g->m);
  k_place_edges<0><<<eb, 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, cnt, nullptr, nullptr,
                                      nullptr, nullptr, st);
  CEL_TRY(exclusive_scan_i32(cnt, boff, C, sc, s));
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  std::vector<int32_t> hb(C + 1);
  CEL_HIP(hipMemcpyAsync(hb.data(), boff, sizeof(int32_t) * (C + 1), hipMemcpyDeviceToHost, s));
  CEL_HIP(hipStreamSynchronize(s));
  const int64_t ncross = hb[C];
  CEL_TRY(sc.get(&keys, ncross));
  CEL_TRY(sc.get(&ids, ncross));
  CEL_TRY(sc.get(&ca, ncross));
  CEL_TRY(sc.get(&cc, ncross));
  CEL_TRY(sc.get(&ecost, m));
  CEL_HIP(hipMemsetAsync(cnt, 0, sizeof(int32_t) * C, s));
  k_place_edges<1><<<eb, 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, cnt, boff, keys, ids, ecost,
                                      st);
  CEL_TRY(segmented_sort(keys, ids, boff, C, ncross, sc, s, st));
  k_place_combine<<<grid_for((int64_t)C * 64, 256, 8192), 256, 0, s>>>(C, boff, keys, ids, ecost,
                                                                      ca, cc, ncp, back, st);
  {
    KTimer kt(s, "k_place");
    k_place<<<1, kPlaceB, 0, s>>>(C, d->D, dcap, W, MEM, boff, ncp, ca, cc, back, cluster_dev,
                                  Fin, bs, bf, (int32_t)bcap, st);
  }
  k_place_out<<<grid_for(n > C ? n : C, 256, 4096), 256, 0, s>>>(n, C, cluster_id, cluster_dev,
                                                                node_dev, Fin, cluster_fin, st);
  CEL_HIP(hipGetLastError());
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  *coarse_makespan = h.s0;
  *best_effort_count = h.i0;
  return CEL_OK;
}
