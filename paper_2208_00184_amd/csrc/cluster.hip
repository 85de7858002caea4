// cel_cluster: memory-capped contiguous clustering of a topological order
// (Section 5.1.3, eq. 4-6).
//
// With PO the prefix sum of each node's out-going comm (outdeg * c) and
// Int(i, j) the comm of edges with both ends inside positions [i, j),
//   cost(i, j) = PO[j] - PO[i] - Int(i, j)            (eq. 4 rewritten)
//   S(j)      = PO[j] + min_i V_j(i),   V_j(i) = S(i) - PO[i] - Int(i, j).
// Moving from j to j+1 only adds the in-edges of the node at position j, each
// lowering V(i) for every i at or before its source (eq. 5's subtracted sum).
// The recurrence is sequential in j, so one wave runs it with the window of
// the last R candidates held 64 lanes wide in registers: per step, a few
// predicated subtractions and one wave-wide (min value, min index) reduction.
// The in-edge lists are staged through LDS in blocks so that no step waits on
// a global load.  The memory bound lo(j) comes from a prefix sum of the
// memory in order (binary search), the greedy mode from the same prefix sums.
#include "cel_internal.h"

namespace cel {

// position arrays: memory, comm, out-going comm
__global__ void k_cluster_pos(int32_t n, const int32_t *order, const int32_t *out_ptr,
                              const int64_t *mem, const int64_t *ob, int64_t bw, int64_t lat,
                              int64_t *memp, int64_t *cq, int64_t *outc, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = order[p];
    const int64_t c = comm_of(ob[v], bw, lat);
    memp[p] = mem[v];
    cq[p] = c;
    outc[p] = c * (int64_t)(out_ptr[v + 1] - out_ptr[v]);
  }
}

// lo[j] (j = 1..n): first feasible start of a cluster ending before j;
// gend[s] (s = 0..n-1): end of the greedy cluster that starts at s.
__global__ void k_cluster_bounds(int32_t n, int32_t R, int64_t M, const int64_t *PM, int32_t *lo,
                                 int32_t *gend, const Status *st) {
  if (failed(st)) return;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < n;
       x += (int64_t)gridDim.x * blockDim.x) {
    {  // j = x + 1: smallest i in [0, j-1] with PM[j] - PM[i] <= M
      const int32_t j = (int32_t)x + 1;
      const int64_t target = PM[j] - M;
      int32_t a = 0, b = j;  // first i with PM[i] >= target (b = j: none)
      while (a < b) {
        const int32_t mid = (a + b) >> 1;
        if (PM[mid] < target) a = mid + 1;
        else b = mid;
      }
      int32_t l = j - R > a ? j - R : a;
      if (l > j - 1) l = j - 1;  // a single node is always a feasible cluster
      if (l < 0) l = 0;
      lo[j] = l;
    }
    {  // greedy: largest e in [s+1, min(n, s+R)] with PM[e] - PM[s] <= M, at least s+1
      const int32_t s = (int32_t)x;
      const int32_t hi = (int64_t)s + R < n ? s + R : n;
      const int64_t lim = PM[s] + M;
      int32_t a = s + 1, b = hi;  // last e in [s+1, hi] with PM[e] <= lim
      if (PM[s + 1] > lim) {
        gend[s] = s + 1;
      } else {
        while (a < b) {
          const int32_t mid = (a + b + 1) >> 1;
          if (PM[mid] <= lim) a = mid;
          else b = mid - 1;
        }
        gend[s] = a;
      }
    }
  }
}

constexpr int kDpBlk = 256;    // DP steps staged per block
constexpr int kDpEcap = 6144;  // in-edges staged per block

template <int SL>
__global__ void __launch_bounds__(64)
    k_cluster_dp(int32_t n, int32_t R, const int32_t *lo, const int32_t *pptr,
                 const int32_t *pidx, const int64_t *cq, const int64_t *PO, int32_t *P,
                 Status *st) {
  constexpr int RW = 64 * SL;
  __shared__ int32_t s_lo[kDpBlk];
  __shared__ int32_t s_ptr[kDpBlk + 1];
  __shared__ int32_t s_q[kDpEcap];
  __shared__ int64_t s_c[kDpEcap];
  if (failed(st)) return;
  (void)R;
  const int lane = threadIdx.x;
  int64_t v[SL];
  int32_t iv[SL];
#pragma unroll
  for (int s = 0; s < SL; s++) {
    v[s] = 0;
    iv[s] = -1;
  }
  if (lane == 0) iv[0] = 0;  // candidate i = 0 with V = S(0) - PO[0] = 0
  int64_t G = 0;
  for (int32_t j0 = 1; j0 <= n;) {
    // block of steps [j0, j1); in-edges of positions [j0, min(j1, n)) staged
    int32_t j1 = j0 + kDpBlk <= n + 1 ? j0 + kDpBlk : n + 1;
    const int32_t eb = pptr[j0 < n ? j0 : n];
    {
      int32_t a = j0 + 1, b = j1;  // largest j1 with staged edges <= cap
      while (a < b) {
        const int32_t mid = (a + b + 1) >> 1;
        if (pptr[mid < n ? mid : n] - eb <= kDpEcap) a = mid;
        else b = mid - 1;
      }
      j1 = a;
    }
    const int32_t ee = pptr[j1 < n ? j1 : n];
    const bool staged = ee - eb <= kDpEcap;
    for (int t = lane; t < j1 - j0; t += 64) s_lo[t] = lo[j0 + t];
    for (int t = lane; t <= j1 - j0; t += 64) {
      const int32_t jj = j0 + t < n ? j0 + t : n;
      s_ptr[t] = pptr[jj] - eb;
    }
    if (staged)
      for (int32_t k = lane; k < ee - eb; k += 64) {
        const int32_t q = pidx[eb + k];
        s_q[k] = q;
        s_c[k] = cq[q];
      }
    __syncthreads();
    for (int32_t j = j0; j < j1; j++) {
      const int32_t lj = s_lo[j - j0];
      int64_t bv = INT64_MAX;
      int32_t bi = INT32_MAX;
#pragma unroll
      for (int s = 0; s < SL; s++) {
        const int32_t i = iv[s];
        if (i >= lj && i < j && (v[s] < bv || (v[s] == bv && i < bi))) {
          bv = v[s];
          bi = i;
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const int64_t ov = __shfl_xor(bv, off);
        const int32_t oi = __shfl_xor(bi, off);
        if (ov < bv || (ov == bv && oi < bi)) {
          bv = ov;
          bi = oi;
        }
      }
      G = bv;
      if (lane == 0) P[j] = bi;
      if (j == n) break;
      // the node at position j joins the target side: subtract its in-edges
      const int32_t k0 = s_ptr[j - j0], k1 = s_ptr[j - j0 + 1];
      if (staged) {
        for (int32_t k = k0; k < k1; k++) {
          const int32_t q = s_q[k];
          const int64_t cu = s_c[k];
#pragma unroll
          for (int s = 0; s < SL; s++)
            if (iv[s] >= 0 && iv[s] <= q) v[s] -= cu;
        }
      } else {
        for (int32_t k = k0; k < k1; k++) {
          const int32_t q = pidx[eb + k];
          const int64_t cu = cq[q];
#pragma unroll
          for (int s = 0; s < SL; s++)
            if (iv[s] >= 0 && iv[s] <= q) v[s] -= cu;
        }
      }
      // new candidate i = j with V = S(j) - PO[j] = G
      const int r = j % RW;
#pragma unroll
      for (int s = 0; s < SL; s++)
        if (lane == (r & 63) && s == (r >> 6)) {
          v[s] = G;
          iv[s] = j;
        }
    }
    __syncthreads();
    j0 = j1;
  }
  if (lane == 0) st->s0 = PO[n] + G;  // S(n): the total inter-cluster comm
}

// breakpoints: follow P from n down to 0, flagging cluster starts
__global__ void k_backtrack(int32_t n, const int32_t *P, int32_t *flag, Status *st) {
  if (failed(st)) return;
  int32_t b = n, C = 0;
  while (b > 0) {
    const int32_t a = P[b];
    if (a < 0 || a >= b) {  // cannot happen: every step has a feasible predecessor
      raise_err(st, EB_ORDER);
      return;
    }
    b = a;
    flag[b] = 1;
    C++;
  }
  st->i0 = C;
}

__global__ void k_greedy_walk(int32_t n, const int32_t *gend, int32_t *flag, Status *st) {
  if (failed(st)) return;
  int32_t s = 0, C = 0;
  while (s < n) {
    flag[s] = 1;
    C++;
    s = gend[s];
  }
  st->i0 = C;
}

// cluster_id[order[p]] = (number of cluster starts at or before p) - 1
__global__ void k_label(int32_t n, const int32_t *order, const int32_t *incl, int32_t *cid,
                        const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x)
    cid[order[p]] = incl[p + 1] - 1;
}

// sum of c[u] over edges u -> v in different clusters (block per 256 sources)
__global__ void k_cut_cost(cel_graph g, int64_t bw, int64_t lat, const int32_t *cid, Status *st) {
  __shared__ int32_t ptr[257];
  __shared__ int64_t red[4];
  if (failed(st)) return;
  int64_t acc = 0;
  for_block_edges(g.out_ptr, g.n, ptr, [&](int32_t u, int32_t e) {
    if (cid[u] != cid[g.out_idx[e]]) acc += comm_of(g.ob[u], bw, lat);
  });
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int64_t t = red[0] + red[1] + red[2] + red[3];
    atomicAdd((unsigned long long *)&st->s0, (unsigned long long)t);
  }
}

template <int SL>
static void launch_dp(int32_t n, int32_t R, const int32_t *lo, const int32_t *pptr,
                      const int32_t *pidx, const int64_t *cq, const int64_t *PO, int32_t *P,
                      Status *st, hipStream_t s) {
  KTimer kt(s, "k_cluster_dp");
  k_cluster_dp<SL><<<1, 64, 0, s>>>(n, R, lo, pptr, pidx, cq, PO, P, st);
}

}  // namespace cel

using namespace cel;

extern "C" int cel_cluster(const cel_graph *g, const cel_devices *d, const int32_t *order,
                           int32_t R, int64_t M, int32_t mode, int32_t *cluster_id,
                           int32_t *n_clusters, int64_t *cut_cost, hipStream_t s) {
  const char *fn = "cel_cluster";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n;
  if (!n_clusters || !cut_cost || (n > 0 && (!order || !cluster_id)))
    return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  if (R < 1 || R > 4096) return set_error(CEL_E_ARG, "%s: R = %d not in [1, 4096]", fn, R);
  if (M < -1) return set_error(CEL_E_ARG, "%s: M < -1", fn);
  if (mode != CEL_CLUSTER_DP && mode != CEL_CLUSTER_GREEDY)
    return set_error(CEL_E_ARG, "%s: unknown mode", fn);
  if (M == -1) {
    int64_t mc = d->cap[0];
    for (int i = 1; i < d->D; i++) mc = d->cap[i] < mc ? d->cap[i] : mc;
    M = mc / 4;
  }
  Scratch sc(s);
  Status *st;
  int32_t *tmp, *pos;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(sc.get(&pos, n));
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, s));
  CEL_TRY(check_topo_order(g, order, pos, st, s));
  if (n == 0) {
    Status h;
    CEL_TRY(read_status(st, &h, s));
    if (h.err) return status_error(h, fn);
    *n_clusters = 0;
    *cut_cost = 0;
    return CEL_OK;
  }
  int64_t *memp, *cq, *outc, *PM, *PO;
  int32_t *lo, *gend, *flag, *incl;
  CEL_TRY(sc.get(&memp, n));
  CEL_TRY(sc.get(&cq, n));
  CEL_TRY(sc.get(&outc, n));
  CEL_TRY(sc.get(&PM, (int64_t)n + 1));
  CEL_TRY(sc.get(&PO, (int64_t)n + 1));
  CEL_TRY(sc.get(&lo, (int64_t)n + 1));
  CEL_TRY(sc.get(&gend, n));
  CEL_TRY(sc.get(&flag, n));
  CEL_TRY(sc.get(&incl, (int64_t)n + 1));
  k_cluster_pos<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, g->out_ptr, g->mem, g->ob, d->bw,
                                                      d->lat, memp, cq, outc, st);
  CEL_TRY(exclusive_scan_i64(memp, PM, n, sc, s));
  CEL_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t) * (size_t)n, s));
  k_cluster_bounds<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, R, M, PM, lo, gend, st);
  if (mode == CEL_CLUSTER_DP) {
    int32_t *pptr, *pidx, *P;
    CEL_TRY(sc.get(&pptr, (int64_t)n + 1));
    CEL_TRY(sc.get(&pidx, g->m));
    CEL_TRY(sc.get(&P, (int64_t)n + 1));
    CEL_TRY(exclusive_scan_i64(outc, PO, n, sc, s));
    CEL_TRY(relabel_csr(n, order, pos, g->in_ptr, g->in_idx, pptr, pidx, sc, s, st));
    if (R <= 64) launch_dp<1>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 128) launch_dp<2>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 256) launch_dp<4>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 512) launch_dp<8>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 1024) launch_dp<16>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 2048) launch_dp<32>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else launch_dp<64>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    k_backtrack<<<1, 1, 0, s>>>(n, P, flag, st);
  } else {
    k_greedy_walk<<<1, 1, 0, s>>>(n, gend, flag, st);
  }
  CEL_TRY(exclusive_scan_i32(flag, incl, n, sc, s));
  k_label<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, incl, cluster_id, st);
  if (mode == CEL_CLUSTER_GREEDY)
    k_cut_cost<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, st);
  CEL_HIP(hipGetLastError());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  *n_clusters = h.i0;
  *cut_cost = h.s0;
  return CEL_OK;
}
