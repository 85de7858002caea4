// cel_blevel: b-level (eq. 3), t-level (eq. 2), critical path and the
// priority order (Section 5.1.3).
//
// Nodes are first relabelled into the positions of the level order, so each
// level is a contiguous range and per-node data is read coalesced.  The
// longest paths are found by policy iteration (lp_policy.hip), which needs
// about ten pointer-jumping passes where the levels are many; when it does
// not converge within its budget, the sweep over levels (sweep.hip) pulls, at
// every node, the values of its successors (b-level, reverse sweep) or
// predecessors (t-level, forward sweep).  Both are exact and independent of
// scheduling.
#include "cel_internal.h"

namespace cel {

// per position: w and w + c (c = 0 with CEL_COMM_OFF)
__global__ void k_node_costs(int32_t n, const int32_t *order, const int64_t *w, const int64_t *ob,
                             int64_t bw, int64_t lat, int comm_off, int64_t *wp, int64_t *wcp,
                             const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = order[p];
    const int64_t wv = w[v];
    wp[p] = wv;
    wcp[p] = comm_off ? wv : wv + comm_of(ob[v], bw, lat);
  }
}

// per position: the weight of the longest-path recurrences, w + c when the
// node has successors, w for a sink
__global__ void k_lp_weights(int32_t n, const int32_t *sptr, const int64_t *wp, const int64_t *wcp,
                             int64_t *wv, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x)
    wv[p] = sptr[p + 1] > sptr[p] ? wcp[p] : wp[p];
}

// out[order[p]] = val[p] (out may be NULL); *maxout = max val
__global__ void k_scatter_max(int32_t n, const int32_t *order, const int64_t *val, int64_t *out,
                              const Status *st, int64_t *maxout) {
  __shared__ int64_t red[4];
  if (failed(st)) return;
  int64_t mx = 0;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int64_t x = val[p];
    if (out) out[order[p]] = x;
    mx = x > mx ? x : mx;
  }
  for (int off = 32; off > 0; off >>= 1) {
    int64_t y = __shfl_xor(mx, off);
    mx = y > mx ? y : mx;
  }
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t r = red[0];
    for (int i = 1; i < (int)(blockDim.x >> 6); i++) r = red[i] > r ? red[i] : r;
    atomicMax((unsigned long long *)maxout, (unsigned long long)r);
  }
}

// priority keys: larger b-level first, then id
__global__ void k_prio_keys(int32_t n, const int32_t *order, const int64_t *blp, uint64_t *keys,
                            uint32_t *ids, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    keys[p] = (uint64_t)(INT64_MAX - blp[p]);
    ids[p] = (uint32_t)order[p];
  }
}

}  // namespace cel

using namespace cel;

CEL_PHASE_READER(cel_debug_phases_blevel)

// How the calling thread's last cel_blevel call found its longest paths.
struct BlInfo {
  int32_t path_b, iters_b, path_t, iters_t;
};
static thread_local BlInfo t_bl_info{1, 0, 2, 0};
static thread_local int t_lp_mode = 1;

namespace cel {
bool policy_iteration_on() { return t_lp_mode > 0; }
bool policy_iteration_packed() { return t_lp_mode == 1; }
}  // namespace cel

extern "C" int cel_blevel_info(int32_t *info) {
  if (!info) return set_error(CEL_E_ARG, "cel_blevel_info: NULL argument");
  info[0] = t_bl_info.path_b;
  info[1] = t_bl_info.iters_b;
  info[2] = t_bl_info.path_t;
  info[3] = t_bl_info.iters_t;
  return CEL_OK;
}

extern "C" int cel_policy_iteration(int mode) {
  if (mode < 0) return set_error(CEL_E_ARG, "cel_policy_iteration: negative mode");
  const int was = t_lp_mode;
  t_lp_mode = mode;
  return was;
}

extern "C" int cel_blevel(const cel_graph *g, const cel_devices *d, const int32_t *level,
                          const int32_t *level_ptr, const int32_t *order_id, int32_t L,
                          int32_t flags, int64_t *blevel, int64_t *tlevel, int32_t *prio_order,
                          int64_t *cp, hipStream_t s) {
  const char *fn = "cel_blevel";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n;
  if (!cp || !level_ptr || (n > 0 && (!level || !order_id || !blevel)))
    return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  if (L < 0 || L > n || (n > 0 && L == 0)) return set_error(CEL_E_ARG, "%s: n_levels out of range", fn);
  if (flags & ~CEL_COMM_OFF) return set_error(CEL_E_ARG, "%s: unknown flags", fn);
  Scratch sc(s);
  Status *st;
  int32_t *tmp, *pos, *sptr, *sidx;
  int64_t *wp, *wcp, *blp;
  CEL_TRY(sc.get(&st, 1));
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(sc.get(&pos, n));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, sc, s));
  CEL_TRY(check_level_order(g, order_id, level, level_ptr, L, pos, st, s));
  CEL_TRY(sc.get(&sptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&sidx, g->m));
  CEL_TRY(sc.get(&wp, n));
  CEL_TRY(sc.get(&wcp, n));
  CEL_TRY(sc.get(&blp, n));
  CEL_TRY(relabel_csr(n, g->m, order_id, pos, g->out_ptr, g->out_idx, sptr, sidx, sc, s, st));
  k_node_costs<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order_id, g->w, g->ob, d->bw, d->lat,
                                                     (flags & CEL_COMM_OFF) ? 1 : 0, wp, wcp, st);
  // Policy iteration first (b-level, then t-level), whole-GPU kernels one
  // after the other; what does not converge takes the level sweep.
  int32_t *pptr = nullptr, *pidx = nullptr;
  int64_t *tlp = nullptr, *wv;
  CEL_TRY(sc.get(&wv, n));
  k_lp_weights<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, sptr, wp, wcp, wv, st);
  if (tlevel && n > 0) {
    CEL_TRY(sc.get(&pptr, (int64_t)n + 1));
    CEL_TRY(sc.get(&pidx, g->m));
    CEL_TRY(sc.get(&tlp, n));
    CEL_TRY(relabel_csr(n, g->m, order_id, pos, g->in_ptr, g->in_idx, pptr, pidx, sc, s, st));
  }
  bool lb = false, lt = false;
  if (policy_iteration_on()) {
    CEL_TRY(lp_policy(n, g->m, L, 0, sptr, sidx, wv, 0, blp, &st->i0, "k_blevel_policy", sc, s,
                      st, &lb));
    if (tlp)
      CEL_TRY(lp_policy(n, g->m, L, 0, pptr, pidx, wv, 1, tlp, &st->i2, "k_tlevel_policy", sc, s,
                        st, &lt));
  }
  bool sweep_b = true, sweep_t = tlp != nullptr;
  t_bl_info = {1, 0, tlp ? 1 : 2, 0};
  // the outputs from the policy-iteration values, queued before the status
  // is read: one host round trip when the iteration converged (a value that
  // did not converge is a real path's length, never above the exact one, so
  // the maxima of the sweep's exact values replace it below)
  auto outputs = [&](bool b, bool t, hipStream_t sb, hipStream_t stt) -> int {
    if (t && tlp)
      k_scatter_max<<<grid_for(n, 256, 2048), 256, 0, stt>>>(n, order_id, tlp, tlevel, st, &st->s1);
    if (b) {
      k_scatter_max<<<grid_for(n, 256, 2048), 256, 0, sb>>>(n, order_id, blp, blevel, st, &st->s0);
      if (prio_order && n > 0) {
        uint64_t *keys;
        CEL_TRY(sc.get(&keys, n));
        uint32_t *ids = reinterpret_cast<uint32_t *>(prio_order);
        k_prio_keys<<<grid_for(n, 256, 4096), 256, 0, sb>>>(n, order_id, blp, keys, ids, st);
        CEL_TRY(segmented_sort(keys, ids, level_ptr, L, n, sc, sb, st));
      }
    }
    CEL_HIP(hipGetLastError());
    return CEL_OK;
  };
  if (lb && (lt || !tlp)) {
    CEL_TRY(outputs(true, true, s, s));
    Status h;
    CEL_TRY(read_status(st, &h, s));
    if (h.err) return status_error(h, fn);
    if (h.i0 && (!tlp || h.i2)) {
      t_bl_info = {0, h.i1, tlp ? 0 : 2, tlp ? h.i3 : 0};
      *cp = h.s0;
      return CEL_OK;
    }
  }
  if (lb || lt) {
    Status h;
    CEL_TRY(read_status(st, &h, s));
    if (h.err) return status_error(h, fn);
    k_fill_i64<<<1, 64, 0, s>>>(&st->s0, 2, 0);  // s0, s1: the maxima, taken again below
    if (lb) {
      sweep_b = !h.i0;
      t_bl_info.path_b = h.i0 ? 0 : 1;
      t_bl_info.iters_b = h.i1;
    }
    if (lt) {
      sweep_t = !h.i2;
      t_bl_info.path_t = h.i2 ? 0 : 1;
      t_bl_info.iters_t = h.i3;
    }
  }
  // The level sweeps: the t-level (eq. 2) needs no b-level, so its sweep runs
  // on a side stream and the two single-workgroup sweeps overlap on two CUs.
  // Both preparations are queued before either plan is read back.
  SideFork fk;
  SweepPlan pt, pb;
  if (sweep_t) {
    CEL_TRY(fk.start(s));
    CEL_TRY(sweep_prepare(pt, false, n, g->m, L, level_ptr, order_id, level, pptr, pidx, wp, wcp,
                          tlp, sc, fk.side(), st));
  }
  if (sweep_b)
    CEL_TRY(sweep_prepare(pb, true, n, g->m, L, level_ptr, order_id, level, sptr, sidx, wp, wcp,
                          blp, sc, s, st));
  if (sweep_t) CEL_TRY(sweep_run(pt, fk.side(), st, "k_tlevel_sweep"));
  if (sweep_b) CEL_TRY(sweep_run(pb, s, st, "k_blevel_sweep"));
  CEL_TRY(outputs(true, true, s, sweep_t ? fk.side() : s));
  CEL_TRY(fk.join());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  *cp = h.s0;
  return CEL_OK;
}
