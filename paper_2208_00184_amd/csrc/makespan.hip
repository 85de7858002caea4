// cel_makespan: makespan of K placements (eq. 7 without insertion).
//
// Sequential definition: nodes in `order`; ready(v) = max over preds p of
// fin(p) + [dev p != dev v] c(p); start(v) = max(ready(v), free(dev v));
// fin(v) = start(v) + w(v); free(dev v) = fin(v).
//
// Level-parallel evaluation.  `order` is level-monotone, so nodes of one level
// have no edges among themselves and every ready() of the level depends only
// on earlier levels: all of them are computed in parallel.  What remains
// sequential is each device's FIFO inside the level.  A node on device d maps
// the device's free time x to max(ready + w, x + w): a function x -> max(a,
// x + b) with a = ready + w, b = w.  Such functions compose associatively,
//   (a1, b1) then (a2, b2)  =  (max(a2, a1 + b2), b1 + b2),
// so after a stable partition of the level's nodes by device, one segmented
// scan (segments = devices) gives every finish time exactly, seeded with the
// device's free time carried from the previous level.
//
// One workgroup evaluates one placement; a batch of K placements runs K
// independent workgroups that share the graph structure through L2/MALL.
#include "cel_internal.h"

namespace cel {

// device per position, with range check (devp[k][p] = node_dev[k][order[p]])
__global__ void k_dev_gather(int32_t K, int32_t n, const int32_t *order, const uint8_t *node_dev,
                             int32_t D, uint8_t *devp, Status *st) {
  if (failed(st)) return;
  uint32_t bad = 0;
  const int64_t tot = (int64_t)K * n;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < tot;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = i / n, p = i - k * n;
    const uint8_t dv = node_dev[k * n + order[p]];
    if (dv >= D) bad |= EB_ARG;
    devp[i] = dv;
  }
  if (bad) raise_err(st, bad);
}

__global__ void k_pos_costs(int32_t n, const int32_t *order, const int64_t *w, const int64_t *ob,
                            int64_t bw, int64_t lat, int64_t *wp, int64_t *cq, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = order[p];
    wp[p] = w[v];
    cq[p] = comm_of(ob[v], bw, lat);
  }
}

template <int B>
__global__ void __launch_bounds__(B)
    k_makespan_sweep(int32_t n, int32_t L, const int32_t *lp, const int32_t *pptr,
                     const int32_t *pidx, const int64_t *wp, const int64_t *cq,
                     const uint8_t *devp, int64_t *finp, int64_t *makespan, const Status *st) {
  constexpr int NW = B / 64;
  static_assert(B >= 256, "device partition uses 256 threads");
  __shared__ int64_t s_avail[256];
  __shared__ int32_t s_wcnt[NW][256];
  __shared__ int32_t s_dbase[256];
  __shared__ int32_t s_dsum[4];
  __shared__ int64_t s_a[B], s_b[B];
  __shared__ int32_t s_pos[B];
  __shared__ uint8_t s_dev[B + 1];
  __shared__ int64_t s_wa[NW], s_wb[NW];
  __shared__ int32_t s_wf[NW];
  __shared__ int64_t s_red[NW];
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t koff = (int64_t)blockIdx.x * n;
  const uint8_t *dk = devp + koff;
  int64_t *fk = finp + koff;
  for (int i = tid; i < 256; i += B) s_avail[i] = 0;
  int64_t mk = 0;
  for (int32_t l = 0; l < L; l++) {
    const int32_t b = lp[l], e = lp[l + 1];
    for (int32_t base = b; base < e; base += B) {
      const int32_t cnt = e - base < B ? e - base : B;
      const bool act = tid < cnt;
      const int32_t p = base + tid;
      for (int i = tid; i < NW * 256; i += B) (&s_wcnt[0][0])[i] = 0;
      __syncthreads();  // earlier finishes and free times visible; counters clear
      // ready time of every node of the chunk (independent within a level)
      int dv = 255;
      int64_t a = 0, w = 0;
      if (act) {
        dv = dk[p];
        int64_t ready = 0;
        const int32_t k1 = pptr[p + 1];
        for (int32_t k = pptr[p]; k < k1; k++) {
          const int32_t q = pidx[k];
          const int64_t f = fk[q] + (dk[q] != dv ? cq[q] : 0);
          ready = f > ready ? f : ready;
        }
        w = wp[p];
        a = ready + w;
      }
      // stable partition by device: rank among same-device lanes of the wave
      uint64_t eq = ~0ull;
      for (int bit = 0; bit < 8; bit++) {
        const int on = (dv >> bit) & 1;
        const uint64_t bb = __ballot(on);
        eq &= on ? bb : ~bb;
      }
      const int rank = __popcll(eq & ((1ull << lane) - 1ull));
      if (act && rank == 0) s_wcnt[wv][dv] = __popcll(eq);
      __syncthreads();
      int32_t tot = 0;
      if (tid < 256) {
        for (int w2 = 0; w2 < NW; w2++) {
          const int32_t c = s_wcnt[w2][tid];
          s_wcnt[w2][tid] = tot;
          tot += c;
        }
      }
      int32_t inc = tot;
      for (int off = 1; off < 64; off <<= 1) {
        const int32_t y = __shfl_up(inc, off);
        if (lane >= off) inc += y;
      }
      if (tid < 256 && lane == 63) s_dsum[wv] = inc;
      __syncthreads();
      if (tid < 256) {
        int32_t bv = inc - tot;
        for (int w2 = 0; w2 < wv; w2++) bv += s_dsum[w2];
        s_dbase[tid] = bv;
      }
      __syncthreads();
      if (act) {
        const int q = s_dbase[dv] + s_wcnt[wv][dv] + rank;
        s_a[q] = a;
        s_b[q] = w;
        s_pos[q] = p;
        s_dev[q] = (uint8_t)dv;
      }
      __syncthreads();
      // segmented scan of (a, b) in device-grouped order
      const bool aq = tid < cnt;
      int64_t sa = 0, sb = 0;
      int dq = 255;
      bool f = true;
      if (aq) {
        sa = s_a[tid];
        sb = s_b[tid];
        dq = s_dev[tid];
        f = (tid == 0) || (s_dev[tid - 1] != dq);
      }
      for (int off = 1; off < 64; off <<= 1) {
        const int64_t ua = __shfl_up(sa, off), ub = __shfl_up(sb, off);
        const int uf = __shfl_up((int)f, off);
        if (lane >= off && !f) {
          sa = (ua + sb) > sa ? ua + sb : sa;
          sb = ub + sb;
          f = uf != 0;
        }
      }
      if (lane == 63) {
        s_wa[wv] = sa;
        s_wb[wv] = sb;
        s_wf[wv] = f ? 1 : 0;
      }
      __syncthreads();
      if (aq && !f && wv > 0) {  // segment began in an earlier wave: prepend their totals
        int64_t ca = s_wa[wv - 1], cb = s_wb[wv - 1];
        bool done = s_wf[wv - 1] != 0;
        for (int w2 = wv - 2; w2 >= 0 && !done; w2--) {
          ca = (s_wa[w2] + cb) > ca ? s_wa[w2] + cb : ca;
          cb = s_wb[w2] + cb;
          done = s_wf[w2] != 0;
        }
        sa = (ca + sb) > sa ? ca + sb : sa;
        sb = cb + sb;
      }
      int64_t fin = 0;
      bool last = false;
      if (aq) {
        const int64_t viafree = s_avail[dq] + sb;
        fin = viafree > sa ? viafree : sa;
        fk[s_pos[tid]] = fin;
        mk = fin > mk ? fin : mk;
        last = (tid + 1 == cnt) || (s_dev[tid + 1] != dq);
      }
      __syncthreads();  // every read of s_avail is done
      if (last) s_avail[dq] = fin;
    }
  }
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t y = __shfl_xor(mk, off);
    mk = y > mk ? y : mk;
  }
  if (lane == 0) s_red[wv] = mk;
  __syncthreads();
  if (tid == 0) {
    int64_t r = s_red[0];
    for (int i = 1; i < NW; i++) r = s_red[i] > r ? s_red[i] : r;
    makespan[blockIdx.x] = r;
  }
}

// finish/start by node id from position-space finishes
__global__ void k_makespan_out(int32_t K, int32_t n, const int32_t *order, const int64_t *finp,
                               const int64_t *wp, int64_t *start, int64_t *finish,
                               const Status *st) {
  if (failed(st)) return;
  const int64_t tot = (int64_t)K * n;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < tot;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = i / n, p = i - k * n;
    const int64_t v = k * n + order[p];
    const int64_t f = finp[i];
    if (finish) finish[v] = f;
    if (start) start[v] = f - wp[p];
  }
}

__global__ void k_fill_i64(int64_t *p, int64_t n, int64_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

}  // namespace cel

using namespace cel;

extern "C" int cel_makespan(const cel_graph *g, const cel_devices *d, const int32_t *order,
                            const int32_t *level, const int32_t *level_ptr, int32_t L, int32_t K,
                            const uint8_t *node_dev, int64_t *start, int64_t *finish,
                            int64_t *makespan, hipStream_t s) {
  const char *fn = "cel_makespan";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n;
  if (!makespan || !level_ptr || K < 1 || (n > 0 && (!order || !level || !node_dev)))
    return set_error(CEL_E_ARG, "%s: NULL argument or K < 1", fn);
  if (L < 0 || L > n || (n > 0 && L == 0)) return set_error(CEL_E_ARG, "%s: n_levels out of range", fn);
  Scratch sc(s);
  Status *st;
  int32_t *tmp, *pos, *pptr, *pidx;
  int64_t *wp, *cq, *finp;
  uint8_t *devp;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  if (n == 0) {
    k_fill_i64<<<grid_for(K, 256, 1024), 256, 0, s>>>(makespan, K, 0);
    CEL_HIP(hipGetLastError());
    CEL_HIP(hipStreamSynchronize(s));
    return CEL_OK;
  }
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(sc.get(&pos, n));
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, s));
  CEL_TRY(check_level_order(g, order, level, level_ptr, L, pos, st, s));
  CEL_TRY(sc.get(&pptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&pidx, g->m));
  CEL_TRY(sc.get(&wp, n));
  CEL_TRY(sc.get(&cq, n));
  CEL_TRY(sc.get(&devp, (int64_t)K * n));
  CEL_TRY(sc.get(&finp, (int64_t)K * n));
  CEL_TRY(relabel_csr(n, order, pos, g->in_ptr, g->in_idx, pptr, pidx, sc, s, st));
  k_pos_costs<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, g->w, g->ob, d->bw, d->lat, wp, cq,
                                                    st);
  k_dev_gather<<<grid_for((int64_t)K * n, 256, 8192), 256, 0, s>>>(K, n, order, node_dev, d->D,
                                                                  devp, st);
  if (K == 1) {
    KTimer kt(s, "k_makespan_sweep");
    k_makespan_sweep<1024><<<1, 1024, 0, s>>>(n, L, level_ptr, pptr, pidx, wp, cq, devp, finp,
                                              makespan, st);
  } else {
    KTimer kt(s, "k_makespan_batch");
    k_makespan_sweep<256><<<(unsigned)K, 256, 0, s>>>(n, L, level_ptr, pptr, pidx, wp, cq, devp,
                                                      finp, makespan, st);
  }
  if (start || finish)
    k_makespan_out<<<grid_for((int64_t)K * n, 256, 8192), 256, 0, s>>>(K, n, order, finp, wp, start,
                                                                      finish, st);
  CEL_HIP(hipGetLastError());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  return CEL_OK;
}
