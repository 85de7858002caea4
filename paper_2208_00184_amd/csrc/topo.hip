// cel_topo_levels: level-synchronous Kahn ordering (Section 4.2.2).
//
// One workgroup runs all levels: a level costs a few dependent L2 round trips
// (frontier id -> adjacency -> in-degree atomic), so keeping the whole loop in
// one workgroup with workgroup barriers is far cheaper than one launch or one
// grid-wide barrier per level.  Frontiers are appended to the caller's
// order_id buffer; each level's slice is then sorted by id.
#include "cel_internal.h"

namespace cel {

constexpr int kKahnB = 1024;
constexpr int kKahnHeavy = 64;    // out-degree above which the whole block shares a node
constexpr int kKahnFront = 8192;  // frontier entries mirrored in LDS
constexpr int kKahnE = 4;         // out-edges per node whose loads and atomics go out together

// Removes edge e's target's in-edge; the node that removes the last one
// appends the target to the next frontier (global order, and the LDS mirror
// while it has room).
__device__ inline void kahn_append(int32_t *F, int32_t *s_front, int32_t *s_tail, int32_t fe,
                                   int32_t v) {
  const int32_t k = atomicAdd(s_tail, 1);
  F[k] = v;
  if (k - fe < kKahnFront) s_front[k - fe] = v;
}

__global__ void __launch_bounds__(kKahnB) k_kahn(cel_graph g, int32_t *cnt, int32_t *F,
                                                 int32_t *level, int32_t *lstart, Status *st) {
  __shared__ int32_t s_tail, s_nheavy;
  __shared__ int32_t s_heavy[kKahnB];
  __shared__ int32_t s_front[2][kKahnFront];  // the frontier being read, the one being built
  if (failed(st)) return;
  const int tid = threadIdx.x;
  const int32_t n = g.n;
  if (tid == 0) s_tail = 0;
  __syncthreads();
  for (int32_t v = tid; v < n; v += kKahnB)
    if (cnt[v] == 0) kahn_append(F, s_front[0], &s_tail, 0, v);
  __syncthreads();
  int32_t fb = 0, fe = s_tail, lvl = 0, cur = 0;
  while (fb < fe) {
    if (tid == 0) lstart[lvl] = fb;
    const int32_t *front = s_front[cur];
    int32_t *next = s_front[cur ^ 1];
    for (int32_t base = fb; base < fe; base += kKahnB) {
      if (tid == 0) s_nheavy = 0;
      __syncthreads();
      const int32_t i = base + tid;
      if (i < fe) {
        const int32_t u = i - fb < kKahnFront ? front[i - fb] : F[i];
        level[u] = lvl;
        const int32_t e0 = g.out_ptr[u], e1 = g.out_ptr[u + 1];
        if (e1 - e0 > kKahnHeavy) {
          s_heavy[atomicAdd(&s_nheavy, 1)] = u;
        } else {
          for (int32_t eb = e0; eb < e1; eb += kKahnE) {
            int32_t v[kKahnE], c[kKahnE];
#pragma unroll
            for (int q = 0; q < kKahnE; q++) v[q] = eb + q < e1 ? g.out_idx[eb + q] : -1;
#pragma unroll
            for (int q = 0; q < kKahnE; q++) c[q] = v[q] >= 0 ? atomicSub(&cnt[v[q]], 1) : 0;
#pragma unroll
            for (int q = 0; q < kKahnE; q++)
              if (c[q] == 1) kahn_append(F, next, &s_tail, fe, v[q]);  // last in-edge removed
          }
        }
      }
      __syncthreads();
      const int32_t nh = s_nheavy;
      for (int32_t h = 0; h < nh; h++) {
        const int32_t u = s_heavy[h];
        for (int32_t e = g.out_ptr[u] + tid; e < g.out_ptr[u + 1]; e += kKahnB) {
          const int32_t v = g.out_idx[e];
          if (atomicSub(&cnt[v], 1) == 1) kahn_append(F, next, &s_tail, fe, v);
        }
      }
      __syncthreads();
    }
    fb = fe;
    fe = s_tail;
    lvl++;
    cur ^= 1;
    __syncthreads();  // everyone has read s_tail before the next level appends
  }
  if (tid == 0) {
    st->i0 = lvl;     // number of levels
    st->i1 = s_tail;  // nodes taken; < n means a cycle
    lstart[lvl] = s_tail;
  }
}

__global__ void k_zero_u64(uint64_t *p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

}  // namespace cel

using namespace cel;

extern "C" int cel_topo_levels(const cel_graph *g, int32_t *level, int32_t *order_id,
                               int32_t *level_ptr, int32_t *n_levels, hipStream_t s) {
  if (!g || !n_levels || !level_ptr) return set_error(CEL_E_ARG, "cel_topo_levels: NULL argument");
  if (g->n < 0 || g->m < 0) return set_error(CEL_E_ARG, "cel_topo_levels: negative size");
  if (!g->out_ptr || !g->in_ptr || (g->m > 0 && (!g->out_idx || !g->in_idx)) ||
      (g->n > 0 && (!g->w || !g->mem || !g->ob || !level || !order_id)))
    return set_error(CEL_E_ARG, "cel_topo_levels: NULL array");
  const int32_t n = g->n;
  Scratch sc(s);
  Status *st;
  int32_t *cnt;
  CEL_TRY(sc.get(&st, 1));
  CEL_TRY(sc.get(&cnt, n));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(check_graph(g, 1, 0, /*bound=*/false, st, cnt, sc, s));
  {
    KTimer kt(s, "k_kahn");
    k_kahn<<<1, kKahnB, 0, s>>>(*g, cnt, order_id, level, level_ptr, st);
  }
  CEL_HIP(hipGetLastError());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, "cel_topo_levels");
  if (h.i1 != n) return set_error(CEL_E_CYCLE, "cel_topo_levels: the graph has a cycle (%d of %d nodes ordered)", h.i1, n);
  const int32_t L = h.i0;
  *n_levels = L;
  if (n == 0) return CEL_OK;
  // sort each level's frontier slice by id
  uint64_t *keys;
  CEL_TRY(sc.get(&keys, n));
  k_zero_u64<<<grid_for(n, 256, 4096), 256, 0, s>>>(keys, n);
  CEL_TRY(segmented_sort(keys, reinterpret_cast<uint32_t *>(order_id), level_ptr, L, n, sc, s, st));
  CEL_HIP(hipStreamSynchronize(s));
  return CEL_OK;
}
