// Ring-buffer level sweep: the b-level (eq. 3, REVERSE) and the t-level
// (eq. 2, forward) of every node in one workgroup.
//
//   b-level: out[p] = cst[p] + max(0, max over successors q of x[q]),  x = out
//            (cst = w for a sink, w + c otherwise)
//   t-level: out[p] = max(0, max over predecessors q of x[q]),  x = out + w + c
//
// Positions are those of a level order, so a level is a contiguous range and
// every neighbour of a level lies in another level.  Levels are dependent
// steps; the sweep keeps them cheap by splitting the work between the waves
// of one workgroup:
//  - wave 0 (the compute wave) runs the levels.  A node's value is its folded
//    far maximum and at most kNear gathers from an LDS ring that holds the
//    pull values x of the last kRing positions computed; it writes its own x
//    there only.  No workgroup barrier inside a run of narrow levels: the
//    compute wave only waits on LDS flags.
//  - the other waves stage positions ahead of it, 256 at a time: they copy
//    each position's precomputed pull record (the ring slots of its near
//    neighbours) and folds the values of its far neighbours (those kRing or
//    more positions away, or outside the run of narrow levels: final long
//    before) into the position's base maximum.  Far values are read from
//    global memory with device-coherent loads; they start as -1, so a value
//    not yet visible is simply read again.  Before a staging task overwrites
//    ring slots it copies the values they hold out to global memory.
// Which neighbours are near, and their ring slots, depend only on the graph
// and the order: a grid-wide pass prepares them for every position before the
// sweep.  Levels wider than kWideW, or holding a node with more than kHeavyDeg
// neighbours, are run by the whole workgroup straight from global memory
// (block mode), between barriers; they split the narrow levels into runs
// (segments) that each start with an empty ring.  A level with at least
// kGridE edges or kGridW nodes (a DNN graph's sources: weights and inputs) is
// more work than one CU should do: it is a grid level, run by kernels over the
// whole GPU between launches of the ring kernel.  The host learns where the
// grid levels are from a small table the preparation writes.
#include "cel_internal.h"

namespace cel {

constexpr int kSwB = 512;               // 8 waves: 1 compute, 7 staging
constexpr int kRing = 2048;             // positions held in the LDS ring
constexpr int kRMask = kRing - 1;
constexpr int kWideW = 1536;            // wider levels run in block mode (< kRing - kStage)
constexpr int kHeavyDeg = 4096;         // a node with more neighbours puts its level in block mode
constexpr int kStage = 256;             // positions per staging task (4 rows)
constexpr int kNF = kRing / kStage;     // staging flags in the ring
constexpr int kNear = 8;                // near neighbours held in a pull record
constexpr int kBP = 8;                  // positions per thread and pass in block mode
static_assert(kWideW + kStage < kRing, "a narrow level and a staging task fit the ring");
constexpr int kGridE = 16384;           // a level of this many edges or nodes is a grid level
constexpr int kGridW = 16384;
constexpr int kGridRow = 64;            // grid levels: larger rows are split into chunks
constexpr int kGridChunk = 4096;        // edges per workgroup of a split row
constexpr int kGridB = 256;
constexpr uint32_t kZeroSlot = kRing;   // ring slot that always reads 0
constexpr int kHeavyNear = 15;          // count field: more near neighbours than kNear

// Pull record of a position (16 bytes): eight 16-bit ring slots of near
// neighbours (kZeroSlot when unused); bits 12..15 of the first entry hold
// their count.  A position with more than kNear near neighbours has count
// kHeavyNear and only kZeroSlot entries; its slot list lies in a global
// array (hidx, from hptr[p]).  Every record thus names in-range slots only.
__device__ inline uint32_t rec_count(const uint4 &r) { return (r.x >> 12) & 15u; }


// -------------------------------------------------------------- preparation

// Levels out of ring mode (wide[l] = 1): wider than kWideW, holding a node
// with more than kHeavyDeg neighbours, or grid levels (grid[l] = 1: at least
// kGridE edges or kGridW nodes).
__global__ void k_sw_wide(int32_t n, int32_t L, const int32_t *lp, const int32_t *rptr,
                          const int32_t *order, const int32_t *level, int32_t *wide,
                          int32_t *grid, const Status *st) {
  if (failed(st)) return;
  const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x, step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t l = i0; l < L; l += step) {
    const int32_t w = lp[l + 1] - lp[l], e = rptr[lp[l + 1]] - rptr[lp[l]];
    const bool g = w >= kGridW || e >= kGridE;
    grid[l] = g ? 1 : 0;
    if (g || w > kWideW) wide[l] = 1;
  }
  for (int64_t p = i0; p < n; p += step)
    if (rptr[p + 1] - rptr[p] > kHeavyDeg) wide[level[order[p]]] = 1;
}

// segment starts: the first level, every block-mode level and the level after one
__global__ void k_sw_segflag(int32_t L, const int32_t *wide, int32_t *flag, const Status *st) {
  if (failed(st)) return;
  for (int64_t l = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; l < L;
       l += (int64_t)gridDim.x * blockDim.x)
    flag[l] = (l == 0 || wide[l] || wide[l - 1]) ? 1 : 0;
}

// seg[k] = first level of segment k, seg[nseg] = L; segid[l] = segment of l
__global__ void k_sw_segfill(int32_t L, const int32_t *flag, const int32_t *pre, int32_t *seg,
                             int32_t *segid, int32_t *nseg, const Status *st) {
  if (failed(st)) return;
  for (int64_t l = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; l < L;
       l += (int64_t)gridDim.x * blockDim.x) {
    const int32_t k = pre[l] + flag[l] - 1;
    segid[l] = k;
    if (flag[l]) seg[k] = (int32_t)l;
    if (l == L - 1) {
      seg[k + 1] = L;
      *nseg = k + 1;
    }
  }
}

// Per position: its pull record, its cost term, and how many far neighbours
// and (past kNear) near neighbours it has.  PASS 1 fills the far lists and the
// long slot lists.  Positions of block-mode levels get neither; those of grid
// levels with more than kGridRow neighbours count their chunks (gk).
template <bool REV, int PASS>
__global__ void k_sw_prep(int32_t n, const int32_t *lp, const int32_t *rptr, const int32_t *ridx,
                          const int32_t *order, const int32_t *level, const int32_t *wide,
                          const int32_t *grid, const int32_t *seg, const int32_t *segid,
                          const int64_t *wp, const int64_t *wcp, uint4 *rec, int64_t *cst,
                          int32_t *fcnt, int32_t *hcnt, int32_t *gk, const int32_t *fptr,
                          int32_t *fidx, const int32_t *hptr, int32_t *hidx, int32_t *rmax,
                          const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t l = level[order[p]];
    const int32_t e0 = rptr[p], e1 = rptr[p + 1];
    if (PASS == 0) {
      cst[p] = (REV && e0 == e1) ? wp[p] : wcp[p];
      gk[p] = (grid[l] && e1 - e0 > kGridRow) ? (e1 - e0 + kGridChunk - 1) / kGridChunk : 0;
    }
    if (wide[l]) {
      if (PASS == 0) {
        rec[p] = make_uint4(kZeroSlot | kZeroSlot << 16, kZeroSlot | kZeroSlot << 16,
                            kZeroSlot | kZeroSlot << 16, kZeroSlot | kZeroSlot << 16);
        fcnt[p] = 0;
        hcnt[p] = 0;
      }
      continue;
    }
    const int32_t k = segid[l];
    const int32_t S0 = lp[seg[k]], S1 = lp[seg[k + 1]];
    int32_t nn = 0, nf = 0;
    uint32_t ent[kNear];
#pragma unroll
    for (int j = 0; j < kNear; j++) ent[j] = kZeroSlot;
    for (int32_t e = e0; e < e1; e++) {
      const int32_t q = ridx[e];
      const bool near = REV ? (q < S1 && q - (int32_t)p < kRing) : (q >= S0 && (int32_t)p - q < kRing);
      if (near) {
        if (PASS == 0) {
#pragma unroll
          for (int j = 0; j < kNear; j++)
            if (j == nn) ent[j] = (uint32_t)(q & kRMask);
        } else if (hptr[p + 1] > hptr[p]) {
          hidx[hptr[p] + nn] = q & kRMask;
        }
        nn++;
      } else {
        if (PASS == 1) fidx[fptr[p] + nf] = q;
        nf++;
      }
    }
    if (PASS == 0) {
      fcnt[p] = nf;
      hcnt[p] = nn > kNear ? nn : 0;
      // the largest count of the row of 64 (from the level's start) holding p
      const int32_t lb = lp[l];
      if (nn > 0) atomicMax(&rmax[lb + ((int32_t)(p - lb) & ~63)], nn > kNear ? kHeavyNear : nn);
      if (nn > kNear)
        rec[p] = make_uint4(kZeroSlot | (uint32_t)kHeavyNear << 12 | kZeroSlot << 16,
                            kZeroSlot | kZeroSlot << 16, kZeroSlot | kZeroSlot << 16,
                            kZeroSlot | kZeroSlot << 16);
      else
        rec[p] = make_uint4(ent[0] | (uint32_t)nn << 12 | ent[1] << 16, ent[2] | ent[3] << 16,
                            ent[4] | ent[5] << 16, ent[6] | ent[7] << 16);
    }
  }
}

// The first position of every row of a narrow level carries the row's
// largest near count in bits 28..31 of its record (kHeavyNear: a position of
// the row has a long slot list), so the compute wave reads it uniformly.
__global__ void k_sw_rowmark(int32_t n, const int32_t *lp, const int32_t *order,
                             const int32_t *level, const int32_t *wide, const int32_t *rmax,
                             uint4 *rec, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t l = level[order[p]];
    if (wide[l] || (((int32_t)p - lp[l]) & 63) != 0) continue;
    rec[p].x = (rec[p].x & 0x0FFFFFFFu) | (uint32_t)rmax[p] << 28;
  }
}

// The plan the host reads back: tab[0] = segments, tab[1] = grid levels G,
// then per grid level (ascending) its segment, width and chunk count.
__global__ void k_sw_gtab(int32_t L, const int32_t *lp, const int32_t *grid, const int32_t *gpre,
                          const int32_t *segid, const int32_t *nseg, const int32_t *gkp,
                          int32_t *tab, const Status *st) {
  if (failed(st)) return;
  for (int64_t l = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; l < L;
       l += (int64_t)gridDim.x * blockDim.x) {
    if (grid[l]) {
      int32_t *t = tab + kPlanHead + kPlanRec * gpre[l];
      t[0] = segid[l];
      t[1] = lp[l + 1] - lp[l];
      t[2] = gkp[lp[l + 1]] - gkp[lp[l]];
    }
    if (l == L - 1) {
      tab[0] = *nseg;
      tab[1] = gpre[l] + grid[l];
    }
  }
}

// ------------------------------------------------------------- grid levels
//
// A grid level [S0, S1) of segment g: every neighbour lies in another level
// and is final (written by an earlier kernel).  k_sw_grid_rows computes the
// rows of at most kGridRow neighbours and zeroes the others' accumulators;
// k_sw_grid_split takes the larger rows in chunks of kGridChunk edges, one
// workgroup each, and folds each chunk's maximum into the accumulator (gx) by
// an atomic maximum; k_sw_grid_fin turns the accumulators into values.

__device__ inline void grid_level(const SweepArgs &a, int32_t g, int32_t *S0, int32_t *S1) {
  const int32_t l = a.seg[g];
  *S0 = a.lp[l];
  *S1 = a.lp[l + 1];
}

template <bool REV>
__global__ void __launch_bounds__(kGridB) k_sw_grid_rows(SweepArgs a, int32_t g, Status *st) {
  if (failed(st)) return;
  int32_t S0, S1;
  grid_level(a, g, &S0, &S1);
  bool bad = false;
  for (int64_t p = S0 + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < S1;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t e0 = a.rptr[p], e1 = a.rptr[p + 1];
    if (e1 - e0 > kGridRow) {
      a.gx[p] = 0;
      continue;
    }
    int64_t m = 0;
    for (int32_t e = e0; e < e1; e += 4) {
      int32_t q[4];
#pragma unroll
      for (int j = 0; j < 4; j++) q[j] = e + j < e1 ? a.ridx[e + j] : -1;
      int64_t x[4];
#pragma unroll
      for (int j = 0; j < 4; j++) x[j] = q[j] >= 0 ? a.gx[q[j]] : 0;
#pragma unroll
      for (int j = 0; j < 4; j++) {
        bad |= x[j] < 0;
        m = x[j] > m ? x[j] : m;
      }
    }
    const int64_t c = a.cst[p];
    const int64_t o = REV ? c + m : m;
    a.gx[p] = REV ? o : o + c;
    if (!REV) a.out[p] = o;
  }
  // a neighbour without its value would be a broken invariant
  if (bad) raise_err(st, EB_WAIT);
}

template <bool REV>
__global__ void __launch_bounds__(kGridB) k_sw_grid_split(SweepArgs a, int32_t g,
                                                          const int32_t *gkp, Status *st) {
  __shared__ int32_t s_p;
  __shared__ int64_t s_red[kGridB / 64];
  if (failed(st)) return;
  int32_t S0, S1;
  grid_level(a, g, &S0, &S1);
  const int32_t i0 = gkp[S0], i1 = gkp[S1];
  const int tid = threadIdx.x, lane = tid & 63;
  constexpr int kPer = kGridChunk / kGridB;
  for (int32_t i = i0 + blockIdx.x; i < i1; i += gridDim.x) {
    // the row holding chunk i: last p in [S0, S1) with gkp[p] <= i
    if (tid < 64) {
      const int32_t u = wave_row_of(gkp + S0, S1 - S0, i, lane);
      if (lane == 0) s_p = S0 + u;
    }
    __syncthreads();
    const int32_t p = s_p;
    const int32_t r1 = a.rptr[p + 1];
    const int32_t e0 = a.rptr[p] + (i - gkp[p]) * kGridChunk;
    const int32_t e1 = e0 + kGridChunk < r1 ? e0 + kGridChunk : r1;
    int32_t q[kPer];
#pragma unroll
    for (int j = 0; j < kPer; j++) q[j] = e0 + tid + j * kGridB < e1 ? a.ridx[e0 + tid + j * kGridB] : -1;
    int64_t m = 0;
    bool bad = false;
#pragma unroll
    for (int j = 0; j < kPer; j++) {
      const int64_t x = q[j] >= 0 ? a.gx[q[j]] : 0;
      bad |= x < 0;
      m = x > m ? x : m;
    }
    if (bad) raise_err(st, EB_WAIT);
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t o = __shfl_xor((long long)m, off);
      m = o > m ? o : m;
    }
    if (lane == 0) s_red[tid >> 6] = m;
    __syncthreads();
    if (tid == 0) {
      for (int w = 1; w < kGridB / 64; w++) m = s_red[w] > m ? s_red[w] : m;
      atomicMax((unsigned long long *)&a.gx[p], (unsigned long long)m);
    }
    __syncthreads();
  }
}

template <bool REV>
__global__ void __launch_bounds__(kGridB) k_sw_grid_fin(SweepArgs a, int32_t g, Status *st) {
  if (failed(st)) return;
  int32_t S0, S1;
  grid_level(a, g, &S0, &S1);
  for (int64_t p = S0 + blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < S1;
       p += (int64_t)gridDim.x * blockDim.x) {
    if (a.rptr[p + 1] - a.rptr[p] <= kGridRow) continue;
    const int64_t m = a.gx[p], c = a.cst[p];
    const int64_t o = REV ? c + m : m;
    a.gx[p] = REV ? o : o + c;
    if (!REV) a.out[p] = o;
  }
}

// ------------------------------------------------------------------- sweep

// ring slot of entry j of a pull record
__device__ inline uint32_t rec_slot(const uint4 &r, int j) {
  const uint32_t w = j < 2 ? r.x : (j < 4 ? r.y : (j < 6 ? r.z : r.w));
  const uint32_t h = (j & 1) ? (w >> 16) : w;
  return h & 0x0FFFu;
}

// Maximum of m and the first K near neighbours' pull values of a record, as a
// tree (the gathers are independent; the maxima form log2 K + 1 steps).  All
// pull values are non-negative.
template <int K>
__device__ inline int64_t near_max(int64_t m, const uint4 &r, const int64_t *s_x) {
  if constexpr (K == 0) {
    return m;
  } else {
    int64_t g[K];
#pragma unroll
    for (int j = 0; j < K; j++) g[j] = s_x[rec_slot(r, j)];
#pragma unroll
    for (int w = 1; w < K; w <<= 1)
#pragma unroll
      for (int j = 0; j + w < K; j += 2 * w) g[j] = max_nonneg(g[j], g[j + w]);
    return max_nonneg(m, g[0]);
  }
}

// Values of the NR rows [r0, r0 + 64 NR) of a narrow level ending at b (the
// compute wave), from their staged data in the ring: the rows' largest near
// count (in their first records) picks how many gathers every lane makes.
// Slots are read unconditionally (every ring slot holds a record with
// in-range slots); lanes past b discard their results.  Only the ring is
// written: staging waves copy values out to global memory when they take
// the slots over (and at the segment's end).
template <bool REV, int NR>
__device__ inline void finish_rows(const SweepArgs &a, int32_t r0, int32_t b, int lane,
                                   int64_t *s_x, const int64_t *s_base, const int64_t *s_cst,
                                   const uint4 *s_rec) {
  uint4 r[NR];
  int64_t m[NR], c[NR];
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int s = (r0 + 64 * u + lane) & kRMask;
    r[u] = s_rec[s];
    m[u] = s_base[s];
    c[u] = s_cst[s];
  }
  uint32_t kmax = 0;
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const uint32_t k = (uint32_t)__builtin_amdgcn_readfirstlane(r[u].x) >> 28;
    kmax = k > kmax ? k : kmax;
  }
  if (kmax == 0) {
    // no near neighbour in these rows
  } else if (kmax <= 2) {
#pragma unroll
    for (int u = 0; u < NR; u++) m[u] = near_max<2>(m[u], r[u], s_x);
  } else if (kmax <= 4) {
#pragma unroll
    for (int u = 0; u < NR; u++) m[u] = near_max<4>(m[u], r[u], s_x);
  } else {
    if (kmax == kHeavyNear) {
      // some position has a long slot list (its record's slots are all
      // kZeroSlot): the wave gathers along each one
#pragma unroll
      for (int u = 0; u < NR; u++) {
        const int32_t p = r0 + 64 * u + lane;
        const bool hv = p < b && rec_count(r[u]) == kHeavyNear;
        const int32_t hs = hv ? a.hptr[p] : 0, he = hv ? a.hptr[p + 1] : 0;
        for (uint64_t hm = __ballot(hv); hm; hm &= hm - 1) {
          const int h = __builtin_ctzll(hm);
          const int32_t g0 = __builtin_amdgcn_readlane(hs, h);
          const int32_t g1 = __builtin_amdgcn_readlane(he, h);
          int64_t mx = 0;
          for (int32_t i = g0 + lane; i < g1; i += 64) {
            const int64_t x = s_x[a.hidx[i]];
            mx = x > mx ? x : mx;
          }
          for (int off = 32; off > 0; off >>= 1) {
            const int64_t o = __shfl_xor((long long)mx, off);
            mx = o > mx ? o : mx;
          }
          if (lane == h) m[u] = mx > m[u] ? mx : m[u];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < NR; u++) m[u] = near_max<kNear>(m[u], r[u], s_x);
  }
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int32_t p = r0 + 64 * u + lane;
    const int64_t o = REV ? c[u] + m[u] : m[u];
    if (p < b) s_x[p & kRMask] = REV ? o : o + c[u];
  }
}

// Copies the computed values of positions [q0, q1) from the ring to global
// memory (x to gx; forward also the result x - cst to out), one wave or block
// striding by `step`.
template <bool REV>
__device__ inline void flush_ring(const SweepArgs &a, int32_t q0, int32_t q1, int t, int step,
                                  const int64_t *s_x, const int64_t *s_cst) {
  for (int32_t q = q0 + t; q < q1; q += step) {
    const int s = q & kRMask;
    const int64_t x = s_x[s];
    st_coherent(&a.gx[q], x);
    if (!REV) a.out[q] = x - s_cst[s];
  }
}

// Segments [k_lo, k_hi) (none a grid level), in sweep order.
template <bool REV>
__global__ void __launch_bounds__(kSwB) k_ring_sweep(SweepArgs a, int32_t k_lo, int32_t k_hi,
                                                     Status *st) {
  __shared__ int64_t s_x[kRing + 1];
  __shared__ int64_t s_base[kRing], s_cst[kRing];
  __shared__ uint4 s_rec[kRing];
  __shared__ int32_t s_flag[kNF];
  __shared__ int32_t s_next, s_cur, s_nh, s_abort;
  __shared__ int32_t s_hl[kBP * kSwB];
  __shared__ int64_t s_red[kSwB / 64];
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) {
    s_x[kRing] = 0;
    s_abort = 0;
  }
  // every ring slot holds a record with in-range slots from the start: the
  // compute wave reads the slots of lanes past a level's end too
  for (int i = tid; i < kRing; i += kSwB) {
    constexpr uint32_t kZ2 = kZeroSlot | kZeroSlot << 16;
    s_rec[i] = make_uint4(kZ2, kZ2, kZ2, kZ2);
    s_x[i] = 0;
  }
  auto aborted = [&]() {
    return __hip_atomic_load(&s_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) != 0;
  };
  auto give_up = [&]() {
    raise_err(st, EB_WAIT);
    __hip_atomic_store(&s_abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  };
  for (int32_t kk = k_lo; kk < k_hi; kk++) {
    const int32_t k = REV ? k_hi - 1 - (kk - k_lo) : kk;
    const int32_t l0 = a.seg[k], l1 = a.seg[k + 1];
    const int32_t S0 = a.lp[l0], S1 = a.lp[l1];
    if (tid < kNF) s_flag[tid] = -1;
    if (tid == 0) {
      s_next = 0;
      s_cur = REV ? S1 : S0;
      s_nh = 0;
    }
    __syncthreads();
    const bool ab = s_abort != 0;
    __syncthreads();  // every wave has read the flag before anyone may set it
    if (ab) break;
    if (a.wide[l0]) {
      // ---------------------------------------------------- block mode
      // one level [S0, S1): every neighbour lies in another level, final.
      // kBP positions per thread and pass, their first 4 neighbours' loads
      // all in flight; nodes of more than 64 neighbours are listed and then
      // taken by the whole block.
      for (int32_t p0 = S0; p0 < S1; p0 += kBP * kSwB) {
        int32_t e0[kBP], e1[kBP];
#pragma unroll
        for (int i = 0; i < kBP; i++) {
          const int32_t p = p0 + i * kSwB + tid;
          e0[i] = p < S1 ? a.rptr[p] : 0;
          e1[i] = p < S1 ? a.rptr[p + 1] : 0;
        }
        int32_t q[kBP * 4];
#pragma unroll
        for (int i = 0; i < kBP; i++)
#pragma unroll
          for (int j = 0; j < 4; j++)
            q[4 * i + j] = (e1[i] - e0[i] <= 64 && e0[i] + j < e1[i]) ? a.ridx[e0[i] + j] : -1;
        int64_t x[kBP * 4];
        ld_many<kBP * 4>(x, q, a.gx, &s_abort, st);
#pragma unroll
        for (int i = 0; i < kBP; i++) {
          const int32_t p = p0 + i * kSwB + tid;
          if (p >= S1) continue;
          if (e1[i] - e0[i] > 64) {
            s_hl[atomicAdd(&s_nh, 1)] = p;
            continue;
          }
          int64_t m = 0;
#pragma unroll
          for (int j = 0; j < 4; j++) m = x[4 * i + j] > m ? x[4 * i + j] : m;
          for (int32_t e = e0[i] + 4; e < e1[i]; e += 4) {
            int32_t qq[4];
#pragma unroll
            for (int j = 0; j < 4; j++) qq[j] = e + j < e1[i] ? a.ridx[e + j] : -1;
            int64_t xx[4];
            ld_many<4>(xx, qq, a.gx, &s_abort, st);
#pragma unroll
            for (int j = 0; j < 4; j++) m = xx[j] > m ? xx[j] : m;
          }
          const int64_t c = a.cst[p];
          const int64_t o = REV ? c + m : m;
          st_coherent(&a.gx[p], REV ? o : o + c);
          if (!REV) a.out[p] = o;
        }
        __syncthreads();
        const int32_t nh = s_nh;
        for (int32_t i = 0; i < nh; i++) {  // nodes of many neighbours: the whole block
          const int32_t p2 = s_hl[i];
          // neighbours stored by other waves before a barrier: a barrier does
          // not wait for those stores, so one still in flight is read again
          const int64_t mx = heavy_max<kHeavyU, kSwB>(
              a.rptr[p2], a.rptr[p2 + 1], tid, [&](int32_t e) { return a.ridx[e]; },
              [&](int32_t qq) { return ld_final(&a.gx[qq], &s_abort, st); });
          if (lane == 0) s_red[wave] = mx;
          __syncthreads();
          if (tid == 0) {
            int64_t m = 0;
            for (int w = 0; w < kSwB / 64; w++) m = s_red[w] > m ? s_red[w] : m;
            const int64_t c = a.cst[p2];
            const int64_t o = REV ? c + m : m;
            st_coherent(&a.gx[p2], REV ? o : o + c);
            if (!REV) a.out[p2] = o;
          }
          __syncthreads();
        }
        if (tid == 0) s_nh = 0;
        __syncthreads();
      }
      continue;
    }
    // --------------------------------------------------------- ring mode
    const int32_t nst = (S1 - S0 + kStage - 1) / kStage;  // staging tasks
    if (wave == 0) {
      // The compute wave: the segment's levels in sweep order.
      __builtin_amdgcn_s_setprio(3);
      int32_t ready = 0;  // staging tasks known complete: [0, ready)
      bool gaveup = false;
      const int32_t nl = l1 - l0;
      for (int32_t lb = 0; lb < nl && !gaveup; lb += 63) {
        // bounds of up to 63 levels: lane i holds lp[l0 + lb + i] (forward)
        // or lp[l1 - lb - 63 + i] (REVERSE, lane 63 the top)
        const int32_t li = REV ? l1 - lb - 63 + lane : l0 + lb + lane;
        const int32_t lcl = li < l0 ? l0 : (li > l1 ? l1 : li);
        const int32_t bnd = a.lp[lcl];
        // wait for the bounds here, once: a wait inside the level loop would
        // also wait for every store the loop has issued
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        const int32_t cnt = nl - lb < 63 ? nl - lb : 63;
        for (int32_t j = 0; j < cnt; j++) {
          const int32_t pa = __builtin_amdgcn_readlane(bnd, REV ? 62 - j : j);
          const int32_t pb = __builtin_amdgcn_readlane(bnd, REV ? 63 - j : j + 1);
          CEL_TSTAMP(t0);
          CEL_TCOUNT(2);
          // every staging task covering [pa, pb) complete
          const int32_t need = (int32_t)((uint32_t)(REV ? S1 - 1 - pa : pb - 1 - S0) / kStage);
          for (int32_t spin = 0; ready <= need;) {
            // lanes 0..kNF-1 look at the next kNF tasks in one LDS round trip
            const int32_t tk = ready + lane;
            const int32_t f = lane < kNF ? __hip_atomic_load(&s_flag[tk % kNF], __ATOMIC_RELAXED,
                                                             __HIP_MEMORY_SCOPE_WORKGROUP)
                                         : -1;
            const uint64_t done = __ballot(lane < kNF && f == tk);
            const int32_t adv = __builtin_ctzll(~done);  // complete tasks in a row from `ready`
            if (adv > 0) {
              ready += adv;
            } else {
              CEL_TCOUNT(3);
              if (++spin == kSpin || aborted()) {
                give_up();
                gaveup = true;
                break;
              }
              __builtin_amdgcn_s_sleep(1);
            }
          }
          if (gaveup) break;
          lds_order();
          CEL_TSTAMP(t1);
          CEL_TADD(0, t0, t1);
          // Rows of 64 from the level's start, one or two at a time (a step's
          // reads before its writes).  REVERSE takes them from the top: a
          // position's slot is the one of the position kRing above it, which
          // a higher position of the same level may still need; going down,
          // every such position has read it first.  Forward, ascending order
          // does the same.
          const int32_t nrow = (pb - pa + 63) >> 6;
          if (REV) {
            int32_t k = nrow;
            for (; k >= 2; k -= 2)
              finish_rows<REV, 2>(a, pa + 64 * (k - 2), pb, lane, s_x, s_base, s_cst, s_rec);
            if (k == 1) finish_rows<REV, 1>(a, pa, pb, lane, s_x, s_base, s_cst, s_rec);
          } else {
            int32_t r0 = pa;
            for (; r0 + 64 < pb; r0 += 128)
              finish_rows<REV, 2>(a, r0, pb, lane, s_x, s_base, s_cst, s_rec);
            if (r0 < pb) finish_rows<REV, 1>(a, r0, pb, lane, s_x, s_base, s_cst, s_rec);
          }
          lds_order();
          CEL_TSTAMP(t2);
          CEL_TADD(1, t1, t2);
          // this level's slots may be staged again: its reads are done
          __hip_atomic_store(&s_cur, REV ? pa : pb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
      }
      __builtin_amdgcn_s_setprio(0);
    } else {
      // staging waves: tasks of kStage positions, in sweep order
      for (;;) {
        int32_t t = 0;
        if (lane == 0) t = atomicAdd(&s_next, 1);
        t = __builtin_amdgcn_readfirstlane(__shfl(t, 0));
        if (t >= nst || aborted()) break;
        const int32_t lo = REV ? (S1 - (t + 1) * kStage > S0 ? S1 - (t + 1) * kStage : S0)
                               : S0 + t * kStage;
        const int32_t hi = REV ? S1 - t * kStage : (lo + kStage < S1 ? lo + kStage : S1);
        // static parts first: they need no free slot
        uint4 r[4];
        int64_t c[4];
        int32_t f0[4], f1[4];
#pragma unroll
        for (int u = 0; u < 4; u++) {
          const int32_t p = lo + 64 * u + lane;
          const bool v = p < hi;
          r[u] = v ? a.rec[p] : make_uint4(0, 0, 0, 0);
          c[u] = v ? a.cst[p] : 0;
          f0[u] = v ? a.fptr[p] : 0;
          f1[u] = v ? a.fptr[p + 1] : 0;
        }
        int32_t q[4][4];
#pragma unroll
        for (int u = 0; u < 4; u++)
#pragma unroll
          for (int j = 0; j < 4; j++) q[u][j] = f0[u] + j < f1[u] ? a.fidx[f0[u] + j] : -1;
        // wait until the compute wave has left the positions whose slots these
        // take over (REVERSE: every position >= lo + kRing computed; forward:
        // every position < hi - kRing)
        for (int32_t spin = 0;; spin++) {
          const int32_t cur = __hip_atomic_load(&s_cur, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_WORKGROUP);
          if (REV ? cur <= lo + kRing : cur >= hi - kRing) break;
          if (spin == kSpin || aborted()) {
            give_up();
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
        if (aborted()) break;
        // the slots' previous positions leave the ring: their values to global
        // memory first (REVERSE: positions [lo, hi) + kRing; forward: - kRing)
        if (REV) flush_ring<REV>(a, lo + kRing, hi + kRing < S1 ? hi + kRing : S1, lane, 64, s_x, s_cst);
        else flush_ring<REV>(a, lo - kRing > S0 ? lo - kRing : S0, hi - kRing, lane, 64, s_x, s_cst);
        int64_t m[4];
        {
          int32_t qa[16];
          int64_t x[16];
#pragma unroll
          for (int u = 0; u < 4; u++)
#pragma unroll
            for (int j = 0; j < 4; j++) qa[4 * u + j] = q[u][j];
          ld_many<16>(x, qa, a.gx, &s_abort, st);
#pragma unroll
          for (int u = 0; u < 4; u++) {
            m[u] = 0;
#pragma unroll
            for (int j = 0; j < 4; j++) m[u] = x[4 * u + j] > m[u] ? x[4 * u + j] : m[u];
          }
        }
        // longer far lists: 4 more at a time per lane up to 64, beyond that the whole wave
#pragma unroll
        for (int u = 0; u < 4; u++) {
          const bool lng = f1[u] - f0[u] > 64;
          for (int32_t e = f0[u] + 4; e < (lng ? f0[u] : f1[u]); e += 4) {
            int32_t qq[4];
#pragma unroll
            for (int j = 0; j < 4; j++) qq[j] = e + j < f1[u] ? a.fidx[e + j] : -1;
            int64_t x[4];
            ld_many<4>(x, qq, a.gx, &s_abort, st);
#pragma unroll
            for (int j = 0; j < 4; j++) m[u] = x[j] > m[u] ? x[j] : m[u];
          }
          for (uint64_t hv = __ballot(lng); hv; hv &= hv - 1) {
            const int h = __builtin_ctzll(hv);
            const int32_t g0 = __builtin_amdgcn_readlane(f0[u], h);
            const int32_t g1 = __builtin_amdgcn_readlane(f1[u], h);
            int64_t mx = 0;
            for (int32_t e = g0 + 4 + lane; e < g1; e += 256) {
              int32_t qq[4];
#pragma unroll
              for (int j = 0; j < 4; j++) qq[j] = e + 64 * j < g1 ? a.fidx[e + 64 * j] : -1;
              int64_t x[4];
              ld_many<4>(x, qq, a.gx, &s_abort, st);
#pragma unroll
              for (int j = 0; j < 4; j++) mx = x[j] > mx ? x[j] : mx;
            }
            for (int off = 32; off > 0; off >>= 1) {
              const int64_t o = __shfl_xor((long long)mx, off);
              mx = o > mx ? o : mx;
            }
            if (lane == h) m[u] = mx > m[u] ? mx : m[u];
          }
        }
#pragma unroll
        for (int u = 0; u < 4; u++) {
          const int32_t p = lo + 64 * u + lane;
          if (p < hi) {
            const int s = p & kRMask;
            s_rec[s] = r[u];
            s_base[s] = m[u];
            s_cst[s] = c[u];
          }
        }
        // the task's slots are written (LDS: in order) before its flag
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        if (lane == 0)
          __hip_atomic_store(&s_flag[t % kNF], t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
    __syncthreads();  // the segment is done: every value in the ring
    // values whose slots were never taken over go out now (REVERSE: the
    // segment's lowest kRing positions; forward: its highest)
    if (REV) flush_ring<REV>(a, S0, S1 < S0 + kRing ? S1 : S0 + kRing, tid, kSwB, s_x, s_cst);
    else flush_ring<REV>(a, S1 - kRing > S0 ? S1 - kRing : S0, S1, tid, kSwB, s_x, s_cst);
    // the stores reach L2 before the next segment's barrier (a barrier alone
    // does not wait for them; readers re-read a value not yet there anyway)
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  }
}

// ------------------------------------------------------------------- host

CEL_PHASE_READER(cel_debug_phases_sweep)

int sweep_prepare(SweepPlan &pl, bool rev, int32_t n, int32_t m, int32_t L, const int32_t *lp,
                  const int32_t *order, const int32_t *level, const int32_t *rptr,
                  const int32_t *ridx, const int64_t *wp, const int64_t *wcp, int64_t *out,
                  Scratch &sc, hipStream_t s, Status *st) {
  pl = SweepPlan{};
  pl.rev = rev;
  if (n == 0) return CEL_OK;
  int32_t *wide, *grid, *gpre, *flag, *pre, *seg, *segid, *nseg, *fcnt, *fptr, *fidx, *hcnt,
      *hptr, *hidx, *rmax, *gk, *gkp, *tab;
  int64_t *cst, *gx;
  uint4 *rec;
  CEL_TRY(sc.get(&wide, L));
  CEL_TRY(sc.get(&grid, L));
  CEL_TRY(sc.get(&gpre, (int64_t)L + 1));
  CEL_TRY(sc.get(&flag, L));
  CEL_TRY(sc.get(&pre, (int64_t)L + 1));
  CEL_TRY(sc.get(&seg, (int64_t)L + 1));
  CEL_TRY(sc.get(&segid, L));
  CEL_TRY(sc.get(&nseg, 1));
  CEL_TRY(sc.get(&fcnt, n));
  CEL_TRY(sc.get(&fptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&hcnt, n));
  CEL_TRY(sc.get(&hptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&gk, n));
  CEL_TRY(sc.get(&gkp, (int64_t)n + 1));
  CEL_TRY(sc.get(&fidx, m));
  CEL_TRY(sc.get(&hidx, m));
  CEL_TRY(sc.get(&cst, n));
  CEL_TRY(sc.get(&rec, n));
  CEL_TRY(sc.get(&rmax, n));
  CEL_TRY(sc.get(&tab, kPlanHead + (int64_t)kPlanRec * L));
  gx = out;
  if (!rev) CEL_TRY(sc.get(&gx, n));
  k_fill_i32<<<grid_for(L, 256, 1024), 256, 0, s>>>(wide, L, 0);
  k_fill_i32<<<1, 64, 0, s>>>(tab, kPlanHead, 0);
  k_fill_i64<<<grid_for(n, 256, 4096), 256, 0, s>>>(gx, n, -1);
  k_fill_i32<<<grid_for(n, 256, 4096), 256, 0, s>>>(rmax, n, 0);
  const int gn = grid_for(n, 256, 4096), gl = grid_for(L, 256, 1024);
  k_sw_wide<<<gn, 256, 0, s>>>(n, L, lp, rptr, order, level, wide, grid, st);
  k_sw_segflag<<<gl, 256, 0, s>>>(L, wide, flag, st);
  CEL_TRY(exclusive_scan_i32(flag, pre, L, sc, s));
  CEL_TRY(exclusive_scan_i32(grid, gpre, L, sc, s));
  k_sw_segfill<<<gl, 256, 0, s>>>(L, flag, pre, seg, segid, nseg, st);
  if (rev) {
    k_sw_prep<true, 0><<<gn, 256, 0, s>>>(n, lp, rptr, ridx, order, level, wide, grid, seg, segid,
                                          wp, wcp, rec, cst, fcnt, hcnt, gk, nullptr, nullptr,
                                          nullptr, nullptr, rmax, st);
  } else {
    k_sw_prep<false, 0><<<gn, 256, 0, s>>>(n, lp, rptr, ridx, order, level, wide, grid, seg, segid,
                                           wp, wcp, rec, cst, fcnt, hcnt, gk, nullptr, nullptr,
                                           nullptr, nullptr, rmax, st);
  }
  CEL_TRY(exclusive_scan_i32(fcnt, fptr, n, sc, s));
  CEL_TRY(exclusive_scan_i32(hcnt, hptr, n, sc, s));
  CEL_TRY(exclusive_scan_i32(gk, gkp, n, sc, s));
  if (rev) {
    k_sw_prep<true, 1><<<gn, 256, 0, s>>>(n, lp, rptr, ridx, order, level, wide, grid, seg, segid,
                                          wp, wcp, rec, cst, fcnt, hcnt, gk, fptr, fidx, hptr, hidx,
                                          rmax, st);
  } else {
    k_sw_prep<false, 1><<<gn, 256, 0, s>>>(n, lp, rptr, ridx, order, level, wide, grid, seg, segid,
                                           wp, wcp, rec, cst, fcnt, hcnt, gk, fptr, fidx, hptr, hidx,
                                           rmax, st);
  }
  k_sw_rowmark<<<gn, 256, 0, s>>>(n, lp, order, level, wide, rmax, rec, st);
  k_sw_gtab<<<gl, 256, 0, s>>>(L, lp, grid, gpre, segid, nseg, gkp, tab, st);
  CEL_HIP(hipGetLastError());
  SweepArgs &a = pl.a;
  a.n = n;
  a.L = L;
  a.lp = lp;
  a.rptr = rptr;
  a.ridx = ridx;
  a.cst = cst;
  a.rec = rec;
  a.fptr = fptr;
  a.fidx = fidx;
  a.hptr = hptr;
  a.hidx = hidx;
  a.seg = seg;
  a.wide = wide;
  a.gx = gx;
  a.out = out;
  pl.gkp = gkp;
  pl.tab = tab;
  return CEL_OK;
}

int sweep_run(SweepPlan &pl, hipStream_t s, Status *st, const char *timer) {
  const SweepArgs &a = pl.a;
  if (a.n == 0) return CEL_OK;
  // the plan: segments, grid levels and, per grid level, segment, width, chunks
  std::vector<int32_t> tab(kPlanFirst);
  CEL_HIP(hipMemcpyAsync(tab.data(), pl.tab, sizeof(int32_t) * kPlanFirst, hipMemcpyDeviceToHost, s));
  CEL_HIP(hipStreamSynchronize(s));
  const int32_t NS = tab[0], G = tab[1];
  // a failed preparation (the status block holds its error) leaves NS = 0
  if (NS <= 0 || NS > a.L || G < 0 || G > NS) return CEL_OK;
  const int64_t len = kPlanHead + (int64_t)kPlanRec * G;
  if (len > kPlanFirst) {
    tab.resize(len);
    CEL_HIP(hipMemcpyAsync(tab.data() + kPlanFirst, pl.tab + kPlanFirst,
                           sizeof(int32_t) * (len - kPlanFirst), hipMemcpyDeviceToHost, s));
    CEL_HIP(hipStreamSynchronize(s));
  }
  auto ring = [&](int32_t lo, int32_t hi) {
    if (lo >= hi) return;
    if (pl.rev) k_ring_sweep<true><<<1, kSwB, 0, s>>>(a, lo, hi, st);
    else k_ring_sweep<false><<<1, kSwB, 0, s>>>(a, lo, hi, st);
  };
  auto gridlev = [&](int32_t j) {
    const int32_t *t = &tab[kPlanHead + kPlanRec * j];
    const int32_t g = t[0], w = t[1], chunks = t[2];
    const int gw = grid_for(w, kGridB, 8192);
    if (pl.rev) k_sw_grid_rows<true><<<gw, kGridB, 0, s>>>(a, g, st);
    else k_sw_grid_rows<false><<<gw, kGridB, 0, s>>>(a, g, st);
    if (chunks > 0) {
      const int gc = chunks < 8192 ? chunks : 8192;
      if (pl.rev) k_sw_grid_split<true><<<gc, kGridB, 0, s>>>(a, g, pl.gkp, st);
      else k_sw_grid_split<false><<<gc, kGridB, 0, s>>>(a, g, pl.gkp, st);
      if (pl.rev) k_sw_grid_fin<true><<<gw, kGridB, 0, s>>>(a, g, st);
      else k_sw_grid_fin<false><<<gw, kGridB, 0, s>>>(a, g, st);
    }
  };
  for (int32_t j = 0; j < G; j++) {
    const int32_t g = tab[kPlanHead + kPlanRec * j];
    const int32_t prev = j > 0 ? tab[kPlanHead + kPlanRec * (j - 1)] : -1;
    if (g <= prev || g >= NS) {
      // only an error raised while the plan was written (on this stream or
      // the other sweep's) leaves it inconsistent: the status reports it
      Status h;
      CEL_TRY(read_status(st, &h, s));
      if (h.err) return CEL_OK;
      return set_error(CEL_E_HIP, "level sweep: inconsistent plan of grid levels");
    }
  }
  KTimer kt(s, timer);
  if (pl.rev) {
    // segments from the top: the part above each grid level, then the level
    int32_t hi = NS;
    for (int32_t j = G - 1; j >= 0; j--) {
      const int32_t g = tab[kPlanHead + kPlanRec * j];
      ring(g + 1, hi);
      gridlev(j);
      hi = g;
    }
    ring(0, hi);
  } else {
    int32_t lo = 0;
    for (int32_t j = 0; j < G; j++) {
      const int32_t g = tab[kPlanHead + kPlanRec * j];
      ring(lo, g);
      gridlev(j);
      lo = g + 1;
    }
    ring(lo, NS);
  }
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

}  // namespace cel
