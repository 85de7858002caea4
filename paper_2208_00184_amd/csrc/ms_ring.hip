// Makespan of one placement (eq. 7, Order-Place's device model) over the
// device-grouped order, with the levels run from an LDS ring.
//
// Slots are the positions of the device-grouped order: a level is a
// contiguous range, and inside it each device's nodes form one run in their
// FIFO order.  With sx(i) the sum of w over the run before slot i and h the
// run's first slot, the device chain unrolls to
//   fin(i) = sx(i) + w(i) + max(free(d) - sx(h), max over h <= j <= i of (ready(j) - sx(j)))
// where ready(j) = max over predecessors q of fin(q) + [dev q != dev j] c(q).
// Per row of 64 slots that is: gather the ready times, one segmented prefix
// maximum over the wave (the run distance decides which lanes combine), the
// carry of a run from the previous row, and the device's free time folded in
// at the run's first slot and updated at its last.
//
// The work is split between the waves of one workgroup as in the level
// sweeps of eq. 2 and 3 (sweep.hip): wave 0 runs the levels from an LDS ring
// of the last kMRing slots' values; the other waves stage slots ahead of it
// (pull records, costs, run data and the folded ready time of predecessors
// too far back for the ring), and copy values out to global memory before
// they take a slot over.  Two values per slot sit in the ring, fin and
// fin + c, so a pull entry (ring slot, plus kMRing when the devices differ)
// is one gather.  Levels wider than kMWideW, or holding a node of more than
// kMHeavyDeg predecessors, are run by the whole workgroup from global memory
// (block mode) and split the rest into segments.
#include "cel_internal.h"

namespace cel {

constexpr int kMsB = 512;               // 8 waves: 1 compute, 7 staging
constexpr int kMRing = 2048;            // slots held in the ring
constexpr int kMRMask = kMRing - 1;
constexpr int kMWideW = 1536;           // wider levels run in block mode
constexpr int kMHeavyDeg = 4096;        // a node with more predecessors puts its level in block mode
constexpr int kMStage = 256;            // slots per staging task (4 rows)
constexpr int kMNF = kMRing / kMStage;  // staging flags
constexpr int kMNear = 8;               // near predecessors in a pull record
constexpr int kMBRow = 64;              // block mode: larger rows are taken by the whole block
static_assert(kMWideW + kMStage < kMRing, "a narrow level and a staging task fit the ring");
constexpr uint32_t kMZero = 2 * kMRing;  // ring index that always reads 0
constexpr uint32_t kMZ2 = kMZero | kMZero << 16;

// Pull record of a slot (16 bytes): eight 16-bit entries, bits 0..12 the ring
// index of a near predecessor's value (its slot, + kMRing when its device
// differs: fin + c), kMZero when unused.  Entry 0 bits 13..15: the class of
// the row of 64 this slot starts (0: no near predecessor, 1: at most 2, 2: at
// most 4, 3: at most 8, 4: a slot of the row has more; 0 for other slots).
// Entry 1 bit 15: this slot has more than kMNear near predecessors; its
// entries are then all kMZero and its list lies in a global array (hidx from
// hptr[p]).
__device__ inline uint32_t ms_entry(const uint4 &r, int j) {
  const uint32_t w = j < 2 ? r.x : (j < 4 ? r.y : (j < 6 ? r.z : r.w));
  return ((j & 1) ? (w >> 16) : w) & 0x1FFFu;
}

struct MsArgs {
  int32_t n;
  const int32_t *lp;              // [L + 1] level starts (slots)
  const int32_t *pptr;            // [n + 1] predecessor rows
  const uint32_t *tidx;           // [m] predecessor slot | devices differ << 31
  const int64_t *wp, *cq, *sxp;   // by slot: w, c, run sum before the slot
  const int32_t *metap;           // by slot: device | run ends << 8 | run distance << 16
  const uint4 *rec;               // [n] pull records
  const int32_t *fptr;            // far predecessors (tagged as tidx)
  const uint32_t *fidx;
  const int32_t *hptr;            // long near lists (ring indices)
  const int32_t *hidx;
  const int32_t *seg;             // [segments + 1] first level of each segment
  const int32_t *nseg;
  const int32_t *wide;            // [L] block-mode levels
  int64_t *gf;                    // [2n] fin, then fin + c; -1 until written
  int64_t *makespan;
};

// value of a tagged predecessor: fin, or fin + c when the devices differ
__device__ inline const int64_t *ms_src(const MsArgs &a, uint32_t t) {
  return a.gf + (int64_t)(t & 0x7FFFFFFFu) + ((t >> 31) ? a.n : 0);
}

// -------------------------------------------------------------- preparation

__global__ void k_ms_wide(int32_t n, int32_t L, const int32_t *lp, const int32_t *pptr,
                          const int32_t *gorder, const int32_t *level, int32_t *wide,
                          const Status *st) {
  if (failed(st)) return;
  const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x, step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t l = i0; l < L; l += step)
    if (lp[l + 1] - lp[l] > kMWideW) wide[l] = 1;
  for (int64_t p = i0; p < n; p += step)
    if (pptr[p + 1] - pptr[p] > kMHeavyDeg) wide[level[gorder[p]]] = 1;
}

// PASS 0: tagged predecessors of every slot; for slots of ring levels the pull
// record, the far count and the long-list count, and the row's largest near
// count (rmax, at the row's first slot).  PASS 1: far lists and long lists.
template <int PASS>
__global__ void k_ms_prep(int32_t n, const int32_t *lp, const int32_t *pptr, const int32_t *pidx,
                          const int32_t *gorder, const int32_t *level, const int32_t *wide,
                          const int32_t *seg, const int32_t *segid, const uint8_t *devp,
                          uint32_t *tidx, uint4 *rec, int32_t *fcnt, int32_t *hcnt,
                          const int32_t *fptr, uint32_t *fidx, const int32_t *hptr, int32_t *hidx,
                          int32_t *rmax, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t l = level[gorder[p]];
    const int32_t e0 = pptr[p], e1 = pptr[p + 1];
    if (PASS == 0) {
      const uint8_t dv = devp[p];
      for (int32_t e = e0; e < e1; e++) {
        const int32_t q = pidx[e];
        tidx[e] = (uint32_t)q | (uint32_t)(devp[q] != dv) << 31;
      }
    }
    if (wide[l]) {
      if (PASS == 0) {
        rec[p] = make_uint4(kMZ2, kMZ2, kMZ2, kMZ2);
        fcnt[p] = 0;
        hcnt[p] = 0;
      }
      continue;
    }
    const int32_t S0 = lp[seg[segid[l]]];
    int32_t nn = 0, nf = 0;
    uint32_t ent[kMNear];
#pragma unroll
    for (int j = 0; j < kMNear; j++) ent[j] = kMZero;
    for (int32_t e = e0; e < e1; e++) {
      const uint32_t t = tidx[e];
      const int32_t q = (int32_t)(t & 0x7FFFFFFFu);
      if (q >= S0 && (int32_t)p - q < kMRing) {
        const uint32_t ix = (uint32_t)(q & kMRMask) + ((t >> 31) ? kMRing : 0);
        if (PASS == 0) {
#pragma unroll
          for (int j = 0; j < kMNear; j++)
            if (j == nn) ent[j] = ix;
        } else if (hptr[p + 1] > hptr[p]) {
          hidx[hptr[p] + nn] = (int32_t)ix;
        }
        nn++;
      } else {
        if (PASS == 1) fidx[fptr[p] + nf] = t;
        nf++;
      }
    }
    if (PASS == 0) {
      fcnt[p] = nf;
      hcnt[p] = nn > kMNear ? nn : 0;
      const int32_t lb = lp[l];
      if (nn > 0) atomicMax(&rmax[lb + ((int32_t)(p - lb) & ~63)], nn);
      if (nn > kMNear)
        rec[p] = make_uint4(kMZ2 | 0x80000000u, kMZ2, kMZ2, kMZ2);
      else
        rec[p] = make_uint4(ent[0] | ent[1] << 16, ent[2] | ent[3] << 16, ent[4] | ent[5] << 16,
                            ent[6] | ent[7] << 16);
    }
  }
}

// the row class (entry 0 bits 13..15) at the first slot of every row of a ring level
__global__ void k_ms_rowmark(int32_t n, const int32_t *lp, const int32_t *gorder,
                             const int32_t *level, const int32_t *wide, const int32_t *rmax,
                             uint4 *rec, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t l = level[gorder[p]];
    if (wide[l] || (((int32_t)p - lp[l]) & 63) != 0) continue;
    const int32_t k = rmax[p];
    const uint32_t cls = k == 0 ? 0u : (k <= 2 ? 1u : (k <= 4 ? 2u : (k <= kMNear ? 3u : 4u)));
    rec[p].x |= cls << 13;
  }
}

// ------------------------------------------------------------------ compute


// max of m and the first K entries' ring values, as a tree (all non-negative)
template <int K>
__device__ inline int64_t ms_near(int64_t m, const uint4 &r, const int64_t *s_x) {
  int64_t g[K];
#pragma unroll
  for (int j = 0; j < K; j++) g[j] = s_x[ms_entry(r, j)];
#pragma unroll
  for (int w = 1; w < K; w <<= 1)
#pragma unroll
    for (int j = 0; j + w < K; j += 2 * w) g[j] = max_nonneg(g[j], g[j + w]);
  return max_nonneg(m, g[0]);
}

// One step of an unsegmented prefix maximum over each of NR rows (lanes
// without a source, or outside the DPP rows the step writes, take 0, the
// identity for non-negative values); the rows' steps are interleaved.
template <int CTRL, int ROWMASK, int NR>
__device__ inline void plain_pmax_step(int64_t (&y)[NR]) {
  int64_t u[NR];
#pragma unroll
  for (int k = 0; k < NR; k++) {
    if constexpr (ROWMASK == 0xF) {
      // every lane is written (bound_ctrl: 0 where the source lane is out of
      // the row), so no old value has to be set up
      const int32_t lo = __builtin_amdgcn_mov_dpp((int32_t)y[k], CTRL, 0xF, 0xF, true);
      const int32_t hi = __builtin_amdgcn_mov_dpp((int32_t)(y[k] >> 32), CTRL, 0xF, 0xF, true);
      u[k] = (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
    } else {
      u[k] = dpp64<CTRL, ROWMASK>(y[k], 0);
    }
  }
#pragma unroll
  for (int k = 0; k < NR; k++) y[k] = max_nonneg(y[k], u[k]);
}

// Finish times of the NR rows [r0, r0 + 64 NR) of a narrow level ending at b,
// by the compute wave from the staged data; carry is the prefix value at the
// end of the previous row of the level (0 before the first).  Lanes past b
// compute from whatever their slots hold (every record names in-range ring
// indices, every meta an in-range device) and write nothing; being the rows'
// last lanes, they never feed a valid lane's prefix.
//
// The prefix runs over y = max(0, ready - sx), with the free time folded in
// at a run's first slot and the carry at lane 0 of a row that continues a
// run: the run's maximum includes the free time, which is never negative, so
// clamping at 0 changes no maximum.  A row that is one run (almost every row
// when a level sits on one device) takes the unsegmented scan.
template <int NR>
__device__ inline void ms_rows(const MsArgs &a, int32_t r0, int32_t b, int lane, int64_t &carry,
                               int64_t &mk, int64_t *s_x, const uint4 *s_rec,
                               const int64_t *s_base, const int64_t *s_sx, const int64_t *s_sxw,
                               const int64_t *s_sxwc, const int32_t *s_meta, int64_t *s_avail) {
  uint4 r[NR];
  int64_t y[NR], sx[NR], av[NR], w[NR], c[NR];  // w: sx + w, c: sx + w + c
  int32_t mt[NR];
  // all staged data in one LDS round trip (the free time's address needs meta)
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int s = (r0 + 64 * u + lane) & kMRMask;
    mt[u] = s_meta[s];
    r[u] = s_rec[s];
    y[u] = s_base[s];
    sx[u] = s_sx[s];
    w[u] = s_sxw[s];
    c[u] = s_sxwc[s];
  }
  lds_order();
  // free times as of the level's start, at a run's first slot (slot 256 of
  // s_avail always holds 0 for the others)
#pragma unroll
  for (int u = 0; u < NR; u++) av[u] = s_avail[(mt[u] >> 16) == 0 ? (mt[u] & 255) : 256];
  uint32_t cls = 0;
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const uint32_t k = ((uint32_t)__builtin_amdgcn_readfirstlane(r[u].x) >> 13) & 7u;
    cls = k > cls ? k : cls;
  }
  if (cls == 1) {
#pragma unroll
    for (int u = 0; u < NR; u++) y[u] = ms_near<2>(y[u], r[u], s_x);
  } else if (cls == 2) {
#pragma unroll
    for (int u = 0; u < NR; u++) y[u] = ms_near<4>(y[u], r[u], s_x);
  } else if (cls >= 3) {
    if (cls == 4) {
      // slots with long near lists (their entries are all kMZero): the wave
      // gathers along each one
#pragma unroll
      for (int u = 0; u < NR; u++) {
        const int32_t p = r0 + 64 * u + lane;
        const bool hv = p < b && (r[u].x >> 31);
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
          if (lane == h) y[u] = max_nonneg(y[u], mx);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < NR; u++) y[u] = ms_near<kMNear>(y[u], r[u], s_x);
  }
  // y = max(0, ready - sx), the free time at a run's first slot; rows with a
  // run starting past lane 0
  bool split = false;
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int32_t hd = mt[u] >> 16;
    // max(0, ready - sx) = max(ready, sx) - sx; sx = 0 at a run's first slot
    y[u] = max_nonneg(max_nonneg(y[u], sx[u]) - sx[u], av[u]);
    split |= __ballot(r0 + 64 * u + lane < b && hd < lane) != 0;
  }
  if (!split) {
    // every row one run: the carry enters at lane 0, then a plain prefix max
    if (lane == 0 && (mt[0] >> 16) > 0) y[0] = max_nonneg(y[0], carry);
    plain_pmax_step<0x111, 0xF, NR>(y);  // row_shr:1
    plain_pmax_step<0x112, 0xF, NR>(y);  // row_shr:2
    plain_pmax_step<0x114, 0xF, NR>(y);  // row_shr:4
    plain_pmax_step<0x118, 0xF, NR>(y);  // row_shr:8
    plain_pmax_step<0x142, 0xA, NR>(y);  // row_bcast:15 into rows 1 and 3
    plain_pmax_step<0x143, 0xC, NR>(y);  // row_bcast:31 into rows 2 and 3
    if constexpr (NR == 2) {
      // the second row takes the first's carry unless a run starts at its lane 0
      if ((__builtin_amdgcn_readfirstlane(mt[1]) >> 16) > 0) {
        y[1] = max_nonneg(y[1], readlane64(y[0], 63));
      }
    }
    carry = readlane64(y[NR - 1], 63);
  } else {
#pragma unroll
    for (int u = 0; u < NR; u++) {
      const int32_t hd = mt[u] >> 16;
      if (lane == 0 && hd > 0) y[u] = max_nonneg(y[u], carry);
      y[u] = wave_seg_pmax(y[u], hd, lane);
      carry = readlane64(y[u], 63);
    }
  }
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int32_t p = r0 + 64 * u + lane;
    if (p < b) {
      const int s = p & kMRMask;
      const int64_t fin = w[u] + y[u];
      s_x[s] = fin;
      s_x[kMRing + s] = c[u] + y[u];
      mk = max_nonneg(mk, fin);
      if (mt[u] & 256) s_avail[mt[u] & 255] = fin;
    }
  }
}

// values of slots [q0, q1) from the ring to global memory, striding by step
__device__ inline void ms_flush(const MsArgs &a, int32_t q0, int32_t q1, int t, int step,
                                const int64_t *s_x) {
  for (int32_t q = q0 + t; q < q1; q += step) {
    const int s = q & kMRMask;
    st_coherent(&a.gf[q], s_x[s]);
    st_coherent(&a.gf[(int64_t)a.n + q], s_x[kMRing + s]);
  }
}

__global__ void __launch_bounds__(kMsB) k_ms_ring(MsArgs a, Status *st) {
  __shared__ int64_t s_x[2 * kMRing + 1];
  __shared__ uint4 s_rec[kMRing];
  __shared__ int64_t s_base[kMRing], s_sx[kMRing];
  __shared__ int64_t s_sxw[kMRing], s_sxwc[kMRing];  // sx + w, sx + w + c
  __shared__ int32_t s_meta[kMRing];
  __shared__ int64_t s_avail[257];
  __shared__ int32_t s_flag[kMNF];
  __shared__ int32_t s_next, s_cur, s_nh, s_abort;
  __shared__ int32_t s_hl[kMsB];
  __shared__ int64_t s_hr[kMsB];
  __shared__ int64_t s_wy[2][kMsB / 64], s_cy[2], s_red[kMsB / 64];
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) {
    s_x[kMZero] = 0;
    s_abort = 0;
  }
  // every slot holds in-range data from the start: the compute wave reads the
  // slots of lanes past a level's end too
  for (int i = tid; i < kMRing; i += kMsB) {
    s_rec[i] = make_uint4(kMZ2, kMZ2, kMZ2, kMZ2);
    s_x[i] = 0;
    s_x[kMRing + i] = 0;
    s_base[i] = 0;
    s_sx[i] = 0;
    s_sxw[i] = 0;
    s_sxwc[i] = 0;
    s_meta[i] = 0;
  }
  for (int i = tid; i < 257; i += kMsB) s_avail[i] = 0;
  auto aborted = [&]() {
    return __hip_atomic_load(&s_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) != 0;
  };
  auto give_up = [&]() {
    raise_err(st, EB_WAIT);
    __hip_atomic_store(&s_abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  };
  int64_t mk = 0;
  const int32_t NS = *a.nseg;
  for (int32_t k = 0; k < NS; k++) {
    const int32_t l0 = a.seg[k], l1 = a.seg[k + 1];
    const int32_t S0 = a.lp[l0], S1 = a.lp[l1];
    if (tid < kMNF) s_flag[tid] = -1;
    if (tid == 0) {
      s_next = 0;
      s_cur = S0;
      s_nh = 0;
    }
    __syncthreads();
    const bool ab = s_abort != 0;
    __syncthreads();  // every wave has read the flag before anyone may set it
    if (ab) break;
    if (a.wide[l0]) {
      // ---------------------------------------------------- block mode
      // one level [S0, S1), kMsB slots per pass in order: ready times from
      // global memory (rows of more than kMBRow predecessors by the whole
      // block), then the prefix maximum across the pass, carried between
      // waves and passes through LDS.  Each pass's per-slot data is loaded
      // during the pass before; the passes' barriers order LDS only (no wave
      // reads this level's finish times).
      struct Pass {
        int32_t e0, e1, meta;
        int64_t sx, w, c;
      };
      auto load_pass = [&](int32_t q0) {
        Pass ps;
        const int32_t p = q0 + tid;
        const bool act = p < S1;
        ps.e0 = act ? a.pptr[p] : 0;
        ps.e1 = act ? a.pptr[p + 1] : 0;
        ps.meta = act ? a.metap[p] : 0;
        ps.sx = act ? a.sxp[p] : 0;
        ps.w = act ? a.wp[p] : 0;
        ps.c = act ? a.cq[p] : 0;
        return ps;
      };
      int par = 0;
      if (tid == 0) s_cy[0] = kNeg;
      Pass cur = load_pass(S0);
      for (int32_t p0 = S0; p0 < S1; p0 += kMsB) {
        const int32_t p = p0 + tid;
        const bool act = p < S1;
        const int32_t e0 = cur.e0, e1 = cur.e1;
        const bool many = e1 - e0 > kMBRow;
        // the first 4 predecessors' values, then the next pass's data, in flight together
        int64_t x[4];
#pragma unroll
        for (int j = 0; j < 4; j++)
          x[j] = (!many && e0 + j < e1) ? ld_coherent(ms_src(a, a.tidx[e0 + j])) : 0;
        const Pass nxt = load_pass(p0 + kMsB);
        int64_t r = 0;
        if (many) {
          s_hl[atomicAdd(&s_nh, 1)] = tid;
        } else {
#pragma unroll
          for (int j = 0; j < 4; j++) {
            if (x[j] < 0) x[j] = ld_final(ms_src(a, a.tidx[e0 + j]), &s_abort, st);
            r = x[j] > r ? x[j] : r;
          }
          for (int32_t e = e0 + 4; e < e1; e += 4) {
            int64_t xx[4];
#pragma unroll
            for (int j = 0; j < 4; j++)
              xx[j] = e + j < e1 ? ld_coherent(ms_src(a, a.tidx[e + j])) : 0;
#pragma unroll
            for (int j = 0; j < 4; j++) {
              if (xx[j] < 0) xx[j] = ld_final(ms_src(a, a.tidx[e + j]), &s_abort, st);
              r = xx[j] > r ? xx[j] : r;
            }
          }
        }
        lds_barrier();
        const int32_t nh = s_nh;
        for (int32_t i = 0; i < nh; i++) {  // rows of many predecessors: the whole block
          const int32_t t2 = s_hl[i];
          const int32_t p2 = p0 + t2;
          // predecessors stored by other waves before a barrier: a barrier
          // does not wait for those stores, so one still in flight is read again
          const int64_t mx = heavy_max<kHeavyU, kMsB>(
              a.pptr[p2], a.pptr[p2 + 1], tid, [&](int32_t e) { return (int32_t)e; },
              [&](int32_t e) { return ld_final(ms_src(a, a.tidx[e]), &s_abort, st); });
          if (lane == 0) s_red[wave] = mx;
          lds_barrier();
          if (tid == 0) {
            int64_t m2 = 0;
            for (int w = 0; w < kMsB / 64; w++) m2 = s_red[w] > m2 ? s_red[w] : m2;
            s_hr[t2] = m2;
          }
          lds_barrier();
        }
        if (act && many) r = s_hr[tid];
        const int32_t meta = cur.meta;
        const int64_t sx = cur.sx;
        const int32_t hd = meta >> 16;
        int64_t y = r - sx;
        if (hd == 0) {
          const int64_t vf = s_avail[meta & 255] - sx;
          y = vf > y ? vf : y;
        }
        y = wave_seg_pmax(y, hd, lane);
        if (lane == 63) s_wy[par][wave] = y;
        lds_barrier();  // every free time read before any is written below
        if (hd > lane) {  // the run began before this wave's row
          const int32_t hs = p - hd;
          int64_t cy = kNeg;
          for (int w2 = wave - 1; w2 >= 0 && p0 + 64 * w2 + 63 >= hs; w2--)
            cy = s_wy[par][w2] > cy ? s_wy[par][w2] : cy;
          if (hs < p0 && s_cy[par] > cy) cy = s_cy[par];
          y = cy > y ? cy : y;
        }
        if (act) {
          const int64_t fin = sx + cur.w + y;
          st_coherent(&a.gf[p], fin);
          st_coherent(&a.gf[(int64_t)a.n + p], fin + cur.c);
          mk = fin > mk ? fin : mk;
          if (meta & 256) s_avail[meta & 255] = fin;
        }
        if (tid == kMsB - 1) s_cy[par ^ 1] = y;
        if (tid == 0) s_nh = 0;
        par ^= 1;
        cur = nxt;
        lds_barrier();
      }
      continue;
    }
    // --------------------------------------------------------- ring mode
    const int32_t nst = (S1 - S0 + kMStage - 1) / kMStage;  // staging tasks
    if (wave == 0) {
      __builtin_amdgcn_s_setprio(3);
      int32_t ready = 0;  // staging tasks known complete: [0, ready)
      bool gaveup = false;
      const int32_t nl = l1 - l0;
      for (int32_t lb = 0; lb < nl && !gaveup; lb += 63) {
        // bounds of up to 63 levels: lane i holds lp[l0 + lb + i]
        const int32_t li = l0 + lb + lane;
        const int32_t bnd = a.lp[li > l1 ? l1 : li];
        // wait for the bounds here, once: a wait inside the level loop would
        // also wait for every store the loop has issued
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        const int32_t cnt = nl - lb < 63 ? nl - lb : 63;
        for (int32_t j = 0; j < cnt; j++) {
          const int32_t pa = __builtin_amdgcn_readlane(bnd, j);
          const int32_t pb = __builtin_amdgcn_readlane(bnd, j + 1);
          // every staging task covering [pa, pb) complete
          const int32_t need = (pb - 1 - S0) / kMStage;
          for (int32_t spin = 0; ready <= need;) {
            // lanes 0..kMNF-1 look at the next kMNF tasks in one LDS round trip
            const int32_t tk = ready + lane;
            const int32_t f = lane < kMNF ? __hip_atomic_load(&s_flag[tk % kMNF], __ATOMIC_RELAXED,
                                                              __HIP_MEMORY_SCOPE_WORKGROUP)
                                          : -1;
            const uint64_t done = __ballot(lane < kMNF && f == tk);
            const int32_t adv = __builtin_ctzll(~done);  // complete tasks in a row from `ready`
            if (adv > 0) {
              ready += adv;
            } else {
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
          // rows of 64 from the level's start, two at a time, in ascending
          // order: a slot's previous position (kMRing back) may still be read
          // by lower slots of the level, which run first
          int64_t carry = 0;
          int32_t r0 = pa;
          for (; r0 + 64 < pb; r0 += 128)
            ms_rows<2>(a, r0, pb, lane, carry, mk, s_x, s_rec, s_base, s_sx, s_sxw, s_sxwc, s_meta, s_avail);
          if (r0 < pb)
            ms_rows<1>(a, r0, pb, lane, carry, mk, s_x, s_rec, s_base, s_sx, s_sxw, s_sxwc, s_meta, s_avail);
          lds_order();
          // this level's slots may be staged again: its reads are done
          __hip_atomic_store(&s_cur, pb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
      }
      __builtin_amdgcn_s_setprio(0);
    } else {
      // staging waves: tasks of kMStage slots, in order
      for (;;) {
        int32_t t = 0;
        if (lane == 0) t = atomicAdd(&s_next, 1);
        t = __builtin_amdgcn_readfirstlane(__shfl(t, 0));
        if (t >= nst || aborted()) break;
        const int32_t lo = S0 + t * kMStage;
        const int32_t hi = lo + kMStage < S1 ? lo + kMStage : S1;
        // static parts first: they need no free slot
        uint4 r[4];
        int64_t sx[4], w[4], c[4];
        int32_t mt[4], f0[4], f1[4];
#pragma unroll
        for (int u = 0; u < 4; u++) {
          const int32_t p = lo + 64 * u + lane;
          const bool v = p < hi;
          r[u] = v ? a.rec[p] : make_uint4(kMZ2, kMZ2, kMZ2, kMZ2);
          sx[u] = v ? a.sxp[p] : 0;
          w[u] = v ? a.wp[p] : 0;
          c[u] = v ? a.cq[p] : 0;
          mt[u] = v ? a.metap[p] : 0;
          f0[u] = v ? a.fptr[p] : 0;
          f1[u] = v ? a.fptr[p + 1] : 0;
        }
        uint32_t q[4][4];
#pragma unroll
        for (int u = 0; u < 4; u++)
#pragma unroll
          for (int j = 0; j < 4; j++) q[u][j] = f0[u] + j < f1[u] ? a.fidx[f0[u] + j] : 0xFFFFFFFFu;
        // wait until the compute wave has left the slots these take over
        // (every position < hi - kMRing computed)
        for (int32_t spin = 0;; spin++) {
          const int32_t cur = __hip_atomic_load(&s_cur, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_WORKGROUP);
          if (cur >= hi - kMRing) break;
          if (spin == kSpin || aborted()) {
            give_up();
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
        if (aborted()) break;
        // the slots' previous positions leave the ring: their values go out first
        ms_flush(a, lo - kMRing > S0 ? lo - kMRing : S0, hi - kMRing, lane, 64, s_x);
        int64_t m[4];
        {
          int64_t x[16];
#pragma unroll
          for (int u = 0; u < 4; u++)
#pragma unroll
            for (int j = 0; j < 4; j++)
              x[4 * u + j] = q[u][j] != 0xFFFFFFFFu ? ld_coherent(ms_src(a, q[u][j])) : 0;
#pragma unroll
          for (int u = 0; u < 4; u++) {
            m[u] = 0;
#pragma unroll
            for (int j = 0; j < 4; j++) {
              int64_t v = x[4 * u + j];
              if (v < 0) v = ld_final(ms_src(a, q[u][j]), &s_abort, st);
              m[u] = v > m[u] ? v : m[u];
            }
          }
        }
        // longer far lists: 4 more at a time per lane up to 64, beyond that the whole wave
#pragma unroll
        for (int u = 0; u < 4; u++) {
          const bool lng = f1[u] - f0[u] > 64;
          for (int32_t e = f0[u] + 4; e < (lng ? f0[u] : f1[u]); e += 4) {
            int64_t x[4];
#pragma unroll
            for (int j = 0; j < 4; j++) x[j] = e + j < f1[u] ? ld_coherent(ms_src(a, a.fidx[e + j])) : 0;
#pragma unroll
            for (int j = 0; j < 4; j++) {
              if (x[j] < 0) x[j] = ld_final(ms_src(a, a.fidx[e + j]), &s_abort, st);
              m[u] = x[j] > m[u] ? x[j] : m[u];
            }
          }
          for (uint64_t hv = __ballot(lng); hv; hv &= hv - 1) {
            const int h = __builtin_ctzll(hv);
            const int32_t g0 = __builtin_amdgcn_readlane(f0[u], h);
            const int32_t g1 = __builtin_amdgcn_readlane(f1[u], h);
            int64_t mx = 0;
            for (int32_t e = g0 + 4 + lane; e < g1; e += 256) {
              int64_t x[4];
#pragma unroll
              for (int j = 0; j < 4; j++)
                x[j] = e + 64 * j < g1 ? ld_coherent(ms_src(a, a.fidx[e + 64 * j])) : 0;
#pragma unroll
              for (int j = 0; j < 4; j++) {
                if (x[j] < 0) x[j] = ld_final(ms_src(a, a.fidx[e + 64 * j]), &s_abort, st);
                mx = x[j] > mx ? x[j] : mx;
              }
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
            const int s = p & kMRMask;
            s_rec[s] = r[u];
            s_base[s] = m[u];
            s_sx[s] = sx[u];
            s_sxw[s] = sx[u] + w[u];
            s_sxwc[s] = sx[u] + w[u] + c[u];
            s_meta[s] = mt[u];
          }
        }
        // the task's slots are written (LDS: in order) before its flag
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        if (lane == 0)
          __hip_atomic_store(&s_flag[t % kMNF], t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
    __syncthreads();  // the segment is done: every value in the ring
    // values whose slots were never taken over: the segment's last kMRing
    ms_flush(a, S1 - kMRing > S0 ? S1 - kMRing : S0, S1, tid, kMsB, s_x);
    // the stores reach L2 before the next segment's barrier (a barrier alone
    // does not wait for them; readers re-read a value not yet there anyway)
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  }
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t o = __shfl_xor((long long)mk, off);
    mk = o > mk ? o : mk;
  }
  __syncthreads();
  if (lane == 0) s_red[wave] = mk;
  __syncthreads();
  if (tid == 0) {
    int64_t r = 0;
    for (int w = 0; w < kMsB / 64; w++) r = s_red[w] > r ? s_red[w] : r;
    a.makespan[0] = r;
  }
}

// ------------------------------------------------------------------- host

int ms_ring(int32_t n, int32_t m, int32_t L, const int32_t *lp, const int32_t *gorder,
            const int32_t *level, const int32_t *pptr, const int32_t *pidx, const int64_t *wp,
            const int64_t *cq, const uint8_t *devp, const int64_t *sxp, const int32_t *metap,
            int64_t *finp, int64_t *makespan, Scratch &sc, hipStream_t s, Status *st) {
  int32_t *wide, *flag, *pre, *seg, *segid, *nseg, *fcnt, *fptr, *hcnt, *hptr, *hidx, *rmax;
  uint32_t *tidx, *fidx;
  uint4 *rec;
  CEL_TRY(sc.get(&wide, L));
  CEL_TRY(sc.get(&flag, L));
  CEL_TRY(sc.get(&pre, (int64_t)L + 1));
  CEL_TRY(sc.get(&seg, (int64_t)L + 1));
  CEL_TRY(sc.get(&segid, L));
  CEL_TRY(sc.get(&nseg, 1));
  CEL_TRY(sc.get(&fcnt, n));
  CEL_TRY(sc.get(&fptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&hcnt, n));
  CEL_TRY(sc.get(&hptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&rmax, n));
  CEL_TRY(sc.get(&tidx, m));
  CEL_TRY(sc.get(&fidx, m));
  CEL_TRY(sc.get(&hidx, m));
  CEL_TRY(sc.get(&rec, n));
  k_fill_i32<<<grid_for(L, 256, 1024), 256, 0, s>>>(wide, L, 0);
  k_fill_i64<<<grid_for(2 * (int64_t)n, 256, 4096), 256, 0, s>>>(finp, 2 * (int64_t)n, -1);
  k_fill_i32<<<grid_for(n, 256, 4096), 256, 0, s>>>(rmax, n, 0);
  const int gn = grid_for(n, 256, 4096), gl = grid_for(L, 256, 1024);
  k_ms_wide<<<gn, 256, 0, s>>>(n, L, lp, pptr, gorder, level, wide, st);
  k_sw_segflag<<<gl, 256, 0, s>>>(L, wide, flag, st);
  CEL_TRY(exclusive_scan_i32(flag, pre, L, sc, s));
  k_sw_segfill<<<gl, 256, 0, s>>>(L, flag, pre, seg, segid, nseg, st);
  k_ms_prep<0><<<gn, 256, 0, s>>>(n, lp, pptr, pidx, gorder, level, wide, seg, segid, devp, tidx,
                                  rec, fcnt, hcnt, nullptr, nullptr, nullptr, nullptr, rmax, st);
  CEL_TRY(exclusive_scan_i32(fcnt, fptr, n, sc, s));
  CEL_TRY(exclusive_scan_i32(hcnt, hptr, n, sc, s));
  k_ms_prep<1><<<gn, 256, 0, s>>>(n, lp, pptr, pidx, gorder, level, wide, seg, segid, devp, tidx,
                                  rec, fcnt, hcnt, fptr, fidx, hptr, hidx, rmax, st);
  k_ms_rowmark<<<gn, 256, 0, s>>>(n, lp, gorder, level, wide, rmax, rec, st);
  MsArgs a{};
  a.n = n;
  a.lp = lp;
  a.pptr = pptr;
  a.tidx = tidx;
  a.wp = wp;
  a.cq = cq;
  a.sxp = sxp;
  a.metap = metap;
  a.rec = rec;
  a.fptr = fptr;
  a.fidx = fidx;
  a.hptr = hptr;
  a.hidx = hidx;
  a.seg = seg;
  a.nseg = nseg;
  a.wide = wide;
  a.gf = finp;
  a.makespan = makespan;
  {
    KTimer kt(s, "k_makespan_one");
    k_ms_ring<<<1, kMsB, 0, s>>>(a, st);
  }
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

}  // namespace cel
