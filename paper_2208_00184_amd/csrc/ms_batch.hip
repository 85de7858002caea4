// Makespan of K placements at once (eq. 7, Order-Place's device model), one
// workgroup per placement, levels run from an LDS ring as in ms_ring.hip but
// over the priority order itself: everything that depends only on the graph
// and the order (pull records of near predecessors, far lists, level sums) is
// prepared once for all placements, and each workgroup's staging waves add
// its placement's part (devices, the devices-differ bit of every pull entry,
// far predecessors' values).
//
// A level's device chains are FIFO in priority order.  When a level sits on
// one device (nearly every level of a clustered placement and of its small
// perturbations) the chain is the level itself, so with sx the sum of w over
// the level's positions before a slot the finish times are the single-run
// prefix maximum of ms_ring.hip.  Otherwise each row of 64 is partitioned by
// device (ballots over the device id's bits, a stable permutation) and run as
// a segmented scan of max-plus maps x -> max(ready + w, x + w) seeded with
// each device's free time; rows go in order, so a device's chain continues
// through its free time.  Wide levels (block mode) partition each pass of the
// workgroup the same way across its waves.
#include "cel_internal.h"

namespace cel {

constexpr int kBB = 512;                // 8 waves: 1 compute, 7 staging
constexpr int kBNW = kBB / 64;
constexpr int kBRing = 2048;            // slots held in the ring
constexpr int kBRMask = kBRing - 1;
constexpr int kBWideW = 1536;           // wider levels run in block mode
constexpr int kBHeavyDeg = 4096;        // a node with more predecessors puts its level in block mode
constexpr int kBStage = 256;            // slots per staging task
constexpr int kBNF = kBRing / kBStage;  // staging flags
constexpr int kBNear = 8;               // near predecessors in a pull record
constexpr int kBBRow = 64;              // block mode: larger rows are taken by the whole block
static_assert(kBWideW + kBStage < kBRing, "a narrow level and a staging task fit the ring");
constexpr uint32_t kBZero = 2 * kBRing;  // ring index that always reads 0
constexpr uint32_t kBZ2 = kBZero | kBZero << 16;
constexpr int64_t kBShift = int64_t(1) << 62;  // map scans: a shifted so the identity is zero

struct MbArgs {
  int32_t n, L;
  const int32_t *lp;              // [L + 1] level starts (positions)
  const int32_t *pptr, *pidx;     // predecessors (positions)
  const int64_t *wp, *cq, *sxl;   // by position: w, c, sum of w over the level before the position
  const uint4 *rec;               // pull records: ring slots of near predecessors, no device bit
  const int32_t *fptr, *fidx;     // far predecessors (positions)
  const int32_t *hptr, *hidx;     // long near lists (positions)
  const int32_t *seg, *nseg, *wide;
  const int32_t *linfo;           // [K][L] gather class | one device << 3 | its device << 8
  const uint8_t *devp;            // [K][n] device by position
  int64_t *fin, *fc;              // [K][n] fin and fin + c by position, -1 until written
  int64_t *makespan;              // [K]
};

__device__ inline uint32_t mb_entry(const uint4 &r, int j) {
  const uint32_t w = j < 2 ? r.x : (j < 4 ? r.y : (j < 6 ? r.z : r.w));
  return ((j & 1) ? (w >> 16) : w) & 0x1FFFu;
}

// -------------------------------------------------------------- preparation

__global__ void k_mb_wide(int32_t n, int32_t L, const int32_t *lp, const int32_t *pptr,
                          const int32_t *order, const int32_t *level, int32_t *wide,
                          const Status *st) {
  if (failed(st)) return;
  const int64_t i0 = blockIdx.x * (int64_t)blockDim.x + threadIdx.x, step = (int64_t)gridDim.x * blockDim.x;
  for (int64_t l = i0; l < L; l += step)
    if (lp[l + 1] - lp[l] > kBWideW) wide[l] = 1;
  for (int64_t p = i0; p < n; p += step)
    if (pptr[p + 1] - pptr[p] > kBHeavyDeg) wide[level[order[p]]] = 1;
}

// PASS 0: per position of a ring level its pull record (ring slots of near
// predecessors), far and long-list counts, the level's largest near count
// (lmax) and sxl.  PASS 1: far lists and long lists (positions).
template <int PASS>
__global__ void k_mb_prep(int32_t n, const int32_t *lp, const int32_t *pptr, const int32_t *pidx,
                          const int32_t *order, const int32_t *level, const int32_t *wide,
                          const int32_t *seg, const int32_t *segid, const int64_t *wx,
                          int64_t *sxl, uint4 *rec, int32_t *fcnt, int32_t *hcnt,
                          const int32_t *fptr, int32_t *fidx, const int32_t *hptr, int32_t *hidx,
                          int32_t *lmax, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t l = level[order[p]];
    const int32_t e0 = pptr[p], e1 = pptr[p + 1];
    if (PASS == 0) sxl[p] = wx[p] - wx[lp[l]];
    if (wide[l]) {
      if (PASS == 0) {
        rec[p] = make_uint4(kBZ2, kBZ2, kBZ2, kBZ2);
        fcnt[p] = 0;
        hcnt[p] = 0;
      }
      continue;
    }
    const int32_t S0 = lp[seg[segid[l]]];
    int32_t nn = 0, nf = 0;
    uint32_t ent[kBNear];
#pragma unroll
    for (int j = 0; j < kBNear; j++) ent[j] = kBZero;
    for (int32_t e = e0; e < e1; e++) {
      const int32_t q = pidx[e];
      if (q >= S0 && (int32_t)p - q < kBRing) {
        if (PASS == 0) {
#pragma unroll
          for (int j = 0; j < kBNear; j++)
            if (j == nn) ent[j] = (uint32_t)(q & kBRMask);
        } else if (hptr[p + 1] > hptr[p]) {
          hidx[hptr[p] + nn] = q;
        }
        nn++;
      } else {
        if (PASS == 1) fidx[fptr[p] + nf] = q;
        nf++;
      }
    }
    if (PASS == 0) {
      fcnt[p] = nf;
      hcnt[p] = nn > kBNear ? nn : 0;
      if (nn > 0) atomicMax(&lmax[l], nn);
      if (nn > kBNear)
        rec[p] = make_uint4(kBZ2 | 0x80000000u, kBZ2, kBZ2, kBZ2);
      else
        rec[p] = make_uint4(ent[0] | ent[1] << 16, ent[2] | ent[3] << 16, ent[4] | ent[5] << 16,
                            ent[6] | ent[7] << 16);
    }
  }
}

// per placement and level: gather class, whether the level lies on one
// device in that placement, and that device
__global__ void k_mb_linfo(int32_t K, int32_t n, int32_t L, const int32_t *lp,
                           const int32_t *wide, const int32_t *lmax, const uint8_t *devp,
                           int32_t *linfo, const Status *st) {
  if (failed(st)) return;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < (int64_t)K * L;
       x += (int64_t)gridDim.x * blockDim.x) {
    const int32_t k = (int32_t)(x / L), l = (int32_t)(x % L);
    if (wide[l]) {
      linfo[x] = 0;
      continue;
    }
    const uint8_t *dk = devp + (int64_t)k * n;
    const int32_t a = lp[l], b = lp[l + 1];
    const uint8_t d0 = dk[a];
    bool one = true;
    for (int32_t p = a + 1; p < b && one; p++) one = dk[p] == d0;
    const int32_t m = lmax[l];
    const int32_t cls = m == 0 ? 0 : (m <= 2 ? 1 : (m <= 4 ? 2 : (m <= kBNear ? 3 : 4)));
    linfo[x] = cls | (one ? 8 : 0) | (int32_t)d0 << 8;
  }
}

// ------------------------------------------------------------------ compute

// The ring and staged arrays in LDS.
struct MbLds {
  int64_t *x;                     // [2 kBRing + 1] fin, fin + c, then 0
  uint4 *rec;                     // pull records with the placement's device bits
  int64_t *base, *sx, *sxw, *c;   // folded far ready time, sx, sx + w, c
  uint8_t *dev;
  int64_t *avail;                 // [257] free time per device, then 0
};

// y[u] = max(y[u], the first K entries' ring values), maxima as trees (all
// values non-negative)
template <int NR, int K>
__device__ inline void mb_near(int64_t (&y)[NR], const uint4 (&r)[NR], const int64_t *s_x) {
  int64_t g[NR][K];
#pragma unroll
  for (int u = 0; u < NR; u++)
#pragma unroll
    for (int j = 0; j < K; j++) g[u][j] = s_x[mb_entry(r[u], j)];
#pragma unroll
  for (int u = 0; u < NR; u++) {
#pragma unroll
    for (int w = 1; w < K; w <<= 1)
#pragma unroll
      for (int j = 0; j + w < K; j += 2 * w) g[u][j] = max_nonneg(g[u][j], g[u][j + w]);
    y[u] = max_nonneg(y[u], g[u][0]);
  }
}

// ready times of NR rows from r0 (all values non-negative): folded far
// maximum, near gathers, and the long lists of slots with more than kBNear
// near predecessors (their devices read from global memory)
template <int NR>
__device__ inline void mb_ready(const MbArgs &a, const uint8_t *dk, int32_t r0, int32_t b,
                                uint32_t cls, int lane, const uint4 (&r)[NR],
                                const uint8_t (&dv)[NR], int64_t (&y)[NR], const MbLds &S) {
  if (cls <= 1) mb_near<NR, 2>(y, r, S.x);
  else if (cls == 2) mb_near<NR, 4>(y, r, S.x);
  else mb_near<NR, kBNear>(y, r, S.x);
  if (cls == 4) {
#pragma unroll
    for (int u = 0; u < NR; u++) {
      const int32_t p = r0 + 64 * u + lane;
      const bool hv = p < b && (r[u].x >> 31);
      const int32_t hs = hv ? a.hptr[p] : 0, he = hv ? a.hptr[p + 1] : 0;
      const int32_t hd = hv ? dv[u] : 0;
      for (uint64_t hm = __ballot(hv); hm; hm &= hm - 1) {
        const int h = __builtin_ctzll(hm);
        const int32_t g0 = __builtin_amdgcn_readlane(hs, h);
        const int32_t g1 = __builtin_amdgcn_readlane(he, h);
        const int32_t dh = __builtin_amdgcn_readlane(hd, h);
        int64_t mx = 0;
        for (int32_t i = g0 + lane; i < g1; i += 64) {
          const int32_t q = a.hidx[i];
          const uint32_t ix = (uint32_t)(q & kBRMask) + (dk[q] != dh ? kBRing : 0);
          mx = max_nonneg(mx, S.x[ix]);
        }
        for (int off = 32; off > 0; off >>= 1) {
          const int32_t lo = __shfl_xor((int32_t)mx, off), hi = __shfl_xor((int32_t)(mx >> 32), off);
          mx = max_nonneg(mx, (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
        }
        if (lane == h) y[u] = max_nonneg(y[u], mx);
      }
    }
  }
}

template <int CTRL, int ROWMASK, int NR>
__device__ inline void mb_pmax_step(int64_t (&y)[NR]) {
  int64_t u[NR];
#pragma unroll
  for (int k = 0; k < NR; k++) {
    if constexpr (ROWMASK == 0xF) {
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

// NR rows [r0, r0 + 64 NR) of a level [pa, b) that lies on device d0: the
// single-run prefix maximum of y = max(0, ready - sx), the free time at the
// level's first slot (where sx = 0) and the carry of the previous rows; the
// free time is updated at the level's last slot.
template <int NR>
__device__ inline void mb_rows_one(const MbArgs &a, const uint8_t *dk, int32_t r0, int32_t pa,
                                   int32_t b, uint32_t cls, int32_t d0, int lane, int64_t &carry,
                                   int64_t &mk, const MbLds &S) {
  uint4 r[NR];
  int64_t y[NR], sx[NR], w[NR], c[NR];
  uint8_t dv[NR];
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int s = (r0 + 64 * u + lane) & kBRMask;
    r[u] = S.rec[s];
    y[u] = S.base[s];
    sx[u] = S.sx[s];
    w[u] = S.sxw[s];
    c[u] = S.c[s];
    dv[u] = (uint8_t)d0;
  }
  lds_order();
  const int64_t av0 = S.avail[d0];
  mb_ready<NR>(a, dk, r0, b, cls, lane, r, dv, y, S);
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int64_t av = (r0 + 64 * u + lane == pa) ? av0 : 0;
    y[u] = max_nonneg(max_nonneg(y[u], sx[u]) - sx[u], av);
  }
  mb_pmax_step<0x111, 0xF, NR>(y);  // row_shr:1
  mb_pmax_step<0x112, 0xF, NR>(y);  // row_shr:2
  mb_pmax_step<0x114, 0xF, NR>(y);  // row_shr:4
  mb_pmax_step<0x118, 0xF, NR>(y);  // row_shr:8
  mb_pmax_step<0x142, 0xA, NR>(y);  // row_bcast:15 into rows 1 and 3
  mb_pmax_step<0x143, 0xC, NR>(y);  // row_bcast:31 into rows 2 and 3
#pragma unroll
  for (int u = 0; u < NR; u++) {  // one run: every row continues the previous ones
    y[u] = max_nonneg(y[u], carry);
    carry = readlane64(y[u], 63);
  }
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int32_t p = r0 + 64 * u + lane;
    if (p < b) {
      const int s = p & kBRMask;
      const int64_t fin = w[u] + y[u];
      S.x[s] = fin;
      S.x[kBRing + s] = fin + c[u];
      mk = max_nonneg(mk, fin);
      if (p == b - 1) S.avail[d0] = fin;
    }
  }
}

// One step of the segmented scan of max-plus maps x -> max(a, x + b), a
// shifted by kBShift so that the identity is all zero and DPP may zero-fill;
// a lane that starts its segment keeps its own map.
template <int CTRL, int ROWMASK>
__device__ inline void mb_segmap_step(int64_t &sa, int64_t &sb, int32_t &f) {
  const int32_t alo = __builtin_amdgcn_update_dpp(0, (int32_t)sa, CTRL, ROWMASK, 0xF, true);
  const int32_t ahi = __builtin_amdgcn_update_dpp(0, (int32_t)(sa >> 32), CTRL, ROWMASK, 0xF, true);
  const int32_t blo = __builtin_amdgcn_update_dpp(0, (int32_t)sb, CTRL, ROWMASK, 0xF, true);
  const int32_t bhi = __builtin_amdgcn_update_dpp(0, (int32_t)(sb >> 32), CTRL, ROWMASK, 0xF, true);
  const int32_t uf = __builtin_amdgcn_update_dpp(0, f, CTRL, ROWMASK, 0xF, true);
  const int64_t ua = (int64_t)(((uint64_t)(uint32_t)ahi << 32) | (uint32_t)alo);
  const int64_t ub = (int64_t)(((uint64_t)(uint32_t)bhi << 32) | (uint32_t)blo);
  const bool keep = f != 0;
  const int64_t cmb = ua + sb;
  sa = (keep || cmb <= sa) ? sa : cmb;
  sb = keep ? sb : ub + sb;
  f = keep ? f : uf;
}
__device__ inline void mb_segmap(int64_t &sa, int64_t &sb, int32_t &f) {
  mb_segmap_step<0x111, 0xF>(sa, sb, f);
  mb_segmap_step<0x112, 0xF>(sa, sb, f);
  mb_segmap_step<0x114, 0xF>(sa, sb, f);
  mb_segmap_step<0x118, 0xF>(sa, sb, f);
  mb_segmap_step<0x142, 0xA>(sa, sb, f);
  mb_segmap_step<0x143, 0xC>(sa, sb, f);
}

// One row [r0, r0 + 64) of a level on several devices (slots past b idle):
// ready times as in the one-device case, then each device's chain through
// the row as a segmented map scan in device-grouped order (a stable
// permutation from ballots over the device id's bits), seeded with the
// device's free time, which the device's last slot of the row updates.
__device__ inline void mb_row_multi(const MbArgs &a, const uint8_t *dk, int32_t r0, int32_t b,
                                    uint32_t cls, int lane, int64_t &mk, const MbLds &S) {
  const int s = (r0 + lane) & kBRMask;
  const bool act = r0 + lane < b;
  uint4 r[1];
  int64_t y[1];
  uint8_t dv[1];
  r[0] = S.rec[s];
  y[0] = S.base[s];
  const int64_t sx = S.sx[s], sxw = S.sxw[s], c = S.c[s];
  dv[0] = S.dev[s];
  lds_order();
  mb_ready<1>(a, dk, r0, b, cls, lane, r, dv, y, S);
  const int dvi = act ? (int)dv[0] : 0;
  const int64_t w = sxw - sx;
  // rank in device-grouped order (devices ascending, positions ascending)
  const uint64_t actm = __ballot(act);
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  uint64_t eq = actm, lt = 0;
  for (int bit = 7; bit >= 0; bit--) {
    const uint32_t on = (dvi >> bit) & 1;
    const uint64_t bb = __ballot(on) & actm;
    if (on) {
      lt |= eq & ~bb;  // same bits above, 0 here where this lane has 1
      eq &= bb;
    } else {
      eq &= ~bb;
    }
  }
  const int below = __popcll(eq & lanemask_lt);
  const int q = act ? __popcll(lt) + below : lane;  // a permutation of the lanes
  const int head = act && below == 0;
  const int tail = act && (eq >> lane) == 1ull;
  const int addr = q << 2;
  const int64_t ash = y[0] + w + kBShift;
  const int32_t meta = dvi | (head << 8) | (tail << 9) | ((int)act << 10);
  const int32_t pa_lo = __builtin_amdgcn_ds_permute(addr, (int32_t)ash);
  const int32_t pa_hi = __builtin_amdgcn_ds_permute(addr, (int32_t)(ash >> 32));
  const int32_t pb_lo = __builtin_amdgcn_ds_permute(addr, (int32_t)w);
  const int32_t pb_hi = __builtin_amdgcn_ds_permute(addr, (int32_t)(w >> 32));
  const int32_t pm = __builtin_amdgcn_ds_permute(addr, meta);
  const bool pact = (pm >> 10) & 1;
  const int dq = pm & 255;
  int64_t sa = pact ? (int64_t)(((uint64_t)(uint32_t)pa_hi << 32) | (uint32_t)pa_lo) : 0;
  int64_t sb = pact ? (int64_t)(((uint64_t)(uint32_t)pb_hi << 32) | (uint32_t)pb_lo) : 0;
  int32_t f = pact ? ((pm >> 8) & 1) : 1;
  mb_segmap(sa, sb, f);
  int64_t fq = 0;
  if (pact) {
    const int64_t viafree = S.avail[dq] + sb;
    const int64_t z = sa - kBShift;
    fq = viafree > z ? viafree : z;
  }
  lds_order();  // every read of a free time before the updates below
  if (pact && ((pm >> 9) & 1)) S.avail[dq] = fq;
  // back to the slot's own lane
  const int32_t flo = __builtin_amdgcn_ds_bpermute(addr, (int32_t)fq);
  const int32_t fhi = __builtin_amdgcn_ds_bpermute(addr, (int32_t)(fq >> 32));
  const int64_t fin = (int64_t)(((uint64_t)(uint32_t)fhi << 32) | (uint32_t)flo);
  if (act) {
    S.x[s] = fin;
    S.x[kBRing + s] = fin + c;
    mk = max_nonneg(mk, fin);
  }
}

// values of positions [q0, q1) from the ring to global memory
__device__ inline void mb_flush(int64_t *fk, int64_t *ck, int32_t q0, int32_t q1, int t, int step,
                                const int64_t *s_x) {
  for (int32_t q = q0 + t; q < q1; q += step) {
    const int s = q & kBRMask;
    st_coherent(&fk[q], s_x[s]);
    st_coherent(&ck[q], s_x[kBRing + s]);
  }
}

// value of predecessor q for a node on device d: fin, or fin + c when the
// devices differ, read again until visible
__device__ inline int64_t mb_pred(const uint8_t *dk, const int64_t *fk, const int64_t *ck, int32_t q,
                                  int d, int32_t *s_abort, Status *st) {
  const int64_t *p = dk[q] != d ? &ck[q] : &fk[q];
  return ld_final(p, s_abort, st);
}

// max of m and the values of predecessors q[j] (q < 0: none) for nodes on
// devices d[j]: every device load, then every value load, is issued before
// the first use; a value not yet visible is read again (rare)
template <int N>
__device__ inline int64_t mb_preds(int64_t m, const int32_t (&q)[N], const int (&d)[N],
                                   const uint8_t *dk, const int64_t *fk, const int64_t *ck,
                                   int32_t *s_abort, Status *st) {
  int dq[N];
#pragma unroll
  for (int j = 0; j < N; j++) dq[j] = q[j] >= 0 ? (int)dk[q[j]] : 0;
  const int64_t *ptr[N];
  int64_t x[N];
#pragma unroll
  for (int j = 0; j < N; j++) {
    ptr[j] = q[j] >= 0 ? (dq[j] != d[j] ? &ck[q[j]] : &fk[q[j]]) : nullptr;
    x[j] = q[j] >= 0 ? ld_coherent(ptr[j]) : 0;
  }
#pragma unroll
  for (int j = 0; j < N; j++) {
    if (x[j] < 0) x[j] = ld_final(ptr[j], s_abort, st);
    m = max_nonneg(m, x[j]);
  }
  return m;
}

__global__ void __launch_bounds__(kBB) k_mb_ring(MbArgs a, Status *st) {
  __shared__ int64_t s_x[2 * kBRing + 1];
  __shared__ uint4 s_rec[kBRing];
  // s_base, s_sx in ring mode; the block-mode scratch otherwise (a segment
  // starts with an empty ring)
  __shared__ int64_t s_pool[2 * kBRing];
  __shared__ int64_t s_sxw[kBRing], s_c[kBRing];
  __shared__ uint8_t s_dev[kBRing];
  __shared__ int64_t s_avail[257];
  __shared__ int32_t s_flag[kBNF];
  __shared__ int32_t s_next, s_cur, s_nh, s_abort;
  __shared__ int32_t s_dbase[256], s_dsum[4];
  __shared__ int64_t s_wa[kBNW], s_wb[kBNW], s_red[kBNW];
  __shared__ int32_t s_wf[kBNW];
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t k = blockIdx.x, n = a.n;
  const uint8_t *dk = a.devp + (int64_t)k * n;
  int64_t *fk = a.fin + (int64_t)k * n;
  int64_t *ck = a.fc + (int64_t)k * n;
  const int32_t *lk = a.linfo + (int64_t)k * a.L;
  int64_t *s_base = s_pool, *s_sx = s_pool + kBRing;
  // block-mode scratch, carved from s_pool (2 x kBRing int64)
  int32_t *s_wcnt = reinterpret_cast<int32_t *>(s_pool);          // [kBNW][256]
  int64_t *s_ga = s_pool + kBNW * 256 / 2;                         // [kBB]
  int64_t *s_gb = s_ga + kBB;                                      // [kBB]
  int64_t *s_hr = s_gb + kBB;                                      // [kBB]
  int32_t *s_gpos = reinterpret_cast<int32_t *>(s_hr + kBB);       // [kBB]
  int32_t *s_hl = s_gpos + kBB;                                    // [kBB]
  uint8_t *s_gdev = reinterpret_cast<uint8_t *>(s_hl + kBB);       // [kBB + 1]
  static_assert(kBNW * 256 / 2 + 3 * kBB + kBB + (kBB + 1 + 7) / 8 <= 2 * kBRing,
                "block-mode scratch fits the pool");
  if (tid == 0) {
    s_x[kBZero] = 0;
    s_abort = 0;
  }
  for (int i = tid; i < kBRing; i += kBB) {
    s_rec[i] = make_uint4(kBZ2, kBZ2, kBZ2, kBZ2);
    s_x[i] = 0;
    s_x[kBRing + i] = 0;
    s_base[i] = 0;
    s_sx[i] = 0;
    s_sxw[i] = 0;
    s_c[i] = 0;
    s_dev[i] = 0;
  }
  for (int i = tid; i < 257; i += kBB) s_avail[i] = 0;
  auto aborted = [&]() {
    return __hip_atomic_load(&s_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) != 0;
  };
  auto give_up = [&]() {
    raise_err(st, EB_WAIT);
    __hip_atomic_store(&s_abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  };
  int64_t mk = 0;
  const int32_t NS = *a.nseg;
  for (int32_t sg = 0; sg < NS; sg++) {
    const int32_t l0 = a.seg[sg], l1 = a.seg[sg + 1];
    const int32_t S0 = a.lp[l0], S1 = a.lp[l1];
    if (tid < kBNF) s_flag[tid] = -1;
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
      // one level [S0, S1), kBB positions per pass in order: ready times from
      // global memory (rows of more than kBBRow predecessors by the whole
      // block), a stable partition of the pass by device across the waves,
      // and each device's chain as a segmented map scan seeded with its free
      // time
      for (int32_t p0 = S0; p0 < S1; p0 += kBB) {
        const int32_t cnt2 = S1 - p0 < kBB ? S1 - p0 : kBB;
        const int32_t p = p0 + tid;
        const bool act = tid < cnt2;
        const int dvi = act ? (int)dk[p] : 255;
        const int32_t e0 = act ? a.pptr[p] : 0, e1 = act ? a.pptr[p + 1] : 0;
        const bool many = e1 - e0 > kBBRow;
        int64_t ready = 0;
        if (many) {
          s_hl[atomicAdd(&s_nh, 1)] = tid;
        } else {
          for (int32_t e = e0; e < e1; e += 4) {
            int32_t qq[4];
            int dd[4];
#pragma unroll
            for (int j = 0; j < 4; j++) {
              qq[j] = e + j < e1 ? a.pidx[e + j] : -1;
              dd[j] = dvi;
            }
            ready = mb_preds<4>(ready, qq, dd, dk, fk, ck, &s_abort, st);
          }
        }
        for (int x = tid; x < kBNW * 256; x += kBB) s_wcnt[x] = 0;
        __syncthreads();
        const int32_t nh = s_nh;
        for (int32_t i = 0; i < nh; i++) {  // rows of many predecessors: the whole block
          const int32_t t2 = s_hl[i];
          const int32_t p2 = p0 + t2;
          const int d2 = dk[p2];
          const int64_t mx = heavy_max<kHeavyU, kBB>(
              a.pptr[p2], a.pptr[p2 + 1], tid, [&](int32_t e) { return a.pidx[e]; },
              [&](int32_t q) { return mb_pred(dk, fk, ck, q, d2, &s_abort, st); });
          if (lane == 0) s_red[wave] = mx;
          __syncthreads();
          if (tid == 0) {
            int64_t m2 = 0;
            for (int w2 = 0; w2 < kBNW; w2++) m2 = s_red[w2] > m2 ? s_red[w2] : m2;
            s_hr[t2] = m2;
          }
          __syncthreads();
        }
        if (act && many) ready = s_hr[tid];
        const int64_t ww = act ? a.wp[p] : 0;
        const int64_t aa = ready + ww;
        // stable partition by device: rank among same-device lanes of the wave
        uint64_t eq = ~0ull;
        for (int bit = 0; bit < 8; bit++) {
          const int on = (dvi >> bit) & 1;
          const uint64_t bb = __ballot(on);
          eq &= on ? bb : ~bb;
        }
        const int rank = __popcll(eq & ((1ull << lane) - 1ull));
        if (act && rank == 0) s_wcnt[wave * 256 + dvi] = __popcll(eq);
        __syncthreads();
        int32_t tot = 0;
        if (tid < 256) {
          for (int w2 = 0; w2 < kBNW; w2++) {
            const int32_t cc = s_wcnt[w2 * 256 + tid];
            s_wcnt[w2 * 256 + tid] = tot;
            tot += cc;
          }
        }
        int32_t inc = tot;
        for (int off = 1; off < 64; off <<= 1) {
          const int32_t yy = __shfl_up(inc, off);
          if (lane >= off) inc += yy;
        }
        if (tid < 256 && lane == 63) s_dsum[wave] = inc;
        __syncthreads();
        if (tid < 256) {
          int32_t bv = inc - tot;
          for (int w2 = 0; w2 < wave; w2++) bv += s_dsum[w2];
          s_dbase[tid] = bv;
        }
        __syncthreads();
        if (act) {
          const int qg = s_dbase[dvi] + s_wcnt[wave * 256 + dvi] + rank;
          s_ga[qg] = aa;
          s_gb[qg] = ww;
          s_gpos[qg] = p;
          s_gdev[qg] = (uint8_t)dvi;
        }
        __syncthreads();
        // segmented scan of (a, b) in device-grouped order
        const bool aq = tid < cnt2;
        int64_t sa = kNeg, sb = 0;
        int dq = 255;
        int32_t f = 1;
        if (aq) {
          sa = s_ga[tid];
          sb = s_gb[tid];
          dq = s_gdev[tid];
          f = (tid == 0) || (s_gdev[tid - 1] != dq);
        }
        wave_seg_scan_dpp(sa, sb, f);
        if (lane == 63) {
          s_wa[wave] = sa;
          s_wb[wave] = sb;
          s_wf[wave] = f;
        }
        __syncthreads();
        if (aq && !f && wave > 0) {  // segment began in an earlier wave: prepend their totals
          int64_t ca = s_wa[wave - 1], cb = s_wb[wave - 1];
          bool done = s_wf[wave - 1] != 0;
          for (int w2 = wave - 2; w2 >= 0 && !done; w2--) {
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
          const int32_t j = s_gpos[tid];
          st_coherent(&fk[j], fin);
          st_coherent(&ck[j], fin + a.cq[j]);
          mk = max_nonneg(mk, fin);
          last = (tid + 1 == cnt2) || (s_gdev[tid + 1] != dq);
        }
        __syncthreads();  // every read of a free time is done
        if (last) s_avail[dq] = fin;
        if (tid == 0) s_nh = 0;
        __syncthreads();
      }
      continue;
    }
    // --------------------------------------------------------- ring mode
    const int32_t nst = (S1 - S0 + kBStage - 1) / kBStage;  // staging tasks
    if (wave == 0) {
      __builtin_amdgcn_s_setprio(3);
      const MbLds S{s_x, s_rec, s_base, s_sx, s_sxw, s_c, s_dev, s_avail};
      int32_t ready = 0;  // staging tasks known complete: [0, ready)
      bool gaveup = false;
      const int32_t nl = l1 - l0;
      for (int32_t lb = 0; lb < nl && !gaveup; lb += 63) {
        // bounds and info of up to 63 levels: lane i holds level l0 + lb + i
        const int32_t li = l0 + lb + lane;
        const int32_t bnd = a.lp[li > l1 ? l1 : li];
        const int32_t inf = lk[li >= l1 ? l1 - 1 : li];
        // wait for them here, once: a wait inside the level loop would also
        // wait for every store the loop has issued
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
        const int32_t cnt = nl - lb < 63 ? nl - lb : 63;
        for (int32_t j = 0; j < cnt; j++) {
          const int32_t pa = __builtin_amdgcn_readlane(bnd, j);
          const int32_t pb = __builtin_amdgcn_readlane(bnd, j + 1);
          const int32_t info = __builtin_amdgcn_readlane(inf, j);
          const uint32_t cls = (uint32_t)info & 7u;
          const bool one = (info >> 3) & 1;
          // every staging task covering [pa, pb) complete
          const int32_t need = (pb - 1 - S0) / kBStage;
          for (int32_t spin = 0; ready <= need;) {
            const int32_t tk = ready + lane;
            const int32_t f = lane < kBNF ? __hip_atomic_load(&s_flag[tk % kBNF], __ATOMIC_RELAXED,
                                                              __HIP_MEMORY_SCOPE_WORKGROUP)
                                          : -1;
            const uint64_t done = __ballot(lane < kBNF && f == tk);
            const int32_t adv = __builtin_ctzll(~done);
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
          // rows of 64 from the level's start, in ascending order: a slot's
          // previous position (kBRing back) may still be read by lower slots
          // of the level, which run first
          if (one) {
            const int32_t d0 = (info >> 8) & 255;
            int64_t carry = 0;
            int32_t r0 = pa;
            for (; r0 + 64 < pb; r0 += 128)
              mb_rows_one<2>(a, dk, r0, pa, pb, cls, d0, lane, carry, mk, S);
            if (r0 < pb) mb_rows_one<1>(a, dk, r0, pa, pb, cls, d0, lane, carry, mk, S);
          } else {
            for (int32_t r0 = pa; r0 < pb; r0 += 64) {
              mb_row_multi(a, dk, r0, pb, cls, lane, mk, S);
              lds_order();
            }
          }
          lds_order();
          // this level's slots may be staged again: its reads are done
          __hip_atomic_store(&s_cur, pb, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        }
      }
      __builtin_amdgcn_s_setprio(0);
    } else {
      // staging waves: tasks of kBStage slots, in order
      for (;;) {
        int32_t t = 0;
        if (lane == 0) t = atomicAdd(&s_next, 1);
        t = __builtin_amdgcn_readfirstlane(__shfl(t, 0));
        if (t >= nst || aborted()) break;
        const int32_t lo = S0 + t * kBStage;
        const int32_t hi = lo + kBStage < S1 ? lo + kBStage : S1;
        // static parts first: they need no free slot
        uint4 r[4];
        int64_t sx[4], w[4], c[4];
        int32_t f0[4], f1[4];
        int dv[4];
#pragma unroll
        for (int u = 0; u < 4; u++) {
          const int32_t p = lo + 64 * u + lane;
          const bool v = p < hi;
          r[u] = v ? a.rec[p] : make_uint4(kBZ2, kBZ2, kBZ2, kBZ2);
          sx[u] = v ? a.sxl[p] : 0;
          w[u] = v ? a.wp[p] : 0;
          c[u] = v ? a.cq[p] : 0;
          dv[u] = v ? (int)dk[p] : 0;
          f0[u] = v ? a.fptr[p] : 0;
          f1[u] = v ? a.fptr[p + 1] : 0;
        }
        // the devices of the near predecessors (position q from ring slot e:
        // the one position in (p - kBRing, p) with that slot)
        uint32_t xb[4] = {0, 0, 0, 0};  // bit j: entry j's predecessor on another device
        {
          int qd[4][kBNear];
#pragma unroll
          for (int u = 0; u < 4; u++) {
            const int32_t p = lo + 64 * u + lane;
#pragma unroll
            for (int j = 0; j < kBNear; j++) {
              const uint32_t e = mb_entry(r[u], j);
              const int32_t q = p - (int32_t)(((uint32_t)(p & kBRMask) - e) & kBRMask);
              qd[u][j] = (p < hi && e != kBZero) ? (int)dk[q] : dv[u];
            }
          }
#pragma unroll
          for (int u = 0; u < 4; u++)
#pragma unroll
            for (int j = 0; j < kBNear; j++) xb[u] |= (uint32_t)(qd[u][j] != dv[u]) << j;
        }
        int32_t q[4][4];
#pragma unroll
        for (int u = 0; u < 4; u++)
#pragma unroll
          for (int j = 0; j < 4; j++) q[u][j] = f0[u] + j < f1[u] ? a.fidx[f0[u] + j] : -1;
        // wait until the compute wave has left the slots these take over
        for (int32_t spin = 0;; spin++) {
          const int32_t cur = __hip_atomic_load(&s_cur, __ATOMIC_RELAXED,
                                                __HIP_MEMORY_SCOPE_WORKGROUP);
          if (cur >= hi - kBRing) break;
          if (spin == kSpin || aborted()) {
            give_up();
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
        if (aborted()) break;
        // the slots' previous positions leave the ring: their values go out first
        mb_flush(fk, ck, lo - kBRing > S0 ? lo - kBRing : S0, hi - kBRing, lane, 64, s_x);
        int64_t m[4];
#pragma unroll
        for (int u = 0; u < 4; u++) {
          int dd[4] = {dv[u], dv[u], dv[u], dv[u]};
          m[u] = mb_preds<4>(0, q[u], dd, dk, fk, ck, &s_abort, st);
        }
        // longer far lists: 4 more at a time per lane up to 64, beyond that the whole wave
#pragma unroll
        for (int u = 0; u < 4; u++) {
          const bool lng = f1[u] - f0[u] > 64;
          for (int32_t e = f0[u] + 4; e < (lng ? f0[u] : f1[u]); e += 4) {
            int32_t qq[4];
            int dd[4];
#pragma unroll
            for (int j = 0; j < 4; j++) {
              qq[j] = e + j < f1[u] ? a.fidx[e + j] : -1;
              dd[j] = dv[u];
            }
            m[u] = mb_preds<4>(m[u], qq, dd, dk, fk, ck, &s_abort, st);
          }
          for (uint64_t hv = __ballot(lng); hv; hv &= hv - 1) {
            const int h = __builtin_ctzll(hv);
            const int32_t g0 = __builtin_amdgcn_readlane(f0[u], h);
            const int32_t g1 = __builtin_amdgcn_readlane(f1[u], h);
            const int dh = __builtin_amdgcn_readlane(dv[u], h);
            int64_t mx = 0;
            for (int32_t e = g0 + 4 + lane; e < g1; e += 64)
              mx = max_nonneg(mx, mb_pred(dk, fk, ck, a.fidx[e], dh, &s_abort, st));
            for (int off = 32; off > 0; off >>= 1) {
              const int32_t lo2 = __shfl_xor((int32_t)mx, off), hi2 = __shfl_xor((int32_t)(mx >> 32), off);
              mx = max_nonneg(mx, (int64_t)(((uint64_t)(uint32_t)hi2 << 32) | (uint32_t)lo2));
            }
            if (lane == h) m[u] = max_nonneg(m[u], mx);
          }
        }
#pragma unroll
        for (int u = 0; u < 4; u++) {
          const int32_t p = lo + 64 * u + lane;
          if (p < hi) {
            const int s = p & kBRMask;
            // pull entries with the device bit: + kBRing reads fin + c
            uint4 rr = r[u];
            uint32_t *wd = reinterpret_cast<uint32_t *>(&rr);
#pragma unroll
            for (int j = 0; j < kBNear; j++)
              if ((xb[u] >> j) & 1) wd[j >> 1] += (uint32_t)kBRing << (16 * (j & 1));
            s_rec[s] = rr;
            s_base[s] = m[u];
            s_sx[s] = sx[u];
            s_sxw[s] = sx[u] + w[u];
            s_c[s] = c[u];
            s_dev[s] = (uint8_t)dv[u];
          }
        }
        // the task's slots are written (LDS: in order) before its flag
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        if (lane == 0)
          __hip_atomic_store(&s_flag[t % kBNF], t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      }
    }
    __syncthreads();  // the segment is done: every value in the ring
    mb_flush(fk, ck, S1 - kBRing > S0 ? S1 - kBRing : S0, S1, tid, kBB, s_x);
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
    for (int w = 0; w < kBNW; w++) r = s_red[w] > r ? s_red[w] : r;
    a.makespan[k] = r;
  }
}

// ------------------------------------------------------------------- host

int mb_ring(int32_t K, int32_t n, int32_t m, int32_t L, const int32_t *lp, const int32_t *order,
            const int32_t *level, const int32_t *pptr, const int32_t *pidx, const int64_t *wp,
            const int64_t *cq, const uint8_t *devp, int64_t *fin, int64_t *fc, int64_t *makespan,
            Scratch &sc, hipStream_t s, Status *st) {
  int32_t *wide, *flag, *pre, *seg, *segid, *nseg, *fcnt, *fptr, *hcnt, *hptr, *fidx, *hidx, *lmax,
      *linfo;
  int64_t *wx, *sxl;
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
  CEL_TRY(sc.get(&fidx, m));
  CEL_TRY(sc.get(&hidx, m));
  CEL_TRY(sc.get(&lmax, L));
  CEL_TRY(sc.get(&linfo, (int64_t)K * L));
  CEL_TRY(sc.get(&wx, (int64_t)n + 1));
  CEL_TRY(sc.get(&sxl, n));
  CEL_TRY(sc.get(&rec, n));
  const int gn = grid_for(n, 256, 4096), gl = grid_for(L, 256, 1024);
  k_fill_i32<<<gl, 256, 0, s>>>(wide, L, 0);
  k_fill_i32<<<gl, 256, 0, s>>>(lmax, L, 0);
  k_fill_i64<<<grid_for((int64_t)K * n, 256, 8192), 256, 0, s>>>(fin, (int64_t)K * n, -1);
  k_fill_i64<<<grid_for((int64_t)K * n, 256, 8192), 256, 0, s>>>(fc, (int64_t)K * n, -1);
  CEL_TRY(exclusive_scan_i64(wp, wx, n, sc, s));
  k_mb_wide<<<gn, 256, 0, s>>>(n, L, lp, pptr, order, level, wide, st);
  k_sw_segflag<<<gl, 256, 0, s>>>(L, wide, flag, st);
  CEL_TRY(exclusive_scan_i32(flag, pre, L, sc, s));
  k_sw_segfill<<<gl, 256, 0, s>>>(L, flag, pre, seg, segid, nseg, st);
  k_mb_prep<0><<<gn, 256, 0, s>>>(n, lp, pptr, pidx, order, level, wide, seg, segid, wx, sxl, rec,
                                  fcnt, hcnt, nullptr, nullptr, nullptr, nullptr, lmax, st);
  CEL_TRY(exclusive_scan_i32(fcnt, fptr, n, sc, s));
  CEL_TRY(exclusive_scan_i32(hcnt, hptr, n, sc, s));
  k_mb_prep<1><<<gn, 256, 0, s>>>(n, lp, pptr, pidx, order, level, wide, seg, segid, wx, sxl, rec,
                                  fcnt, hcnt, fptr, fidx, hptr, hidx, lmax, st);
  k_mb_linfo<<<grid_for((int64_t)K * L, 256, 8192), 256, 0, s>>>(K, n, L, lp, wide, lmax, devp,
                                                                 linfo, st);
  MbArgs a{};
  a.n = n;
  a.L = L;
  a.lp = lp;
  a.pptr = pptr;
  a.pidx = pidx;
  a.wp = wp;
  a.cq = cq;
  a.sxl = sxl;
  a.rec = rec;
  a.fptr = fptr;
  a.fidx = fidx;
  a.hptr = hptr;
  a.hidx = hidx;
  a.seg = seg;
  a.nseg = nseg;
  a.wide = wide;
  a.linfo = linfo;
  a.devp = devp;
  a.fin = fin;
  a.fc = fc;
  a.makespan = makespan;
  {
    KTimer kt(s, "k_makespan_batch");
    k_mb_ring<<<(unsigned)K, kBB, 0, s>>>(a, st);
  }
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

}  // namespace cel
