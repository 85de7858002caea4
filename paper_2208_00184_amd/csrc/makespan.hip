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
#include <map>
#include <mutex>
#include <type_traits>

#include "cel_internal.h"

namespace cel {

// device per position, with range check (devp[k][p] = node_dev[k][order[p]]);
// x runs over positions, y over placements
__global__ void k_dev_gather(int32_t K, int32_t n, const int32_t *order, const uint8_t *node_dev,
                             int32_t D, uint8_t *devp, Status *st) {
  if (failed(st)) return;
  uint32_t bad = 0;
  for (int32_t p = blockIdx.x * blockDim.x + threadIdx.x; p < n; p += gridDim.x * blockDim.x) {
    const int32_t v = order[p];
    for (int32_t k = blockIdx.y; k < K; k += gridDim.y) {
      const uint8_t dv = node_dev[(int64_t)k * n + v];
      if (dv >= D) bad |= EB_ARG;
      devp[(int64_t)k * n + p] = dv;
    }
  }
  if (bad) raise_err(st, bad);
}

// The same gather for a batch: one workgroup per placement stages the
// devices of up to kGRowNodes nodes at a time in LDS (read once, coalesced)
// and serves the positions whose node lies in that range from there; a
// direct gather would move one cache line per byte.
constexpr int kGRowB = 1024;
constexpr int kGRowNodes = 131072;
template <bool VEC>
__global__ void __launch_bounds__(kGRowB) k_dev_rows(int32_t n, const int32_t *order,
                                                     const uint8_t *node_dev, int32_t D,
                                                     uint8_t *devp, Status *st) {
  __shared__ uint32_t s_dev4[kGRowNodes / 4];
  uint8_t *s_dev = (uint8_t *)s_dev4;
  if (failed(st)) return;
  const int64_t koff = (int64_t)blockIdx.x * n;
  const uint8_t *row = node_dev + koff;
  uint8_t *out = devp + koff;
  uint32_t bad = 0;
  for (int32_t v0 = 0; v0 < n; v0 += kGRowNodes) {
    const int32_t cnt = n - v0 < kGRowNodes ? n - v0 : kGRowNodes;
    if (VEC) {  // n, the row and order aligned: words of 4 devices, quads of positions
      const uint32_t *row4 = (const uint32_t *)(row + v0);
#pragma unroll 4
      for (int32_t i = threadIdx.x; i < (cnt >> 2); i += kGRowB) {
        const uint32_t w = row4[i];
#pragma unroll
        for (int j = 0; j < 4; j++)
          if ((int32_t)((w >> (8 * j)) & 255u) >= D) bad |= EB_ARG;
        s_dev4[i] = w;
      }
      __syncthreads();
      const int4 *order4 = (const int4 *)order;
#pragma unroll 2
      for (int32_t i = threadIdx.x; i < (n >> 2); i += kGRowB) {
        const int4 o = order4[i];
        const int32_t v[4] = {o.x - v0, o.y - v0, o.z - v0, o.w - v0};
#pragma unroll
        for (int j = 0; j < 4; j++)
          if ((uint32_t)v[j] < (uint32_t)cnt) out[4 * i + j] = s_dev[v[j]];
      }
    } else {
#pragma unroll 4
      for (int32_t i = threadIdx.x; i < cnt; i += kGRowB) {
        const uint8_t dv = row[v0 + i];
        if (dv >= D) bad |= EB_ARG;
        s_dev[i] = dv;
      }
      __syncthreads();
#pragma unroll 4
      for (int32_t p = threadIdx.x; p < n; p += kGRowB) {
        const int32_t v = order[p] - v0;
        if ((uint32_t)v < (uint32_t)cnt) out[p] = s_dev[v];
      }
    }
    __syncthreads();
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

// Windowed sweep, one workgroup per placement.  Positions are taken in
// windows of at most NC consecutive positions (EC in-edges, kMsL levels).
// Staging folds every predecessor outside the window (its finish time is
// final) into a partial ready time per node, records each edge's owner and
// the owner's device, keeps the window's costs and devices in LDS and the
// per-level ranges in registers (lane l holds levels l, l+64, ...).  Each
// level of the window is then evaluated from LDS only: predecessors inside
// the window edge-parallel (atomic max into the owner's ready time), then the
// device-FIFO chains as a segmented max-plus scan over the level's nodes in
// device-grouped order.  A level of at most 256 nodes and 512 edges is run by
// wave 0 alone in rows of 64, without workgroup barriers; wider levels use
// the whole block.  A node with more than EC predecessors forms a window of
// its own.
constexpr int kMsL = 256;
constexpr int64_t kShift = int64_t(1) << 62;

// packed in-edge words of edges [ea, eb) (at most 512), 8 per lane
__device__ inline void load_epk(int32_t (&pk)[8], const int32_t *s_epk, int32_t ea, int32_t eb,
                                int lane) {
#pragma unroll
  for (int q = 0; q < 8; q++) {
    const int32_t e = ea + lane + 64 * q;
    pk[q] = (ea + 64 * q < eb && e < eb) ? s_epk[e] : 0;
  }
}

// One step of the segmented scan of max-plus maps x -> max(a, x + b) with a
// shifted by +2^62, so that the identity (a, b, no start) is all zero and DPP
// may zero-fill: combine with the lane selected by CTRL unless this lane
// already starts its segment.
template <int CTRL, int ROWMASK>
__device__ inline void segz_step(int64_t &a, int64_t &b, int32_t &f) {
  const int32_t alo = __builtin_amdgcn_update_dpp(0, (int32_t)a, CTRL, ROWMASK, 0xF, true);
  const int32_t ahi = __builtin_amdgcn_update_dpp(0, (int32_t)(a >> 32), CTRL, ROWMASK, 0xF, true);
  const int32_t blo = __builtin_amdgcn_update_dpp(0, (int32_t)b, CTRL, ROWMASK, 0xF, true);
  const int32_t bhi = __builtin_amdgcn_update_dpp(0, (int32_t)(b >> 32), CTRL, ROWMASK, 0xF, true);
  const int32_t uf = __builtin_amdgcn_update_dpp(0, f, CTRL, ROWMASK, 0xF, true);
  const int64_t ua = (int64_t)(((uint64_t)(uint32_t)ahi << 32) | (uint32_t)alo);
  const int64_t ub = (int64_t)(((uint64_t)(uint32_t)bhi << 32) | (uint32_t)blo);
  const bool keep = f != 0;
  const int64_t c = ua + b;
  a = (keep || c <= a) ? a : c;
  b = keep ? b : ub + b;
  f = keep ? f : uf;
}
__device__ inline void wave_seg_scan_maxplus_z(int64_t &a, int64_t &b, int32_t &f) {
  segz_step<0x111, 0xF>(a, b, f);  // row_shr:1
  segz_step<0x112, 0xF>(a, b, f);  // row_shr:2
  segz_step<0x114, 0xF>(a, b, f);  // row_shr:4
  segz_step<0x118, 0xF>(a, b, f);  // row_shr:8
  segz_step<0x142, 0xA>(a, b, f);  // row_bcast:15 into rows 1 and 3
  segz_step<0x143, 0xC>(a, b, f);  // row_bcast:31 into rows 2 and 3
}

// The same scan over one segment (no start flags): every lane combines.
template <int CTRL, int ROWMASK>
__device__ inline void mpz_step(int64_t &a, int64_t &b) {
  const int32_t alo = __builtin_amdgcn_update_dpp(0, (int32_t)a, CTRL, ROWMASK, 0xF, true);
  const int32_t ahi = __builtin_amdgcn_update_dpp(0, (int32_t)(a >> 32), CTRL, ROWMASK, 0xF, true);
  const int32_t blo = __builtin_amdgcn_update_dpp(0, (int32_t)b, CTRL, ROWMASK, 0xF, true);
  const int32_t bhi = __builtin_amdgcn_update_dpp(0, (int32_t)(b >> 32), CTRL, ROWMASK, 0xF, true);
  const int64_t ua = (int64_t)(((uint64_t)(uint32_t)ahi << 32) | (uint32_t)alo);
  const int64_t ub = (int64_t)(((uint64_t)(uint32_t)bhi << 32) | (uint32_t)blo);
  const int64_t c = ua + b;
  a = c <= a ? a : c;
  b = ub + b;
}
__device__ inline void wave_scan_maxplus_z(int64_t &a, int64_t &b) {
  mpz_step<0x111, 0xF>(a, b);
  mpz_step<0x112, 0xF>(a, b);
  mpz_step<0x114, 0xF>(a, b);
  mpz_step<0x118, 0xF>(a, b);
  mpz_step<0x142, 0xA>(a, b);
  mpz_step<0x143, 0xC>(a, b);
}
constexpr int kBatchWide = 384;  // batches up to this size get one CU-sized window per placement
constexpr int kWideLevels = 256;  // mean level width from which batches skip the windows

template <int B, int NC, int EC>
__global__ void __launch_bounds__(B)
    k_makespan_sweep(int32_t n, int32_t L, int32_t dbits, const int32_t *lp, const int32_t *pptr,
                     const int32_t *pidx, const int64_t *wp, const int64_t *cq,
                     const uint8_t *devp, int64_t *finp, int64_t *makespan, const Status *st) {
  constexpr int NW = B / 64;
  static_assert(B >= 256, "device partition uses 256 threads");
  __shared__ int32_t s_lv[kMsL + 2];
  __shared__ int32_t s_rp[NC + 1];
  __shared__ int32_t s_epk[EC];  // per in-edge: pred slot + 1 (0: before the window), owner, owner's device
  __shared__ int16_t s_own[EC];
  __shared__ int64_t s_pm[NC], s_f[NC], s_w[NC], s_c[NC];
  __shared__ uint8_t s_dv[NC];
  __shared__ int32_t s_la[kMsL], s_lb[kMsL], s_lea[kMsL], s_leb[kMsL], s_lend[kMsL];
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
  __shared__ int32_t s_cut;
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const bool wave0 = tid < 64;
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  const int64_t koff = (int64_t)blockIdx.x * n;
  const uint8_t *dk = devp + koff;
  int64_t *fk = finp + koff;
  for (int i = tid; i < 256; i += B) s_avail[i] = 0;
  int64_t mk = 0;
  int32_t P0 = 0, lcur = 0;
  while (P0 < n) {
    CEL_TSTAMP(t0);
    CEL_TCOUNT(6);
    const int32_t Pc1 = P0 + NC < n ? P0 + NC : n;
    for (int t = tid; t <= Pc1 - P0; t += B) s_rp[t] = pptr[P0 + t];
    for (int k = tid; k <= kMsL + 1; k += B) {
      const int32_t l = lcur + k;  // level lcur + k is [s_lv[k], s_lv[k+1])
      s_lv[k] = lp[l > L ? L : l];
    }
    if (tid == 0) s_cut = 0;
    __syncthreads();
    int32_t cnt = 0;
    for (int t = tid; t < Pc1 - P0; t += B) cnt += (s_rp[t + 1] - s_rp[0] <= EC) ? 1 : 0;
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
    if (lane == 0 && cnt) atomicAdd(&s_cut, cnt);
    __syncthreads();
    int32_t P1 = P0 + s_cut;
    const int32_t lvcap = (lcur + kMsL < L) ? s_lv[kMsL] : n;
    if (P1 > lvcap) P1 = lvcap;
    const bool heavy = (P1 == P0);  // one node with more than EC predecessors
    if (heavy) P1 = P0 + 1;
    const int32_t E0 = s_rp[0], E1 = s_rp[P1 - P0];
    for (int32_t i = tid; i < P1 - P0; i += B) {
      const uint8_t dv = dk[P0 + i];
      s_pm[i] = 0;
      s_w[i] = wp[P0 + i];
      s_c[i] = cq[P0 + i];
      s_dv[i] = dv;
      if (!heavy)
        for (int32_t q = s_rp[i] - E0; q < s_rp[i + 1] - E0; q++) s_own[q] = (int16_t)i;
    }
    for (int32_t k = tid; k < kMsL; k += B) {
      const int32_t lb = s_lv[k], le = s_lv[k + 1];
      int32_t a = lb < P0 ? P0 : (lb > P1 ? P1 : lb);
      const int32_t b = le < P0 ? P0 : (le > P1 ? P1 : le);
      if (a > b) a = b;
      s_la[k] = a - P0;
      s_lb[k] = b - P0;
      s_lea[k] = heavy ? 0 : s_rp[a - P0] - E0;
      s_leb[k] = heavy ? 0 : s_rp[b - P0] - E0;
      s_lend[k] = le >= P1;
    }
    __syncthreads();
    CEL_TSTAMP(t1);
    CEL_TADD(0, t0, t1);
    // predecessors before the window are final: fold them into s_pm
    for (int32_t e = E0 + tid; e < E1; e += B) {
      const int32_t q = pidx[e];
      const int32_t own = heavy ? 0 : s_own[e - E0];
      if (!heavy)
        s_epk[e - E0] = (q >= P0 ? q - P0 + 1 : 0) | (own << 12) | ((int32_t)s_dv[own] << 24);
      if (q < P0) {
        const int64_t x = fk[q] + (dk[q] != s_dv[own] ? cq[q] : 0);
        atomicMax((long long *)&s_pm[own], (long long)x);
      }
    }
    __syncthreads();
    CEL_TSTAMP(t2);
    CEL_TADD(1, t1, t2);
    int32_t ma[4], mb[4], mea[4], meb[4], mend[4];
#pragma unroll
    for (int u = 0; u < 4; u++) {
      const int k = lane + 64 * u;
      ma[u] = s_la[k];
      mb[u] = s_lb[k];
      mea[u] = s_lea[k];
      meb[u] = s_leb[k];
      mend[u] = s_lend[k];
    }
    bool synced = true;
    CEL_TSTAMP(t3);
    CEL_TADD(2, t2, t3);
    for (int32_t k = 0; k < kMsL; k++) {
      const int u = k >> 6, ln = k & 63;
      int32_t a0, b0, ea, eb, stop;
      switch (u) {
        case 0: a0 = ma[0]; b0 = mb[0]; ea = mea[0]; eb = meb[0]; stop = mend[0]; break;
        case 1: a0 = ma[1]; b0 = mb[1]; ea = mea[1]; eb = meb[1]; stop = mend[1]; break;
        case 2: a0 = ma[2]; b0 = mb[2]; ea = mea[2]; eb = meb[2]; stop = mend[2]; break;
        default: a0 = ma[3]; b0 = mb[3]; ea = mea[3]; eb = meb[3]; stop = mend[3]; break;
      }
      a0 = __builtin_amdgcn_readlane(a0, ln);
      b0 = __builtin_amdgcn_readlane(b0, ln);
      ea = __builtin_amdgcn_readlane(ea, ln);
      eb = __builtin_amdgcn_readlane(eb, ln);
      stop = __builtin_amdgcn_readlane(stop, ln);
      if (a0 < b0) {
        const bool narrow = (b0 - a0 <= 256) && (eb - ea <= 512);
        CEL_TSTAMP(tl0);
        if (narrow) {
          if (wave0) {
            // predecessors inside the window: up to 8 edges per lane (one
            // packed word each: predecessor slot, owner, owner's device)
            int32_t pk[8];
            load_epk(pk, s_epk, ea, eb, lane);
            int64_t x[8];
            int32_t ow[8];
#pragma unroll
            for (int q = 0; q < 8; q++) {
              ow[q] = -1;
              x[q] = 0;
              if (ea + 64 * q < eb) {
                const int32_t wd = pk[q];
                const int32_t jp = wd & 0xFFF;
                const int32_t j = jp ? jp - 1 : 0;
                ow[q] = jp ? (wd >> 12) & 0xFFF : -1;
                x[q] = s_f[j] + (s_dv[j] != ((wd >> 24) & 255) ? s_c[j] : 0);
              }
            }
#pragma unroll
            for (int q = 0; q < 8; q++)
              if (ow[q] >= 0) atomicMax((long long *)&s_pm[ow[q]], (long long)x[q]);
            // One wave's LDS operations complete in issue order, so the rows
            // below see these updates; only the compiler must not reorder.
            lds_order();
            CEL_TSTAMP(te);
            CEL_TADD(9, tl0, te);
            for (int32_t row = a0; row < b0; row += 64) {
              CEL_TCOUNT(11);
              const int32_t cnt2 = b0 - row < 64 ? b0 - row : 64;
              const bool act = lane < cnt2;
              const int32_t i = row + lane;
              int dv = 0;
              int64_t aa = 0, ww = 0;
              if (act) {
                dv = s_dv[i];
                ww = s_w[i];
                aa = s_pm[i] + ww;
              }
              // Rows whose nodes all sit on one device (nearly every row of
              // a clustered placement): device-grouped order is lane order
              // and the row is one segment, so no permutation is needed.
              const int dv0 = __builtin_amdgcn_readfirstlane(dv);  // lane 0 is active
              if (__ballot(act && dv != dv0) == 0) {
                int64_t sa = act ? aa + kShift : 0, sb = act ? ww : 0;
                wave_scan_maxplus_z(sa, sb);
                sa -= kShift;
                int64_t fin = 0;
                if (act) {
                  const int64_t viafree = s_avail[dv0] + sb;
                  fin = viafree > sa ? viafree : sa;
                  s_f[i] = fin;
                  fk[P0 + i] = fin;
                  mk = fin > mk ? fin : mk;
                }
                lds_order();  // every lane's read of s_avail precedes the update
                if (lane == cnt2 - 1) s_avail[dv0] = fin;
              } else {
                // slot in device-grouped order (devices ascending, positions
                // ascending): ballots over the device id's bits, high to low
                const uint64_t actm = __ballot(act);
                uint32_t eql = (uint32_t)actm, eqh = (uint32_t)(actm >> 32), ltl = 0, lth = 0;
                for (int bit = dbits - 1; bit >= 0; bit--) {
                  const uint32_t on = (dv >> bit) & 1;
                  const uint64_t bb = __ballot(on) & actm;
                  const uint32_t bl = (uint32_t)bb, bh = (uint32_t)(bb >> 32);
                  const uint32_t keep0 = on - 1u;  // ~0 when the bit is 0, else 0
                  ltl |= (eql & ~bl) & ~keep0;     // equal so far, bit 0 there, 1 here
                  lth |= (eqh & ~bh) & ~keep0;
                  eql &= bl ^ keep0;
                  eqh &= bh ^ keep0;
                }
                const uint64_t eq = ((uint64_t)eqh << 32) | eql;
                const int below = __popcll(eq & lanemask_lt);
                const int q = act ? __popc(ltl) + __popc(lth) + below : lane;  // a permutation
                const int head = act && below == 0;                // first of its device
                const int tail = act && (eq >> lane) == 1ull;      // last of its device
                const int addr = q << 2;
                const int64_t ash = aa + kShift;  // shifted: the scan identity is all zero
                const int32_t meta = dv | (head << 8) | (tail << 9) | ((int)act << 10);
                const int32_t pa_lo = __builtin_amdgcn_ds_permute(addr, (int32_t)ash);
                const int32_t pa_hi = __builtin_amdgcn_ds_permute(addr, (int32_t)(ash >> 32));
                const int32_t pb_lo = __builtin_amdgcn_ds_permute(addr, (int32_t)ww);
                const int32_t pb_hi = __builtin_amdgcn_ds_permute(addr, (int32_t)(ww >> 32));
                const int32_t pm = __builtin_amdgcn_ds_permute(addr, meta);
                const int32_t pj = __builtin_amdgcn_ds_permute(addr, i);
                const bool pact = (pm >> 10) & 1;
                const int dq = pm & 255;
                int64_t sa = pact ? (int64_t)(((uint64_t)(uint32_t)pa_hi << 32) | (uint32_t)pa_lo) : 0;
                int64_t sb = pact ? (int64_t)(((uint64_t)(uint32_t)pb_hi << 32) | (uint32_t)pb_lo) : 0;
                int32_t f = pact ? ((pm >> 8) & 1) : 1;
                wave_seg_scan_maxplus_z(sa, sb, f);
                sa -= kShift;
                if (pact) {
                  const int64_t viafree = s_avail[dq] + sb;
                  const int64_t fin = viafree > sa ? viafree : sa;
                  s_f[pj] = fin;
                  fk[P0 + pj] = fin;
                  mk = fin > mk ? fin : mk;
                  lds_order();  // every lane's read of s_avail precedes the update
                  if ((pm >> 9) & 1) s_avail[dq] = fin;
                }

              }
              lds_order();
            }
            CEL_TSTAMP(tr);
            CEL_TADD(10, te, tr);
          }
          synced = false;
          CEL_TSTAMP(tl1);
          CEL_TADD(7, tl0, tl1);

          CEL_TCOUNT(4);
        } else {
          if (!synced) __syncthreads();
          for (int32_t e = ea + tid; e < eb; e += B) {
            const int32_t wd = s_epk[e];
            const int32_t jp = wd & 0xFFF;
            if (jp) {
              const int32_t j = jp - 1;
              const int64_t x = s_f[j] + (s_dv[j] != ((wd >> 24) & 255) ? s_c[j] : 0);
              atomicMax((long long *)&s_pm[(wd >> 12) & 0xFFF], (long long)x);
            }
          }
          __syncthreads();
          for (int32_t base = a0; base < b0; base += B) {
            const int32_t cnt2 = b0 - base < B ? b0 - base : B;
            const bool act = tid < cnt2;
            const int32_t i = base + tid;
            for (int x = tid; x < NW * 256; x += B) (&s_wcnt[0][0])[x] = 0;
            __syncthreads();
            int dv = 255;
            int64_t aa = 0, ww = 0;
            if (act) {
              dv = s_dv[i];
              ww = s_w[i];
              aa = s_pm[i] + ww;
            }
            // stable partition by device: rank among same-device lanes of the wave
            uint64_t eq = ~0ull;
            for (int bit = 0; bit < 8; bit++) {
              const int on = (dv >> bit) & 1;
              const uint64_t bb = __ballot(on);
              eq &= on ? bb : ~bb;
            }
            const int rank = __popcll(eq & lanemask_lt);
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
              s_a[q] = aa;
              s_b[q] = ww;
              s_pos[q] = i;
              s_dev[q] = (uint8_t)dv;
            }
            __syncthreads();
            // segmented scan of (a, b) in device-grouped order
            const bool aq = tid < cnt2;
            int64_t sa = kNeg, sb = 0;
            int dq = 255;
            int32_t f = 1;
            if (aq) {
              sa = s_a[tid];
              sb = s_b[tid];
              dq = s_dev[tid];
              f = (tid == 0) || (s_dev[tid - 1] != dq);
            }
            wave_seg_scan_dpp(sa, sb, f);
            if (lane == 63) {
              s_wa[wv] = sa;
              s_wb[wv] = sb;
              s_wf[wv] = f;
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
              const int32_t j = s_pos[tid];
              s_f[j] = fin;
              fk[P0 + j] = fin;
              mk = fin > mk ? fin : mk;
              last = (tid + 1 == cnt2) || (s_dev[tid + 1] != dq);
            }
            __syncthreads();  // every read of s_avail is done
            if (last) s_avail[dq] = fin;
            __syncthreads();
          }
          synced = true;
          CEL_TSTAMP(tl1);
          CEL_TADD(8, tl0, tl1);
          CEL_TCOUNT(5);
        }
      }
      if (stop) break;  // the window ends inside this level
    }
    CEL_TSTAMP(t4);
    CEL_TADD(3, t3, t4);
    // next window starts at P1; move the level cursor to the level holding P1
    if (P1 < n) {
      int32_t k = 0;
      while (k < kMsL && lcur + k + 1 < L && s_lv[k + 1] <= P1) k++;
      lcur += k;
    }
    P0 = P1;
    __syncthreads();
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

// ---------------------------------------------------------------------------
// Single placement (K = 1) over the device-grouped order: inside every level
// the nodes are sorted by device, priority order kept within a device, so each
// device's FIFO chain in a level is one run of consecutive slots.  k_runs
// precomputes the run data; the sweep itself is ms_ring (ms_ring.hip).

// Run structure of the device-grouped order, per slot s: sx = exclusive sum
// of w over the slot's run, meta = device | run ends here << 8 |
// min(distance to the run's first slot, 32767) << 16.
__global__ void k_runs(int32_t n, const int32_t *lp, const int32_t *level, const int32_t *gorder,
                       const uint8_t *gdev, const int64_t *wx, int64_t *sx, int32_t *meta,
                       const Status *st) {
  if (failed(st)) return;
  for (int32_t s = blockIdx.x * blockDim.x + threadIdx.x; s < n; s += gridDim.x * blockDim.x) {
    const int32_t l = level[gorder[s]];
    const int32_t lo = lp[l], hi = lp[l + 1];
    const int d = gdev[s];
    int32_t a = lo, b = s;  // first slot of the level with device d (devices ascend)
    while (a < b) {
      const int32_t mid = (a + b) >> 1;
      if (gdev[mid] < d) a = mid + 1;
      else b = mid;
    }
    sx[s] = wx[s] - wx[a];
    const int32_t hd = s - a < 32767 ? s - a : 32767;
    const int tl = (s + 1 == hi) || gdev[s + 1] != d;
    meta[s] = d | (tl << 8) | (hd << 16);
  }
}

// keys for the device-grouped order: device of each position, id = position
__global__ void k_dev_keys(int32_t n, const uint8_t *devp, uint64_t *keys, uint32_t *ids,
                           const Status *st) {
  if (failed(st)) return;
  for (int32_t p = blockIdx.x * blockDim.x + threadIdx.x; p < n; p += gridDim.x * blockDim.x) {
    keys[p] = devp[p];
    ids[p] = (uint32_t)p;
  }
}

// grouped order: node, device and inverse position of every slot
__global__ void k_grouped(int32_t n, const int32_t *order, const uint32_t *sig,
                          const uint8_t *devp, int32_t *gorder, int32_t *gpos, uint8_t *gdev,
                          const Status *st) {
  if (failed(st)) return;
  for (int32_t s = blockIdx.x * blockDim.x + threadIdx.x; s < n; s += gridDim.x * blockDim.x) {
    const uint32_t p = sig[s];
    const int32_t v = order[p];
    gorder[s] = v;
    gpos[v] = s;
    gdev[s] = devp[p];
  }
}

// ---------------------------------------------------------------------------
// Batches over graphs with wide levels: one workgroup of B threads per
// placement walks the levels in order with no LDS window.  Predecessors of a
// level all lie in earlier levels, whose finish times this workgroup already
// wrote to global memory, so every ready() of a level is gathered at once:
// each thread takes PT nodes per pass, loads their first kRnd in-edge indices,
// then all predecessor finish, device and comm values, in flight together (a
// node with more in-edges finishes in a loop).  Each chunk of B nodes is then
// partitioned by device (stable: ballots per wave, per-wave device counts in
// LDS) and scanned as max-plus maps per device run, seeded with the device's
// free time, which the run's last node updates.
template <int B, int PT, int kRnd>
__global__ void __launch_bounds__(B)
    k_makespan_levels(int32_t n, int32_t L, int32_t dbits, const int32_t *lp, const int32_t *pptr,
                      const int32_t *pidx, const int64_t *wp, const int64_t *cq,
                      const uint8_t *devp, int64_t *finp, int64_t *makespan, const Status *st) {
  constexpr int NW = B / 64;
  static_assert(B >= 256 && B % 64 == 0, "the device prefix uses one thread per device id");
  __shared__ int64_t s_avail[256];
  __shared__ int32_t s_wcnt[NW][256];
  __shared__ int32_t s_dbase[256];
  __shared__ int32_t s_dsum[4];
  __shared__ int64_t s_a[B], s_b[B];
  __shared__ int32_t s_pos[B];
  __shared__ uint8_t s_dev[B];
  __shared__ int64_t s_wa[NW], s_wb[NW];
  __shared__ int32_t s_wf[NW];
  __shared__ int64_t s_red[NW];
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const uint64_t lanemask_lt = (1ull << lane) - 1ull;
  const int64_t koff = (int64_t)blockIdx.x * n;
  const uint8_t *dk = devp + koff;
  int64_t *fk = finp + koff;
  const bool dlane = tid < 256;  // threads that own a device id in the prefix steps
  if (dlane) {
    s_avail[tid] = 0;
    for (int w2 = 0; w2 < NW; w2++) s_wcnt[w2][tid] = 0;
  }
  __syncthreads();
  int64_t mk = 0;
  for (int32_t l = 0; l < L; l++) {
    const int32_t a = lp[l], b = lp[l + 1];
    for (int32_t base = a; base < b; base += B * PT) {
      // ---- gather: a = ready + w and w of PT nodes per thread
      int32_t dv[PT], e0[PT], e1[PT];
      int64_t w[PT], rdy[PT];
#pragma unroll
      for (int j = 0; j < PT; j++) {
        const int32_t p = base + j * B + tid;
        const bool act = p < b;
        const int32_t ps = act ? p : a;
        dv[j] = act ? dk[ps] : 255;
        w[j] = wp[ps];
        e0[j] = pptr[ps];
        e1[j] = act ? pptr[ps + 1] : e0[j];
        rdy[j] = 0;
      }
      int32_t q[PT][kRnd];
#pragma unroll
      for (int j = 0; j < PT; j++)
#pragma unroll
        for (int r = 0; r < kRnd; r++) {
          const bool ok = e0[j] + r < e1[j];
          const int32_t v = pidx[ok ? e0[j] + r : 0];  // pidx holds at least one element
          q[j][r] = ok ? v : 0;                         // node 0 stands in for absent edges
        }
      int64_t fq[PT][kRnd], cc[PT][kRnd];
      int32_t dq[PT][kRnd];
#pragma unroll
      for (int j = 0; j < PT; j++)
#pragma unroll
        for (int r = 0; r < kRnd; r++) {
          fq[j][r] = fk[q[j][r]];
          dq[j][r] = dk[q[j][r]];
          cc[j][r] = cq[q[j][r]];
        }
#pragma unroll
      for (int j = 0; j < PT; j++) {
#pragma unroll
        for (int r = 0; r < kRnd; r++) {
          if (e0[j] + r < e1[j]) {
            const int64_t x = fq[j][r] + (dq[j][r] != dv[j] ? cc[j][r] : 0);
            rdy[j] = x > rdy[j] ? x : rdy[j];
          }
        }
        for (int32_t e = e0[j] + kRnd; e < e1[j]; e++) {  // in-edges past the first kRnd
          const int32_t qq = pidx[e];
          const int64_t x = fk[qq] + (dk[qq] != dv[j] ? cq[qq] : 0);
          rdy[j] = x > rdy[j] ? x : rdy[j];
        }
      }
      // ---- per chunk of B nodes: stable partition by device, then scan
#pragma unroll
      for (int j = 0; j < PT; j++) {
        const int32_t cbase = base + j * B;
        if (cbase >= b) break;  // uniform
        const int32_t cnt = b - cbase < B ? b - cbase : B;
        const bool act = tid < cnt;
        const int d = dv[j];
        const uint64_t actm = __ballot(act);
        uint64_t eq = actm;
        for (int bit = 0; bit < dbits; bit++) {
          const int on = (d >> bit) & 1;
          const uint64_t bb = __ballot(on);
          eq &= on ? bb : ~bb;
        }
        const int rank = __popcll(eq & lanemask_lt);
        if (act && rank == 0) s_wcnt[wv][d] = __popcll(eq);
        __syncthreads();
        // per device: exclusive bases over the waves, then over the devices
        int32_t tot = 0;
        if (dlane)
          for (int w2 = 0; w2 < NW; w2++) {
            const int32_t c = s_wcnt[w2][tid];
            s_wcnt[w2][tid] = tot;
            tot += c;
          }
        int32_t inc = tot;
        for (int off = 1; off < 64; off <<= 1) {
          const int32_t y = __shfl_up(inc, off);
          if (lane >= off) inc += y;
        }
        if (dlane && lane == 63) s_dsum[wv] = inc;
        __syncthreads();
        if (dlane) {
          int32_t bv = inc - tot;
          for (int w2 = 0; w2 < wv; w2++) bv += s_dsum[w2];
          s_dbase[tid] = bv;
        }
        __syncthreads();
        if (act) {
          const int slot = s_dbase[d] + s_wcnt[wv][d] + rank;
          s_a[slot] = rdy[j] + w[j];
          s_b[slot] = w[j];
          s_pos[slot] = cbase + tid;
          s_dev[slot] = (uint8_t)d;
        }
        __syncthreads();
        if (dlane)
          for (int w2 = 0; w2 < NW; w2++) s_wcnt[w2][tid] = 0;  // ready for the next chunk
        // segmented scan of (a, b) over the device runs
        int64_t sa = kNeg, sb = 0;
        int dq2 = 0;
        int32_t f = 1;
        if (act) {
          sa = s_a[tid];
          sb = s_b[tid];
          dq2 = s_dev[tid];
          f = (tid == 0) || (s_dev[tid - 1] != dq2);
        }
        wave_seg_scan_dpp(sa, sb, f);
        if (lane == 63) {
          s_wa[wv] = sa;
          s_wb[wv] = sb;
          s_wf[wv] = f;
        }
        __syncthreads();
        if (act && !f && wv > 0) {  // the run began in an earlier wave: prepend their totals
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
        if (act) {
          const int64_t viafree = s_avail[dq2] + sb;
          fin = viafree > sa ? viafree : sa;
          fk[s_pos[tid]] = fin;
          mk = fin > mk ? fin : mk;
          last = (tid + 1 == cnt) || (s_dev[tid + 1] != dq2);
        }
        __syncthreads();  // every read of s_avail, s_a, s_b, s_dev is done
        if (last) s_avail[dq2] = fin;
      }
    }
    // the next level gathers these finish times from global memory
    __syncthreads();
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

CEL_PHASE_READER(cel_debug_phases_makespan)

static int check_makespan_args(const char *fn, const cel_graph *g, const cel_devices *d,
                               const int32_t *order, const int32_t *level,
                               const int32_t *level_ptr, int32_t L, int32_t K,
                               const uint8_t *node_dev, const int64_t *makespan) {
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n;
  if (!makespan || !level_ptr || K < 1 || (n > 0 && (!order || !level || !node_dev)))
    return set_error(CEL_E_ARG, "%s: NULL argument or K < 1", fn);
  if (L < 0 || L > n || (n > 0 && L == 0)) return set_error(CEL_E_ARG, "%s: n_levels out of range", fn);
  return CEL_OK;
}

// How the calling thread's last makespan call ran (cel_makespan_info).
struct MsInfo {
  int32_t path, rounds;
};
static thread_local MsInfo t_ms_info{2, 0};
static thread_local int t_ms_relax = 1;

extern "C" int cel_makespan_relax(int mode) {
  if (mode < 0) return set_error(CEL_E_ARG, "cel_makespan_relax: negative mode");
  const int was = t_ms_relax;
  t_ms_relax = mode;
  return was;
}

extern "C" int cel_makespan_info(int32_t *path, int32_t *rounds) {
  if (!path || !rounds) return set_error(CEL_E_ARG, "cel_makespan_info: NULL argument");
  *path = t_ms_info.path;
  *rounds = t_ms_info.rounds;
  return CEL_OK;
}

// The whole call on scratch from `sc` (the arena, or the fixed array of
// cel_makespan_noalloc).
static int makespan_impl(const char *fn, const cel_graph *g, const cel_devices *d,
                         const int32_t *order, const int32_t *level, const int32_t *level_ptr,
                         int32_t L, int32_t K, const uint8_t *node_dev, int64_t *start,
                         int64_t *finish, int64_t *makespan, Scratch &sc, hipStream_t s) {
  const int32_t n = g->n;
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
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, sc, s));
  CEL_TRY(check_level_order(g, order, level, level_ptr, L, pos, st, s));
  CEL_TRY(sc.get(&pptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&pidx, g->m));
  CEL_TRY(sc.get(&wp, n));
  CEL_TRY(sc.get(&cq, n));
  CEL_TRY(sc.get(&devp, (int64_t)K * n));
  CEL_TRY(sc.get(&finp, 2 * (int64_t)K * n));  // fin, then fin + c (the ring sweeps)
  const int gx = grid_for(n, 256, 1024);
  if (K == 1) {
    uint8_t *dev0;
    CEL_TRY(sc.get(&dev0, n));
    {
      KTimer kt(s, "k_dev_gather");
      k_dev_gather<<<dim3(gx, 1), 256, 0, s>>>(1, n, order, node_dev, d->D, dev0, st);
    }
    // First the relaxation over cross-device edges; it converges in a few
    // rounds unless the placement changes device along most long paths.
    const Scratch::Mark mk = sc.mark();
    bool launched = false;
    if (t_ms_relax > 0)
      CEL_TRY(ms_relax(g, d, L, order, node_dev, dev0, start, finish, makespan,
                       t_ms_relax > 1 ? t_ms_relax : 0, sc, s, st, &launched));
    if (launched) {
      Status h;
      CEL_TRY(read_status(st, &h, s));
      if (h.err) return status_error(h, fn);
      t_ms_info = {0, h.i2};
      if (h.i3) return CEL_OK;
      t_ms_info = {1, h.i2};
    } else {
      t_ms_info = {1, 0};
    }
    sc.release(mk);
    // Device-grouped order: inside each level, nodes sorted by (device,
    // position in `order`).  Every device keeps its FIFO order, so the
    // makespan is unchanged, and each device's chain in a level is one run.
    uint64_t *keys;
    uint32_t *sig;
    int32_t *gorder, *meta;
    int64_t *wx, *sx;
    CEL_TRY(sc.get(&keys, n));
    CEL_TRY(sc.get(&sig, n));
    CEL_TRY(sc.get(&gorder, n));
    CEL_TRY(sc.get(&meta, n));
    CEL_TRY(sc.get(&wx, (int64_t)n + 1));
    CEL_TRY(sc.get(&sx, n));
    k_dev_keys<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, dev0, keys, sig, st);
    CEL_TRY(segmented_sort(keys, sig, level_ptr, L, n, sc, s, st));
    k_grouped<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, sig, dev0, gorder, pos, devp, st);
    CEL_TRY(relabel_csr(n, g->m, gorder, pos, g->in_ptr, g->in_idx, pptr, pidx, sc, s, st));
    k_pos_costs<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, gorder, g->w, g->ob, d->bw, d->lat, wp,
                                                      cq, st);
    CEL_TRY(exclusive_scan_i64(wp, wx, n, sc, s));
    k_runs<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, level_ptr, level, gorder, devp, wx, sx, meta,
                                                 st);
    CEL_TRY(ms_ring(n, g->m, L, level_ptr, gorder, level, pptr, pidx, wp, cq, devp, sx, meta, finp,
                    makespan, sc, s, st));
    if (start || finish)
      k_makespan_out<<<grid_for(n, 256, 8192), 256, 0, s>>>(1, n, gorder, finp, wp, start, finish,
                                                            st);
  } else {
    t_ms_info = {2, 0};
    CEL_TRY(relabel_csr(n, g->m, order, pos, g->in_ptr, g->in_idx, pptr, pidx, sc, s, st));
    k_pos_costs<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, g->w, g->ob, d->bw, d->lat, wp,
                                                      cq, st);
    {
      KTimer kt(s, "k_dev_gather");
      if (K >= 64 && n <= 2 * kGRowNodes) {  // rows staged in at most two passes
        const bool vec = (n & 3) == 0 && ((uintptr_t)order & 15) == 0 &&
                         ((uintptr_t)node_dev & 3) == 0;
        if (vec) k_dev_rows<true><<<(unsigned)K, kGRowB, 0, s>>>(n, order, node_dev, d->D, devp, st);
        else k_dev_rows<false><<<(unsigned)K, kGRowB, 0, s>>>(n, order, node_dev, d->D, devp, st);
      } else {
        const int gy = K < 1024 ? K : 1024;
        k_dev_gather<<<dim3(gx, gy), 256, 0, s>>>(K, n, order, node_dev, d->D, devp, st);
      }
    }
    const bool wide = (int64_t)n >= (int64_t)kWideLevels * L;  // gathers from global memory
    int dbits = 0;  // bits of the largest device id
    while ((1 << dbits) < d->D) dbits++;
    if (wide && d->D <= kWDev && n <= kWMaxN) {
      CEL_TRY(mw_batch(K, n, L, d->D, level_ptr, pptr, pidx, wp, cq, devp, finp, makespan, sc, s,
                       st));
    } else if (wide) {
      KTimer kt(s, "k_makespan_batch");
      k_makespan_levels<512, 1, 3><<<(unsigned)K, 512, 0, s>>>(n, L, dbits, level_ptr, pptr, pidx,
                                                              wp, cq, devp, finp, makespan, st);
    } else if (K <= kBatchWide) {
      CEL_TRY(mb_ring(K, n, g->m, L, level_ptr, order, level, pptr, pidx, wp, cq, devp, finp,
                      finp + (int64_t)K * n, makespan, sc, s, st));
    } else {
      // more placements than CUs: small windows (about 35 KB of LDS) so that
      // several placements share a CU and hide each other's memory latency
      KTimer kt(s, "k_makespan_batch");
      k_makespan_sweep<256, 256, 1024><<<(unsigned)K, 256, 0, s>>>(n, L, dbits, level_ptr, pptr,
                                                                   pidx, wp, cq, devp, finp,
                                                                   makespan, st);
    }
    if (start || finish)
      k_makespan_out<<<grid_for((int64_t)K * n, 256, 8192), 256, 0, s>>>(K, n, order, finp, wp,
                                                                        start, finish, st);
  }
  CEL_HIP(hipGetLastError());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  return CEL_OK;
}

extern "C" int cel_makespan(const cel_graph *g, const cel_devices *d, const int32_t *order,
                            const int32_t *level, const int32_t *level_ptr, int32_t L, int32_t K,
                            const uint8_t *node_dev, int64_t *start, int64_t *finish,
                            int64_t *makespan, hipStream_t s) {
  const char *fn = "cel_makespan";
  CEL_TRY(check_makespan_args(fn, g, d, order, level, level_ptr, L, K, node_dev, makespan));
  Scratch sc(s);
  return makespan_impl(fn, g, d, order, level, level_ptr, L, K, node_dev, start, finish, makespan,
                       sc, s);
}

// ----------------------------------------------- the allocation-free variant
//
// Its scratch is one fixed device array per GPU, a module-scope __device__
// variable: the runtime creates it when it loads the library's code object on
// a device and keeps it until the process ends.  Host code may not use the
// array's name as a device address; the address comes from
// hipGetSymbolAddress, taken once per device with that device current.
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace {
std::mutex g_fixed_mu;               // one call at a time per process (the array is shared)
std::map<int, char *> g_fixed_ptr;   // device ordinal -> address of that device's array
}  // namespace

static int fixed_scratch(char **out) {  // g_fixed_mu held
  int dev = 0;
  CEL_HIP(hipGetDevice(&dev));
  auto it = g_fixed_ptr.find(dev);
  if (it == g_fixed_ptr.end()) {
    void *p = nullptr;
    CEL_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return set_error(CEL_E_HIP, "hipGetSymbolAddress returned NULL for the fixed scratch");
    it = g_fixed_ptr.emplace(dev, (char *)p).first;
  }
  *out = it->second;
  return CEL_OK;
}

// A bound on the scratch one call takes: per node at most 200 bytes (position
// maps, relabelled CSR rows, costs, the device-grouped order and its sort
// buffers, per-level tile lists, and for K = 1 the ring sweep's pull records,
// list offsets, level and segment tables and the second finish array), 16
// bytes per edge (relabelled in-edges; for K = 1 tagged, far and long lists),
// 21 bytes per node and placement (devices, finish times, finish + c, level
// information), and 64 KiB for block partials and 256-byte rounding.
static uint64_t makespan_scratch_bound(int64_t n, int64_t m, int64_t K) {
  return 65536ull + 200ull * (uint64_t)(n + 1) + 16ull * (uint64_t)m + 21ull * (uint64_t)K * (uint64_t)n;
}

extern "C" int cel_makespan_noalloc(const cel_graph *g, const cel_devices *d, const int32_t *order,
                                    const int32_t *level, const int32_t *level_ptr, int32_t L,
                                    int32_t K, const uint8_t *node_dev, int64_t *start,
                                    int64_t *finish, int64_t *makespan, hipStream_t s) {
  const char *fn = "cel_makespan_noalloc";
  CEL_TRY(check_makespan_args(fn, g, d, order, level, level_ptr, L, K, node_dev, makespan));
  const uint64_t need = makespan_scratch_bound(g->n, g->m, K);
  if (need > kNoAllocScratchBytes)
    return set_error(CEL_E_ARG,
                     "%s: n = %d, m = %d, K = %d may need %llu bytes of scratch, above the fixed "
                     "%llu (use cel_makespan)",
                     fn, g->n, g->m, K, (unsigned long long)need,
                     (unsigned long long)kNoAllocScratchBytes);
  std::lock_guard<std::mutex> lk(g_fixed_mu);
  char *base = nullptr;
  CEL_TRY(fixed_scratch(&base));
  Scratch sc(s, base, kNoAllocScratchBytes);
  const int rc = makespan_impl(fn, g, d, order, level, level_ptr, L, K, node_dev, start, finish,
                               makespan, sc, s);
  // a failed call may leave kernels queued that use the array: drain them
  // before the next call may take it
  if (rc != CEL_OK) (void)hipStreamSynchronize(s);
  return rc;
}
