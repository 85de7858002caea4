// cel_blevel: b-level (eq. 3), t-level (eq. 2), critical path and the
// priority order (Section 5.1.3).
//
// Nodes are first relabelled into the positions of the level order, so each
// level is a contiguous range and per-node data is read coalesced.  The sweep
// over levels runs in one workgroup (a level is a dependent step; workgroup
// barriers cost tens of ns where a grid barrier costs microseconds).  Inside a
// level every node pulls the values of its successors (b-level, reverse
// sweep) or predecessors (t-level, forward sweep): no atomics, so the result
// is exact and independent of scheduling.
#include "cel_internal.h"

namespace cel {

constexpr int kSweepB = 1024;

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

// Windowed level sweep.
//
// REVERSE = true:  val[p] = wp[p] for a sink, else wcp[p] + max val[successor]   (eq. 3)
// REVERSE = false: val[p] = 0 for a source, else max (val[pred] + wcp[pred])       (eq. 2)
//
// Positions are processed in windows of at most kWinN consecutive positions
// (kWinE edges, kWinL levels), from the top for REVERSE, from the bottom
// otherwise.  Staging a window reads its rows and edge targets.  A neighbour
// outside the window already has its final value, which is folded into the
// node's partial maximum in LDS right away.  Neighbours inside the window are
// counted per node with an LDS atomic: the first kPullB of them form the
// node's pull list (window slots), the rest (rare) become packed overflow
// words (neighbour | owner << 16) that a per-level edge-parallel atomic max
// applies first.  A node's value is then a few independent LDS gathers and a
// max, unrolled to the largest pull count in its wave.  A level of at most
// kNarrowB nodes is run by wave 0 alone in rows of 64 with no workgroup
// barrier (a wave sees its own LDS writes in order); wider levels use the
// whole block.  A node with more than kWinE edges forms a window of its own,
// all of whose neighbours lie outside it.
constexpr int kWinN = 2048, kWinE = 8192, kWinL = 256, kPullB = 6, kNarrowB = 256;

// Gathered value of a window slot: s_x[j] = val(j) (REVERSE) or val(j) +
// wcp(j) (forward), what a neighbour's pull needs; -1 at the dummy slot.
//
// Pull maxima of NR rows of 64 slots at once (slot si[u] of row u; kWinN for
// idle lanes), K gathers per slot: every gather of the rows is issued before
// the first use (the compiler would otherwise chain the cases of the caller's
// switch into serial round trips).
template <int NR, int K, int K0 = 0>
__device__ inline void rows_pull(int64_t (&r)[NR], const int32_t (&si)[NR],
                                 const int16_t (*pw)[kWinN + 1], const int64_t *s_x) {
  int32_t j[NR][K];
#pragma unroll
  for (int u = 0; u < NR; u++)
#pragma unroll
    for (int k = 0; k < K; k++) j[u][k] = pw[K0 + k][si[u]];
  int64_t x[NR][K];
#pragma unroll
  for (int u = 0; u < NR; u++)
#pragma unroll
    for (int k = 0; k < K; k++) x[u][k] = s_x[j[u][k]];
  asm volatile("" ::: "memory");
#pragma unroll
  for (int u = 0; u < NR; u++)
#pragma unroll
    for (int k = 0; k < K; k++) r[u] = x[u][k] > r[u] ? x[u][k] : r[u];
}

// Values of the NR rows of slots starting at a (slots past b idle); the
// gathers are unrolled to the largest pull count among the rows' lanes.
// Returns the values; the caller stores them.
template <bool REVERSE, int NR>
__device__ inline void rows_val(int32_t a, int32_t b, int lane, const int16_t (*pw)[kWinN + 1],
                                const int32_t *s_pc, const int64_t *s_pm, const int64_t *s_x,
                                const int64_t *s_wc, int64_t (&v)[NR], int64_t (&wc)[NR]) {
  int32_t si[NR];
  int64_t r[NR];
  int32_t c = 0;
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int32_t s = a + lane + 64 * u;
    si[u] = s < b ? s : kWinN;
    const int32_t pc = s_pc[si[u]];
    r[u] = s_pm[si[u]];
    wc[u] = s_wc[si[u]];
    c = pc > c ? pc : c;
  }
  c = c < kPullB ? c : kPullB;
  int kmax = 0;
  while (kmax < kPullB && __ballot(c > kmax)) kmax++;
  // one batch holds at most 12 gathers per lane (registers); more take two
  constexpr int KB = 12 / NR < kPullB ? 12 / NR : kPullB;
  switch (kmax) {
    case 0: break;
    case 1: rows_pull<NR, 1>(r, si, pw, s_x); break;
    case 2: rows_pull<NR, 2>(r, si, pw, s_x); break;
    case 3: rows_pull<NR, (3 < KB ? 3 : KB)>(r, si, pw, s_x);
      if constexpr (KB < 3) rows_pull<NR, 3 - KB, KB>(r, si, pw, s_x);
      break;
    case 4: rows_pull<NR, (4 < KB ? 4 : KB)>(r, si, pw, s_x);
      if constexpr (KB < 4) rows_pull<NR, 4 - KB, KB>(r, si, pw, s_x);
      break;
    case 5: rows_pull<NR, (5 < KB ? 5 : KB)>(r, si, pw, s_x);
      if constexpr (KB < 5) rows_pull<NR, 5 - KB, KB>(r, si, pw, s_x);
      break;
    default: rows_pull<NR, (6 < KB ? 6 : KB)>(r, si, pw, s_x);
      if constexpr (KB < 6) rows_pull<NR, 6 - KB, KB>(r, si, pw, s_x);
      break;
  }
#pragma unroll
  for (int u = 0; u < NR; u++) v[u] = REVERSE ? wc[u] + r[u] : (r[u] > 0 ? r[u] : 0);
}

// Narrow level [a, b) of at most 4 rows, run by one wave: values, then the
// window copy (the pull value) and the global output
template <bool REVERSE, int NR>
__device__ inline void narrow_level(int32_t a, int32_t b, int lane, const int16_t (*pw)[kWinN + 1],
                                    const int32_t *s_pc, const int64_t *s_pm, int64_t *s_x,
                                    const int64_t *s_wc, int64_t *valP0) {
  int64_t v[NR], wc[NR];
  rows_val<REVERSE, NR>(a, b, lane, pw, s_pc, s_pm, s_x, s_wc, v, wc);
#pragma unroll
  for (int u = 0; u < NR; u++) {
    const int32_t s = a + lane + 64 * u;
    if (s < b) {
      s_x[s] = REVERSE ? v[u] : v[u] + wc[u];
      valP0[s] = v[u];
    }
  }
}

template <bool REVERSE>
__global__ void __launch_bounds__(kSweepB)
    k_level_sweep(int32_t n, int32_t L, const int32_t *lp, const int32_t *rptr,
                  const int32_t *ridx, const int64_t *wp, const int64_t *wcp, int64_t *val,
                  const Status *st) {
  constexpr int32_t kNoop = (kWinN << 16) | kWinN;  // overflow word that changes nothing
  __shared__ int32_t s_lv[kWinL + 2];  // level boundaries near the cursor
  __shared__ int32_t s_rp[kWinN + 1];  // rows of the candidate window (absolute edge offsets)
  __shared__ int16_t s_own[kWinE];     // owner slot of each edge (-1: past kOwnFill of its row)
  __shared__ int32_t s_epk[kWinE];     // overflow words (kNoop for the other edges)
  __shared__ int16_t s_pw[kPullB][kWinN + 1];  // pull lists
  __shared__ int32_t s_pc[kWinN + 1];  // in-window neighbours per slot
  __shared__ int64_t s_pm[kWinN + 1];  // partial max over neighbours, -1 if none yet
  __shared__ int64_t s_x[kWinN + 1];   // pull values of this window's slots (-1 at the dummy)
  __shared__ int64_t s_wc[kWinN + 1];  // wcp (w for a sink in REVERSE) of the window's nodes
  __shared__ int32_t s_la[kWinL], s_lb[kWinL], s_lea[kWinL], s_leb[kWinL], s_lend[kWinL];
  __shared__ int32_t s_lov[kWinL];
  __shared__ int32_t s_cut;
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const bool wave0 = tid < 64;
  if (tid == 0) {
    s_pc[kWinN] = 0;
    s_pm[kWinN] = -1;
    s_x[kWinN] = -1;
    s_wc[kWinN] = 0;
  }
  if (tid < kPullB) s_pw[tid][kWinN] = kWinN;
  int32_t edge_lo = REVERSE ? n : 0;   // boundary of the processed region
  int32_t lcur = REVERSE ? L - 1 : 0;  // level holding the next position to process
  while (REVERSE ? edge_lo > 0 : edge_lo < n) {
    CEL_TSTAMP(t0);
    CEL_TCOUNT(REVERSE ? 6 : 16 + 6);
    const int32_t Pc0 = REVERSE ? (edge_lo - kWinN > 0 ? edge_lo - kWinN : 0) : edge_lo;
    const int32_t Pc1 = REVERSE ? edge_lo : (edge_lo + kWinN < n ? edge_lo + kWinN : n);
    for (int t = tid; t <= Pc1 - Pc0; t += kSweepB) s_rp[t] = rptr[Pc0 + t];
    for (int t = tid; t < kWinE; t += kSweepB) s_own[t] = -1;
    for (int k = tid; k <= kWinL + 1; k += kSweepB) {
      // REVERSE: s_lv[k] = lp[lcur + 1 - k], so level lcur - k is [s_lv[k+1], s_lv[k]);
      // forward: s_lv[k] = lp[lcur + k], so level lcur + k is [s_lv[k], s_lv[k+1])
      const int32_t l = REVERSE ? lcur + 1 - k : lcur + k;
      s_lv[k] = lp[l < 0 ? 0 : (l > L ? L : l)];
    }
    if (tid == 0) s_cut = 0;
    __syncthreads();
    // window bounds: edge cap (counted from the boundary) and level cap
    int32_t cnt = 0;
    for (int t = tid; t < Pc1 - Pc0; t += kSweepB) {
      if (REVERSE) cnt += (s_rp[Pc1 - Pc0] - s_rp[t] > kWinE) ? 1 : 0;  // too far below P1
      else cnt += (s_rp[t + 1] - s_rp[0] <= kWinE) ? 1 : 0;            // fits above P0
    }
    for (int off = 32; off > 0; off >>= 1) cnt += __shfl_xor(cnt, off);
    if ((tid & 63) == 0 && cnt) atomicAdd(&s_cut, cnt);
    __syncthreads();
    int32_t P0, P1;
    if (REVERSE) {
      P1 = Pc1;
      P0 = Pc0 + s_cut;
      const int32_t lvcap = (lcur - kWinL + 1 > 0) ? s_lv[kWinL] : 0;  // start of level lcur-kWinL+1
      if (P0 < lvcap) P0 = lvcap;
    } else {
      P0 = Pc0;
      P1 = Pc0 + s_cut;
      const int32_t lvcap = (lcur + kWinL < L) ? s_lv[kWinL] : n;  // end of level lcur+kWinL-1
      if (P1 > lvcap) P1 = lvcap;
    }
    const bool heavy = (P0 == P1);  // one node with more than kWinE edges
    if (heavy) {
      if (REVERSE) P0 = P1 - 1;
      else P1 = P0 + 1;
    }
    const int32_t NN = P1 - P0;
    const int32_t R0 = P0 - Pc0;  // row of P0 in s_rp
    const int32_t E0 = s_rp[R0], E1 = s_rp[R0 + NN];
    CEL_TSTAMP(t1);
    CEL_TADD(REVERSE ? 0 : 16 + 0, t0, t1);
    // stage nodes: costs, partials (0 for a REVERSE sink: its value is w),
    // pull counters and lists
    for (int32_t i = tid; i < NN; i += kSweepB) {
      const bool sink = s_rp[R0 + i] == s_rp[R0 + i + 1];
      s_pm[i] = (REVERSE && sink) ? 0 : -1;
      s_wc[i] = (REVERSE && sink) ? wp[P0 + i] : wcp[P0 + i];
      s_pc[i] = 0;
#pragma unroll
      for (int k = 0; k < kPullB; k++) s_pw[k][i] = kWinN;  // rows gather past a short list
      if (!heavy) {  // owners of the row's first kOwnFill edges
        const int32_t k0 = s_rp[R0 + i] - E0, k1 = s_rp[R0 + i + 1] - E0;
        const int32_t kc = k1 - k0 < kOwnFill ? k1 : k0 + kOwnFill;
        for (int32_t q = k0; q < kc; q++) s_own[q] = (int16_t)i;
      }
    }
    // per-level ranges of the window: nodes [a, b), edges [ea, eb) (window-relative)
    for (int32_t k = tid; k < kWinL; k += kSweepB) {
      const int32_t lb = REVERSE ? s_lv[k + 1] : s_lv[k];
      const int32_t le = REVERSE ? s_lv[k] : s_lv[k + 1];
      // clamp to the window: levels outside it become empty ranges at its edge
      int32_t a = lb < P0 ? P0 : (lb > P1 ? P1 : lb);
      const int32_t b = le < P0 ? P0 : (le > P1 ? P1 : le);
      if (a > b) a = b;
      s_la[k] = a - P0;
      s_lb[k] = b - P0;
      s_lea[k] = heavy ? 0 : s_rp[a - Pc0] - E0;
      s_leb[k] = heavy ? 0 : s_rp[b - Pc0] - E0;
      s_lend[k] = REVERSE ? (lb <= P0) : (le >= P1);
      s_lov[k] = 0;
    }
    __syncthreads();
    CEL_TSTAMP(t2);
    CEL_TADD(REVERSE ? 1 : 16 + 1, t1, t2);
    // stage edges: neighbours outside the window are final (each thread takes
    // EU edges per pass: all index loads, then all value gathers, in flight
    // together)
    if (heavy) {  // a single node with more than kWinE edges, all outside the window
      const int64_t mx = heavy_max<kHeavyU, kSweepB>(
          E0, E1, tid, [&](int32_t e) { return ridx[e]; },
          [&](int32_t r) { return REVERSE ? val[r] : val[r] + wcp[r]; });
      if ((tid & 63) == 0 && mx >= 0) atomicMax((long long *)&s_pm[0], (long long)mx);
    }
    constexpr int EU = (kWinE + kSweepB - 1) / kSweepB;
    for (int32_t e0 = E0 + tid; !heavy && e0 < E1; e0 += EU * kSweepB) {
      int32_t rr[EU];
#pragma unroll
      for (int u = 0; u < EU; u++) {
        const int32_t e = e0 + u * kSweepB;
        rr[u] = e < E1 ? ridx[e] : P0;
      }
      int64_t xv[EU];
#pragma unroll
      for (int u = 0; u < EU; u++) {  // unconditional: in-window neighbours read a final slot
        const bool in = REVERSE ? (rr[u] < P1) : (rr[u] >= P0);
        const int32_t rs = in ? 0 : rr[u];
        xv[u] = REVERSE ? val[rs] : val[rs] + wcp[rs];
      }
#pragma unroll
      for (int u = 0; u < EU; u++) {
        const int32_t e = e0 + u * kSweepB;
        if (e >= E1) break;
        const int32_t r = rr[u];
        const int32_t own = heavy ? 0 : owner_of(&s_rp[R0], NN, s_own[e - E0], e);
        const bool in = REVERSE ? (r < P1) : (r >= P0);
        int32_t word = kNoop;
        if (in) {
          const int32_t j = r - P0;
          const int32_t kk = atomicAdd(&s_pc[own], 1);
          if (kk < kPullB) {
            s_pw[kk][own] = (int16_t)j;
          } else {
            word = j | (own << 16);
            // the owner's level: REVERSE levels run down the table, forward up
            int32_t lo = 0, hi = kWinL - 1;
            while (lo < hi) {
              if (REVERSE) {
                const int32_t mid = (lo + hi) >> 1;
                if (s_la[mid] <= own) hi = mid;
                else lo = mid + 1;
              } else {
                const int32_t mid = (lo + hi + 1) >> 1;
                if (s_la[mid] <= own) lo = mid;
                else hi = mid - 1;
              }
            }
            s_lov[lo] = 1;
          }
        } else {
          atomicMax((long long *)&s_pm[own], (long long)xv[u]);
        }
        if (!heavy) s_epk[e - E0] = word;
      }
    }
    __syncthreads();
    CEL_TSTAMP(t3);
    CEL_TADD(REVERSE ? 2 : 16 + 2, t2, t3);
    // level metadata in registers: lane l holds levels l, l+64, l+128, l+192
    int32_t ma[4], mb[4], mea[4], meb[4], mend[4];
#pragma unroll
    for (int u = 0; u < 4; u++) {
      const int k = (tid & 63) + 64 * u;
      ma[u] = s_la[k];
      mb[u] = s_lb[k];
      mea[u] = s_lea[k];
      meb[u] = s_leb[k];
      mend[u] = s_lend[k] | (s_lov[k] << 1);
    }
    uint64_t vis[4];  // levels the whole block visits: wide ones and the window's end
#pragma unroll
    for (int u = 0; u < 4; u++)
      vis[u] = __ballot((mb[u] - ma[u] > kNarrowB) || (mend[u] & 1));
    for (int32_t k = wave0 ? 0 : next_marked(vis, 0); k < kWinL;
         k = wave0 ? k + 1 : next_marked(vis, k + 1)) {
      const int u = k >> 6, ln = k & 63;
      int32_t a, b, ea, eb, fl;
      switch (u) {  // uniform: pick the register set, then read lane ln
        case 0: a = ma[0]; b = mb[0]; ea = mea[0]; eb = meb[0]; fl = mend[0]; break;
        case 1: a = ma[1]; b = mb[1]; ea = mea[1]; eb = meb[1]; fl = mend[1]; break;
        case 2: a = ma[2]; b = mb[2]; ea = mea[2]; eb = meb[2]; fl = mend[2]; break;
        default: a = ma[3]; b = mb[3]; ea = mea[3]; eb = meb[3]; fl = mend[3]; break;
      }
      a = __builtin_amdgcn_readlane(a, ln);
      b = __builtin_amdgcn_readlane(b, ln);
      ea = __builtin_amdgcn_readlane(ea, ln);
      eb = __builtin_amdgcn_readlane(eb, ln);
      fl = __builtin_amdgcn_readlane(fl, ln);
      if (a < b) {
        CEL_TSTAMP(tl0);
        if (b - a <= kNarrowB) {
          CEL_TCOUNT(REVERSE ? 4 : 16 + 4);
          if (wave0) {
            if (fl & 2) {  // in-window neighbours past the pull lists
              for (int32_t e = ea + lane; e < eb; e += 64) {
                const int32_t wd = s_epk[e];
                atomicMax((long long *)&s_pm[wd >> 16], (long long)s_x[wd & 0xFFFF]);
              }
              lds_order();
            }
            // all rows of the level at once: their gathers share round trips
            switch ((b - a + 63) >> 6) {
              case 1: narrow_level<REVERSE, 1>(a, b, lane, s_pw, s_pc, s_pm, s_x, s_wc, val + P0); break;
              case 2: narrow_level<REVERSE, 2>(a, b, lane, s_pw, s_pc, s_pm, s_x, s_wc, val + P0); break;
              case 3: narrow_level<REVERSE, 3>(a, b, lane, s_pw, s_pc, s_pm, s_x, s_wc, val + P0); break;
              default: narrow_level<REVERSE, 4>(a, b, lane, s_pw, s_pc, s_pm, s_x, s_wc, val + P0); break;
            }
            lds_order();
          }
          CEL_TSTAMP(tl1);
          CEL_TADD(REVERSE ? 7 : 16 + 7, tl0, tl1);
        } else {
          CEL_TCOUNT(REVERSE ? 5 : 16 + 5);
          __syncthreads();  // wave 0's narrow levels before this one
          if (fl & 2) {
            for (int32_t e = ea + tid; e < eb; e += kSweepB) {
              const int32_t wd = s_epk[e];
              atomicMax((long long *)&s_pm[wd >> 16], (long long)s_x[wd & 0xFFFF]);
            }
            __syncthreads();
          }
          for (int32_t i0 = a + (tid & ~63); i0 < b; i0 += kSweepB) {  // a row per wave
            int64_t v[1], wc[1];
            rows_val<REVERSE, 1>(i0, b, lane, s_pw, s_pc, s_pm, s_x, s_wc, v, wc);
            const int32_t i = i0 + lane;
            if (i < b) {
              s_x[i] = REVERSE ? v[0] : v[0] + wc[0];
              val[P0 + i] = v[0];
            }
          }
          __syncthreads();
          CEL_TSTAMP(tl1);
          CEL_TADD(REVERSE ? 8 : 16 + 8, tl0, tl1);
        }
      }
      if (fl & 1) break;  // the window ends inside this level
    }
    CEL_TSTAMP(t4);
    CEL_TADD(REVERSE ? 3 : 16 + 3, t3, t4);
    // advance the cursor to the level holding the next unprocessed position
    // (s_lv still covers every level the window touched)
    if (REVERSE) {
      edge_lo = P0;
      if (P0 > 0) {
        int32_t k = 1;  // smallest k >= 1 with start(lcur + 1 - k) <= P0 - 1
        while (k <= kWinL + 1 && s_lv[k] > P0 - 1) k++;
        if (k <= kWinL + 1) {
          lcur = lcur + 1 - k;
        } else {  // only past a run of empty levels
          int32_t l = lcur - kWinL - 1;
          while (l > 0 && lp[l] > P0 - 1) l--;
          lcur = l;
        }
      }
    } else {
      edge_lo = P1;
      if (P1 < n) {
        int32_t k = 0;  // largest k with start(lcur + k) <= P1
        while (k < kWinL && lcur + k + 1 < L && s_lv[k + 1] <= P1) k++;
        lcur = lcur + k;
      }
    }
    __syncthreads();
  }
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
  // The t-level (eq. 2) needs no b-level: its relabelling and sweep run on a
  // side stream, so the two single-workgroup sweeps overlap on two CUs.
  SideFork fk;
  if (tlevel && n > 0) {
    int32_t *pptr, *pidx;
    int64_t *tlp;
    CEL_TRY(sc.get(&pptr, (int64_t)n + 1));
    CEL_TRY(sc.get(&pidx, g->m));
    CEL_TRY(sc.get(&tlp, n));
    CEL_TRY(fk.start(s));
    const hipStream_t t = fk.side();
    CEL_TRY(relabel_csr(n, g->m, order_id, pos, g->in_ptr, g->in_idx, pptr, pidx, sc, t, st));
    {
      KTimer kt(t, "k_tlevel_sweep");
      k_level_sweep<false><<<1, kSweepB, 0, t>>>(n, L, level_ptr, pptr, pidx, wp, wcp, tlp, st);
    }
    k_scatter_max<<<grid_for(n, 256, 2048), 256, 0, t>>>(n, order_id, tlp, tlevel, st, &st->s1);
  }
  {
    KTimer kt(s, "k_blevel_sweep");
    k_level_sweep<true><<<1, kSweepB, 0, s>>>(n, L, level_ptr, sptr, sidx, wp, wcp, blp, st);
  }
  k_scatter_max<<<grid_for(n, 256, 2048), 256, 0, s>>>(n, order_id, blp, blevel, st, &st->s0);
  if (prio_order && n > 0) {
    uint64_t *keys;
    CEL_TRY(sc.get(&keys, n));
    uint32_t *ids = reinterpret_cast<uint32_t *>(prio_order);
    k_prio_keys<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order_id, blp, keys, ids, st);
    CEL_TRY(segmented_sort(keys, ids, level_ptr, L, n, sc, s, st));
  }
  CEL_HIP(hipGetLastError());
  CEL_TRY(fk.join());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  *cp = h.s0;
  return CEL_OK;
}
