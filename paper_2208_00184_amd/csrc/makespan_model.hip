// cel_makespan_model: makespan of K placements under richer device models.
// INSERT applies the slot rule of eq. 7 (Section 5.2) to single nodes: a node
// starts in the first idle slot of its device, at or after its ready time,
// that holds it.  COMM_TASKS makes every transfer a task (the runtime model of
// Section 6.1): one transfer of a producer's output to each other device that
// holds one of its successors, in increasing device order, occupying the
// producer device's send channel and the target device's receive channel.
//
// Under either model a node's start depends on everything placed before it on
// its device, so a placement is a walk in order.  One wave walks one
// placement, 64 consecutive positions (a window) at a time:
//  A. lane j folds slot j's inputs from before the window (finish times, or
//     arrivals of transfers: final by now) into a partial ready time and
//     marks its in-window predecessors in a 64-bit mask.  Its own w, c,
//     device, row and first four inputs (a per-position table) were loaded
//     during the previous window.  Rows with many inputs are folded by the
//     whole wave.
//  B. the window splits into segments, runs of consecutive slots with no
//     edge among them, taken in order.  A segment's slots add their inputs
//     from earlier segments (shuffles), then are placed: with FIFO devices
//     by one segmented max-plus scan over the slots sorted by (device,
//     position); with insertion by lane d for device d's slots, in order.
//     Device d's state (free time or end of its last task, gap count and
//     ring head, channel free times) lives in lane d.  The segment's
//     transfers are then issued in slot order.
//  C. the window's finish times are stored.
//
// Idle gaps: device d keeps the idle intervals before its last task, sorted,
// in its segment of a per-placement global array (a task adds at most one gap,
// so the segment holds as many entries as d has nodes), and its newest 64
// again in an LDS ring (written through to the array).  A node ready at or
// after the last gap's end goes after the device's last task with no search.
// Otherwise lane d binary-searches its device's ring for the first gap that
// holds the node and shrinks or empties it.  A split (which moves the ring),
// or a ring whose oldest gap already ends after the ready time (an older gap
// may hold the node), goes to the whole wave: the ring one gap per lane with
// a ballot, after walking the global segment, 64 gaps per round trip.
// Transfers: a producer's destination devices form a mask; its arrivals sit
// in a pool at off[p] + (rank of the device in the mask).
// Heterogeneous devices (HET): device d runs a node of w in ceil(w tmul[d] /
// 1024), computed as (w >> 10) tmul + ceil((w & 1023) tmul / 1024) so that
// no product leaves 64 bits; a transfer from a to b takes ceil(ob / bw[a][b])
// + lat[a][b], the link tables staged in LDS.
//
// cel_colocate (co-location groups, Section 6.1): the first member of each
// group in the order (smallest position, by atomicMin) leads, and every
// member takes its device.
#include "cel_internal.h"

namespace cel {

constexpr int kMmLight = 16;  // rows with more inputs are folded by the whole wave

struct MmArgs {
  int32_t n, D;
  const int32_t *iptr, *iidx;  // predecessors in position space
  const int64_t *wp, *cq;      // w, c by position
  const uint8_t *devp;         // [K][n] device by position
  const uint64_t *dmask;       // [K][n] destination devices by position (transfers)
  const int64_t *aoff;         // [K][n] arrival pool offsets (transfers)
  int64_t *pool;               // arrivals (transfers)
  const int64_t *goff;         // [K][D] start of each device's gap segment (insertion)
  int64_t *ga, *gb;            // gap starts and ends (insertion)
  int64_t *finp;               // [K][n] finish by position
  int64_t *makespan;           // [K]
  const int64_t *obp;          // ob by position (HET)
  const int64_t *tmul;         // [D] time multipliers, 1/1024 (HET)
  const int64_t *lbw, *llat;   // [D][D] links (HET)
  const int4 *ipre;            // first 4 inputs of each position (-1 past the row's end)
};

constexpr int kHetD = 64;  // link table stride

// ceil(w * tm / 1024) for w >= 0, 1 <= tm <= 65536, without a 128-bit product
__device__ inline int64_t dur_on(int64_t w, int64_t tm) {
  return (w >> 10) * tm + (((w & 1023) * tm + 1023) >> 10);
}

__device__ inline int64_t link_c(int64_t ob, int32_t bw, int32_t lat) {
  return ob / bw + (ob % bw != 0 ? 1 : 0) + lat;
}

// Lane l of a register replaced by v (uniform l and v): a lane compare and a
// select, no memory.
template <class T>
__device__ inline T setlane(T old, T v, int l) {
  return (int)threadIdx.x == l ? v : old;
}

__device__ inline uint64_t below(int b) { return (uint64_t(1) << b) - 1; }

// Ready-time contribution of the inputs iidx[e] for e = e0, e0 + step, ...
// < e1 of a node on device dv: inputs before the window (position < P0) are
// folded into ext, the others marked in msk (bit = position - P0).  An input
// on another device contributes f + c (contention-free) or, with transfers,
// the arrival of its output on dv: pool[off + rank of dv in its mask].
template <bool TASKS, bool HET>
__device__ inline void fold_batch(const MmArgs &a, const uint8_t *dev, const int64_t *fin,
                                  const uint64_t *dm, const int64_t *of, const int32_t *s_bw,
                                  const int32_t *s_lat, int32_t P0, const int32_t (&q)[4],
                                  int32_t dv, int64_t &ext, uint64_t &msk, uint32_t &bad) {
  int64_t f[4], x[4];
  int32_t dq[4];
#pragma unroll
  for (int u = 0; u < 4; u++) {  // first round: all loads that need only q
    dq[u] = dv;
    f[u] = x[u] = 0;
    if (q[u] >= 0 && q[u] < P0) {
      dq[u] = dev[q[u]];
      f[u] = fin[q[u]];
      if (TASKS) {  // -1: dv missing from the mask (CSR and CSC disagree)
        const uint64_t mq = dm[q[u]];
        x[u] = (mq >> dv) & 1 ? of[q[u]] + __builtin_popcountll(mq & below(dv)) : -1;
      } else {
        x[u] = HET ? a.obp[q[u]] : a.cq[q[u]];
      }
    }
  }
#pragma unroll
  for (int u = 0; u < 4; u++) {  // second round: arrivals of transfers
    if (q[u] < 0) continue;
    if (q[u] >= P0) {
      msk |= uint64_t(1) << (q[u] - P0);
      continue;
    }
    int64_t t;
    if (dq[u] == dv) {
      t = f[u];
    } else if (TASKS) {
      if (x[u] < 0) {
        bad |= EB_ARG;
        continue;
      }
      t = a.pool[x[u]];
    } else if (HET) {
      t = f[u] + link_c(x[u], s_bw[dq[u] * kHetD + dv], s_lat[dq[u] * kHetD + dv]);
    } else {
      t = f[u] + x[u];
    }
    ext = t > ext ? t : ext;
  }
}

// Ready-time contribution of the inputs iidx[e] for e = e0, e0 + step, ...
// < e1 of a node on device dv: inputs before the window (position < P0) are
// folded into ext, the others marked in msk (bit = position - P0).  An input
// on another device contributes f + c (contention-free) or, with transfers,
// the arrival of its output on dv: pool[off + rank of dv in its mask].
template <bool TASKS, bool HET>
__device__ inline void fold_inputs(const MmArgs &a, const uint8_t *dev, const int64_t *fin,
                                   const uint64_t *dm, const int64_t *of, const int32_t *s_bw,
                                   const int32_t *s_lat, int32_t P0, int32_t e0, int32_t e1,
                                   int32_t step, int32_t dv, int64_t &ext, uint64_t &msk,
                                   uint32_t &bad) {
  for (int32_t e = e0; e < e1; e += 4 * step) {
    int32_t q[4];
#pragma unroll
    for (int u = 0; u < 4; u++) q[u] = e + u * step < e1 ? a.iidx[e + u * step] : -1;
    fold_batch<TASKS, HET>(a, dev, fin, dm, of, s_bw, s_lat, P0, q, dv, ext, msk, bad);
  }
}

constexpr int kTail = 64;  // most recent idle gaps of each device kept in LDS

// Device d's idle gaps: the full sorted list in global memory (A / B [0, G),
// written through), and its newest t = min(G, kTail) entries again in an LDS
// ring (ta / tb), logical tail index i at slot (h + i) mod kTail.

// Appends the idle gap [a, b) after the G gaps.
__device__ inline void gap_append(int64_t *A, int64_t *B, int64_t *ta, int64_t *tb, int32_t G,
                                  int32_t &h, int64_t a, int64_t b, int lane) {
  const int32_t slot = G < kTail ? G : h;  // a full ring overwrites its oldest gap
  if (lane == 0) {
    A[G] = a;
    B[G] = b;
    ta[slot] = a;
    tb[slot] = b;
  }
  if (G >= kTail) h = (h + 1) & (kTail - 1);
  lds_order();
}

// First-fit slot of a node (w > 0, ready r); L, G, gl, h are the device's
// last end, gap count, last gap end and ring head (uniform), updated in
// place.  Returns the start.
__device__ inline int64_t insert_slot(int64_t *A, int64_t *B, int64_t *ta, int64_t *tb, int64_t r,
                                      int64_t w, int64_t &L, int32_t &G, int64_t &gl, int32_t &h,
                                      int lane) {
  if (G == 0 || r >= gl) {  // no idle gap ends after r: go after the last task
    const int64_t s = r > L ? r : L;
    if (s > L) {
      gap_append(A, B, ta, tb, G, h, L, s, lane);
      G++;
      gl = s;
    }
    L = s + w;
    return s;
  }
  const int32_t t = G < kTail ? G : kTail, g0 = G - t;
  int64_t ca = 0, cb = 0;  // the tail in logical order, one gap per lane
  if (lane < t) {
    const int slot = (h + lane) & (kTail - 1);
    ca = ta[slot];
    cb = tb[slot];
  }
  int32_t q = -1;
  int64_t qa = 0, qb = 0;
  bool glob = false;
  if (g0 > 0 && readlane64(cb, 0) > r) {
    // the tail's oldest gap ends after r: an older one may hold the node.
    // Gaps stored by earlier steps must be visible here.
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    CEL_TCOUNT(5);
    int32_t lo = g0 > 64 ? g0 - 64 : 0;
    int64_t ga_ = 0, gb_ = 0;
    for (;;) {  // walk back to the chunk holding the first gap that ends after r
      const int32_t i = lo + lane;
      ga_ = gb_ = 0;
      if (i < g0) {
        ga_ = A[i];
        gb_ = B[i];
      }
      if (lo == 0 || !(__builtin_amdgcn_readfirstlane((int32_t)(gb_ > r)))) break;
      lo = lo > 64 ? lo - 64 : 0;
      CEL_TCOUNT(6);
    }
    for (;;) {  // scan forward, over the gaps older than the tail, for one that holds it
      const int32_t i = lo + lane;
      const int64_t x = ga_ > r ? ga_ : r;
      const uint64_t fit = __ballot(i < g0 && gb_ > r && x + w <= gb_);
      if (fit) {
        const int l = __builtin_ctzll(fit);
        q = lo + l;
        qa = readlane64(ga_, l);
        qb = readlane64(gb_, l);
        glob = true;
        break;
      }
      lo += 64;
      if (lo >= g0) break;
      CEL_TCOUNT(7);
      ga_ = gb_ = 0;
      if (lo + lane < g0) {
        ga_ = A[lo + lane];
        gb_ = B[lo + lane];
      }
    }
  }
  if (q < 0) {  // the tail
    const int64_t x = ca > r ? ca : r;
    const uint64_t fit = __ballot(lane < t && cb > r && x + w <= cb);
    if (fit) {
      q = __builtin_ctzll(fit);
      qa = readlane64(ca, q);
      qb = readlane64(cb, q);
    }
  }
  if (q < 0) {  // none holds it: after the last task (r < gl <= L)
    CEL_TCOUNT(10);
    const int64_t s = L;
    L = s + w;
    return s;
  }
  const int64_t s = qa > r ? qa : r, e = s + w;
  const bool left = s > qa, right = e < qb;
  if (glob) {  // a gap older than the tail (global only)
    if (left && right) {  // split: move gaps q+1 .. G-1 up by one, top chunk first
      for (int32_t hi = G; hi > q + 1;) {
        const int32_t l0 = hi - 64 > q + 1 ? hi - 64 : q + 1;
        const int32_t i = l0 + lane;
        int64_t xa = 0, xb = 0;
        if (i < hi) {
          xa = A[i];
          xb = B[i];
        }
        if (i < hi) {
          A[i + 1] = xa;
          B[i + 1] = xb;
        }
        hi = l0;
        CEL_TCOUNT(9);
      }
      if (lane == 0) {
        B[q] = s;
        A[q + 1] = e;
        B[q + 1] = qb;
      }
      G++;  // the newest t gaps, and so the ring, are unchanged
      CEL_TCOUNT(8);
    } else if (left) {
      if (lane == 0) B[q] = s;
    } else if (right) {
      if (lane == 0) A[q] = e;
    } else {  // filled exactly: leave an empty gap [qb, qb)
      if (lane == 0) A[q] = qb;
    }
    return s;
  }
  if (left && right) {  // split inside the tail: t + 1 gaps, the oldest leaves a full ring
    const int drop = t == kTail ? 1 : 0;
    const int k = lane + drop;  // lane i takes gap k of the new sequence (global g0 + k)
    const int src = k < q ? k : k - 1;
    const int64_t xa = __shfl(ca, src < 0 ? 0 : src), xb = __shfl(cb, src < 0 ? 0 : src);
    int64_t na = xa, nb = xb;
    if (k == q) {
      na = qa;
      nb = s;
    } else if (k == q + 1) {
      na = e;
      nb = qb;
    }
    const int32_t h2 = (h + drop) & (kTail - 1);
    if (lane < t + 1 - drop) {
      const int slot = (h2 + lane) & (kTail - 1);
      ta[slot] = na;
      tb[slot] = nb;
      if (k >= q) {  // write the changed part through
        A[g0 + k] = na;
        B[g0 + k] = nb;
      }
    }
    if (drop && q == 0 && lane == 0) {  // the dropped gap is the split's first part
      A[g0] = qa;
      B[g0] = s;
    }
    lds_order();
    h = h2;
    G++;
    CEL_TCOUNT(8);
  } else {
    const int slot = (h + q) & (kTail - 1);
    if (left) {  // the node ends the gap
      if (lane == 0) {
        tb[slot] = s;
        B[g0 + q] = s;
      }
      if (q == t - 1) gl = s;
    } else if (right) {  // the node starts the gap
      if (lane == 0) {
        ta[slot] = e;
        A[g0 + q] = e;
      }
    } else {  // filled exactly: leave an empty gap [qb, qb)
      if (lane == 0) {
        ta[slot] = qb;
        A[g0 + q] = qb;
      }
    }
    lds_order();
  }
  return s;
}

// First fit run by the lane that holds the device (its own state, its own
// gap segment and ring).  Returns false, leaving everything unchanged, when
// the whole wave must place the node: a split, which moves the ring, or a
// ring whose oldest gap already ends after r, so that an older gap may hold it.
__device__ inline bool lane_insert(int64_t *A, int64_t *B, int64_t *ta, int64_t *tb, int64_t r,
                                   int64_t w, int64_t &L, int32_t &G, int64_t &gl, int32_t &h,
                                   int64_t &s) {
  if (w == 0) {
    s = r;
    return true;
  }
  if (G == 0 || r >= gl) {  // after the last task, maybe leaving a new gap
    s = r > L ? r : L;
    if (s > L) {
      const int32_t slot = G < kTail ? G : h;
      A[G] = L;
      B[G] = s;
      ta[slot] = L;
      tb[slot] = s;
      if (G >= kTail) h = (h + 1) & (kTail - 1);
      G++;
      gl = s;
    }
    L = s + w;
    return true;
  }
  const int32_t t = G < kTail ? G : kTail, g0 = G - t;
  if (g0 > 0 && tb[h] > r) return false;
  int32_t lo = 0, hi = t - 1;  // first gap of the ring that ends after r (the last one does)
  while (lo < hi) {
    const int32_t mid = (lo + hi) >> 1;
    if (tb[(h + mid) & (kTail - 1)] > r) hi = mid;
    else lo = mid + 1;
  }
  for (int32_t i = lo; i < t; i++) {
    const int sl = (h + i) & (kTail - 1);
    const int64_t ga = ta[sl], gb = tb[sl], x = ga > r ? ga : r, e = x + w;
    if (e > gb) continue;
    const bool left = x > ga, right = e < gb;
    if (left && right) return false;
    if (left) {  // the node ends the gap
      tb[sl] = x;
      B[g0 + i] = x;
      if (i == t - 1) gl = x;
    } else if (right) {  // the node starts the gap
      ta[sl] = e;
      A[g0 + i] = e;
    } else {  // filled exactly: an empty gap [gb, gb)
      ta[sl] = gb;
      A[g0 + i] = gb;
    }
    s = x;
    return true;
  }
  s = L;  // none holds it: after the last task
  L = s + w;
  return true;
}

template <bool INS, bool TASKS, bool HET, bool BLOCK = false>
__global__ void __launch_bounds__(64) k_makespan_model(MmArgs a, Status *st) {
  // transfers whose arrivals the inputs read: on channels (TASKS) or on the
  // devices' compute queues (BLOCK)
  constexpr bool ARR = TASKS || BLOCK;
  static_assert(!(BLOCK && (INS || TASKS)), "the blocking model combines with no other bit");
  __shared__ int64_t s_T[ARR ? 64 * 64 : 1];  // arrival of slot j's output on device b
  __shared__ int32_t s_bw[HET ? kHetD * kHetD : 1], s_lat[HET ? kHetD * kHetD : 1];
  __shared__ int64_t s_ta[INS ? 64 * kTail : 1], s_tb[INS ? 64 * kTail : 1];  // gap tails
  __shared__ unsigned long long s_lst[64];  // slots of the segment by device
  __shared__ int64_t s_fin[64];             // finish of the segment's slots
  if (failed(st)) return;
  const int lane = threadIdx.x;
  s_lst[lane] = 0;
  int64_t tmr = 1024;  // device `lane`'s time multiplier
  if (HET) {
    for (int i = lane; i < a.D * a.D; i += 64) {
      const int x = i / a.D, y = i - x * a.D;
      s_bw[x * kHetD + y] = (int32_t)a.lbw[i];
      s_lat[x * kHetD + y] = (int32_t)a.llat[i];
    }
    if (lane < a.D) tmr = a.tmul[lane];
    __syncthreads();
  }
  const int64_t k = blockIdx.x;
  const int32_t n = a.n;
  const uint8_t *dev = a.devp + k * n;
  int64_t *fin = a.finp + k * n;
  const uint64_t *dm = ARR ? a.dmask + k * n : nullptr;
  const int64_t *of = ARR ? a.aoff + k * n : nullptr;
  // device `lane`'s state
  int64_t last = 0;   // free time (FIFO) or end of the last task (insertion)
  int32_t gcnt = 0;   // idle gaps stored
  int64_t glast = 0;  // end of the last stored gap
  int64_t gbase = INS && lane < a.D ? a.goff[k * a.D + lane] : 0;
  int32_t ghead = 0;  // ring head of the gap tail
  int64_t snd = 0, rcv = 0, tcur = 0;
  int64_t span = 0;
  uint32_t bad = 0;
  // A slot's own values and its first 4 inputs depend on nothing computed
  // here: they are loaded for the next window while this one is placed.
  int32_t nx_dv = 0, nx_i0 = 0, nx_i1 = 0, nx_q[4] = {-1, -1, -1, -1};
  int64_t nx_w = 0, nx_c = 0, nx_off = 0;
  uint64_t nx_dm = 0;
  auto load_own = [&](int32_t P) {
    const int32_t q = P + lane;
    nx_dv = nx_i0 = nx_i1 = 0;
    nx_w = nx_c = nx_off = 0;
    nx_dm = 0;
    nx_q[0] = nx_q[1] = nx_q[2] = nx_q[3] = -1;
    if (q < n) {
      nx_dv = dev[q];
      nx_w = a.wp[q];
      nx_c = HET ? a.obp[q] : a.cq[q];  // ob under HET: the comm depends on the link
      nx_i0 = a.iptr[q];
      nx_i1 = a.iptr[q + 1];
      const int4 f4 = a.ipre[q];
      nx_q[0] = f4.x;
      nx_q[1] = f4.y;
      nx_q[2] = f4.z;
      nx_q[3] = f4.w;
      if (ARR) {
        nx_dm = dm[q];
        nx_off = of[q];
      }
    }
  };
  load_own(0);
  for (int32_t P0 = 0; P0 < n; P0 += 64) {
    const int32_t nw = n - P0 < 64 ? n - P0 : 64;
    const int32_t p = P0 + lane;
    const bool act = lane < nw;
    CEL_TSTAMP(t_a);
    const int32_t dv = nx_dv, i0 = nx_i0, i1 = nx_i1;
    const int64_t w = nx_w, c = nx_c, myoff = nx_off;
    const uint64_t mydm = nx_dm;
    int32_t q4[4];
#pragma unroll
    for (int u = 0; u < 4; u++) q4[u] = nx_q[u];
    int64_t ext = 0;
    uint64_t msk = 0;
    // A: inputs from before the window
    const bool heavy = i1 - i0 > kMmLight;
    if (!heavy) {
      fold_batch<ARR, HET>(a, dev, fin, dm, of, s_bw, s_lat, P0, q4, dv, ext, msk, bad);
      fold_inputs<ARR, HET>(a, dev, fin, dm, of, s_bw, s_lat, P0, i0 + 4, i1, 1, dv, ext, msk,
                            bad);
    }
    for (uint64_t hv = __ballot(heavy); hv; hv &= hv - 1) {
      const int h = __builtin_ctzll(hv);
      const int32_t e0 = __builtin_amdgcn_readlane(i0, h), e1 = __builtin_amdgcn_readlane(i1, h);
      const int32_t dh = __builtin_amdgcn_readlane(dv, h);
      int64_t mx = 0;
      uint64_t mk = 0;
      fold_inputs<ARR, HET>(a, dev, fin, dm, of, s_bw, s_lat, P0, e0 + lane, e1, 64, dh, mx, mk,
                            bad);
      for (int off = 32; off > 0; off >>= 1) {
        const int64_t o = __shfl_xor(mx, off);
        mx = o > mx ? o : mx;
        mk |= __shfl_xor(mk, off);
      }
      if (lane == h) {
        ext = mx;
        msk = mk;
      }
    }
    // B: segments of consecutive slots with no edge among them, in order.
    // Inside a segment every slot's ready time is known once the earlier
    // segments are placed, and devices are independent but for the transfer
    // channels: lane d places device d's slots of the segment in order, then
    // the segment's transfers are issued in slot order.
    CEL_TSTAMP(t_b);
    CEL_TADD(0, t_a, t_b);
    load_own(P0 + 64);
    int64_t finw = 0;
    const int64_t wd = HET ? dur_on(w, __shfl(tmr, dv)) : w;  // slot duration on its device
    for (int32_t s0 = 0; s0 < nw;) {
      const uint64_t cut = __ballot(lane > s0 && lane < nw && (msk & ~below(s0)) != 0);
      const int32_t s1 = cut ? __builtin_ctzll(cut) : nw;
      const bool inseg = lane >= s0 && lane < s1;
      CEL_TCOUNT(11);
      int64_t r = ext;  // + inputs from the earlier segments of this window
      for (uint64_t mm = inseg ? msk : 0; __ballot(mm != 0);) {
        const bool has = mm != 0;
        const int q = has ? __builtin_ctzll(mm) : lane;
        mm &= mm - 1;
        const int64_t fq = __shfl(finw, q), xq = __shfl(c, q);
        const int32_t dq = __shfl(dv, q);
        int64_t t = fq;
        if (dq != dv) {
          if (ARR) t = s_T[q * 64 + dv];
          else if (HET) t = fq + link_c(xq, s_bw[dq * kHetD + dv], s_lat[dq * kHetD + dv]);
          else t = fq + xq;
        }
        if (has && t > r) r = t;
      }
      if (BLOCK) {
        // Transfers sit on the compute queues: a slot's transfers delay the
        // devices of later slots of the segment, so its slots are placed one
        // at a time, in order, each followed by its transfers (one per
        // destination device, increasing), from device states held in lanes
        for (uint64_t sm = __ballot(inseg); sm; sm &= sm - 1) {
          const int j = __builtin_ctzll(sm);
          CEL_TCOUNT(14);
          const int32_t dj = __builtin_amdgcn_readlane(dv, j);
          const int64_t rj = readlane64(r, j), wj = readlane64(wd, j);
          const int64_t lj = readlane64(last, dj);
          const int64_t f = (rj > lj ? rj : lj) + wj;
          int64_t qe = f;  // end of the sending device's queue
          const uint64_t dmj = (uint64_t)readlane64((int64_t)mydm, j);
          const int64_t cj = readlane64(c, j);
          for (uint64_t x = dmj; x; x &= x - 1) {
            const int b = __builtin_ctzll(x);
            const int64_t lb = readlane64(last, b);
            const int64_t t0 = qe > lb ? qe : lb;
            qe = t0 + (HET ? link_c(cj, s_bw[dj * kHetD + b], s_lat[dj * kHetD + b]) : cj);
            last = setlane<int64_t>(last, qe, b);
            tcur = setlane<int64_t>(tcur, qe, b);
          }
          last = setlane<int64_t>(last, qe, dj);
          finw = setlane<int64_t>(finw, f, j);
          if ((dmj >> lane) & 1) {
            s_T[j * 64 + lane] = tcur;
            a.pool[readlane64(myoff, j) + __builtin_popcountll(dmj & below(lane))] = tcur;
          }
          lds_order();
        }
        s0 = s1;
        continue;
      }
      if (inseg) atomicOr(&s_lst[dv], 1ull << lane);
      wave_lds_sync();
      uint64_t mine = lane < a.D ? s_lst[lane] : 0;
      if (!INS) {
        // FIFO devices: a device's chain last' = max(r, last) + w composes
        // maps x -> max(r + w, x + w); with the segment's slots sorted by
        // (device, position), one segmented max-plus scan places them all.
        const int32_t cnt = __builtin_popcountll(mine);
        int32_t inc = cnt;
        for (int off = 1; off < 64; off <<= 1) {
          const int32_t o = __shfl_up(inc, off);
          if (lane >= off) inc += o;
        }
        const int32_t first = inc - cnt;  // lane d: where device d's slots start
        int32_t rank = 0;
        const int32_t fd = __shfl(first, dv);
        if (inseg) {
          rank = fd + __builtin_popcountll(s_lst[dv] & below(lane));
          s_fin[rank] = lane;  // sorted position -> slot (s_fin reused as scratch)
        }
        wave_lds_sync();
        const int32_t ns = s1 - s0;
        const int32_t jj = lane < ns ? (int32_t)s_fin[lane] : lane;
        const int32_t dd = __shfl(dv, jj);
        const int64_t rr = __shfl(r, jj), ww = __shfl(wd, jj), l0 = __shfl(last, dd);
        const int32_t dprev = __shfl_up(dd, 1);
        int64_t ma = kNeg, mb = 0;
        int32_t fl = 1;
        if (lane < ns) {
          ma = rr + ww;
          mb = ww;
          fl = lane == 0 || dprev != dd;
        }
        wave_seg_scan_dpp(ma, mb, fl);
        const int64_t fs = ma > l0 + mb ? ma : l0 + mb;  // finish of sorted slot `lane`
        const int64_t nl = __shfl(fs, cnt > 0 ? inc - 1 : 0);  // device `lane`'s last finish
        if (lane < a.D && cnt > 0) last = nl;
        const int64_t myf = __shfl(fs, rank);
        if (inseg) finw = myf;
        lds_order();
        s_lst[lane] = 0;
        mine = 0;
      } else {
        lds_order();
        s_lst[lane] = 0;
      }
      while (__ballot(mine != 0)) {
        const bool has = mine != 0;
        const int j = has ? __builtin_ctzll(mine) : lane;
        mine &= mine - 1;
        const int64_t rj = __shfl(r, j), wj = __shfl(wd, j);
        CEL_TCOUNT(12);
        int64_t f = 0;
        bool done = true;
        if (has) {
          if (!INS) {
            last = (rj > last ? rj : last) + wj;
            f = last;
          } else {
            int64_t s_;
            done = lane_insert(a.ga + gbase, a.gb + gbase, s_ta + lane * kTail,
                               s_tb + lane * kTail, rj, wj, last, gcnt, glast, ghead, s_);
            f = s_ + wj;
          }
        }
        if (INS) {
          lds_order();
          for (uint64_t dl = __ballot(has && !done); dl; dl &= dl - 1) {  // the whole wave
            const int d = __builtin_ctzll(dl);
            CEL_TCOUNT(13);
            const int64_t rr = readlane64(rj, d), ww = readlane64(wj, d);
            int64_t L = readlane64(last, d), gl = readlane64(glast, d);
            int32_t G = __builtin_amdgcn_readlane(gcnt, d), hd = __builtin_amdgcn_readlane(ghead, d);
            const int64_t base = readlane64(gbase, d);
            const int64_t s_ = insert_slot(a.ga + base, a.gb + base, s_ta + d * kTail,
                                           s_tb + d * kTail, rr, ww, L, G, gl, hd, lane);
            last = setlane<int64_t>(last, L, d);
            glast = setlane<int64_t>(glast, gl, d);
            gcnt = setlane<int32_t>(gcnt, G, d);
            ghead = setlane<int32_t>(ghead, hd, d);
            f = setlane<int64_t>(f, s_ + ww, d);
          }
        }
        if (has) s_fin[j] = f;
      }
      if (INS) {
        wave_lds_sync();
        if (inseg) finw = s_fin[lane];
        lds_order();
      }
      if (TASKS) {  // the segment's transfers in slot order
        for (uint64_t pm = __ballot(inseg && mydm != 0); pm; pm &= pm - 1) {
          const int j = __builtin_ctzll(pm);
          const int32_t dj = __builtin_amdgcn_readlane(dv, j);
          const int64_t f = readlane64(finw, j), cj = readlane64(c, j);
          const uint64_t dmj = (uint64_t)readlane64((int64_t)mydm, j);
          int64_t sf = readlane64(snd, dj);
          for (uint64_t x = dmj; x; x &= x - 1) {
            const int b = __builtin_ctzll(x);
            const int64_t rb = readlane64(rcv, b);
            int64_t t0 = f > sf ? f : sf;
            t0 = rb > t0 ? rb : t0;
            sf = t0 + (HET ? link_c(cj, s_bw[dj * kHetD + b], s_lat[dj * kHetD + b]) : cj);
            rcv = setlane<int64_t>(rcv, sf, b);
            tcur = setlane<int64_t>(tcur, sf, b);
          }
          snd = setlane<int64_t>(snd, sf, dj);
          if ((dmj >> lane) & 1) {
            s_T[j * 64 + lane] = tcur;
            a.pool[readlane64(myoff, j) + __builtin_popcountll(dmj & below(lane))] = tcur;
          }
          lds_order();
        }
      }
      s0 = s1;
    }
    if (act) span = finw > span ? finw : span;
    // C: finish times of the window
    CEL_TSTAMP(t_c);
    CEL_TADD(1, t_b, t_c);
    if (act) fin[p] = finw;
    // the next window reads these finish times and arrivals
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
    CEL_TSTAMP(t_d);
    CEL_TADD(2, t_c, t_d);
    CEL_TCOUNT(3);
  }
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t o = __shfl_xor(span, off);
    span = o > span ? o : span;
  }
  if (lane == 0) a.makespan[k] = span;
  if (bad) raise_err(st, bad);
}

// First 4 inputs of each position (position space, -1 past the row's end),
// so that a window's inputs load with its other per-slot values.
__global__ void k_mm_ipre(int32_t n, const int32_t *iptr, const int32_t *iidx, int4 *ipre,
                          const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t e0 = iptr[p], e1 = iptr[p + 1];
    ipre[p] = make_int4(e0 < e1 ? iidx[e0] : -1, e0 + 1 < e1 ? iidx[e0 + 1] : -1,
                        e0 + 2 < e1 ? iidx[e0 + 2] : -1, e0 + 3 < e1 ? iidx[e0 + 3] : -1);
  }
}

// Per placement, nodes per device (gap segment sizes); blocks take chunks of
// positions and add an LDS histogram into cnt[k][D].
__global__ void k_mm_devcount(int32_t K, int32_t n, int32_t D, const uint8_t *devp, int32_t *cnt,
                              const Status *st) {
  __shared__ int32_t h[64];
  if (failed(st)) return;
  for (int64_t k = blockIdx.y; k < K; k += gridDim.y) {
    if (threadIdx.x < 64) h[threadIdx.x] = 0;
    __syncthreads();
    for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
         p += (int64_t)gridDim.x * blockDim.x)
      atomicAdd(&h[devp[k * n + p]], 1);
    __syncthreads();
    if (threadIdx.x < D && h[threadIdx.x]) atomicAdd(&cnt[k * D + threadIdx.x], h[threadIdx.x]);
    __syncthreads();
  }
}

// goff[k][d] = k * n + nodes of placement k on devices below d.
__global__ void k_mm_goff(int32_t K, int32_t n, int32_t D, const int32_t *cnt, int64_t *goff,
                          const Status *st) {
  if (failed(st)) return;
  for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < K;
       k += (int64_t)gridDim.x * blockDim.x) {
    int64_t acc = k * n;
    for (int32_t d = 0; d < D; d++) {
      goff[k * D + d] = acc;
      acc += cnt[k * D + d];
    }
  }
}

// Destination devices of every producer: for each edge u -> v and placement
// k with v on another device, set that device's bit in u's mask (by u's
// position); reading first keeps heavy rows from hammering one word.
__global__ void k_mm_dmask(cel_graph g, int32_t K, const int32_t *pos, const uint8_t *node_dev,
                           unsigned long long *dmask, const Status *st) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  if (failed(st)) return;
  const int64_t n = g.n;
  for_edges_balanced(g.out_ptr, g.n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    const int32_t v = g.out_idx[e];
    const int64_t pu = pos[u];
    for (int64_t k = blockIdx.y; k < K; k += gridDim.y) {
      const int du = node_dev[k * n + u], dv = node_dev[k * n + v];
      if (du == dv) continue;
      const unsigned long long bit = 1ull << dv;
      unsigned long long *x = &dmask[k * n + pu];
      if (!(__atomic_load_n(x, __ATOMIC_RELAXED) & bit)) atomicOr(x, bit);
    }
  });
}

__global__ void k_mm_popc(int64_t N, const uint64_t *dmask, int64_t *cntv, const Status *st) {
  if (failed(st)) return;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < N;
       i += (int64_t)gridDim.x * blockDim.x)
    cntv[i] = __builtin_popcountll(dmask[i]);
}

// Start and finish by node id: start = finish - the node's duration on its
// device (w, or ceil(w tmul / 1024) with tmul).
__global__ void k_mm_out(int32_t K, int32_t n, const int32_t *order, const int64_t *finp,
                         const int64_t *wp, const uint8_t *devp, const int64_t *tmul,
                         int64_t *start, int64_t *finish, const Status *st) {
  if (failed(st)) return;
  const int64_t tot = (int64_t)K * n;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < tot;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = i / n, p = i - k * n;
    const int64_t v = k * n + order[p];
    const int64_t f = finp[i];
    if (finish) finish[v] = f;
    if (start) start[v] = f - (tmul ? dur_on(wp[p], tmul[devp[i]]) : wp[p]);
  }
}

// lead[g] = smallest position of a member of group g (INT32_MAX initially).
__global__ void k_colo_lead(int32_t n, int32_t G, const int32_t *group, const int32_t *pos,
                            int32_t *lead, Status *st) {
  if (failed(st)) return;
  uint32_t bad = 0;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t x = group[v];
    if (x < -1 || x >= G) bad |= EB_ARG;
    else if (x >= 0) atomicMin(&lead[x], pos[v]);
  }
  if (bad) raise_err(st, bad);
}

// Every member takes its group leader's device (the leader keeps its own).
__global__ void k_colo_apply(int32_t K, int32_t n, const int32_t *group, const int32_t *lead,
                             const int32_t *order, uint8_t *node_dev, const Status *st) {
  if (failed(st)) return;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t x = group[v];
    if (x < 0) continue;
    const int32_t u = order[lead[x]];
    if (u == v) continue;
    for (int64_t k = blockIdx.y; k < K; k += gridDim.y)
      node_dev[k * n + v] = node_dev[k * n + u];
  }
}

}  // namespace cel

using namespace cel;

// Host checks of a heterogeneous descriptor; fills the worst link (smallest
// bandwidth, largest latency) and the largest multiplier.
int cel::check_hetero(const cel_hetero *h, const cel_devices *d, const char *fn, int64_t *bwmin,
                      int64_t *latmax, int64_t *tmax) {
  const int32_t D = d->D;
  *bwmin = d->bw;
  *latmax = d->lat;
  *tmax = 1024;
  if (h->tmul) {
    *tmax = 0;
    for (int32_t x = 0; x < D; x++) {
      if (h->tmul[x] < 1 || h->tmul[x] > 65536)
        return set_error(CEL_E_ARG, "%s: tmul[%d] outside [1, 65536]", fn, x);
      *tmax = h->tmul[x] > *tmax ? h->tmul[x] : *tmax;
    }
  }
  if (h->bw) *bwmin = INT32_MAX;
  if (h->lat) *latmax = 0;
  for (int32_t i = 0; i < D * D; i++) {
    if (i / D == i % D) continue;
    if (h->bw) {
      if (h->bw[i] < 1 || h->bw[i] > INT32_MAX)
        return set_error(CEL_E_ARG, "%s: link bandwidth %d outside [1, 2^31)", fn, i);
      *bwmin = h->bw[i] < *bwmin ? h->bw[i] : *bwmin;
    }
    if (h->lat) {
      if (h->lat[i] < 0 || h->lat[i] > INT32_MAX)
        return set_error(CEL_E_ARG, "%s: link latency %d outside [0, 2^31)", fn, i);
      *latmax = h->lat[i] > *latmax ? h->lat[i] : *latmax;
    }
  }
  if (D == 1) *bwmin = d->bw;
  return CEL_OK;
}

extern "C" int cel_makespan_model(const cel_graph *g, const cel_devices *d, const cel_hetero *h,
                                  const int32_t *order, int32_t K, const uint8_t *node_dev,
                                  int32_t model, int64_t *start, int64_t *finish,
                                  int64_t *makespan, hipStream_t s) {
  const char *fn = "cel_makespan_model";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n, D = d->D;
  if (!makespan || K < 1 || (n > 0 && (!order || !node_dev)))
    return set_error(CEL_E_ARG, "%s: NULL argument or K < 1", fn);
  if (model & ~(CEL_MODEL_INSERT | CEL_MODEL_COMM_TASKS | CEL_MODEL_COMM_BLOCK))
    return set_error(CEL_E_ARG, "%s: unknown model bits 0x%x", fn, model);
  if ((model & CEL_MODEL_COMM_BLOCK) && (model & (CEL_MODEL_INSERT | CEL_MODEL_COMM_TASKS)))
    return set_error(CEL_E_ARG, "%s: CEL_MODEL_COMM_BLOCK combines with no other bit", fn);
  if (D > 64) return set_error(CEL_E_ARG, "%s: D = %d above 64", fn, D);
  const bool ins = model & CEL_MODEL_INSERT, tasks = model & CEL_MODEL_COMM_TASKS;
  const bool block = model & CEL_MODEL_COMM_BLOCK;
  const bool het = h && (h->tmul || h->bw || h->lat);
  int64_t bwmin = d->bw, latmax = d->lat, tmax = 1024;
  if (het) {
    CEL_TRY(check_hetero(h, d, fn, &bwmin, &latmax, &tmax));
    // overflow bound with the slowest device and the worst link: every time
    // is a sum of durations and transfers along one chain
    cel_devices worst = *d;
    worst.bw = bwmin;
    worst.lat = latmax;
    int64_t ec = 0, ws = 0;
    CEL_TRY(cel_comm_sums(g, &worst, nullptr, &ec, &ws, s));
    const __int128 tot = (__int128)ws * ((tmax + 1023) / 1024) + ec;
    if (tot >= ((__int128)1 << 62))
      return set_error(CEL_E_OVERFLOW, "%s: times could reach 2^62", fn);
  }
  Scratch sc(s);
  Status *st;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  if (n == 0) {
    k_fill_i64<<<grid_for(K, 256, 1024), 256, 0, s>>>(makespan, K, 0);
    CEL_HIP(hipGetLastError());
    CEL_HIP(hipStreamSynchronize(s));
    return CEL_OK;
  }
  int32_t *tmp, *pos, *iptr, *iidx;
  int64_t *wp, *cq, *finp;
  uint8_t *devp;
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(sc.get(&pos, n));
  CEL_TRY(check_graph(g, bwmin, latmax, true, st, tmp, sc, s));
  CEL_TRY(check_topo_order(g, order, pos, st, s));
  const int64_t Kn = (int64_t)K * n;
  CEL_TRY(sc.get(&iptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&iidx, g->m));
  CEL_TRY(sc.get(&wp, n));
  CEL_TRY(sc.get(&cq, n));
  CEL_TRY(sc.get(&devp, Kn));
  CEL_TRY(sc.get(&finp, Kn));
  CEL_TRY(relabel_csr(n, g->m, order, pos, g->in_ptr, g->in_idx, iptr, iidx, sc, s, st));
  // under HET cq holds ob (bandwidth 1, latency 0): the link decides the comm
  k_pos_costs<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, g->w, g->ob, het ? 1 : d->bw,
                                                    het ? 0 : d->lat, wp, cq, st);
  const int gx = grid_for(n, 256, 1024), gy = K < 1024 ? K : 1024;
  k_dev_gather<<<dim3(gx, gy), 256, 0, s>>>(K, n, order, node_dev, D, devp, st);
  int4 *ipre;
  CEL_TRY(sc.get(&ipre, n));
  k_mm_ipre<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, iptr, iidx, ipre, st);
  MmArgs a{};
  a.ipre = ipre;
  a.n = n;
  a.D = D;
  a.iptr = iptr;
  a.iidx = iidx;
  a.wp = wp;
  a.cq = cq;
  a.devp = devp;
  a.finp = finp;
  a.makespan = makespan;
  int64_t *tmul_d = nullptr;
  if (het) {
    int64_t *lbw, *llat;
    CEL_TRY(sc.get(&tmul_d, D));
    CEL_TRY(sc.get(&lbw, (int64_t)D * D));
    CEL_TRY(sc.get(&llat, (int64_t)D * D));
    std::vector<int64_t> ht(D), hb((size_t)D * D), hl((size_t)D * D);
    for (int32_t x = 0; x < D; x++) ht[x] = h->tmul ? h->tmul[x] : 1024;
    for (int32_t i = 0; i < D * D; i++) {
      const bool diag = i / D == i % D;
      hb[i] = diag ? 1 : (h->bw ? h->bw[i] : d->bw);
      hl[i] = diag ? 0 : (h->lat ? h->lat[i] : d->lat);
      if (!h->bw && hb[i] > INT32_MAX) return set_error(CEL_E_ARG, "%s: bw above 2^31", fn);
      if (!h->lat && hl[i] > INT32_MAX) return set_error(CEL_E_ARG, "%s: lat above 2^31", fn);
    }
    CEL_HIP(hipMemcpyAsync(tmul_d, ht.data(), sizeof(int64_t) * D, hipMemcpyHostToDevice, s));
    CEL_HIP(hipMemcpyAsync(lbw, hb.data(), sizeof(int64_t) * D * D, hipMemcpyHostToDevice, s));
    CEL_HIP(hipMemcpyAsync(llat, hl.data(), sizeof(int64_t) * D * D, hipMemcpyHostToDevice, s));
    a.obp = cq;
    a.tmul = tmul_d;
    a.lbw = lbw;
    a.llat = llat;
  }
  if (ins) {
    int32_t *cnt;
    int64_t *goff, *ga, *gb;
    CEL_TRY(sc.get(&cnt, (int64_t)K * D));
    CEL_TRY(sc.get(&goff, (int64_t)K * D));
    CEL_TRY(sc.get(&ga, Kn));
    CEL_TRY(sc.get(&gb, Kn));
    CEL_HIP(hipMemsetAsync(cnt, 0, sizeof(int32_t) * K * D, s));
    k_mm_devcount<<<dim3(grid_for(n, 256, 64), gy), 256, 0, s>>>(K, n, D, devp, cnt, st);
    k_mm_goff<<<grid_for(K, 256, 1024), 256, 0, s>>>(K, n, D, cnt, goff, st);
    a.goff = goff;
    a.ga = ga;
    a.gb = gb;
  }
  if (tasks || block) {
    uint64_t *dmask;
    int64_t *pc, *aoff, *pool;
    CEL_TRY(sc.get(&dmask, Kn));
    CEL_TRY(sc.get(&pc, Kn));
    CEL_TRY(sc.get(&aoff, Kn + 1));
    CEL_HIP(hipMemsetAsync(dmask, 0, sizeof(uint64_t) * Kn, s));
    k_mm_dmask<<<dim3(edge_blocks(g->m), gy), 256, 0, s>>>(*g, K, pos, node_dev,
                                                           (unsigned long long *)dmask, st);
    k_mm_popc<<<grid_for(Kn, 256, 8192), 256, 0, s>>>(Kn, dmask, pc, st);
    CEL_TRY(exclusive_scan_i64(pc, aoff, Kn, sc, s));
    int64_t total = 0;  // transfers of all placements (valid once the checks passed)
    CEL_HIP(hipMemcpyAsync(&total, aoff + Kn, sizeof(int64_t), hipMemcpyDeviceToHost, s));
    Status h0;
    CEL_TRY(read_status(st, &h0, s));
    if (h0.err) return status_error(h0, fn);
    CEL_TRY(sc.get(&pool, total > 0 ? total : 1));
    a.dmask = dmask;
    a.aoff = aoff;
    a.pool = pool;
  }
  {
    KTimer kt(s, "k_makespan_model");
    const unsigned gk = (unsigned)K;
    if (block) {
      if (het) k_makespan_model<false, false, true, true><<<gk, 64, 0, s>>>(a, st);
      else k_makespan_model<false, false, false, true><<<gk, 64, 0, s>>>(a, st);
    } else if (het) {
      if (!ins && !tasks) k_makespan_model<false, false, true><<<gk, 64, 0, s>>>(a, st);
      else if (ins && !tasks) k_makespan_model<true, false, true><<<gk, 64, 0, s>>>(a, st);
      else if (!ins) k_makespan_model<false, true, true><<<gk, 64, 0, s>>>(a, st);
      else k_makespan_model<true, true, true><<<gk, 64, 0, s>>>(a, st);
    } else {
      if (!ins && !tasks) k_makespan_model<false, false, false><<<gk, 64, 0, s>>>(a, st);
      else if (ins && !tasks) k_makespan_model<true, false, false><<<gk, 64, 0, s>>>(a, st);
      else if (!ins) k_makespan_model<false, true, false><<<gk, 64, 0, s>>>(a, st);
      else k_makespan_model<true, true, false><<<gk, 64, 0, s>>>(a, st);
    }
  }
  if (start || finish)
    k_mm_out<<<grid_for(Kn, 256, 8192), 256, 0, s>>>(K, n, order, finp, wp, devp, tmul_d, start,
                                                    finish, st);
  CEL_HIP(hipGetLastError());
  Status hs;
  CEL_TRY(read_status(st, &hs, s));
  if (hs.err) return status_error(hs, fn);
  return CEL_OK;
}

CEL_PHASE_READER(cel_debug_phases_model)

extern "C" int cel_colocate(const cel_graph *g, const int32_t *order, const int32_t *group,
                            int32_t n_groups, int32_t K, uint8_t *node_dev, hipStream_t s) {
  const char *fn = "cel_colocate";
  CEL_TRY(check_host_graph(g, fn));
  const int32_t n = g->n;
  if (K < 1 || n_groups < 0 || (n > 0 && (!order || !group || !node_dev)))
    return set_error(CEL_E_ARG, "%s: NULL argument, K < 1 or n_groups < 0", fn);
  if (n == 0) return CEL_OK;
  Scratch sc(s);
  Status *st;
  int32_t *tmp, *pos, *lead;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(sc.get(&pos, n));
  CEL_TRY(check_graph(g, 1, 0, false, st, tmp, sc, s));
  CEL_TRY(check_topo_order(g, order, pos, st, s));
  if (n_groups > 0) {
    CEL_TRY(sc.get(&lead, n_groups));
    k_fill_i32<<<grid_for(n_groups, 256, 1024), 256, 0, s>>>(lead, n_groups, INT32_MAX);
    k_colo_lead<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, n_groups, group, pos, lead, st);
    const int gy = K < 1024 ? K : 1024;
    k_colo_apply<<<dim3(grid_for(n, 256, 1024), gy), 256, 0, s>>>(K, n, group, lead, order,
                                                                 node_dev, st);
  } else {
    k_colo_lead<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, 0, group, pos, nullptr, st);
  }
  CEL_HIP(hipGetLastError());
  Status hs;
  CEL_TRY(read_status(st, &hs, s));
  if (hs.err) return status_error(hs, fn);
  return CEL_OK;
}
