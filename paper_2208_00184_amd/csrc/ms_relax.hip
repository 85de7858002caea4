// Makespan of one placement (eq. 7 without insertion, Order-Place's device
// model: each device runs its nodes in the given order, one after another) by
// relaxation over the edges that cross devices.
//
// Each device's nodes, in the order given, form one chain.  With S(k) the
// sum of w over the chain through node k and Sx(k) = S(k) - w(k), the FIFO
// rule fin(k) = max(ready(k), fin(previous on the chain)) + w(k) unrolls to
//   fin(k) = S(k) + max(0, max over chain nodes j up to k of ready(j) - Sx(j)).
// An edge between two nodes of one device never decides a ready time: its
// source lies earlier on the same chain and finishes no later than the
// chain's node just before the target, whose finish already bounds the
// target's start.  So only edges whose ends sit on different devices count:
//   ready(j) = max(0, max over such predecessors p of fin(p) + c(p)).
// Start from fin = S (no cross-device waits) and repeat "ready times from
// the current fin, then each chain's prefix maximum".  Every iterate is a
// lower bound of the true finish times (the map is monotone and the true
// times are its fixed point), and after t rounds every node whose finish is
// decided by a path with fewer than t device changes is exact.  A round that
// changes nothing has reached the unique fixed point: the schedule is exact.
// The rounds needed are the longest run of device changes along a deciding
// path plus two, far fewer than the levels on placements that keep most
// edges on one device (Adjusting Placement keeps whole clusters together).
//
// Layout.  Slots are the chain order: device 0's nodes in the given order,
// then device 1's, ... (a stable counting sort of the order by device).  Per
// slot: wxa = exclusive prefix sum of w over all slots (the chain sums are
// differences of it), wxc = wxa(q + 1) + c(q), the list of cross-device
// predecessor slots (CSR).  With V(j) = ready(j) - wxa(j), and at a chain's
// first slot h also -wxa(h), fin(q) = wxa(q + 1) + PM(q), PM the prefix
// maximum of V along the chain; the rounds store fin + c (finc) per slot, the
// value a cross-device successor gathers.
//
// One persistent kernel runs every round.  Workgroup b owns slots
// [b T, (b + 1) T) as NT tiles of kRxB, one slot per thread and tile, and
// keeps its in-block prefix maxima in registers.  A round: gather the
// predecessors' finc (every load issued before the first use), per tile a
// segmented wave scan (DPP) and the wave tails through LDS, publish the
// block's tail, grid barrier, the carry from earlier blocks of the chain,
// fin + c stored where it changed, grid barrier, and every block reads
// whether any slot changed.  The converged round writes start, finish and
// the makespan directly.  Each grid barrier waits a bounded time; a wait
// that outlasts it raises EB_WAIT and ends every workgroup.
#include <map>
#include <mutex>

#include "cel_internal.h"

namespace cel {

constexpr int kRxB = 1024;       // threads per workgroup (16 waves)
constexpr int kRxW = kRxB / 64;
constexpr int kRxCB = 1024;      // positions per block of the counting sort
constexpr int kRxGroup = 4;      // tiles whose gathers are in flight together
constexpr int kRxHeavy = 8;      // more predecessors: the whole wave gathers them

__device__ inline uint64_t lanemask_le(int lane) {
  return lane == 63 ? ~0ull : ((1ull << (lane + 1)) - 1);
}

// Lanes of the wave that are active and hold the same device as this lane
// (one ballot per bit of the id).
__device__ inline uint64_t same_device_lanes(uint32_t d, bool act) {
  uint64_t m = __ballot(act);
#pragma unroll
  for (int b = 0; b < 8; b++) {
    const bool bit = (d >> b) & 1u;
    const uint64_t x = __ballot(act && bit);
    m &= bit ? x : ~x;
  }
  return m;
}

// ------------------------------------------------- chain order (counting sort)

// cnt[d * nb + b] = nodes of device d among positions [b kRxCB, (b+1) kRxCB)
__global__ void __launch_bounds__(kRxCB) k_rx_count(int32_t n, int32_t D, int32_t nb,
                                                   const uint8_t *devp, int32_t *cnt,
                                                   const Status *st) {
  __shared__ int32_t h[256];
  if (failed(st)) return;
  for (int i = threadIdx.x; i < D; i += kRxCB) h[i] = 0;
  __syncthreads();
  const int64_t p = (int64_t)blockIdx.x * kRxCB + threadIdx.x;
  const bool act = p < n;
  const uint32_t d = act ? devp[p] : 0u;
  const uint64_t peers = same_device_lanes(d, act);
  const int lane = threadIdx.x & 63;
  if (act && lane == __builtin_ctzll(peers)) atomicAdd(&h[d], __popcll(peers));
  __syncthreads();
  for (int i = threadIdx.x; i < D; i += kRxCB) cnt[(int64_t)i * nb + blockIdx.x] = h[i];
}

// Slot of every position: off[d * nb + b] (exclusive scan of cnt) + the
// nodes of device d before it in its block.  Writes the node of each slot,
// the slot of each node, and w and c by slot (c = 0 for a node without
// successors).
__global__ void __launch_bounds__(kRxCB) k_rx_scatter(int32_t n, int32_t D, int32_t nb,
                                                     const uint8_t *devp, const int32_t *order,
                                                     const int32_t *off, const int64_t *w,
                                                     const int64_t *ob, const int32_t *out_ptr,
                                                     int64_t bw, int64_t lat, int32_t *gnode,
                                                     int32_t *nslot, int64_t *wq, int64_t *cq,
                                                     const Status *st) {
  __shared__ int32_t wc[kRxCB / 64][256];
  if (failed(st)) return;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  for (int i = lane; i < D; i += 64) wc[wv][i] = 0;
  __syncthreads();
  const int64_t p = (int64_t)blockIdx.x * kRxCB + threadIdx.x;
  const bool act = p < n;
  const uint32_t d = act ? devp[p] : 0u;
  const uint64_t peers = same_device_lanes(d, act);
  if (act && lane == __builtin_ctzll(peers)) wc[wv][d] = __popcll(peers);
  __syncthreads();
  if (!act) return;
  int32_t q = off[(int64_t)d * nb + blockIdx.x] + __popcll(peers & (lanemask_le(lane) >> 1));
  for (int i = 0; i < wv; i++) q += wc[i][d];
  const int32_t v = order[p];
  gnode[q] = v;
  nslot[v] = q;
  wq[q] = w[v];
  // a sink's c is never paid (and the overflow bound does not cover it)
  cq[q] = out_ptr[v + 1] > out_ptr[v] ? comm_of(ob[v], bw, lat) : 0;
}

// Cross-device in-edges counted per target slot (edge-balanced over the CSC).
__global__ void k_rx_xcount(int32_t n, int32_t m, const int32_t *in_ptr, const int32_t *in_idx,
                            const uint8_t *node_dev, const int32_t *nslot, int32_t *xcnt,
                            const Status *st) {
  __shared__ int32_t rp[kRowsPB + 1], su[2];
  if (failed(st)) return;
  for_edges_balanced(in_ptr, n, m, rp, su, [&](int32_t v, int32_t e) {
    const int32_t u = in_idx[e];
    if (node_dev[u] != node_dev[v]) atomicAdd(&xcnt[nslot[v]], 1);
  });
}

// The lists: xsrc[xptr[q] ..) = slots of q's cross-device predecessors, in
// any order (xcnt counts down to 0 as the cursor).
__global__ void k_rx_xfill(int32_t n, int32_t m, const int32_t *in_ptr, const int32_t *in_idx,
                           const uint8_t *node_dev, const int32_t *nslot, const int32_t *xptr,
                           int32_t *xcnt, int32_t *xsrc, const Status *st) {
  __shared__ int32_t rp[kRowsPB + 1], su[2];
  if (failed(st)) return;
  for_edges_balanced(in_ptr, n, m, rp, su, [&](int32_t v, int32_t e) {
    const int32_t u = in_idx[e];
    if (node_dev[u] != node_dev[v]) {
      const int32_t q = nslot[v];
      xsrc[xptr[q] + atomicSub(&xcnt[q], 1) - 1] = nslot[u];
    }
  });
}

// Per slot: rec = {first cross-device predecessor slot or -1, second or -1,
// count, start of the list}, wxc = wxa(q + 1) + c(q).
__global__ void k_rx_rec(int32_t n, const int32_t *xptr, const int32_t *xsrc, const int64_t *wxa,
                         const int64_t *cq, int4 *rec, int64_t *wxc, const Status *st) {
  if (failed(st)) return;
  for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n;
       q += (int64_t)gridDim.x * blockDim.x) {
    const int32_t b = xptr[q], c = xptr[q + 1] - b;
    rec[q] = make_int4(c > 0 ? xsrc[b] : -1, c > 1 ? xsrc[b + 1] : -1, c, b);
    wxc[q] = wxa[q + 1] + cq[q];
  }
}

// ------------------------------------------------------------ relaxation

struct RxArgs {
  int32_t n, D, nb, cap;
  const int32_t *off;     // [D nb + 1] chain starts: off[d nb]; off[D nb] = n
  const int64_t *wxa;     // [n + 1]
  const int64_t *wxc;     // [n]
  const int4 *rec;        // [n]
  const int32_t *xsrc;    // cross-device predecessor slots
  const int32_t *gnode;   // [n] node of each slot
  int64_t *finc;          // [n] fin + c by slot
  int64_t *tail;          // [gridDim] each block's running maximum at its end
  int32_t *bar;           // [0] released barrier (k << 1 | OR of the bits), [1] abort,
                          // [2 + b] workgroup b's arrival (k << 1 | its bit)
  int64_t *start, *finish, *makespan;
};

template <int NT>
__global__ void __launch_bounds__(kRxB) k_rx_relax(RxArgs a, Status *st) {
  __shared__ uint32_t s_head[NT * kRxB / 32];  // chain starts among the block's slots
  __shared__ int64_t s_wt[2][kRxW];            // per tile parity: each wave's tail value
  __shared__ int32_t s_wh[2][kRxW];            // ... and whether the wave holds a chain start
  __shared__ int64_t s_red[kRxW];
  __shared__ int64_t s_prev[NT][kRxB];         // PM stored last round (kInf before the first)
  __shared__ int32_t s_sb, s_ok, s_bit, s_chg;
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int32_t n = a.n;
  const int64_t T = (int64_t)NT * kRxB;
  const int64_t lo = (int64_t)blockIdx.x * T;

  for (int i = tid; i < NT * kRxB / 32; i += kRxB) s_head[i] = 0;
  if (tid == 0) {
    s_sb = -1;
    s_chg = 0;
  }
  __syncthreads();
  // chain starts inside [lo, lo + T), and the start of the chain through lo
  for (int d = tid; d < a.D; d += kRxB) {
    const int64_t h = a.off[(int64_t)d * a.nb];
    if (h >= lo && h < lo + T && h < n)
      atomicOr(&s_head[(h - lo) >> 5], 1u << ((h - lo) & 31));
    if (h <= lo) atomicMax(&s_sb, (int32_t)h);  // the largest chain start at or before lo
  }
  __syncthreads();
  // block of the chain start before lo (-1: lo starts a chain, no carry)
  const int32_t sb = s_sb == (int32_t)lo ? -1 : (int32_t)(s_sb / T);

  // per tile: pv = this round's value (ready - wxa, then its prefix maximum PM)
  int64_t pv[NT];
  uint32_t hbits = 0;  // bit k: a chain starts in the block at or before this thread's slot of tile k
#pragma unroll
  for (int k = 0; k < NT; k++) s_prev[k][tid] = kInf;
  int32_t bar = 0;  // grid barriers passed
  int32_t r = 0;
  for (; r < a.cap; r++) {
    // ready(q) - wxa(q) for every slot, gathers in groups of kRxGroup tiles
#pragma unroll
    for (int g0 = 0; g0 < NT; g0 += kRxGroup) {
      constexpr int GR = NT < kRxGroup ? NT : kRxGroup;
      int4 rc[GR];
      int64_t wa[GR], f0[GR], f1[GR];
#pragma unroll
      for (int j = 0; j < GR; j++) {
        const int64_t q = lo + (int64_t)(g0 + j) * kRxB + tid;
        rc[j] = make_int4(-1, -1, 0, 0);
        wa[j] = 0;
        if (g0 + j < NT && q < n) {
          wa[j] = a.wxa[q];
          if (r > 0) rc[j] = a.rec[q];
        }
      }
#pragma unroll
      for (int j = 0; j < GR; j++) {
        f0[j] = rc[j].x >= 0 ? ld_coherent(&a.finc[rc[j].x]) : -1;
        f1[j] = rc[j].y >= 0 ? ld_coherent(&a.finc[rc[j].y]) : -1;
      }
#pragma unroll
      for (int j = 0; j < GR; j++) {
        if (g0 + j >= NT) continue;
        int64_t rd = f0[j] > f1[j] ? f0[j] : f1[j];
        const int32_t cnt = rc[j].z, xb = rc[j].w;
        if (cnt > 2 && cnt <= kRxHeavy)  // the rest, one by one
          for (int32_t e = xb + 2; e < xb + cnt; e++) {
            const int64_t y = ld_coherent(&a.finc[a.xsrc[e]]);
            rd = y > rd ? y : rd;
          }
        // rows of many predecessors: the whole wave takes each in turn
        uint64_t heavy = __ballot(cnt > kRxHeavy);
        while (heavy) {
          const int l = __builtin_ctzll(heavy);
          heavy &= heavy - 1;
          const int32_t h0 = __builtin_amdgcn_readlane(xb, l);
          const int32_t h1 = h0 + __builtin_amdgcn_readlane(cnt, l);
          int64_t mx = -1;
          for (int32_t e = h0 + lane; e < h1; e += 64) {
            const int64_t y = ld_coherent(&a.finc[a.xsrc[e]]);
            mx = y > mx ? y : mx;
          }
          for (int o = 32; o > 0; o >>= 1) {
            const int64_t y = __shfl_xor((long long)mx, o);
            mx = y > mx ? y : mx;
          }
          if (lane == l) rd = mx;
        }
        const int64_t ql = (int64_t)(g0 + j) * kRxB + tid;
        int64_t v = rd >= 0 ? rd - wa[j] : kNeg;
        if (lo + ql < n && ((s_head[ql >> 5] >> (ql & 31)) & 1u)) v = -wa[j] > v ? -wa[j] : v;
        pv[g0 + j] = v;
      }
    }
    // per tile: segmented prefix maximum along the chains, carried across
    // waves and tiles of the block
    int64_t tcar = kNeg;
    bool tseen = false;
    hbits = 0;
#pragma unroll
    for (int k = 0; k < NT; k++) {
      const int64_t ql = (int64_t)k * kRxB + tid;
      const bool head = lo + ql < n && ((s_head[ql >> 5] >> (ql & 31)) & 1u);
      const uint64_t hm = __ballot(head);
      const uint64_t le = hm & lanemask_le(lane);
      const int32_t hd = le ? lane - (63 - __builtin_clzll(le)) : 64;
      int64_t y = wave_seg_pmax(pv[k], hd, lane);
      const int par = k & 1;
      if (lane == 63) s_wt[par][wv] = y;
      if (lane == 0) s_wh[par][wv] = hm != 0;
      lds_barrier();
      // lanes 0..kRxW-1 of every wave: segmented inclusive scan of the wave tails
      const int64_t t = lane < kRxW ? s_wt[par][lane] : kNeg;
      const uint64_t thm = __ballot(lane < kRxW && s_wh[par][lane] != 0);
      const uint64_t tle = thm & lanemask_le(lane);
      const int32_t thd = tle ? lane - (63 - __builtin_clzll(tle)) : 64;
      const int64_t inc = wave_seg_pmax(t, thd, lane);
      int64_t cw = wv > 0 ? readlane64(inc, wv - 1) : kNeg;  // waves before this one
      bool sw = (thm & ((1ull << wv) - 1)) != 0;
      if (!sw) {
        cw = tcar > cw ? tcar : cw;
        sw = tseen;
      }
      if (!le) y = cw > y ? cw : y;  // the chain runs in from before the wave
      pv[k] = y;
      hbits |= (le || sw) ? 1u << k : 0u;
      const int64_t all = readlane64(inc, kRxW - 1);  // the block's running value after this tile
      if (thm) {
        tcar = all;
        tseen = true;
      } else {
        tcar = all > tcar ? all : tcar;
      }
    }
    if (tid == 0) st_coherent(&a.tail[blockIdx.x], tcar);
    int64_t wc[NT];
#pragma unroll
    for (int k = 0; k < NT; k++) {
      const int64_t q = lo + (int64_t)k * kRxB + tid;
      wc[k] = q < n ? a.wxc[q] : 0;
    }
    int32_t any;
    if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &any)) return;
    // carry from the earlier blocks of the chain through lo
    int64_t carry = kNeg;
    if (sb >= 0) {
      int64_t c = kNeg;
      for (int32_t b2 = sb + tid; b2 < (int32_t)blockIdx.x; b2 += kRxB) {
        const int64_t t = ld_coherent(&a.tail[b2]);
        c = t > c ? t : c;
      }
      for (int o = 32; o > 0; o >>= 1) {
        const int64_t t = __shfl_xor((long long)c, o);
        c = t > c ? t : c;
      }
      if (lane == 0) s_red[wv] = c;
      lds_barrier();
      carry = lane < kRxW ? s_red[lane] : kNeg;
      for (int o = 32; o > 0; o >>= 1) {
        const int64_t t = __shfl_xor((long long)carry, o);
        carry = t > carry ? t : carry;
      }
    }
    // PM with the carry; fin + c stored where PM changed
    bool chg = false;
#pragma unroll
    for (int k = 0; k < NT; k++) {
      const int64_t q = lo + (int64_t)k * kRxB + tid;
      const int64_t pm = ((hbits >> k) & 1u) ? pv[k] : (carry > pv[k] ? carry : pv[k]);
      pv[k] = pm;
      if (q < n && pm != s_prev[k][tid]) {
        s_prev[k][tid] = pm;
        chg = true;
        st_coherent(&a.finc[q], wc[k] + pm);
      }
    }
    if (__ballot(chg) && lane == 0) s_chg = 1;  // LDS store; read after the barrier's __syncthreads
    __syncthreads();
    const int32_t mychg = s_chg;
    if (!grid_sync(a.bar, ++bar, mychg, &s_ok, &s_bit, st, &any)) return;
    if (tid == 0) s_chg = 0;  // the next round's flag (read only after two more barriers)
    if (!any) break;
  }
  if (r == a.cap) {  // not converged: the caller runs the level sweep instead
    if (blockIdx.x == 0 && tid == 0) {
      st->i2 = r;
      st->i3 = 0;
    }
    return;
  }
  // converged: pv holds PM; fin = wxa(q + 1) + PM, start = wxa(q) + PM
  int64_t mk = 0;
#pragma unroll
  for (int k = 0; k < NT; k++) {
    const int64_t q = lo + (int64_t)k * kRxB + tid;
    if (q >= n) continue;
    const int64_t fin = a.wxa[q + 1] + pv[k];
    mk = fin > mk ? fin : mk;
    if (a.finish || a.start) {
      const int32_t v = a.gnode[q];
      if (a.finish) a.finish[v] = fin;
      if (a.start) a.start[v] = a.wxa[q] + pv[k];
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const int64_t t = __shfl_xor((long long)mk, o);
    mk = t > mk ? t : mk;
  }
  if (lane == 0 && mk > 0) atomicMax((unsigned long long *)a.makespan, (unsigned long long)mk);
  if (blockIdx.x == 0 && tid == 0) {
    st->i2 = r + 1;
    st->i3 = 1;
  }
}

// ------------------------------------------------------------------- host

namespace {
constexpr int kRxNT[] = {1, 2, 3, 4, 5, 6, 8};  // tiles per thread of the instantiations
constexpr int kRxNV = sizeof(kRxNT) / sizeof(kRxNT[0]);
struct RxDev {
  int cus = 0;
  int occ[kRxNV] = {};  // co-resident workgroups per CU for each instantiation
};
std::mutex g_rx_mu;
std::map<int, RxDev> g_rx_dev;

const void *rx_kernel(int i) {
  switch (i) {
    case 0: return (const void *)k_rx_relax<1>;
    case 1: return (const void *)k_rx_relax<2>;
    case 2: return (const void *)k_rx_relax<3>;
    case 3: return (const void *)k_rx_relax<4>;
    case 4: return (const void *)k_rx_relax<5>;
    case 5: return (const void *)k_rx_relax<6>;
    default: return (const void *)k_rx_relax<8>;
  }
}

int rx_device(RxDev *out) {
  int dev = 0;
  CEL_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_rx_mu);
  auto it = g_rx_dev.find(dev);
  if (it == g_rx_dev.end()) {
    RxDev r;
    CEL_HIP(hipDeviceGetAttribute(&r.cus, hipDeviceAttributeMultiprocessorCount, dev));
    for (int i = 0; i < kRxNV; i++) {
      int nb = 0;
      CEL_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, rx_kernel(i), kRxB, 0));
      r.occ[i] = nb;
    }
    it = g_rx_dev.emplace(dev, r).first;
  }
  *out = it->second;
  return CEL_OK;
}
}  // namespace

int ms_relax(const cel_graph *g, const cel_devices *d, int32_t L, const int32_t *order,
             const uint8_t *node_dev, const uint8_t *devp, int64_t *start, int64_t *finish,
             int64_t *makespan, int max_groups, Scratch &sc, hipStream_t s, Status *st,
             bool *launched) {
  *launched = false;
  const int32_t n = g->n, m = g->m, D = d->D;
  RxDev rd;
  CEL_TRY(rx_device(&rd));
  // the fewest tiles per thread whose grid fits the co-resident workgroups
  // (one workgroup per CU at most: the grid barrier's cost grows with it)
  int ti = -1, G = 0;
  for (int i = 0; i < kRxNV && ti < 0; i++) {
    const int64_t T = (int64_t)kRxB * kRxNT[i];
    const int64_t need = ((int64_t)n + T - 1) / T;
    int64_t fit = (int64_t)(rd.occ[i] < 1 ? rd.occ[i] : 1) * rd.cus;
    if (max_groups > 0 && fit > max_groups) fit = max_groups;
    if (need <= fit) {
      ti = i;
      G = (int)need;
    }
  }
  if (ti < 0) return CEL_OK;  // too large for one co-resident grid
  // The grid is at most one workgroup per CU, within what the occupancy
  // calculator says fits: on an idle GPU every workgroup is resident at once,
  // which the grid barriers need.  Their waits are bounded (kGridSpin), so a
  // workgroup kept off the GPU by other work ends the call with an error
  // instead of hanging it.
  // Rounds allowed before the level sweep is cheaper: a round costs a few
  // microseconds of barriers plus its bytes at a few TB/s; the sweep about
  // 0.85 us per level after some 0.5 ms of preparation.
  const double round_us = 6.0 + (32.0 * n + 12.0 * m) / 4.0e6;
  const double sweep_us = 500.0 + 0.85 * L;
  int32_t cap = (int32_t)(sweep_us / round_us);
  if (cap < 4) cap = 4;
  if (cap > 1 << 20) cap = 1 << 20;

  const int32_t nb = (n + kRxCB - 1) / kRxCB;
  int32_t *cnt, *off, *gnode, *nslot, *xcnt, *xptr, *xsrc, *bar;
  int64_t *wq, *cq, *wxa, *wxc, *finc, *tail;
  int4 *rec;
  CEL_TRY(sc.get(&cnt, (int64_t)D * nb));
  CEL_TRY(sc.get(&off, (int64_t)D * nb + 1));
  CEL_TRY(sc.get(&gnode, n));
  CEL_TRY(sc.get(&nslot, n));
  CEL_TRY(sc.get(&xcnt, n));
  CEL_TRY(sc.get(&xptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&xsrc, m));
  CEL_TRY(sc.get(&bar, 2 + (int64_t)G));
  CEL_TRY(sc.get(&wq, n));
  CEL_TRY(sc.get(&cq, n));
  CEL_TRY(sc.get(&wxa, (int64_t)n + 1));
  CEL_TRY(sc.get(&wxc, n));
  CEL_TRY(sc.get(&finc, n));
  CEL_TRY(sc.get(&tail, G));
  CEL_TRY(sc.get(&rec, n));
  k_rx_count<<<nb, kRxCB, 0, s>>>(n, D, nb, devp, cnt, st);
  CEL_TRY(exclusive_scan_i32(cnt, off, (int64_t)D * nb, sc, s));
  k_rx_scatter<<<nb, kRxCB, 0, s>>>(n, D, nb, devp, order, off, g->w, g->ob, g->out_ptr, d->bw,
                                    d->lat, gnode, nslot, wq, cq, st);
  CEL_TRY(exclusive_scan_i64(wq, wxa, n, sc, s));
  k_fill_i32<<<grid_for(n, 256, 4096), 256, 0, s>>>(xcnt, n, 0);
  k_fill_i32<<<grid_for(2 + (int64_t)G, 256, 64), 256, 0, s>>>(bar, 2 + (int64_t)G, 0);
  k_fill_i64<<<1, 64, 0, s>>>(makespan, 1, 0);
  k_rx_xcount<<<edge_blocks(m), 256, 0, s>>>(n, m, g->in_ptr, g->in_idx, node_dev, nslot, xcnt,
                                             st);
  CEL_TRY(exclusive_scan_i32(xcnt, xptr, n, sc, s));
  k_rx_xfill<<<edge_blocks(m), 256, 0, s>>>(n, m, g->in_ptr, g->in_idx, node_dev, nslot, xptr,
                                            xcnt, xsrc, st);
  k_rx_rec<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, xptr, xsrc, wxa, cq, rec, wxc, st);
  CEL_HIP(hipGetLastError());
  RxArgs a{};
  a.n = n;
  a.D = D;
  a.nb = nb;
  a.cap = cap;
  a.off = off;
  a.wxa = wxa;
  a.wxc = wxc;
  a.rec = rec;
  a.xsrc = xsrc;
  a.gnode = gnode;
  a.finc = finc;
  a.tail = tail;
  a.bar = bar;
  a.start = start;
  a.finish = finish;
  a.makespan = makespan;
  {
    KTimer kt(s, "k_makespan_one");
    switch (ti) {
      case 0: k_rx_relax<1><<<G, kRxB, 0, s>>>(a, st); break;
      case 1: k_rx_relax<2><<<G, kRxB, 0, s>>>(a, st); break;
      case 2: k_rx_relax<3><<<G, kRxB, 0, s>>>(a, st); break;
      case 3: k_rx_relax<4><<<G, kRxB, 0, s>>>(a, st); break;
      case 4: k_rx_relax<5><<<G, kRxB, 0, s>>>(a, st); break;
      case 5: k_rx_relax<6><<<G, kRxB, 0, s>>>(a, st); break;
      default: k_rx_relax<8><<<G, kRxB, 0, s>>>(a, st); break;
    }
  }
  CEL_HIP(hipGetLastError());
  *launched = true;
  return CEL_OK;
}

}  // namespace cel
