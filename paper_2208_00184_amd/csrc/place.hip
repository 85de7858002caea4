// cel_place: coarse graph + Adjusting Placement (Section 5.2, eq. 7-9,
// Algorithm 2); also the Order-Place baseline (Sections 5.2, 6.2.2) and the
// CCR parts (Section 5.1.1, eq. 1) used to compare them.
//
// Coarse graph (data-parallel): cluster sums by atomics; every edge between
// two clusters is bucketed by its target cluster, each bucket sorted by
// (source cluster, edge id) and runs of equal source cluster summed, which
// gives each cluster its list of coarse in-edges (pred, comm) in a fixed order.
//
// Placement (sequential over clusters, as the algorithm is): one wave.  For
// cluster t, pre_t on device x is max over preds of Fin[p] + I(dev p != x)
// cc; it is evaluated for all devices at once from the largest Fin + cc over
// the preds, one device reaching it, and two more maxima (wave reductions
// over the preds, one per lane).  Lane x then finds the first-fit start on
// device x in that device's sorted list of busy blocks (touching intervals
// are merged, so the list holds one block per idle gap), and a wave
// reduction picks the device.
#include <type_traits>

#include "cel_internal.h"

namespace cel {

__global__ void k_place_nodes(int32_t n, int32_t C, const int32_t *cid, const int64_t *w,
                              const int64_t *mem, uint64_t *W, uint64_t *MEM, Status *st) {
  if (failed(st)) return;
  uint32_t bad = 0;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t c = cid[v];
    if (c < 0 || c >= C) {
      bad |= EB_ARG;
      continue;
    }
    atomicAdd((unsigned long long *)&W[c], (unsigned long long)w[v]);
    atomicAdd((unsigned long long *)&MEM[c], (unsigned long long)mem[v]);
  }
  if (bad) raise_err(st, bad);
}

// Edges between clusters, edge-balanced blocks.  PASS 0
// counts per target cluster (and checks cid[u] <= cid[v]); PASS 1 writes
// (source cluster, edge id) into the target's bucket and the edge's comm.
template <int PASS>
__global__ void k_place_edges(cel_graph g, int64_t bw, int64_t lat, const int32_t *cid,
                              int32_t *cnt, const int32_t *boff, uint64_t *keys, uint32_t *ids,
                              int64_t *ecost, Status *st) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  if (failed(st)) return;
  uint32_t bad = 0;
  for_edges_balanced(g.out_ptr, g.n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    const int32_t a = cid[u], b = cid[g.out_idx[e]];
    if (a == b) return;
    if (a > b) {
      bad |= EB_ORDER;
      return;
    }
    if (PASS == 0) {
      atomicAdd(&cnt[b], 1);
    } else {
      const int32_t slot = boff[b] + atomicAdd(&cnt[b], 1);
      keys[slot] = (uint64_t)a;
      ids[slot] = (uint32_t)e;
      ecost[e] = comm_of(g.ob[u], bw, lat);
    }
  });
  if (bad) raise_err(st, bad);
}

// Per target cluster (one wave each): sum runs of equal source cluster into
// coarse in-edges, written in order at the bucket's front, and raise the
// source's back_cost.  64 bucket entries at a time: run heads from the
// neighbouring key, a segmented sum over the wave, run tails compacted by a
// ballot; a run that reaches the end of a batch carries into the next.
__global__ void k_place_combine(int32_t C, const int32_t *boff, const uint64_t *keys,
                                const uint32_t *ids, const int64_t *ecost, int32_t *ca,
                                int64_t *cc, int32_t *ncp, uint64_t *back, const Status *st) {
  if (failed(st)) return;
  const int lane = threadIdx.x & 63;
  const uint64_t lt = (1ull << lane) - 1ull;
  const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t b = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6; b < C; b += nw) {
    const int32_t k0 = boff[b], k1 = boff[b + 1];
    int32_t out = k0;
    uint64_t ckey = ~0ull;  // run carried from the previous batch (none: ~0)
    int64_t csum = 0;
    for (int32_t base = k0; base < k1; base += 64) {
      const int32_t k = base + lane;
      const bool v = k < k1;
      const uint64_t key = v ? keys[k] : ~0ull;
      const int64_t c = v ? ecost[ids[k]] : 0;
      const uint64_t first = __shfl(key, 0);
      if (ckey != ~0ull && first != ckey) {  // the carried run ended with the last batch
        if (lane == 0) {
          ca[out] = (int32_t)ckey;
          cc[out] = csum;
          atomicMax((unsigned long long *)&back[ckey], (unsigned long long)csum);
        }
        out++;
        ckey = ~0ull;
        csum = 0;
      }
      const uint64_t prev = __shfl_up(key, 1);
      const uint64_t pk = lane == 0 ? ckey : prev;
      const int32_t head = v && key != pk;
      // segmented inclusive sum (segments start at heads)
      int64_t x = c;
      int32_t f = head;
      for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_up(x, d);
        const int32_t g = __shfl_up(f, d);
        if (lane >= d && !f) {
          x += y;
          f = g;
        }
      }
      if (!f) x += csum;  // still in the run carried into this batch
      const uint64_t next = __shfl_down(key, 1);
      const bool last_valid = k1 - base <= 64 ? lane == k1 - base - 1 : lane == 63;
      const bool more = k1 - base > 64;  // the batch's last run may continue
      const bool tail = v && (last_valid ? !more : next != key);
      const uint64_t tm = __ballot(tail);
      if (tail) {
        const int32_t o = out + __popcll(tm & lt);
        ca[o] = (int32_t)key;
        cc[o] = x;
        atomicMax((unsigned long long *)&back[key], (unsigned long long)x);
      }
      out += __popcll(tm);
      // carry: the run open at the end of the batch
      const int src = k1 - base < 64 ? k1 - base - 1 : 63;
      ckey = __shfl(key, src);
      const int64_t xs = __shfl(x, src);
      const bool open = more && !__shfl((int)tail, src);
      csum = open ? xs : 0;
      if (!open) ckey = ~0ull;
    }
    if (lane == 0) ncp[b] = out - k0;
  }
}

constexpr int kPlaceBlk = 5120;  // busy blocks held in LDS, shared evenly by the devices
constexpr int kPlaceLds = 8192;  // clusters whose Fin and device are kept in LDS too (155,648 B of LDS in all)

__device__ inline void argmax_i64(int64_t &v, int32_t &i) {  // wave: largest v, then smallest i
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t ov = __shfl_xor((long long)v, off);
    const int32_t oi = __shfl_xor(i, off);
    if (ov > v || (ov == v && oi < i)) {
      v = ov;
      i = oi;
    }
  }
}

// Number of blocks of a sorted busy list (ends xf[0..nb)) that end at or
// before s, searched from the end: ready times mostly fall near the end of
// the list, so a galloping step back brackets them in a few reads.
__device__ inline int32_t blocks_ending_by(const int64_t *xf, int32_t nb, int64_t s) {
  int32_t hi = nb, step = 1;
  while (hi > 0 && xf[hi - 1] > s) {  // xf[hi - 1] > s: the answer is below hi
    const int32_t lo = hi - step > 0 ? hi - step : 0;
    if (xf[lo] <= s) {  // answer in (lo, hi): binary search
      int32_t a = lo + 1, b = hi - 1;  // first index in [a, b] ending after s, else b + 1
      while (a <= b) {
        const int32_t mid = (a + b) >> 1;
        if (xf[mid] <= s) a = mid + 1;
        else b = mid - 1;
      }
      return a;
    }
    hi = lo;
    step <<= 1;
  }
  return hi;
}

// Inserts [s0, f) into a sorted list of merged busy blocks (xs, xf, nb of
// them, room for cap): touching blocks merge, so the list keeps one block
// per idle gap.  Returns the end of the last block.
__device__ inline int64_t busy_insert(int64_t *xs, int64_t *xf, int32_t &nb, int32_t cap,
                                      int64_t s0, int64_t f, Status *st) {
  const int32_t k = blocks_ending_by(xf, nb, s0);
  const bool left = k > 0 && xf[k - 1] == s0;
  const bool right = k < nb && xs[k] == f;
  if (left && right) {
    xf[k - 1] = xf[k];
    for (int32_t q = k; q + 1 < nb; q++) {
      xs[q] = xs[q + 1];
      xf[q] = xf[q + 1];
    }
    nb--;
  } else if (left) {
    xf[k - 1] = f;
  } else if (right) {
    xs[k] = s0;
  } else if (nb < cap) {
    for (int32_t q = nb; q > k; q--) {
      xs[q] = xs[q - 1];
      xf[q] = xf[q - 1];
    }
    xs[k] = s0;
    xf[k] = f;
    nb++;
  } else {
    raise_err(st, EB_ARG);  // cannot happen: the list moves out of LDS when full
  }
  return nb > 0 ? xf[nb - 1] : 0;
}

// Wave reductions for the placement: the largest of the lanes' non-negative
// values below 2^62 (max_nonneg: such bit patterns order as doubles), by DPP
// row shifts and broadcasts with zero fill (0 is the identity, so no lane
// needs an initial value) and one v_max_f64 per step.  Lane 63, or lane 15
// for lanes 0-15 only, ends with the result; lanes outside the chain that
// feeds it may hold anything.
template <int CTRL, int ROWMASK>
__device__ inline int64_t dpp64z(int64_t v) {
  const int32_t lo = __builtin_amdgcn_mov_dpp((int32_t)v, CTRL, ROWMASK, 0xF, true);
  const int32_t hi = __builtin_amdgcn_mov_dpp((int32_t)(v >> 32), CTRL, ROWMASK, 0xF, true);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
template <bool ALL>
__device__ inline int64_t wave_max_nonneg(int64_t y) {
  y = max_nonneg(y, dpp64z<0x111, 0xF>(y));  // row_shr:1
  y = max_nonneg(y, dpp64z<0x112, 0xF>(y));  // row_shr:2
  y = max_nonneg(y, dpp64z<0x114, 0xF>(y));  // row_shr:4
  y = max_nonneg(y, dpp64z<0x118, 0xF>(y));  // row_shr:8
  if (!ALL) return readlane64(y, 15);
  y = max_nonneg(y, dpp64z<0x142, 0xA>(y));  // row_bcast:15 into rows 1 and 3
  y = max_nonneg(y, dpp64z<0x143, 0xC>(y));  // row_bcast:31 into rows 2 and 3
  return readlane64(y, 63);
}
// two at once (independent chains, interleaved)
__device__ inline void wave_max_nonneg2(int64_t &y, int64_t &z) {
  y = max_nonneg(y, dpp64z<0x111, 0xF>(y));
  z = max_nonneg(z, dpp64z<0x111, 0xF>(z));
  y = max_nonneg(y, dpp64z<0x112, 0xF>(y));
  z = max_nonneg(z, dpp64z<0x112, 0xF>(z));
  y = max_nonneg(y, dpp64z<0x114, 0xF>(y));
  z = max_nonneg(z, dpp64z<0x114, 0xF>(z));
  y = max_nonneg(y, dpp64z<0x118, 0xF>(y));
  z = max_nonneg(z, dpp64z<0x118, 0xF>(z));
  y = max_nonneg(y, dpp64z<0x142, 0xA>(y));
  z = max_nonneg(z, dpp64z<0x142, 0xA>(z));
  y = max_nonneg(y, dpp64z<0x143, 0xC>(y));
  z = max_nonneg(z, dpp64z<0x143, 0xC>(z));
  y = readlane64(y, 63);
  z = readlane64(z, 63);
}
constexpr int64_t kPlaceFull = int64_t(1) << 62;  // EST of a device without room
constexpr int kPlaceQ = 4;                        // preds per lane held in registers
constexpr int kPlacePad = 64 * kPlaceQ;           // entries read past the end of a pred list

// Placement, one wave (its LDS accesses are in program order, so no barrier
// is needed).  For cluster t, pre_t on device x is the largest of 0, Fin[p]
// over preds p on x and Fin[p] + cc over preds on other devices.  With m1 the
// largest Fin + cc over all preds and d1 the device of one pred reaching it,
// every device other than d1 has pre_t = m1 (a pred's Fin never exceeds its
// Fin + cc); d1 itself takes the larger of m2, the largest Fin + cc over
// preds on other devices, and g, the largest Fin over its own preds.  So one
// pass over the preds, kPQ per lane, and three wave reductions give every
// device's pre_t; device x's free memory and busy-list state sit in the
// registers of lane x mod 64, so each lane then finds its device's first-fit
// start and EST (eq. 7) and a wave reduction the smallest EST.  Each device's
// busy list (merged intervals: one block per idle gap) lives in LDS
// (kPlaceBlk / D blocks) until it outgrows that share; it then moves to its
// global list.  A start at or after the list's last end (the usual case)
// extends or appends without reading the list.
//
// A step's only memory round trips are LDS ones: the preds of the cluster
// two steps ahead are loaded into registers at the end of a step (two
// register sets, the loop unrolled by two, and the sizes of 64 clusters moved
// between register blocks only between blocks of 64 steps, so no register
// copy waits for a load in flight: a wait for the vector memory counter waits
// for every load and store issued before it), and with LDSF every cluster's
// Fin and device stay in LDS (C <= kPlaceLds) and go to global memory after
// the loop.  GL = false keeps every busy list in LDS and takes at most 64 kPQ
// preds per cluster, so that a step issues no global memory access at all;
// a list that outgrows its share, or a longer pred list, stops the kernel
// with st->i1 = 1, and the caller runs the GL = true kernel, whose lists move
// to global memory when full and whose long pred lists are read in passes.
template <bool LDSF, bool GL, int NI>  // NI: devices per lane (D <= 64 NI)
__global__ void __launch_bounds__(64)
    k_place(int32_t C, int32_t D, const int64_t *cap, const uint64_t *W, const uint64_t *MEM,
            const int32_t *boff, const int32_t *ncp, const int32_t *ca, const int64_t *cc,
            const uint64_t *back, uint8_t *cdev, int64_t *Fin, int64_t *bs, int64_t *bf,
            int32_t bcap, Status *st) {
  __shared__ int64_t s_bs[kPlaceBlk], s_bf[kPlaceBlk];
  __shared__ int64_t s_fin[LDSF ? kPlaceLds : 1];
  __shared__ uint8_t s_cd[LDSF ? kPlaceLds : 1];
  if (failed(st)) return;
  const int lane = threadIdx.x;
  const int32_t capL = kPlaceBlk / D;
  int64_t ava[NI], last[NI];  // device lane + 64 i: free memory, end of its last busy block
  int32_t nbl[NI], glob[NI];  // its busy-block count; list moved to global memory
#pragma unroll
  for (int i = 0; i < NI; i++) {
    const int x = lane + 64 * i;
    ava[i] = x < D ? cap[x] : 0;
    last[i] = 0;
    nbl[i] = 0;
    glob[i] = 0;
  }
  int32_t prev = 0, be = 0;
  int64_t span = 0;
  // The sizes of 64 clusters at a time, one per lane, a block of 64 ahead
  // (read back with readlane).  Loads here are never predicated (indexes are
  // clamped instead), so each goes straight into the register that keeps it
  // and nothing waits for it before its use.
  constexpr int kPQ = kPlaceQ;
  auto bulk = [&](int32_t t0, int32_t &zb, int32_t &zn, int64_t &zw, int64_t &zm, int64_t &zk) {
    const int32_t t = t0 + lane < C ? t0 + lane : C - 1;  // past C: never read
    zb = boff[t];
    zn = ncp[t];
    zw = (int64_t)W[t];
    zm = (int64_t)MEM[t];
    zk = (int64_t)back[t];
  };
  int32_t ub, un, vb, vn;  // sizes of clusters [T, T + 64) (u*) and [T + 64, T + 128) (v*)
  int64_t uw, um, uk, vw, vm, vk;
  bulk(0, ub, un, uw, um, uk);
  bulk(64, vb, vn, vw, vm, vk);
  // preds 64 q + lane of the cluster t' in the block of ub (lane t' & 63);
  // lanes past its count read on into the next clusters' lists (the lists
  // are allocated with 64 kPQ entries to spare), and the step masks them.
  // Past C the sizes repeat cluster C - 1's, so no call is ever skipped: a
  // load that may or may not have been issued makes later waits for earlier
  // loads wait for it too.  Only ub is read here, never the block in flight.
  auto preds = [&](int32_t tp, int32_t (&pa)[kPQ], int64_t (&pc)[kPQ]) {
    const int32_t k = __builtin_amdgcn_readlane(ub, tp & 63) + lane;
#pragma unroll
    for (int q = 0; q < kPQ; q++) {
      pa[q] = ca[k + 64 * q];
      pc[q] = cc[k + 64 * q];
    }
  };
  // Fin and device of pred cluster a (every lane that has one)
  auto fin_dev = [&](int32_t a, int64_t &f, int32_t &d) {
    f = LDSF ? s_fin[a] : Fin[a];
    d = LDSF ? s_cd[a] : cdev[a];
  };
  // first-fit start on device x (lane x mod 64) at or after sv for a cluster
  // of length Wt, in a list held in LDS (GL = false) or in global memory
  auto first_fit = [&](const int64_t *xs, const int64_t *xf, int32_t nb, int64_t sv, int64_t Wt) {
    for (int32_t k = blocks_ending_by(xf, nb, sv); k < nb && xs[k] < sv + Wt; k++) sv = xf[k];
    return sv;
  };
  // one cluster; false when the kernel has to stop (GL = false, a full list)
  auto step = [&](int32_t t, const int32_t (&pa)[kPQ], const int64_t (&pcv)[kPQ]) -> bool {
    const int l = t & 63;
    const int32_t b0 = __builtin_amdgcn_readlane(ub, l), np = __builtin_amdgcn_readlane(un, l);
    const int64_t Wt = readlane64(uw, l), Mt = readlane64(um, l), bk = readlane64(uk, l);
    // ---- pre_t by device: m1, d1, m2, g over the preds (0 when none)
    int64_t m1 = 0, m2 = 0, g = 0;
    int32_t d1 = -1;
    // one chunk (np <= 64: most clusters) or kPQ of them, in registers
    auto in_regs = [&](auto nq) {
      constexpr int NQ = decltype(nq)::value;
      int64_t f[NQ], fc[NQ];
      int32_t d[NQ];
#pragma unroll
      for (int q = 0; q < NQ; q++)  // every lane loads (pred 0 past np), then masks
        fin_dev(64 * q + lane < np ? pa[q] : 0, f[q], d[q]);
      int64_t bfc = 0;
      int32_t bd = 255;
#pragma unroll
      for (int q = 0; q < NQ; q++) {
        const bool in = 64 * q + lane < np;
        f[q] = in ? f[q] : 0;
        d[q] = in ? d[q] : 255;  // no device
        fc[q] = in ? f[q] + pcv[q] : 0;
        if (fc[q] > bfc) {
          bfc = fc[q];
          bd = d[q];
        }
      }
      m1 = wave_max_nonneg<true>(bfc);
      if (m1 > 0) {
        d1 = __builtin_amdgcn_readlane(bd, (int)__builtin_ctzll(__ballot(bfc == m1)));
        int64_t y = 0, z = 0;
#pragma unroll
        for (int q = 0; q < NQ; q++) {
          if (d[q] != d1 && fc[q] > y) y = fc[q];
          if (d[q] == d1 && f[q] > z) z = f[q];
        }
        wave_max_nonneg2(y, z);
        m2 = y;
        g = z;
      }
    };
    if (np > 0 && np <= 64) {
      in_regs(std::integral_constant<int, 1>());
    } else if (np > 0 && np <= 64 * kPQ) {
      in_regs(std::integral_constant<int, kPQ>());
    } else if (!GL && np > 0) {
      return false;  // long pred list: the caller runs the GL = true kernel
    } else if (GL && np > 0) {  // long pred lists: two passes over them, 64 at a time
      int64_t bfc = 0;
      int32_t bd = 255;
      for (int32_t k0 = 0; k0 < np; k0 += 64) {
        if (k0 + lane < np) {
          int64_t f;
          int32_t d;
          fin_dev(ca[b0 + k0 + lane], f, d);
          const int64_t fc = f + cc[b0 + k0 + lane];
          if (fc > bfc) {
            bfc = fc;
            bd = d;
          }
        }
      }
      m1 = wave_max_nonneg<true>(bfc);
      if (m1 > 0) {
        d1 = __builtin_amdgcn_readlane(bd, (int)__builtin_ctzll(__ballot(bfc == m1)));
        int64_t y = 0, z = 0;
        for (int32_t k0 = 0; k0 < np; k0 += 64) {
          if (k0 + lane < np) {
            int64_t f;
            int32_t d;
            fin_dev(ca[b0 + k0 + lane], f, d);
            const int64_t fc = f + cc[b0 + k0 + lane];
            if (d != d1 && fc > y) y = fc;
            if (d == d1 && f > z) z = f;
          }
        }
        wave_max_nonneg2(y, z);
        m2 = y;
        g = z;
      }
    }
    const int64_t pre1 = m2 > g ? m2 : g;  // pre_t on d1
    // ---- device x: first-fit start and EST (eq. 7); kPlaceFull without room
    int64_t slot[NI], est[NI];
#pragma unroll
    for (int i = 0; i < NI; i++) {
      slot[i] = 0;
      est[i] = kPlaceFull;
      const int x = lane + 64 * i;
      if (x < D) {
        int64_t sv = x == d1 ? pre1 : m1;
        const int32_t nb = nbl[i];
        if (Wt > 0 && nb > 0 && sv < last[i]) {
          if (!GL || !glob[i])
            sv = first_fit(s_bs + x * capL, s_bf + x * capL, nb, sv, Wt);
          else
            sv = first_fit(bs + (int64_t)x * bcap, bf + (int64_t)x * bcap, nb, sv, Wt);
        }
        slot[i] = sv;
        est[i] = ava[i] < Mt ? kPlaceFull : sv;
      }
    }
    // ---- device of smallest EST (lowest id on ties): the largest
    // kPlaceFull - EST, so that the reduction's identity is 0
    int64_t e = kPlaceFull - est[0];
#pragma unroll
    for (int i = 1; i < NI; i++) e = max_nonneg(e, kPlaceFull - est[i]);
    const int64_t ev = kPlaceFull - (D <= 16 ? wave_max_nonneg<false>(e) : wave_max_nonneg<true>(e));
    int32_t ei = 0;
    if (ev < kPlaceFull) {
#pragma unroll
      for (int i = NI - 1; i >= 0; i--) {  // the lowest i with a hit, then its lowest lane
        const uint64_t hit = __ballot(est[i] == ev);
        if (hit) ei = 64 * i + (int32_t)__builtin_ctzll(hit);
      }
    }
    // ---- the choice (eq. 8-9), uniform over the wave
    const int32_t dk = t == 0 ? 0 : prev;
    int64_t edk = kPlaceFull;
#pragma unroll
    for (int i = 0; i < NI; i++)
      if (i == (dk >> 6)) edk = readlane64(est[i], dk & 63);
    int32_t pick;
    if (ev >= kPlaceFull) {  // every device full: most remaining memory (best effort)
      int64_t av = INT64_MIN;  // free memory can be negative after best-effort picks
      int32_t ai = INT32_MAX;
#pragma unroll
      for (int i = 0; i < NI; i++)
        if (lane + 64 * i < D && ava[i] > av) {
          av = ava[i];
          ai = lane + 64 * i;
        }
      argmax_i64(av, ai);
      pick = ai;
      be++;
    } else if (edk >= kPlaceFull || edk - ev > bk) {
      pick = ei;
    } else {
      pick = dk;
    }
    const int ip = pick >> 6, lp = pick & 63;
    int64_t slp = 0, lst = 0;
    int32_t nb = 0, gl = 0;
#pragma unroll
    for (int i = 0; i < NI; i++)
      if (i == ip) {
        slp = slot[i];
        lst = last[i];
        nb = nbl[i];
        gl = glob[i];
      }
    const int64_t s0 = readlane64(slp, lp), f = s0 + Wt;
    const int64_t lastp = readlane64(lst, lp);
    nb = __builtin_amdgcn_readlane(nb, lp);
    gl = __builtin_amdgcn_readlane(gl, lp);
    span = f > span ? f : span;
    prev = pick;
    if (Wt > 0) {  // insert [s0, f) into the device's merged busy blocks
      int64_t lastv = lastp;
      if (nb > 0 && s0 == lastp) {  // touches the last block: extend it
        if (lane == 0) {
          if (!GL || !gl) s_bf[pick * capL + nb - 1] = f;
          else bf[(int64_t)pick * bcap + nb - 1] = f;
        }
        lastv = f;
      } else {
        if (!gl && nb == capL) {  // the LDS share is full
          if (!GL) return false;  // stop: the caller runs the GL = true kernel
          for (int32_t q = lane; q < nb; q += 64) {  // move the list out
            bs[(int64_t)pick * bcap + q] = s_bs[pick * capL + q];
            bf[(int64_t)pick * bcap + q] = s_bf[pick * capL + q];
          }
          gl = 1;
        }
        if (nb == 0 || s0 > lastp) {  // after the last block: a new block at the end
          if (lane == 0) {
            if (!GL || !gl) {
              s_bs[pick * capL + nb] = s0;
              s_bf[pick * capL + nb] = f;
            } else {
              bs[(int64_t)pick * bcap + nb] = s0;
              bf[(int64_t)pick * bcap + nb] = f;
            }
          }
          nb++;
          lastv = f;
        } else {  // into an idle gap
          if (lane == 0) {
            if (!GL || !gl)
              lastv = busy_insert(s_bs + pick * capL, s_bf + pick * capL, nb, capL, s0, f, st);
            else
              lastv = busy_insert(bs + (int64_t)pick * bcap, bf + (int64_t)pick * bcap, nb, bcap,
                                  s0, f, st);
          }
          nb = __builtin_amdgcn_readlane(nb, 0);
          lastv = readlane64(lastv, 0);
        }
      }
#pragma unroll
      for (int i = 0; i < NI; i++)
        if (i == ip && lane == lp) {
          nbl[i] = nb;
          last[i] = lastv;
          glob[i] = gl;
        }
    }
#pragma unroll
    for (int i = 0; i < NI; i++)
      if (i == ip && lane == lp) ava[i] -= Mt;
    if (lane == 0) {  // later steps of this wave read these back, in program order
      if (LDSF) {
        s_fin[t] = f;
        s_cd[t] = (uint8_t)pick;
      } else {
        cdev[t] = (uint8_t)pick;
        Fin[t] = f;
      }
    }
    return true;
  };
  int32_t pa0[kPQ], pa1[kPQ];
  int64_t pc0[kPQ], pc1[kPQ];
  preds(0, pa0, pc0);
  preds(1, pa1, pc1);
  bool ok = true;
  for (int32_t T = 0; T < C && ok; T += 64) {  // blocks of 64 clusters: ub / vb hold T, T + 64
    const int32_t te = T + 64 < C ? T + 64 : C;
    int32_t t = T;  // even: pa0 holds cluster t, pa1 cluster t + 1
    for (; t + 2 < T + 64 && t < te; t += 2) {  // the next pair in this block too
      if (!step(t, pa0, pc0)) {
        ok = false;
        break;
      }
      preds(t + 2, pa0, pc0);  // a whole step before its use
      if (t + 1 < te && !step(t + 1, pa1, pc1)) {
        ok = false;
        break;
      }
      preds(t + 3, pa1, pc1);
    }
    if (ok && t < te) ok = step(t, pa0, pc0) && (t + 1 >= te || step(t + 1, pa1, pc1));
    ub = vb;
    un = vn;
    uw = vw;
    um = vm;
    uk = vk;
    bulk(T + 128, vb, vn, vw, vm, vk);
    preds(T + 64, pa0, pc0);  // from the new ub (past C: cluster C - 1's sizes)
    preds(T + 65, pa1, pc1);
  }
  if (!ok) {  // a busy list outgrew its LDS share, or a long pred list (GL = false)
    if (lane == 0) st->i1 = 1;
    return;
  }
  if (LDSF) {  // every cluster's Fin and device, from LDS
    for (int32_t t = lane; t < C; t += 64) {
      Fin[t] = s_fin[t];
      cdev[t] = s_cd[t];
    }
  }
  if (lane == 0) {
    st->s0 = span;
    st->i0 = be;
  }
}

// ----------------------------------- extended placement: devices, links, groups
//
// Algorithm 2 with per-device cluster durations, per-link coarse-edge costs
// and co-location groups (cel_place_ext).  Cluster t's duration on device x
// is the sum of its members' durations there; devices are compared on the
// earliest finish time (start + duration: the order of eq. 7's start times
// when devices are identical).  Under link tables a coarse edge (OB = summed
// ob of its N member edges) costs ceil(OB / bw[y][x]) + N lat[y][x] on the
// link y -> x: in pre_t from each predecessor's device, in back_cost (eq. 8)
// on the link from the best device back to the previous cluster's.  A group
// follows its smallest cluster; its other members' memory is charged to that
// cluster's device when their own cluster is placed.

__device__ inline int64_t dur_tm(int64_t w, int64_t tm) {  // ceil(w * tm / 1024)
  return (w >> 10) * tm + (((w & 1023) * tm + 1023) >> 10);
}

// Per node: the cluster's duration on every device (atomics into W2[t][x]),
// its own memory (followers excluded) and follower counts per cluster.
__global__ void k_pe_nodes(int32_t n, int32_t C, int32_t D, const int32_t *cid, const int64_t *w,
                           const int64_t *mem, const int32_t *group, const int32_t *lead,
                           const int64_t *tmul, uint64_t *W2, uint64_t *MEMo, int32_t *fcnt,
                           Status *st) {
  if (failed(st)) return;
  uint32_t bad = 0;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t c = cid[v];
    if (c < 0 || c >= C) {
      bad |= EB_ARG;
      continue;
    }
    const int64_t wv = w[v];
    for (int32_t x = 0; x < D; x++)
      atomicAdd((unsigned long long *)&W2[(int64_t)c * D + x],
                (unsigned long long)(tmul ? dur_tm(wv, tmul[x]) : wv));
    const int32_t gv = group ? group[v] : -1;
    if (gv >= 0 && lead[gv] < c) atomicAdd(&fcnt[c], 1);
    else atomicAdd((unsigned long long *)&MEMo[c], (unsigned long long)mem[v]);
  }
  if (bad) raise_err(st, bad);
}

// Follower entries (leading cluster, mem) in their own cluster's slice.
__global__ void k_pe_followers(int32_t n, const int32_t *cid, const int64_t *mem,
                               const int32_t *group, const int32_t *lead, const int32_t *foff,
                               int32_t *fill, int32_t *fl, int64_t *fm, const Status *st) {
  if (failed(st)) return;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t gv = group[v], c = cid[v];
    if (gv < 0 || lead[gv] >= c) continue;
    const int32_t k = foff[c] + atomicAdd(&fill[c], 1);
    fl[k] = lead[gv];
    fm[k] = mem[v];
  }
}

// Per edge id: the source's output bytes and a count of one (summed per
// coarse edge by k_place_combine into OB and N).
__global__ void k_pe_edge_ob(cel_graph g, int64_t *eob, int64_t *eone, const Status *st) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  if (failed(st)) return;
  for_edges_balanced(g.out_ptr, g.n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    eob[e] = g.ob[u];
    eone[e] = 1;
  });
}

// Successor lists of the coarse graph (by source cluster) from the
// predecessor buckets: PASS 0 counts, PASS 1 writes (OB, N).
template <int PASS>
__global__ void k_pe_succ(int32_t C, const int32_t *boff, const int32_t *ncp, const int32_t *ca,
                          const int64_t *cob, const int64_t *cnum, int32_t *scnt,
                          const int32_t *soff, int64_t *sob, int64_t *snum, const Status *st) {
  if (failed(st)) return;
  for (int64_t b = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; b < C;
       b += (int64_t)gridDim.x * blockDim.x) {
    for (int32_t k = boff[b]; k < boff[b] + ncp[b]; k++) {
      const int32_t a = ca[k];
      if (PASS == 0) {
        atomicAdd(&scnt[a], 1);
      } else {
        const int32_t q = soff[a] + atomicAdd(&scnt[a], 1);
        sob[q] = cob[k];
        snum[q] = cnum[k];
      }
    }
  }
}

struct PeArgs {
  int32_t C, D;
  bool links;                      // per-link tables given
  const int64_t *cap;              // [D]
  const uint64_t *W2, *MEMo;       // [C][D] durations, [C] own memory
  const int32_t *boff, *ncp, *ca;  // coarse in-edges (bucket start, count, source)
  const int64_t *cc, *cob, *cnum;  // their summed c, ob and member count
  const uint64_t *back;            // max summed c over out-edges (no link tables)
  const int32_t *soff;             // [C + 1] out-edges (link tables): OB, N
  const int64_t *sob, *snum;
  const int32_t *foff, *fl;        // [C + 1] followers: leading cluster, memory
  const int64_t *fm;
  const int64_t *lbw, *llat;       // [D][D] link tables
  uint8_t *cdev;
  int64_t *Fin, *bs, *bf;          // busy lists [D][bcap]
  int32_t bcap;
};

constexpr int kPeLds = 8192;  // clusters whose Fin and device stay in LDS too

__device__ inline int64_t link_cost(int64_t ob, int64_t cnt, int32_t bw, int32_t lat) {
  return (int64_t)(((uint64_t)ob + (uint64_t)bw - 1) / (uint64_t)bw) + cnt * lat;
}

// One wave; device x's free memory, busy-list size and last end sit in lane
// x (D <= 64), its busy blocks in its global list, which only lane x reads
// and writes.
template <bool LDSF>
__global__ void __launch_bounds__(64) k_place_ext(PeArgs a, Status *st) {
  __shared__ int32_t s_bw[64 * 64], s_lat[64 * 64];
  __shared__ int64_t s_fin[LDSF ? kPeLds : 1];
  __shared__ uint8_t s_cd[LDSF ? kPeLds : 1];
  if (failed(st)) return;
  const int lane = threadIdx.x;
  const int32_t C = a.C, D = a.D;
  const bool mine = lane < D;
  if (a.links)
    for (int i = lane; i < D * D; i += 64) {
      s_bw[i] = (int32_t)a.lbw[i];
      s_lat[i] = (int32_t)a.llat[i];
    }
  lds_order();
  wave_lds_sync();
  int64_t ava = mine ? a.cap[lane] : 0;
  int32_t nb = 0;
  int64_t lastb = 0;
  int64_t *xs = a.bs + (int64_t)(mine ? lane : 0) * a.bcap, *xf = a.bf + (int64_t)(mine ? lane : 0) * a.bcap;
  int32_t prev = 0, be = 0;
  int64_t span = 0;
  auto finof = [&](int32_t c) -> int64_t { return LDSF ? s_fin[c] : a.Fin[c]; };
  auto devof = [&](int32_t c) -> int32_t { return LDSF ? (int32_t)s_cd[c] : (int32_t)a.cdev[c]; };
  for (int32_t t = 0; t < C; t++) {
    // followers of earlier groups: their memory on their leading device
    const int32_t f0 = a.foff[t], f1 = a.foff[t + 1];
    for (int32_t k0 = f0; k0 < f1; k0 += 64) {
      const int32_t k = k0 + lane;
      int32_t fd = -1;
      int64_t fmv = 0;
      if (k < f1) {
        fd = devof(a.fl[k]);
        fmv = a.fm[k];
      }
      const int nk = f1 - k0 < 64 ? f1 - k0 : 64;
      for (int j = 0; j < nk; j++) {
        const int32_t dj = __builtin_amdgcn_readlane(fd, j);
        const int64_t mj = readlane64(fmv, j);
        if (lane == dj) ava -= mj;
      }
    }
    const int64_t Mt = (int64_t)a.MEMo[t];
    const int64_t Wx = mine ? (int64_t)a.W2[(int64_t)t * D + lane] : 0;
    // pre_t on device `lane` (eq. 7)
    int64_t pre = 0;
    const int32_t b0 = a.boff[t], np = a.ncp[t];
    for (int32_t k0 = 0; k0 < np; k0 += 64) {
      const int32_t k = k0 + lane;
      int64_t pf = 0, pc = 0, po = 0, pn = 0;
      int32_t pd = 0;
      if (k < np) {
        const int32_t pa = a.ca[b0 + k];
        pf = finof(pa);
        pd = devof(pa);
        pc = a.cc[b0 + k];
        if (a.links) {
          po = a.cob[b0 + k];
          pn = a.cnum[b0 + k];
        }
      }
      const int nk = np - k0 < 64 ? np - k0 : 64;
      for (int j = 0; j < nk; j++) {
        const int64_t fj = readlane64(pf, j);
        const int32_t dj = __builtin_amdgcn_readlane(pd, j);
        int64_t cost = 0;
        if (dj != lane) {
          if (a.links)
            cost = link_cost(readlane64(po, j), readlane64(pn, j), s_bw[dj * D + (mine ? lane : 0)],
                             s_lat[dj * D + (mine ? lane : 0)]);
          else
            cost = readlane64(pc, j);
        }
        pre = fj + cost > pre ? fj + cost : pre;
      }
    }
    // first fit on device `lane`
    int64_t sv = pre;
    if (mine && Wx > 0 && nb > 0 && sv < lastb)
      for (int32_t q = blocks_ending_by(xf, nb, sv); q < nb && xs[q] < sv + Wx; q++) sv = xf[q];
    const int64_t eft = (mine && ava >= Mt) ? sv + Wx : kInf;
    // best device (lowest id on ties)
    int64_t ev = eft;
    int32_t ei = lane;
    for (int off = 32; off > 0; off >>= 1) {
      const int64_t ov = __shfl_xor((long long)ev, off);
      const int32_t oi = __shfl_xor(ei, off);
      if (ov < ev || (ov == ev && oi < ei)) {
        ev = ov;
        ei = oi;
      }
    }
    const int32_t dk = t == 0 ? 0 : prev;
    const int64_t edk = readlane64(eft, dk);
    int32_t pick;
    if (ev == kInf) {  // every device full: most remaining memory (best effort)
      int64_t av = mine ? ava : INT64_MIN;
      int32_t ai = mine ? lane : INT32_MAX;
      argmax_i64(av, ai);
      pick = ai;
      be++;
    } else if (edk == kInf || ei == dk) {
      pick = ei;
    } else {
      int64_t bk = 0;  // back_cost (eq. 8)
      if (!a.links) {
        bk = (int64_t)a.back[t];
      } else {
        const int32_t bw = s_bw[ei * D + dk], lt = s_lat[ei * D + dk];
        for (int32_t k = a.soff[t] + lane; k < a.soff[t + 1]; k += 64) {
          const int64_t c = link_cost(a.sob[k], a.snum[k], bw, lt);
          bk = c > bk ? c : bk;
        }
        for (int off = 32; off > 0; off >>= 1) {
          const int64_t o = __shfl_xor((long long)bk, off);
          bk = o > bk ? o : bk;
        }
      }
      pick = edk - ev > bk ? ei : dk;
    }
    const int64_t s0 = readlane64(sv, pick), wp = readlane64(Wx, pick), f = s0 + wp;
    span = f > span ? f : span;
    prev = pick;
    if (lane == pick) {
      if (wp > 0) lastb = busy_insert(xs, xf, nb, a.bcap, s0, f, st);
      ava -= Mt;
    }
    if (lane == 0) {  // later steps of this wave read these back, in program order
      a.cdev[t] = (uint8_t)pick;
      a.Fin[t] = f;
      if (LDSF) {
        s_fin[t] = f;
        s_cd[t] = (uint8_t)pick;
      }
    }
    if (LDSF) lds_order();
  }
  if (lane == 0) {
    st->s0 = span;
    st->i0 = be;
  }
}

// node_dev: a group member takes its leading cluster's device, every other
// node its own cluster's; cluster finish times out.
__global__ void k_pe_out(int32_t n, int32_t C, const int32_t *cid, const int32_t *group,
                         const int32_t *lead, const uint8_t *cdev, uint8_t *node_dev,
                         const int64_t *Fin, int64_t *fin_out, const Status *st) {
  if (failed(st)) return;
  const int64_t tot = n > C ? n : C;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < tot;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i < n) {
      const int32_t gv = group ? group[i] : -1;
      node_dev[i] = cdev[gv >= 0 ? lead[gv] : cid[i]];
    }
    if (fin_out && i < C) fin_out[i] = Fin[i];
  }
}

__global__ void k_place_out(int32_t n, int32_t C, const int32_t *cid, const uint8_t *cdev,
                            uint8_t *node_dev, const int64_t *Fin, int64_t *fin_out,
                            const Status *st) {
  if (failed(st)) return;
  const int64_t tot = n > C ? n : C;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < tot;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i < n) node_dev[i] = cdev[cid[i]];
    if (fin_out && i < C) fin_out[i] = Fin[i];
  }
}

// CCR parts (Section 5.1.1, eq. 1): the comm of the edges (only between clusters when cid is
// given) and the total compute; edge-balanced blocks, block sums in LDS, one
// atomic per block.
__global__ void k_comm_sums(cel_graph g, int64_t bw, int64_t lat, const int32_t *cid,
                            unsigned long long *sums, const Status *st) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  __shared__ unsigned long long s_e, s_w;
  if (failed(st)) return;
  if (threadIdx.x == 0) s_e = s_w = 0;
  __syncthreads();
  unsigned long long ec = 0, ws = 0;
  for_edges_balanced(g.out_ptr, g.n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    if (!cid || cid[u] != cid[g.out_idx[e]]) ec += (unsigned long long)comm_of(g.ob[u], bw, lat);
  });
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < g.n;
       v += (int64_t)gridDim.x * blockDim.x)
    ws += (unsigned long long)g.w[v];
  if (ec) atomicAdd(&s_e, ec);
  if (ws) atomicAdd(&s_w, ws);
  __syncthreads();
  if (threadIdx.x == 0) {
    atomicAdd(&sums[0], s_e);
    atomicAdd(&sums[1], s_w);
  }
}

// Order-Place (the baseline of Sections 5.2, 6.2.2): clusters in index order fill one
// device until the next cluster does not fit its remaining memory, then the
// next device; the last device takes the rest (best effort, counted).  One
// wave: the fill state is uniform, cluster sizes come 64 at a time.
__global__ void __launch_bounds__(64)
    k_order_place(int32_t C, int32_t D, const int64_t *cap, const uint64_t *MEM, uint8_t *cdev,
                  Status *st) {
  if (failed(st)) return;
  const int lane = threadIdx.x;
  int32_t dev = 0, be = 0;
  int64_t used = 0, capd = cap[0];
  for (int32_t t0 = 0; t0 < C; t0 += 64) {
    const int64_t mv = t0 + lane < C ? (int64_t)MEM[t0 + lane] : 0;
    const int nt = C - t0 < 64 ? C - t0 : 64;
    int32_t mine = 0;
    for (int l = 0; l < nt; l++) {
      const int64_t mt = readlane64(mv, l);
      while (used + mt > capd && dev + 1 < D) {  // full: the next device
        dev++;
        used = 0;
        capd = cap[dev];
      }
      if (used + mt > capd) be++;  // the last device, over its cap
      used += mt;
      if (lane == l) mine = dev;
    }
    if (t0 + lane < C) cdev[t0 + lane] = (uint8_t)mine;
  }
  if (lane == 0) st->i0 = be;
}

}  // namespace cel

using namespace cel;

extern "C" int cel_place(const cel_graph *g, const cel_devices *d, const int32_t *cluster_id,
                         int32_t C, uint8_t *cluster_dev, uint8_t *node_dev,
                         int64_t *cluster_fin, int64_t *coarse_makespan,
                         int32_t *best_effort_count, hipStream_t s) {
  const char *fn = "cel_place";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n;
  if (!coarse_makespan || !best_effort_count || (n > 0 && (!cluster_id || !node_dev)) ||
      (C > 0 && !cluster_dev))
    return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  if (C < 0 || (n > 0 && C < 1) || C > (n > 0 ? n : 0))
    return set_error(CEL_E_ARG, "%s: n_clusters = %d out of range", fn, C);
  const int64_t bcap = C;
  if ((int64_t)d->D * bcap > (int64_t)1 << 28)
    return set_error(CEL_E_NOMEM, "%s: D * n_clusters too large for the busy lists", fn);
  Scratch sc(s);
  Status *st;
  int32_t *tmp;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, sc, s));
  if (C == 0) {
    Status h;
    CEL_TRY(read_status(st, &h, s));
    if (h.err) return status_error(h, fn);
    *coarse_makespan = 0;
    *best_effort_count = 0;
    return CEL_OK;
  }
  uint64_t *W, *MEM, *back, *keys;
  int32_t *cnt, *boff, *ca, *ncp;
  int64_t *ecost, *cc, *Fin, *bs, *bf, *dcap;
  uint32_t *ids;
  const int64_t m = g->m;
  CEL_TRY(sc.get(&W, C));
  CEL_TRY(sc.get(&MEM, C));
  CEL_TRY(sc.get(&back, C));
  CEL_TRY(sc.get(&cnt, C));
  CEL_TRY(sc.get(&boff, (int64_t)C + 1));
  CEL_TRY(sc.get(&ncp, C));
  CEL_TRY(sc.get(&Fin, C));
  CEL_TRY(sc.get(&dcap, d->D));
  CEL_TRY(sc.get(&bs, d->D * bcap));
  CEL_TRY(sc.get(&bf, d->D * bcap));
  CEL_HIP(hipMemsetAsync(W, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(MEM, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(back, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(cnt, 0, sizeof(int32_t) * C, s));
  CEL_HIP(hipMemcpyAsync(dcap, d->cap, sizeof(int64_t) * d->D, hipMemcpyHostToDevice, s));
  k_place_nodes<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, C, cluster_id, g->w, g->mem, W, MEM, st);
  const unsigned eb = edge_blocks(g->m);
  k_place_edges<0><<<eb, 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, cnt, nullptr, nullptr,
                                      nullptr, nullptr, st);
  CEL_TRY(exclusive_scan_i32(cnt, boff, C, sc, s));
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  std::vector<int32_t> hb(C + 1);
  CEL_HIP(hipMemcpyAsync(hb.data(), boff, sizeof(int32_t) * (C + 1), hipMemcpyDeviceToHost, s));
  CEL_HIP(hipStreamSynchronize(s));
  const int64_t ncross = hb[C];
  CEL_TRY(sc.get(&keys, ncross));
  CEL_TRY(sc.get(&ids, ncross));
  CEL_TRY(sc.get(&ca, ncross + kPlacePad));  // k_place reads up to kPlacePad past a list
  CEL_TRY(sc.get(&cc, ncross + kPlacePad));
  CEL_TRY(sc.get(&ecost, m));
  CEL_HIP(hipMemsetAsync(cnt, 0, sizeof(int32_t) * C, s));
  k_place_edges<1><<<eb, 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, cnt, boff, keys, ids, ecost,
                                      st);
  CEL_TRY(segmented_sort(keys, ids, boff, C, ncross, sc, s, st));
  k_place_combine<<<grid_for((int64_t)C * 64, 256, 8192), 256, 0, s>>>(C, boff, keys, ids, ecost,
                                                                      ca, cc, ncp, back, st);
  // Busy lists in LDS only first; if one outgrows its share (st->i1 set, the
  // outputs not written), the placement again with lists that move to global
  // memory when full.
  for (int gl = 0; gl < 2; gl++) {
    {
      KTimer kt(s, "k_place");
#define CEL_PLACE_LAUNCH(LDSF, GL, NI)                                                          \
  k_place<LDSF, GL, NI><<<1, 64, 0, s>>>(C, d->D, dcap, W, MEM, boff, ncp, ca, cc, back,        \
                                         cluster_dev, Fin, bs, bf, (int32_t)bcap, st)
      const bool lds = C <= kPlaceLds, one = d->D <= 64;
      if (lds && !gl) {
        if (one) CEL_PLACE_LAUNCH(true, false, 1);
        else CEL_PLACE_LAUNCH(true, false, 4);
      } else if (lds) {
        if (one) CEL_PLACE_LAUNCH(true, true, 1);
        else CEL_PLACE_LAUNCH(true, true, 4);
      } else if (!gl) {
        if (one) CEL_PLACE_LAUNCH(false, false, 1);
        else CEL_PLACE_LAUNCH(false, false, 4);
      } else {
        if (one) CEL_PLACE_LAUNCH(false, true, 1);
        else CEL_PLACE_LAUNCH(false, true, 4);
      }
#undef CEL_PLACE_LAUNCH
    }
    k_place_out<<<grid_for(n > C ? n : C, 256, 4096), 256, 0, s>>>(n, C, cluster_id, cluster_dev,
                                                                  node_dev, Fin, cluster_fin, st);
    CEL_HIP(hipGetLastError());
    CEL_TRY(read_status(st, &h, s));
    if (h.err) return status_error(h, fn);
    if (gl || !h.i1) break;  // the GL = true kernel never stops early
  }
  *coarse_makespan = h.s0;
  *best_effort_count = h.i0;
  return CEL_OK;
}

extern "C" int cel_comm_sums(const cel_graph *g, const cel_devices *d, const int32_t *cluster_id,
                             int64_t *edge_comm, int64_t *w_sum, hipStream_t s) {
  const char *fn = "cel_comm_sums";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  if (!edge_comm || !w_sum) return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  Scratch sc(s);
  Status *st;
  int32_t *tmp;
  unsigned long long *sums;
  CEL_TRY(sc.get(&st, 1));
  CEL_TRY(sc.get(&tmp, g->n));
  CEL_TRY(sc.get(&sums, 2));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_HIP(hipMemsetAsync(sums, 0, 2 * sizeof(unsigned long long), s));
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, sc, s));
  k_comm_sums<<<edge_blocks(g->m), 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, sums, st);
  CEL_HIP(hipGetLastError());
  unsigned long long h2[2] = {0, 0};
  CEL_HIP(hipMemcpyAsync(h2, sums, sizeof h2, hipMemcpyDeviceToHost, s));
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  *edge_comm = (int64_t)h2[0];
  *w_sum = (int64_t)h2[1];
  return CEL_OK;
}

extern "C" int cel_order_place(const cel_graph *g, const cel_devices *d, const int32_t *cluster_id,
                               int32_t C, uint8_t *cluster_dev, uint8_t *node_dev,
                               int32_t *best_effort_count, hipStream_t s) {
  const char *fn = "cel_order_place";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n;
  if (!best_effort_count || (n > 0 && (!cluster_id || !node_dev)) || (C > 0 && !cluster_dev))
    return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  if (C < 0 || (n > 0 && C < 1))
    return set_error(CEL_E_ARG, "%s: n_clusters = %d out of range", fn, C);
  Scratch sc(s);
  Status *st;
  int32_t *tmp;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(check_graph(g, d->bw, d->lat, false, st, tmp, sc, s));
  if (C == 0) {
    Status h;
    CEL_TRY(read_status(st, &h, s));
    if (h.err) return status_error(h, fn);
    *best_effort_count = 0;
    return CEL_OK;
  }
  uint64_t *W, *MEM;
  int64_t *dcap;
  CEL_TRY(sc.get(&W, C));
  CEL_TRY(sc.get(&MEM, C));
  CEL_TRY(sc.get(&dcap, d->D));
  CEL_HIP(hipMemsetAsync(W, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(MEM, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemcpyAsync(dcap, d->cap, sizeof(int64_t) * d->D, hipMemcpyHostToDevice, s));
  k_place_nodes<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, C, cluster_id, g->w, g->mem, W, MEM, st);
  k_order_place<<<1, 64, 0, s>>>(C, d->D, dcap, MEM, cluster_dev, st);
  k_place_out<<<grid_for(n > C ? n : C, 256, 4096), 256, 0, s>>>(n, C, cluster_id, cluster_dev,
                                                                node_dev, nullptr, nullptr, st);
  CEL_HIP(hipGetLastError());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  *best_effort_count = h.i0;
  return CEL_OK;
}

extern "C" int cel_place_ext(const cel_graph *g, const cel_devices *d, const cel_hetero *h,
                             const int32_t *group, int32_t n_groups, const int32_t *cluster_id,
                             int32_t C, uint8_t *cluster_dev, uint8_t *node_dev,
                             int64_t *cluster_fin, int64_t *coarse_makespan,
                             int32_t *best_effort_count, hipStream_t s) {
  const char *fn = "cel_place_ext";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n, D = d->D;
  if (!coarse_makespan || !best_effort_count || (n > 0 && (!cluster_id || !node_dev)) ||
      (C > 0 && !cluster_dev) || n_groups < 0 || (n_groups > 0 && n > 0 && !group))
    return set_error(CEL_E_ARG, "%s: NULL argument or n_groups < 0", fn);
  if (C < 0 || (n > 0 && C < 1) || C > (n > 0 ? n : 0))
    return set_error(CEL_E_ARG, "%s: n_clusters = %d out of range", fn, C);
  if (D > 64) return set_error(CEL_E_ARG, "%s: D = %d above 64", fn, D);
  const bool het = h && (h->tmul || h->bw || h->lat);
  const bool links = het && (h->bw || h->lat);
  int64_t bwmin = d->bw, latmax = d->lat, tmax = 1024;
  if (het) {
    CEL_TRY(check_hetero(h, d, fn, &bwmin, &latmax, &tmax));
    // overflow bound with the slowest device and the worst link: every time
    // is a sum of cluster durations and coarse-edge costs along one chain,
    // each coarse cost at most the sum of its member edges' worst-link c
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
  int32_t *tmp;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, sc, s));
  if (C == 0) {
    Status hs;
    CEL_TRY(read_status(st, &hs, s));
    if (hs.err) return status_error(hs, fn);
    *coarse_makespan = 0;
    *best_effort_count = 0;
    return CEL_OK;
  }
  const bool grp = n_groups > 0;
  const int64_t m = g->m, bcap = C;
  uint64_t *W2, *MEMo, *back, *keys;
  int32_t *cnt, *boff, *ca, *ncp, *lead, *fcnt, *foff, *fl, *soff, *scnt;
  int64_t *ecost, *eob, *eone, *cc, *cob, *cnum, *Fin, *bs, *bf, *dcap, *tm_d = nullptr, *fm;
  int64_t *sob = nullptr, *snum = nullptr, *lbw = nullptr, *llat = nullptr;
  uint32_t *ids;
  CEL_TRY(sc.get(&W2, (int64_t)C * D));
  CEL_TRY(sc.get(&MEMo, C));
  CEL_TRY(sc.get(&back, C));
  CEL_TRY(sc.get(&cnt, C));
  CEL_TRY(sc.get(&boff, (int64_t)C + 1));
  CEL_TRY(sc.get(&ncp, C));
  CEL_TRY(sc.get(&Fin, C));
  CEL_TRY(sc.get(&dcap, D));
  CEL_TRY(sc.get(&bs, D * bcap));
  CEL_TRY(sc.get(&bf, D * bcap));
  CEL_TRY(sc.get(&lead, grp ? n_groups : 1));
  CEL_TRY(sc.get(&fcnt, C));
  CEL_TRY(sc.get(&foff, (int64_t)C + 1));
  CEL_TRY(sc.get(&soff, (int64_t)C + 1));
  CEL_TRY(sc.get(&scnt, C));
  CEL_HIP(hipMemsetAsync(W2, 0, sizeof(uint64_t) * C * D, s));
  CEL_HIP(hipMemsetAsync(MEMo, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(back, 0, sizeof(uint64_t) * C, s));
  CEL_HIP(hipMemsetAsync(cnt, 0, sizeof(int32_t) * C, s));
  CEL_HIP(hipMemsetAsync(fcnt, 0, sizeof(int32_t) * C, s));
  CEL_HIP(hipMemcpyAsync(dcap, d->cap, sizeof(int64_t) * D, hipMemcpyHostToDevice, s));
  std::vector<int64_t> ht, hb, hl;
  if (het && h->tmul) {
    CEL_TRY(sc.get(&tm_d, D));
    ht.assign(h->tmul, h->tmul + D);
    CEL_HIP(hipMemcpyAsync(tm_d, ht.data(), sizeof(int64_t) * D, hipMemcpyHostToDevice, s));
  }
  if (links) {
    CEL_TRY(sc.get(&lbw, (int64_t)D * D));
    CEL_TRY(sc.get(&llat, (int64_t)D * D));
    hb.resize((size_t)D * D);
    hl.resize((size_t)D * D);
    for (int32_t i = 0; i < D * D; i++) {
      const bool diag = i / D == i % D;
      hb[i] = diag ? 1 : (h->bw ? h->bw[i] : d->bw);
      hl[i] = diag ? 0 : (h->lat ? h->lat[i] : d->lat);
      if (hb[i] < 1 || hb[i] > INT32_MAX || hl[i] < 0 || hl[i] > INT32_MAX)
        return set_error(CEL_E_ARG, "%s: link %d: bw in [1, 2^31) and lat in [0, 2^31) needed", fn, i);
    }
    CEL_HIP(hipMemcpyAsync(lbw, hb.data(), sizeof(int64_t) * D * D, hipMemcpyHostToDevice, s));
    CEL_HIP(hipMemcpyAsync(llat, hl.data(), sizeof(int64_t) * D * D, hipMemcpyHostToDevice, s));
  }
  if (group && n > 0) {  // group ids checked even when there are no groups
    if (grp) k_fill_i32<<<grid_for(n_groups, 256, 1024), 256, 0, s>>>(lead, n_groups, INT32_MAX);
    k_colo_lead<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, n_groups, group, cluster_id,
                                                      grp ? lead : nullptr, st);
  }
  k_pe_nodes<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, C, D, cluster_id, g->w, g->mem,
                                                    grp ? group : nullptr, lead, tm_d, W2, MEMo,
                                                    fcnt, st);
  CEL_TRY(exclusive_scan_i32(fcnt, foff, C, sc, s));
  const unsigned eb = edge_blocks(g->m);
  k_place_edges<0><<<eb, 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, cnt, nullptr, nullptr,
                                      nullptr, nullptr, st);
  CEL_TRY(exclusive_scan_i32(cnt, boff, C, sc, s));
  Status hs;
  CEL_TRY(read_status(st, &hs, s));
  if (hs.err) return status_error(hs, fn);
  int32_t counts[2];  // coarse-edge slots, followers
  CEL_HIP(hipMemcpyAsync(&counts[0], boff + C, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  CEL_HIP(hipMemcpyAsync(&counts[1], foff + C, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  CEL_HIP(hipStreamSynchronize(s));
  const int64_t ncross = counts[0], nfol = counts[1];
  CEL_TRY(sc.get(&keys, ncross));
  CEL_TRY(sc.get(&ids, ncross));
  CEL_TRY(sc.get(&ca, ncross));
  CEL_TRY(sc.get(&cc, ncross));
  CEL_TRY(sc.get(&ecost, m));
  CEL_TRY(sc.get(&fl, nfol));
  CEL_TRY(sc.get(&fm, nfol));
  if (nfol > 0) {
    CEL_HIP(hipMemsetAsync(fcnt, 0, sizeof(int32_t) * C, s));
    k_pe_followers<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, cluster_id, g->mem, group, lead, foff,
                                                          fcnt, fl, fm, st);
  }
  CEL_HIP(hipMemsetAsync(cnt, 0, sizeof(int32_t) * C, s));
  k_place_edges<1><<<eb, 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, cnt, boff, keys, ids, ecost,
                                      st);
  CEL_TRY(segmented_sort(keys, ids, boff, C, ncross, sc, s, st));
  const int cg = grid_for((int64_t)C * 64, 256, 8192);
  k_place_combine<<<cg, 256, 0, s>>>(C, boff, keys, ids, ecost, ca, cc, ncp, back, st);
  cob = cnum = nullptr;
  if (links) {
    int32_t *ca2, *ncp2;
    uint64_t *back2;
    CEL_TRY(sc.get(&eob, m));
    CEL_TRY(sc.get(&eone, m));
    CEL_TRY(sc.get(&cob, ncross));
    CEL_TRY(sc.get(&cnum, ncross));
    CEL_TRY(sc.get(&ca2, ncross));
    CEL_TRY(sc.get(&ncp2, C));
    CEL_TRY(sc.get(&back2, C));
    CEL_TRY(sc.get(&sob, ncross));
    CEL_TRY(sc.get(&snum, ncross));
    k_pe_edge_ob<<<eb, 256, 0, s>>>(*g, eob, eone, st);
    // the same runs summed over ob and over a count of one (their sources
    // and run counts are those of the first pass)
    k_place_combine<<<cg, 256, 0, s>>>(C, boff, keys, ids, eob, ca2, cob, ncp2, back2, st);
    k_place_combine<<<cg, 256, 0, s>>>(C, boff, keys, ids, eone, ca2, cnum, ncp2, back2, st);
    CEL_HIP(hipMemsetAsync(scnt, 0, sizeof(int32_t) * C, s));
    k_pe_succ<0><<<grid_for(C, 256, 4096), 256, 0, s>>>(C, boff, ncp, ca, cob, cnum, scnt, nullptr,
                                                       nullptr, nullptr, st);
    CEL_TRY(exclusive_scan_i32(scnt, soff, C, sc, s));
    CEL_HIP(hipMemsetAsync(scnt, 0, sizeof(int32_t) * C, s));
    k_pe_succ<1><<<grid_for(C, 256, 4096), 256, 0, s>>>(C, boff, ncp, ca, cob, cnum, scnt, soff,
                                                       sob, snum, st);
  }
  PeArgs pa{};
  pa.C = C;
  pa.D = D;
  pa.links = links;
  pa.cap = dcap;
  pa.W2 = W2;
  pa.MEMo = MEMo;
  pa.boff = boff;
  pa.ncp = ncp;
  pa.ca = ca;
  pa.cc = cc;
  pa.cob = cob;
  pa.cnum = cnum;
  pa.back = back;
  pa.soff = soff;
  pa.sob = sob;
  pa.snum = snum;
  pa.foff = foff;
  pa.fl = fl;
  pa.fm = fm;
  pa.lbw = lbw;
  pa.llat = llat;
  pa.cdev = cluster_dev;
  pa.Fin = Fin;
  pa.bs = bs;
  pa.bf = bf;
  pa.bcap = (int32_t)bcap;
  {
    KTimer kt(s, "k_place_ext");
    if (C <= kPeLds) k_place_ext<true><<<1, 64, 0, s>>>(pa, st);
    else k_place_ext<false><<<1, 64, 0, s>>>(pa, st);
  }
  k_pe_out<<<grid_for(n > C ? n : C, 256, 4096), 256, 0, s>>>(n, C, cluster_id,
                                                             grp ? group : nullptr, lead,
                                                             cluster_dev, node_dev, Fin,
                                                             cluster_fin, st);
  CEL_HIP(hipGetLastError());
  CEL_TRY(read_status(st, &hs, s));
  if (hs.err) return status_error(hs, fn);
  *coarse_makespan = hs.s0;
  *best_effort_count = hs.i0;
  return CEL_OK;
}
