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
// cc; it is evaluated for all devices at once from per-device maxima of Fin
// and of Fin + cc over the preds, and the best and second-best devices of
// the latter.  Lane x then finds the first-fit start on device x in that
// device's sorted list of busy blocks (touching intervals are merged, so the
// list holds one block per idle gap), and a wave argmin picks the device.
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
constexpr int kPlaceLds = 8192;  // clusters whose Fin and device are kept in LDS too (161,792 B of LDS in all)

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

// Placement, one wave (its LDS accesses are in program order, so no barrier
// is needed).  For cluster t, one pass over its coarse preds leaves per device
// y the largest Fin and the largest Fin + cc of the preds on y; pre_t on
// device x is then max(0, the first at x, the largest second over devices
// other than x), from the best and second-best devices.  Device x's free
// memory and busy-list state sit in the registers of lane x mod 64; values
// every lane needs are read from LDS in unrolled groups, all requests out
// before the first use.  Each device's busy list lives in LDS
// (kPlaceBlk / D blocks) until it outgrows that share; it then moves to its
// global list.  LDSF keeps every cluster's Fin and device in LDS as well
// (C <= kPlaceLds).
template <bool LDSF>
__global__ void __launch_bounds__(64)
    k_place(int32_t C, int32_t D, const int64_t *cap, const uint64_t *W, const uint64_t *MEM,
            const int32_t *boff, const int32_t *ncp, const int32_t *ca, const int64_t *cc,
            const uint64_t *back, uint8_t *cdev, int64_t *Fin, int64_t *bs, int64_t *bf,
            int32_t bcap, Status *st) {
  constexpr int G = 16;  // devices per group of LDS reads
  __shared__ int64_t s_bs[kPlaceBlk], s_bf[kPlaceBlk];
  __shared__ int64_t s_fin[LDSF ? kPlaceLds : 1];
  __shared__ uint8_t s_cd[LDSF ? kPlaceLds : 1];
  // per device: max Fin and max Fin + cc of the preds on it (-1: none), EST
  // (kInf past D)
  __shared__ int64_t s_dm[256], s_dmc[256], s_est[256];
  if (failed(st)) return;
  const int lane = threadIdx.x;
  const int32_t capL = kPlaceBlk / D;
  int64_t ava[4], last[4];  // device lane + 64 i: free memory, end of its last busy block
  int32_t nbl[4], glob[4];  // its busy-block count; list moved to global memory
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int x = lane + 64 * i;
    ava[i] = x < D ? cap[x] : 0;
    last[i] = 0;
    nbl[i] = 0;
    glob[i] = 0;
    s_dm[x] = -1;
    s_dmc[x] = -1;
    s_est[x] = kInf;
  }
  int32_t prev = 0, be = 0;
  int64_t span = 0;
  // Loads run ahead of their use: the sizes of 64 clusters at a time, one per
  // lane, a block of 64 ahead (read back with readlane), and the first 64
  // preds of a cluster kPD steps ahead; their Fin and device come from LDS
  // (LDSF), else from global memory at the step.
  constexpr int kPD = 3;
  auto bulk = [&](int32_t t0, int32_t &zb, int32_t &zn, int64_t &zw, int64_t &zm, int64_t &zk) {
    const int32_t t = t0 + lane;
    zb = t < C ? boff[t] : 0;
    zn = t < C ? ncp[t] : 0;
    zw = t < C ? (int64_t)W[t] : 0;
    zm = t < C ? (int64_t)MEM[t] : 0;
    zk = t < C ? (int64_t)back[t] : 0;
  };
  int32_t ub, un, vb, vn;  // sizes of clusters [T, T + 64) (u*) and [T + 64, T + 128) (v*)
  int64_t uw, um, uk, vw, vm, vk;
  bulk(0, ub, un, uw, um, uk);
  bulk(64, vb, vn, vw, vm, vk);
  // first preds of the cluster t' (t' < T + 128), by lane
  auto preds = [&](int32_t tp, int32_t T, int32_t &pa, int64_t &pc) {
    pa = 0;
    pc = 0;
    if (tp >= C) return;
    const bool in_u = tp - T < 64;
    const int l = (tp - T) & 63;
    const int32_t b = __builtin_amdgcn_readlane(in_u ? ub : vb, l);
    const int32_t nn = __builtin_amdgcn_readlane(in_u ? un : vn, l);
    if (lane < nn) {
      pa = ca[b + lane];
      pc = cc[b + lane];
    }
  };
  int32_t pa[kPD];
  int64_t pcv[kPD];
#pragma unroll
  for (int q = 0; q < kPD; q++) preds(q, 0, pa[q], pcv[q]);
  for (int32_t t = 0; t < C; t++) {
    const int32_t T = t & ~63;
    if (t > 0 && (t & 63) == 0) {  // next block of sizes
      ub = vb;
      un = vn;
      uw = vw;
      um = vm;
      uk = vk;
      bulk(t + 64, vb, vn, vw, vm, vk);
    }
    const int l = t & 63;
    const int32_t b0 = __builtin_amdgcn_readlane(ub, l), np = __builtin_amdgcn_readlane(un, l);
    const int64_t Wt = readlane64(uw, l), Mt = readlane64(um, l), bk = readlane64(uk, l);
    int32_t a0 = pa[0];
    int64_t c0 = pcv[0];
#pragma unroll
    for (int q = 0; q + 1 < kPD; q++) {
      pa[q] = pa[q + 1];
      pcv[q] = pcv[q + 1];
    }
    preds(t + kPD, T, pa[kPD - 1], pcv[kPD - 1]);
    // per-device maxima over the preds
    for (int32_t k0 = 0; k0 < np; k0 += 64) {
      if (k0 > 0) {
        a0 = k0 + lane < np ? ca[b0 + k0 + lane] : 0;
        c0 = k0 + lane < np ? cc[b0 + k0 + lane] : 0;
      }
      if (k0 + lane < np) {
        const int64_t f0 = LDSF ? s_fin[a0] : Fin[a0];
        const int32_t d0 = LDSF ? s_cd[a0] : cdev[a0];
        atomicMax((long long *)&s_dm[d0], (long long)f0);
        atomicMax((long long *)&s_dmc[d0], (long long)(f0 + c0));
      }
    }
    // best device by Fin + cc (lowest id on ties) and the best of the others,
    // by every lane
    int64_t m1 = -1, m2 = -1;
    int32_t d1 = INT32_MAX;
    for (int32_t x0 = 0; x0 < D; x0 += G) {
      int64_t v[G];
#pragma unroll
      for (int q = 0; q < G; q++) v[q] = s_dmc[x0 + q];
#pragma unroll
      for (int q = 0; q < G; q++) {
        if (v[q] > m1) {
          m2 = m1;
          m1 = v[q];
          d1 = x0 + q;
        } else if (v[q] > m2) {
          m2 = v[q];
        }
      }
    }
    // device x: pre_t, first-fit slot and EST (eq. 7)
    int64_t slot[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
      slot[i] = 0;
      const int x = lane + 64 * i;
      if (64 * i >= D) continue;  // uniform
      if (x < D) {
        int64_t pre = 0;
        const int64_t other = x != d1 ? m1 : m2;
        pre = other > pre ? other : pre;
        pre = s_dm[x] > pre ? s_dm[x] : pre;
        int64_t sv = pre;
        const int32_t nb = nbl[i];
        if (Wt > 0 && nb > 0 && sv < last[i]) {  // LDS and global lists in separate code
          if (!glob[i]) {
            const int64_t *xs = s_bs + x * capL, *xf = s_bf + x * capL;
            for (int32_t k = blocks_ending_by(xf, nb, sv); k < nb && xs[k] < sv + Wt; k++)
              sv = xf[k];
          } else {
            const int64_t *xs = bs + (int64_t)x * bcap, *xf = bf + (int64_t)x * bcap;
            for (int32_t k = blocks_ending_by(xf, nb, sv); k < nb && xs[k] < sv + Wt; k++)
              sv = xf[k];
          }
        }
        slot[i] = sv;
        s_est[x] = ava[i] < Mt ? kInf : sv;
        s_dm[x] = -1;  // cleared for the next cluster
        s_dmc[x] = -1;
      }
    }
    // device of smallest EST (lowest id on ties), by every lane
    int64_t ev = kInf;
    int32_t ei = INT32_MAX;
    for (int32_t x0 = 0; x0 < D; x0 += G) {
      int64_t v[G];
#pragma unroll
      for (int q = 0; q < G; q++) v[q] = s_est[x0 + q];
#pragma unroll
      for (int q = 0; q < G; q++)
        if (v[q] < ev) {
          ev = v[q];
          ei = x0 + q;
        }
    }
    // the choice (eq. 8-9), uniform over the wave
    const int32_t dk = t == 0 ? 0 : prev;
    const int64_t edk = s_est[dk];
    int32_t pick;
    if (ev == kInf) {  // every device full: most remaining memory (best effort)
      int64_t av = INT64_MIN;  // free memory can be negative after best-effort picks
      int32_t ai = INT32_MAX;
#pragma unroll
      for (int i = 0; i < 4; i++)
        if (lane + 64 * i < D && ava[i] > av) {
          av = ava[i];
          ai = lane + 64 * i;
        }
      argmax_i64(av, ai);
      pick = ai;
      be++;
    } else if (edk == kInf || edk - ev > bk) {
      pick = ei;
    } else {
      pick = dk;
    }
    const int ip = pick >> 6, lp = pick & 63;
    int64_t slp = 0;
    int32_t nb = 0, gl = 0;
#pragma unroll
    for (int i = 0; i < 4; i++)
      if (i == ip) {
        slp = slot[i];
        nb = nbl[i];
        gl = glob[i];
      }
    const int64_t s0 = readlane64(slp, lp), f = s0 + Wt;
    nb = __builtin_amdgcn_readlane(nb, lp);
    gl = __builtin_amdgcn_readlane(gl, lp);
    span = f > span ? f : span;
    prev = pick;
    if (Wt > 0) {  // insert [s0, f) into the device's merged busy blocks
      if (!gl && nb == capL) {  // the LDS share is full: move the list out
        for (int32_t q = lane; q < nb; q += 64) {
          bs[(int64_t)pick * bcap + q] = s_bs[pick * capL + q];
          bf[(int64_t)pick * bcap + q] = s_bf[pick * capL + q];
        }
        gl = 1;
      }
      int64_t lastv = 0;
      if (lane == 0) {
        if (!gl) lastv = busy_insert(s_bs + pick * capL, s_bf + pick * capL, nb, capL, s0, f, st);
        else lastv = busy_insert(bs + (int64_t)pick * bcap, bf + (int64_t)pick * bcap, nb, bcap,
                                 s0, f, st);
      }
      nb = __builtin_amdgcn_readlane(nb, 0);
      lastv = readlane64(lastv, 0);
#pragma unroll
      for (int i = 0; i < 4; i++)
        if (i == ip && lane == lp) {
          nbl[i] = nb;
          last[i] = lastv;
          glob[i] = gl;
        }
    }
#pragma unroll
    for (int i = 0; i < 4; i++)
      if (i == ip && lane == lp) ava[i] -= Mt;
    if (lane == 0) {  // later steps of this wave read these back, in program order
      cdev[t] = (uint8_t)pick;
      Fin[t] = f;
      if (LDSF) {
        s_fin[t] = f;
        s_cd[t] = (uint8_t)pick;
      }
    }
  }
  if (lane == 0) {
    st->s0 = span;
    st->i0 = be;
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
  CEL_TRY(sc.get(&ca, ncross));
  CEL_TRY(sc.get(&cc, ncross));
  CEL_TRY(sc.get(&ecost, m));
  CEL_HIP(hipMemsetAsync(cnt, 0, sizeof(int32_t) * C, s));
  k_place_edges<1><<<eb, 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, cnt, boff, keys, ids, ecost,
                                      st);
  CEL_TRY(segmented_sort(keys, ids, boff, C, ncross, sc, s, st));
  k_place_combine<<<grid_for((int64_t)C * 64, 256, 8192), 256, 0, s>>>(C, boff, keys, ids, ecost,
                                                                      ca, cc, ncp, back, st);
  {
    KTimer kt(s, "k_place");
    if (C <= kPlaceLds)
      k_place<true><<<1, 64, 0, s>>>(C, d->D, dcap, W, MEM, boff, ncp, ca, cc, back, cluster_dev,
                                     Fin, bs, bf, (int32_t)bcap, st);
    else
      k_place<false><<<1, 64, 0, s>>>(C, d->D, dcap, W, MEM, boff, ncp, ca, cc, back,
                                      cluster_dev, Fin, bs, bf, (int32_t)bcap, st);
  }
  k_place_out<<<grid_for(n > C ? n : C, 256, 4096), 256, 0, s>>>(n, C, cluster_id, cluster_dev,
                                                                node_dev, Fin, cluster_fin, st);
  CEL_HIP(hipGetLastError());
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
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
