// cel_cluster: memory-capped contiguous clustering of a topological order
// (Section 5.1.3, eq. 4-6).
//
// With PO the prefix sum of each node's out-going comm (outdeg * c) and
// Int(i, j) the comm of edges with both ends inside positions [i, j),
//   cost(i, j) = PO[j] - PO[i] - Int(i, j)            (eq. 4 rewritten)
//   S(j)      = PO[j] + min_i V_j(i),   V_j(i) = S(i) - PO[i] - Int(i, j),
// over lo(j) <= i < j (window R, memory cap M); ties go to the smallest i.
//
// The recurrence is sequential in j.  One workgroup runs it in blocks of 64
// targets, one lane per target:
//  * the candidates below the block ("old" ones, at most R) are split evenly
//    over waves 1..NW-1 (about 16 each, up to 15 waves), in chunks of at most
//    64; each wave sweeps its candidates in
//    descending order, merging the block's edge list (sorted by source,
//    descending), so that every lane keeps the running Int of its own target
//    and a running (min, argmin); per-wave offsets are added afterwards;
//  * wave 0 meanwhile gathers, in registers, Int(i, j) for the candidates and
//    targets inside the block, then runs the 64 in-block steps (one lane
//    broadcast per step).
// H(i) = V_{j0}(i) for the old candidates lives in an LDS ring and moves to
// the next block by subtracting the comm of the block's edges whose source is
// at or after i.  Only edges whose source lies in the window can change a
// candidate, so each block's list holds only those; it is built and sorted by
// a parallel pass and staged one block ahead.  A block whose list exceeds the
// staging size is taken target by target by the whole workgroup from the
// in-edge lists; totals of comm too large for the packed keys take a
// step-wise kernel that keeps the window in registers.
//
// The memory bound lo(j) comes from a prefix sum of the memory in order
// (binary search), the greedy mode from the same prefix sums.
#include "cel_internal.h"

namespace cel {

// position arrays: memory, comm, out-going comm
__global__ void k_cluster_pos(int32_t n, const int32_t *order, const int32_t *out_ptr,
                              const int64_t *mem, const int64_t *ob, int64_t bw, int64_t lat,
                              int64_t *memp, int64_t *cq, int64_t *outc, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t v = order[p];
    const int64_t c = comm_of(ob[v], bw, lat);
    memp[p] = mem[v];
    cq[p] = c;
    outc[p] = c * (int64_t)(out_ptr[v + 1] - out_ptr[v]);
  }
}

// lo[j] (j = 1..n): first feasible start of a cluster ending before j;
// gend[s] (s = 0..n-1): end of the greedy cluster that starts at s.
__global__ void k_cluster_bounds(int32_t n, int32_t R, int64_t M, const int64_t *PM, int32_t *lo,
                                 int32_t *gend, const Status *st) {
  if (failed(st)) return;
  for (int64_t x = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; x < n;
       x += (int64_t)gridDim.x * blockDim.x) {
    {  // j = x + 1: smallest i in [0, j-1] with PM[j] - PM[i] <= M
      const int32_t j = (int32_t)x + 1;
      const int64_t target = PM[j] - M;
      int32_t a = 0, b = j;  // first i with PM[i] >= target (b = j: none)
      while (a < b) {
        const int32_t mid = (a + b) >> 1;
        if (PM[mid] < target) a = mid + 1;
        else b = mid;
      }
      int32_t l = j - R > a ? j - R : a;
      if (l > j - 1) l = j - 1;  // a single node is always a feasible cluster
      if (l < 0) l = 0;
      lo[j] = l;
    }
    {  // greedy: largest e in [s+1, min(n, s+R)] with PM[e] - PM[s] <= M, at least s+1
      const int32_t s = (int32_t)x;
      const int32_t hi = (int64_t)s + R < n ? s + R : n;
      const int64_t lim = PM[s] + M;
      int32_t a = s + 1, b = hi;  // last e in [s+1, hi] with PM[e] <= lim
      if (PM[s + 1] > lim) {
        gend[s] = s + 1;
      } else {
        while (a < b) {
          const int32_t mid = (a + b + 1) >> 1;
          if (PM[mid] <= lim) a = mid;
          else b = mid - 1;
        }
        gend[s] = a;
      }
    }
  }
}

// ---------------------------------------------------- step-wise DP (fallback)
// One wave; the window of the last R candidates is held 64 lanes wide in
// registers: per step a few predicated subtractions and one wave-wide
// (min value, min index) reduction.  In-edge lists are staged through LDS.
constexpr int kDpBlk = 256;    // DP steps staged per block
constexpr int kDpEcap = 6144;  // in-edges staged per block

template <int SL>
__global__ void __launch_bounds__(64)
    k_cluster_dp_step(int32_t n, int32_t R, const int32_t *lo, const int32_t *pptr,
                 const int32_t *pidx, const int64_t *cq, const int64_t *PO, int32_t *P,
                 Status *st) {
  constexpr int RW = 64 * SL;
  __shared__ int32_t s_lo[kDpBlk];
  __shared__ int32_t s_ptr[kDpBlk + 1];
  __shared__ int32_t s_q[kDpEcap];
  __shared__ int64_t s_c[kDpEcap];
  if (failed(st)) return;
  (void)R;
  const int lane = threadIdx.x;
  int64_t v[SL];
  int32_t iv[SL];
#pragma unroll
  for (int s = 0; s < SL; s++) {
    v[s] = 0;
    iv[s] = -1;
  }
  if (lane == 0) iv[0] = 0;  // candidate i = 0 with V = S(0) - PO[0] = 0
  int64_t G = 0;
  for (int32_t j0 = 1; j0 <= n;) {
    // block of steps [j0, j1); in-edges of positions [j0, min(j1, n)) staged
    int32_t j1 = j0 + kDpBlk <= n + 1 ? j0 + kDpBlk : n + 1;
    const int32_t eb = pptr[j0 < n ? j0 : n];
    {
      int32_t a = j0 + 1, b = j1;  // largest j1 with staged edges <= cap
      while (a < b) {
        const int32_t mid = (a + b + 1) >> 1;
        if (pptr[mid < n ? mid : n] - eb <= kDpEcap) a = mid;
        else b = mid - 1;
      }
      j1 = a;
    }
    const int32_t ee = pptr[j1 < n ? j1 : n];
    const bool staged = ee - eb <= kDpEcap;
    for (int t = lane; t < j1 - j0; t += 64) s_lo[t] = lo[j0 + t];
    for (int t = lane; t <= j1 - j0; t += 64) {
      const int32_t jj = j0 + t < n ? j0 + t : n;
      s_ptr[t] = pptr[jj] - eb;
    }
    if (staged)
      for (int32_t k = lane; k < ee - eb; k += 64) {
        const int32_t q = pidx[eb + k];
        s_q[k] = q;
        s_c[k] = cq[q];
      }
    __syncthreads();
    for (int32_t j = j0; j < j1; j++) {
      const int32_t lj = s_lo[j - j0];
      int64_t bv = INT64_MAX;
      int32_t bi = INT32_MAX;
#pragma unroll
      for (int s = 0; s < SL; s++) {
        const int32_t i = iv[s];
        if (i >= lj && i < j && (v[s] < bv || (v[s] == bv && i < bi))) {
          bv = v[s];
          bi = i;
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const int64_t ov = __shfl_xor(bv, off);
        const int32_t oi = __shfl_xor(bi, off);
        if (ov < bv || (ov == bv && oi < bi)) {
          bv = ov;
          bi = oi;
        }
      }
      G = bv;
      if (lane == 0) P[j] = bi;
      if (j == n) break;
      // the node at position j joins the target side: subtract its in-edges
      const int32_t k0 = s_ptr[j - j0], k1 = s_ptr[j - j0 + 1];
      if (staged) {
        for (int32_t k = k0; k < k1; k++) {
          const int32_t q = s_q[k];
          const int64_t cu = s_c[k];
#pragma unroll
          for (int s = 0; s < SL; s++)
            if (iv[s] >= 0 && iv[s] <= q) v[s] -= cu;
        }
      } else {
        for (int32_t k = k0; k < k1; k++) {
          const int32_t q = pidx[eb + k];
          const int64_t cu = cq[q];
#pragma unroll
          for (int s = 0; s < SL; s++)
            if (iv[s] >= 0 && iv[s] <= q) v[s] -= cu;
        }
      }
      // new candidate i = j with V = S(j) - PO[j] = G
      const int r = j % RW;
#pragma unroll
      for (int s = 0; s < SL; s++)
        if (lane == (r & 63) && s == (r >> 6)) {
          v[s] = G;
          iv[s] = j;
        }
    }
    __syncthreads();
    j0 = j1;
  }
  if (lane == 0) st->s0 = PO[n] + G;  // S(n): the total inter-cluster comm
}

// ------------------------------------------------------------ blocked DP
constexpr int kRingBig = 8192;  // LDS ring of H over positions (window R + 64 <= 4160)
constexpr int kRingSmall = 2048;  // the same for R + 64 <= 2048, with room for the in-block table
constexpr int kTS = 65;  // row stride of the in-block table (int64; odd: rows start in other banks)
constexpr int kEC = 1024;    // staged edges of one block
constexpr int kPF = 4;       // prefetched edges per thread of waves 1..NW-1
constexpr int kMaxW = 15;    // candidate waves (with wave 0: 16 values in the minimum tree)

__device__ inline int32_t rl32(int32_t v, int32_t l) { return __builtin_amdgcn_readlane(v, l); }
__device__ inline int64_t rl64(int64_t v, int32_t l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int32_t)(v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
template <int RING>
__device__ inline int rmod(int32_t p) { return p & (RING - 1); }

// first k in [0, cnt) with q[k] <= thr (q descending), cnt if none; wave-uniform
__device__ inline int32_t first_le(const int32_t *q, int32_t cnt, int32_t thr, int lane) {
  for (int32_t base = 0; base < cnt; base += 64) {
    const int32_t k = base + lane;
    const uint64_t m = __ballot(k < cnt && q[k] <= thr);
    if (m) return base + (int32_t)__builtin_ctzll(m);
  }
  return cnt;
}

// Per block of 64 targets (block b: j in [64b, 64b + 64)): the number of
// in-edges of positions [64b, min(64b + 64, n)) whose source is at or after
// lo(64b), and the largest such count.  One wave per block.
__global__ void k_dp_count(int32_t n, int32_t nb, const int32_t *pptr, const int32_t *pidx,
                           const int32_t *lo, int32_t *cnt, int32_t *mx, const Status *st) {
  if (failed(st)) return;
  const int lane = threadIdx.x & 63;
  const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t b = (blockIdx.x * (int64_t)blockDim.x + threadIdx.x) >> 6; b < nb; b += nw) {
    const int32_t j0 = (int32_t)b * 64, pe = j0 + 64 < n ? j0 + 64 : n;
    const int32_t lo0 = b == 0 ? 0 : lo[j0];
    const int32_t e1 = pptr[pe];
    int32_t c = 0;
    for (int32_t e = pptr[j0] + lane; e < e1; e += 64) c += pidx[e] >= lo0;
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
    if (lane == 0) {
      cnt[b] = c;
      atomicMax(mx, c);
    }
  }
}

// Builds each block's edge list: (source position q, target offset t) sorted
// by q descending then t ascending, the source's comm c and the exclusive
// prefix sum E of c along the list.  One workgroup per block, rank sort in
// LDS.  Blocks above kEC edges are skipped (the step-wise kernel runs then).
__global__ void __launch_bounds__(256)
    k_dp_fill(int32_t n, int32_t nb, const int32_t *pptr, const int32_t *pidx, const int32_t *lo,
              const int64_t *cq, const int32_t *boff, int32_t *eq, int32_t *et, int64_t *ec,
              int64_t *eE, const Status *st) {
  __shared__ int32_t s_ptr[65];
  __shared__ int32_t s_q[kEC];
  __shared__ int32_t s_t[kEC];
  __shared__ int64_t s_c[kEC];
  __shared__ int32_t s_n;
  if (failed(st)) return;
  const int lane = threadIdx.x & 63;
  for (int32_t b = blockIdx.x; b < nb; b += gridDim.x) {
    const int32_t o = boff[b], c = boff[b + 1] - o;
    if (c > kEC) continue;
    const int32_t j0 = b * 64, pe = j0 + 64 < n ? j0 + 64 : n, rows = pe - j0;
    const int32_t lo0 = b == 0 ? 0 : lo[j0];
    for (int t = threadIdx.x; t <= rows; t += blockDim.x) s_ptr[t] = pptr[j0 + t];
    if (threadIdx.x == 0) s_n = 0;
    __syncthreads();
    for (int32_t e = s_ptr[0] + threadIdx.x; e < s_ptr[rows]; e += blockDim.x) {
      const int32_t q = pidx[e];
      if (q >= lo0) {
        int r = 0, h = rows - 1;  // target row: last r with s_ptr[r] <= e
        while (r < h) {
          const int mid = (r + h + 1) >> 1;
          if (s_ptr[mid] <= e) r = mid;
          else h = mid - 1;
        }
        const int32_t k = atomicAdd(&s_n, 1);
        if (k < kEC) {
          s_q[k] = q;
          s_t[k] = r;
        }
      }
    }
    __syncthreads();
    for (int32_t k = threadIdx.x; k < c; k += blockDim.x) {
      const int32_t q = s_q[k], t = s_t[k];
      int32_t r = 0;
      for (int32_t k2 = 0; k2 < c; k2++) {
        const int32_t q2 = s_q[k2], t2 = s_t[k2];
        r += (q2 > q) || (q2 == q && (t2 < t || (t2 == t && k2 < k)));
      }
      eq[o + r] = q;
      et[o + r] = t;
      s_c[r] = cq[q];
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      int64_t run = 0;
      for (int32_t base = 0; base < c; base += 64) {
        const int32_t k = base + lane;
        const int64_t v = k < c ? s_c[k] : 0;
        int64_t x = v;
        for (int d = 1; d < 64; d <<= 1) {
          const int64_t y = __shfl_up(x, d);
          if (lane >= d) x += y;
        }
        if (k < c) {
          ec[o + k] = v;
          eE[o + k] = run + x - v;
        }
        run += __shfl(x, 63);
      }
    }
    __syncthreads();
  }
}

// Candidate keys: (V << 13) + (i - base), base = j0 - kBaseOff, so that one
// signed 64-bit minimum picks the smallest V and, among equal V, the smallest
// i.  Valid while every |V| stays below 2^48 (the host checks the total comm
// PO[n] against kPackLim).
constexpr int kIdxBits = 13;
constexpr int64_t kIdxMask = (int64_t(1) << kIdxBits) - 1;
constexpr int32_t kBaseOff = 4160;
constexpr int64_t kKeyInf = int64_t(1) << 62;
constexpr int64_t kPackLim = int64_t(1) << 46;
constexpr int kMaxRuns = 12;  // in-block runs handled by scans (more: one step per target)

// One Hillis-Steele step of a segmented inclusive min-scan (f = 1 starts a
// segment); lanes without a source combine with the identity.
template <int CTRL, int ROWMASK>
__device__ inline void segmin_step(int64_t &x, int32_t &f) {
  const int64_t ux = dpp64<CTRL, ROWMASK>(x, kKeyInf);
  const int32_t uf = dpp32<CTRL, ROWMASK>(f, 0);
  if (!f) {
    x = ux < x ? ux : x;
    f = uf;
  }
}
__device__ inline void wave_segmin(int64_t &x, int32_t f) {
  segmin_step<0x111, 0xF>(x, f);
  segmin_step<0x112, 0xF>(x, f);
  segmin_step<0x114, 0xF>(x, f);
  segmin_step<0x118, 0xF>(x, f);
  segmin_step<0x142, 0xA>(x, f);
  segmin_step<0x143, 0xC>(x, f);
}
// inclusive prefix sums over the wave
__device__ inline int32_t wave_incl_sum32(int32_t x) {
  x += dpp32<0x111, 0xF>(x, 0);
  x += dpp32<0x112, 0xF>(x, 0);
  x += dpp32<0x114, 0xF>(x, 0);
  x += dpp32<0x118, 0xF>(x, 0);
  x += dpp32<0x142, 0xA>(x, 0);
  x += dpp32<0x143, 0xC>(x, 0);
  return x;
}
__device__ inline int64_t wave_incl_sum64(int64_t x) {
  x += dpp64<0x111, 0xF>(x, 0);
  x += dpp64<0x112, 0xF>(x, 0);
  x += dpp64<0x114, 0xF>(x, 0);
  x += dpp64<0x118, 0xF>(x, 0);
  x += dpp64<0x142, 0xA>(x, 0);
  x += dpp64<0x143, 0xC>(x, 0);
  return x;
}

__device__ inline int64_t wave_prefix_min(int64_t x) {
  int64_t y;
  y = dpp64<0x111, 0xF>(x, kKeyInf);
  x = y < x ? y : x;
  y = dpp64<0x112, 0xF>(x, kKeyInf);
  x = y < x ? y : x;
  y = dpp64<0x114, 0xF>(x, kKeyInf);
  x = y < x ? y : x;
  y = dpp64<0x118, 0xF>(x, kKeyInf);
  x = y < x ? y : x;
  y = dpp64<0x142, 0xA>(x, kKeyInf);
  x = y < x ? y : x;
  y = dpp64<0x143, 0xC>(x, kKeyInf);
  x = y < x ? y : x;
  return x;
}

// Key of candidate position j0 + s carrying value G (the index field replaced).
__device__ inline int64_t relabel(int64_t key, int32_t s) {
  return (key & ~kIdxMask) | (int64_t)(s + kBaseOff);
}

// One chunk of candidates [cb, ct] (at most 64, lane l <-> i = ct - l) for
// the 64 targets of the block.  The chunk's edges split its candidates into
// segments (a segment starts at each candidate with edges); inside one the
// lane's running comm accS is constant, so a segmented min-scan gives every
// segment's best key.  The loop then walks the edges in order (sources
// descending): add the edge to the lanes above its target, evaluate its
// segment.  A segment evaluated before its last edge only overestimates.
// H moves to the next block.  FULL: every target may use every candidate.
template <bool FULL, int RING>
__device__ inline void dp_chunk(int32_t ct, int32_t cb, int32_t base, int32_t lo_t, int32_t *hist,
                                int64_t *H, const int32_t *Q, const int32_t *T, const int64_t *C,
                                const int64_t *E, int32_t cnt, int32_t &kk, int64_t &best,
                                int64_t &accS, int lane) {
  const int32_t nc = ct - cb + 1;
  const int32_t k0 = kk;
  int32_t k1 = k0;
  for (;;) {  // edges of the chunk: [k0, k1); per-candidate counts in LDS
    const int32_t e = k1 + lane;
    const bool in = e < cnt && Q[e] >= cb;
    const uint64_t m = __ballot(in);
    if (in) atomicAdd(&hist[ct - Q[e]], 1);
    k1 += __popcll(m);
    if (m != ~0ull) break;
  }
  wave_lds_sync();
  const int32_t ecnt = hist[lane];
  hist[lane] = 0;
  const int32_t i = ct - lane;
  const int64_t h = lane < nc ? H[rmod<RING>(i)] : 0;
  int64_t sx = lane < nc ? (int64_t)((uint64_t)h << kIdxBits) + (i - base) : kKeyInf;
  const uint64_t F = __ballot(ecnt > 0) | 1ull;
  wave_segmin(sx, (int32_t)((F >> lane) & 1));
  const uint64_t above = lane == 63 ? 0ull : F & ~((2ull << lane) - 1);
  const int32_t en_l = above ? (int32_t)__builtin_ctzll(above) - 1 : nc - 1;  // segment end
  int32_t lmax = 63;
  int64_t Pt = 0;
  if (!FULL) {
    lmax = ct - lo_t < nc - 1 ? ct - lo_t : nc - 1;  // last candidate lane valid for the target
    Pt = __shfl(sx, lmax < 0 ? 0 : lmax);
  }
  {  // segment of lane 0 before the chunk's edges
    const int32_t en0 = rl32(en_l, 0);
    const int64_t sk = rl64(sx, en0);
    if (FULL) {
      const int64_t kv = sk - accS;
      best = kv < best ? kv : best;
    } else {
      const int64_t kv = (lmax >= en0 ? sk : Pt) - accS;
      if (lmax >= 0 && kv < best) best = kv;
    }
  }
  for (int32_t kb0 = k0; kb0 < k1; kb0 += 64) {
    const int32_t nE = k1 - kb0 < 64 ? k1 - kb0 : 64;
    const bool v = lane < nE;
    const int32_t x = v ? kb0 + lane : k0;
    const int32_t stx = v ? ct - Q[x] : 0;
    const int32_t tx = v ? T[x] : 64;
    const int64_t cx = v ? (int64_t)((uint64_t)C[x] << kIdxBits) : 0;
    const int32_t enx = __shfl(en_l, stx);
    const int64_t skx = __shfl(sx, enx);
    for (int32_t y = 0; y < nE; y++) {
      const int32_t tk = rl32(tx, y);
      const int64_t ck = rl64(cx, y);
      const int64_t sk = rl64(skx, y);
      accS += lane > tk ? ck : 0;
      if (FULL) {
        const int64_t kv = sk - accS;
        best = kv < best ? kv : best;
      } else {
        const int32_t st = rl32(stx, y), en = rl32(enx, y);
        const int64_t kv = (lmax >= en ? sk : Pt) - accS;
        if (lmax >= st && kv < best) best = kv;
      }
    }
  }
  kk = k1;
  // H(i) for the next block: minus the comm of the block's edges with source >= i
  const int32_t kl = k0 + wave_incl_sum32(ecnt);
  if (lane < nc) H[rmod<RING>(i)] = h - E[kl];
}

// In-block steps, one target at a time: lane t takes candidate j0 + s at step
// s (s < t, and j0 + s >= lo when GEN); RS holds the lane's Int(j0 + s, j0 +
// t) shifted, reduced past each in-block source.
template <bool GEN>
__device__ inline void dp_inblock(int64_t &best, int64_t RS, int32_t smin, int32_t j0, int32_t ein,
                                  const int32_t *Q, const int32_t *T, const int64_t *C, int lane) {
  int32_t kbase = ein - 64 > 0 ? ein - 64 : 0;
  int32_t qb = kbase + lane < ein ? Q[kbase + lane] : -1;
  int32_t tb = kbase + lane < ein ? T[kbase + lane] : 0;
  int64_t cb = kbase + lane < ein ? C[kbase + lane] : 0;
  int32_t ke = ein - 1;
  int32_t nsrc = ke >= 0 ? rl32(qb, ke - kbase) - j0 : 64;
  int32_t lv = lane;
  asm volatile("" : "+v"(lv));  // keeps the per-step lane tests inside the loop
  const uint32_t len = (uint32_t)(lv - smin);
#pragma unroll
  for (int s = 0; s < 64; s++) {
    const int64_t Gs = relabel(rl64(best, s), s);
    const int64_t kv = Gs - RS;
    const bool valid = GEN ? ((uint32_t)(s - smin) < len) : (lv > s);
    if (valid && kv < best) best = kv;
    while (nsrc == s) {
      const int32_t tk = rl32(tb, ke - kbase);
      const int64_t ck = rl64(cb, ke - kbase) << kIdxBits;
      if (lane > tk) RS -= ck;
      ke--;
      if (ke >= 0 && ke < kbase) {
        kbase = ke - 63 > 0 ? ke - 63 : 0;
        qb = Q[kbase + lane < ein ? kbase + lane : 0];
        tb = T[kbase + lane < ein ? kbase + lane : 0];
        cb = C[kbase + lane < ein ? kbase + lane : 0];
      }
      nsrc = ke >= 0 ? rl32(qb, ke - kbase) - j0 : 64;
    }
  }
}

// In-block table (SMALL kernel): tab[s * kTS + t] = the comm, shifted by
// kIdxBits, of the block's edges whose source offset is at least s and whose
// target offset is below t: Int(j0 + s, j0 + t) over sources inside the
// block, what the in-block step s subtracts for target t.  Built by one wave
// from the block's in-block edges (the first ein of the list): scatter each
// edge's comm at (source, target), an exclusive prefix over targets per row
// (lane = row), then a suffix over rows per column (lane = column).
__device__ inline void dp_table(int64_t *tab, int32_t j0, int32_t ein, const int32_t *Q,
                                const int32_t *T, const int64_t *C, int lane) {
  uint4 *z = reinterpret_cast<uint4 *>(tab);
  for (int k = lane; k < 64 * kTS / 2; k += 64) z[k] = make_uint4(0, 0, 0, 0);
  for (int32_t k = lane; k < ein; k += 64)
    atomicAdd((unsigned long long *)&tab[(Q[k] - j0) * kTS + T[k]],
              (unsigned long long)C[k] << kIdxBits);
  // 16 entries at a time: every load of a chunk is issued before the first
  // use, so the running sum does not wait on one LDS round trip per entry
  int64_t run = 0;
  for (int t0 = 0; t0 < 64; t0 += 16) {
    int64_t a[16];
#pragma unroll
    for (int k = 0; k < 16; k++) a[k] = tab[lane * kTS + t0 + k];
#pragma unroll
    for (int k = 0; k < 16; k++) {
      tab[lane * kTS + t0 + k] = run;
      run += a[k];
    }
  }
  run = 0;
  for (int s0 = 63; s0 >= 0; s0 -= 16) {
    int64_t a[16];
#pragma unroll
    for (int k = 0; k < 16; k++) a[k] = tab[(s0 - k) * kTS + lane];
#pragma unroll
    for (int k = 0; k < 16; k++) {
      run += a[k];
      tab[(s0 - k) * kTS + lane] = run;
    }
  }
}

// In-block steps from the table: lane t takes candidate j0 + s at step s (s <
// t, and j0 + s >= lo when GEN) at its key less tab[s][t].  The steps form
// one dependent chain through the candidates' keys; the table rows are read
// eight steps ahead.
template <bool GEN>
__device__ inline void dp_inblock_tab(int64_t &best, int32_t smin, const int64_t *tab, int lane) {
  int32_t lv = lane;
  asm volatile("" : "+v"(lv));  // keeps the per-step lane tests inside the loop
  const uint32_t len = (uint32_t)(lv - smin);
  int64_t row[8], nrow[8];
#pragma unroll
  for (int k = 0; k < 8; k++) row[k] = tab[k * kTS + lane];
#pragma unroll
  for (int s8 = 0; s8 < 64; s8 += 8) {
#pragma unroll
    for (int k = 0; k < 8; k++) nrow[k] = s8 + 8 < 64 ? tab[(s8 + 8 + k) * kTS + lane] : 0;
#pragma unroll
    for (int k = 0; k < 8; k++) {
      const int s = s8 + k;
      const int64_t kv = relabel(rl64(best, s), s) - row[k];
      const bool valid = GEN ? ((uint32_t)(s - smin) < len) : (lv > s);
      if (valid && kv < best) best = kv;
    }
#pragma unroll
    for (int k = 0; k < 8; k++) row[k] = nrow[k];
  }
}

// In-block steps by runs: the targets between two consecutive in-block edge
// targets form a run.  Inside a run no in-block edge lies within [s, t) for
// candidates s of the run, so the run's targets take, besides their own best
// key U_t, either the best earlier candidate K (one reduction) or the best
// candidate s in [start, t) of the run, whose value is the prefix minimum of
// U: one exclusive prefix-min scan.  Y holds the finished candidates' keys as
// seen by the current run.  Requires ein <= 64 and no memory bound in-block.
__device__ inline void dp_inblock_runs(int64_t &best, uint64_t runs, int32_t j0, int32_t ein,
                                       const int32_t *Q, const int32_t *T, const int64_t *C,
                                       int lane) {
  const bool v = lane < ein;
  const int32_t se = v ? Q[lane] - j0 : 0;
  const int32_t te = v ? T[lane] : -2;
  const int64_t ce = v ? (int64_t)((uint64_t)C[lane] << kIdxBits) : 0;
  int64_t Y = kKeyInf;
  while (runs) {
    const int32_t ta = (int32_t)__builtin_ctzll(runs);
    runs &= runs - 1;
    const int32_t tb = runs ? (int32_t)__builtin_ctzll(runs) : 64;
    int64_t K = kKeyInf;
    if (ta > 0) {
      for (uint64_t m = __ballot(te == ta - 1); m; m &= m - 1) {  // edges now inside [s, t)
        const int32_t x = (int32_t)__builtin_ctzll(m);
        const int32_t sx = rl32(se, x);
        const int64_t cx = rl64(ce, x);
        if (lane <= sx) Y -= cx;
      }
      K = rl64(wave_prefix_min(Y), 63);
    }
    const bool in = lane >= ta && lane < tb;
    const int64_t U = K < best ? K : best;
    const int64_t W = in ? relabel(U, lane) : kKeyInf;
    const int64_t inc = wave_prefix_min(W);
    const int64_t X0 = __shfl(inc, lane > 0 ? lane - 1 : 0);
    const int64_t X = lane > 0 ? X0 : kKeyInf;
    const int64_t G = X < U ? X : U;
    if (in) {
      best = G;
      Y = relabel(G, lane);
    }
  }
}

// The blocked DP.  blockDim = 64 * NW: wave 0 runs the in-block steps, waves
// 1..NW-1 the candidates below the block.  SMALL (R + 64 <= kRingSmall): a
// smaller ring of H, and blocks whose in-block steps cannot go by runs take
// them from the in-block table, which wave 0 builds while the candidate waves
// work.
template <bool SMALL>
__global__ void __launch_bounds__(1024)
    k_cluster_dp(int32_t n, int32_t nb, const int32_t *lo, const int32_t *boff, const int32_t *eq,
                 const int32_t *et, const int64_t *ec, const int64_t *eE, const int64_t *PO,
                 const int32_t *pptr, const int32_t *pidx, const int64_t *cq, int32_t *P,
                 Status *st) {
  constexpr int RING = SMALL ? kRingSmall : kRingBig;
  __shared__ int64_t s_h[RING];
  __shared__ __align__(16) int64_t s_tab[SMALL ? 64 * kTS + 1 : 2];
  __shared__ int32_t s_eq[2][kEC];
  __shared__ int32_t s_et[2][kEC];
  __shared__ int64_t s_ec[2][kEC];
  __shared__ int64_t s_eE[2][kEC + 1];
  __shared__ int32_t s_lo[2][64];
  __shared__ int64_t s_wb[kMaxW][64];  // per wave: min key relative to the wave's offset
  __shared__ int64_t s_wa[kMaxW][64];  // per wave: comm (shifted) of its edges counted by the lane
  __shared__ int32_t s_hist[kMaxW + 1][64];
  __shared__ int64_t s_hc[64];
  __shared__ int64_t s_bm[16];  // per wave: the minimum key of a dense block's target
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int W = (int)(blockDim.x >> 6) - 1, NT = W * 64;

  // block 0 staged by everyone; histograms cleared
  int32_t o0 = 0, o1 = boff[1 < nb ? 1 : nb], o2 = boff[2 < nb ? 2 : nb];
  {
    const int32_t c0 = o1 <= kEC ? o1 : 0;  // a dense block 0 is not staged
    for (int32_t k = tid; k < c0; k += blockDim.x) {
      s_eq[0][k] = eq[k];
      s_et[0][k] = et[k];
      s_ec[0][k] = ec[k];
      s_eE[0][k] = eE[k];
      if (k == c0 - 1) s_eE[0][c0] = eE[k] + ec[k];
    }
    if (tid == 0 && c0 == 0) s_eE[0][0] = 0;
    if (tid < 64) s_lo[0][tid] = tid == 0 ? 0 : lo[tid <= n ? tid : n];
    for (int k = tid; k < (kMaxW + 1) * 64; k += blockDim.x) (&s_hist[0][0])[k] = 0;
    if (tid < 64) s_hc[tid] = 0;
    for (int k = W * 64 + tid; k < kMaxW * 64; k += blockDim.x) {  // rows of absent waves
      (&s_wb[0][0])[k] = kKeyInf;
      (&s_wa[0][0])[k] = 0;
    }
  }

#ifdef CEL_PHASE_TIMERS
  unsigned long long tp_prev = wall_clock64();
#endif
  for (int32_t b = 0; b < nb; b++) {
    __syncthreads();  // staging of block b and H of block b - 1 visible
    CEL_TSTAMP(tp_a);
#ifdef CEL_PHASE_TIMERS
    if (tid == 0) {
      atomicAdd(&g_cel_phase[3], tp_a - tp_prev);
      atomicAdd(&g_cel_phase[6], 1ull);
    }
#endif
    const int buf = b & 1;
    const int32_t j0 = b * 64, base = j0 - kBaseOff;
    const int32_t cnt = o1 - o0;
    const int32_t o3 = boff[b + 3 < nb ? b + 3 : nb];
    const bool more = b + 1 < nb;
    if (cnt > kEC) {
      // A dense block (more window edges than the staging holds): its targets
      // one at a time by the whole workgroup, straight from the in-edge lists.
      // Before target j, H(i) = V_j(i); S(j) takes the smallest key over the
      // candidates [lo(j), j); then H(j) = S(j) - PO[j] and every candidate i
      // loses the comm of j's in-edges from sources at or after i.
      const int nwv = (int)(blockDim.x >> 6);
      for (int t = 0; t < 64; t++) {
        const int32_t j = j0 + t;
        if (j > n) break;
        const int32_t loj = j == 0 ? 0 : lo[j];
        int64_t key = j == 0 ? (int64_t)kBaseOff : kKeyInf;  // S(0) = 0
        for (int32_t i = loj + tid; i < j; i += blockDim.x) {
          const int64_t kv = (int64_t)((uint64_t)s_h[rmod<RING>(i)] << kIdxBits) + (i - base);
          key = kv < key ? kv : key;
        }
        for (int off = 32; off > 0; off >>= 1) {
          const int64_t o = __shfl_xor((long long)key, off);
          key = o < key ? o : key;
        }
        if (lane == 0) s_bm[wave] = key;
        __syncthreads();
        key = s_bm[0];
        for (int w = 1; w < nwv; w++) key = s_bm[w] < key ? s_bm[w] : key;
        const int64_t G = key >> kIdxBits;
        if (tid == 0) {
          if (j >= 1) P[j] = (int32_t)(key & kIdxMask) + base;
          if (j == n) st->s0 = PO[n] + G;
        }
        if (j < n) {
          const int32_t e0 = pptr[j], e1 = pptr[j + 1];
          for (int32_t i = loj + tid; i < j; i += blockDim.x) {
            int64_t d = 0;
            for (int32_t e = e0; e < e1; e++) {
              const int32_t q = pidx[e];
              if (q >= i) d += cq[q];
            }
            if (d) s_h[rmod<RING>(i)] -= d;
          }
          if (tid == 0) s_h[rmod<RING>(j)] = G;
        }
        __syncthreads();  // H and s_bm settled before the next target
      }
      // stage block b + 1 (unless it is dense too)
      const int nbuf = buf ^ 1;
      const int32_t c1 = o2 - o1;
      if (more && c1 <= kEC) {
        for (int32_t k = tid; k < c1; k += blockDim.x) {
          const int32_t e = o1 + k;
          s_eq[nbuf][k] = eq[e];
          s_et[nbuf][k] = et[e];
          s_ec[nbuf][k] = ec[e];
          s_eE[nbuf][k] = eE[e];
          if (k == c1 - 1) s_eE[nbuf][c1] = eE[e] + ec[e];
        }
        if (tid == 0 && c1 == 0) s_eE[nbuf][0] = 0;
      }
      if (more && tid < 64) {
        const int32_t jj = j0 + 64 + tid;
        s_lo[nbuf][tid] = lo[jj <= n ? jj : n];
      }
      o0 = o1;
      o1 = o2;
      o2 = o3;
      continue;
    }
    const int32_t *Q = s_eq[buf];
    const int32_t *T = s_et[buf];
    const int64_t *Cc = s_ec[buf];
    const int64_t *E = s_eE[buf];
    const int32_t lo_t = s_lo[buf][lane];
    const int32_t lo_hi = s_lo[buf][63];  // lo is nondecreasing: the block's largest

    // prefetch of block b + 1 into registers (waves 1..W)
    int32_t pq[kPF], pt[kPF], plo = 0;
    int64_t pc[kPF], pE[kPF];
#pragma unroll
    for (int r = 0; r < kPF; r++) {
      pq[r] = pt[r] = 0;
      pc[r] = pE[r] = 0;
    }
    if (wave >= 1 && more) {
      const int x = tid - 64;
#pragma unroll
      for (int r = 0; r < kPF; r++) {
        const int32_t e = o1 + x + r * NT;
        if (e < o2) {
          pq[r] = eq[e];
          pt[r] = et[e];
          pc[r] = ec[e];
          pE[r] = eE[e];
        }
      }
      if (x < 64) {
        const int32_t jj = j0 + 64 + x;
        plo = lo[jj <= n ? jj : n];
      }
    }

    int32_t ein = 0;
    int64_t XS = 0, Nt = 0;
    uint64_t runs = 1;
    if (wave == 0) {
      // in-block edges: per-source counts and per-target comm
      ein = first_le(Q, cnt, j0 - 1, lane);
      for (int32_t k = lane; k < ein; k += 64) {
        atomicAdd(&s_hist[kMaxW][Q[k] - j0], 1);
        atomicAdd((unsigned long long *)&s_hc[T[k]], (unsigned long long)Cc[k]);
      }
      wave_lds_sync();
      const int32_t sc = s_hist[kMaxW][lane];
      const int64_t hc = s_hc[lane];
      s_hist[kMaxW][lane] = 0;
      s_hc[lane] = 0;
      XS = (int64_t)((uint64_t)(wave_incl_sum64(hc) - hc) << kIdxBits);  // edges with t_e < t
      const int32_t ks = ein - (wave_incl_sum32(sc) - sc);                 // edges with q >= j0 + t
      Nt = E[ks];
      runs = (__ballot(hc > 0) << 1) | 1ull;  // a run starts after each in-block edge target
      if (SMALL && (lo_hi > j0 || ein > 64 || __popcll(runs) > kMaxRuns))
        dp_table(s_tab, j0, ein, Q, T, Cc, lane);
    } else {
      // candidates below the block: chunks [ka, kb) of 64, descending
      const int w = wave - 1;
      int64_t best = kKeyInf, accS = 0;
      if (j0 > 0) {
        // the candidates [lo0, j0), split evenly: wave w takes the w-th range
        // from the top, in chunks of at most 64
        const int32_t lo0 = s_lo[buf][0];
        const int32_t Nc = j0 - lo0;
        const int32_t sa = (int32_t)((int64_t)w * Nc / W), sb = (int32_t)((int64_t)(w + 1) * Nc / W);
        if (sa < sb) {
          const int32_t top = j0 - 1 - sa;
          const int32_t bot = j0 - sb;
          int32_t kk = first_le(Q, cnt, top, lane);
          for (int32_t ct = top; ct >= bot; ct -= 64) {
            const int32_t cb = ct - 63 > bot ? ct - 63 : bot;
            if (lo_hi <= cb)
              dp_chunk<true, RING>(ct, cb, base, lo_t, s_hist[w], s_h, Q, T, Cc, E, cnt, kk, best,
                                   accS, lane);
            else
              dp_chunk<false, RING>(ct, cb, base, lo_t, s_hist[w], s_h, Q, T, Cc, E, cnt, kk, best,
                                    accS, lane);
          }
        }
      }
      s_wb[w][lane] = best;
      s_wa[w][lane] = accS;
    }
#ifdef CEL_PHASE_TIMERS
    {
      const unsigned long long t = wall_clock64();
      if (lane == 0 && wave < 6) atomicAdd(&g_cel_phase[8 + wave], t - tp_a);
    }
#endif
    __syncthreads();  // wave results visible
    CEL_TSTAMP(tp_b);
#ifdef CEL_PHASE_TIMERS
    if (tid == 0) atomicAdd(&g_cel_phase[1], tp_b - tp_a);
#endif

    if (wave == 0) {
      const int32_t j = j0 + lane;
      int64_t best = j == 0 ? (int64_t)kBaseOff : kKeyInf;  // S(0) = 0
      int64_t off = XS;
      // every wave's results read at once (rows past W: kKeyInf and 0)
      int64_t wb[kMaxW], wa[kMaxW];
#pragma unroll
      for (int w = 0; w < kMaxW; w++) {
        wb[w] = s_wb[w][lane];
        wa[w] = s_wa[w][lane];
      }
      // key of wave w's best relative to the offset of the waves above it: a
      // prefix sum of the offsets, then a minimum tree
      int64_t kv[16];
#pragma unroll
      for (int w = 0; w < kMaxW; w++) {
        kv[w] = wb[w] - off;  // rows past W: kKeyInf - off, above every real key
        off += wa[w];
      }
      kv[15] = best;
#pragma unroll
      for (int h = 8; h > 0; h >>= 1)
#pragma unroll
        for (int w = 0; w < h; w++) kv[w] = kv[w + h] < kv[w] ? kv[w + h] : kv[w];
      best = kv[0];
      const int32_t smin = lo_t - j0 > 0 ? lo_t - j0 : 0;
      CEL_TSTAMP(tq0);
      CEL_TADD(20, tp_b, tq0);
      if (SMALL && lo_hi > j0) {
        dp_inblock_tab<true>(best, smin, s_tab, lane);
        CEL_TSTAMP(tq1);
        CEL_TADD(14, tq0, tq1);
        CEL_TCOUNT(15);
      } else if (SMALL && (ein > 64 || __popcll(runs) > kMaxRuns)) {
        dp_inblock_tab<false>(best, smin, s_tab, lane);
        CEL_TSTAMP(tq1);
        CEL_TADD(18, tq0, tq1);
        CEL_TCOUNT(19);
      } else if (lo_hi > j0) {
        dp_inblock<true>(best, XS, smin, j0, ein, Q, T, Cc, lane);
        CEL_TSTAMP(tq1);
        CEL_TADD(14, tq0, tq1);
        CEL_TCOUNT(15);
      } else if (ein <= 64 && __popcll(runs) <= kMaxRuns) {
        dp_inblock_runs(best, runs, j0, ein, Q, T, Cc, lane);
        CEL_TSTAMP(tq1);
        CEL_TADD(16, tq0, tq1);
        CEL_TCOUNT(17);
      } else {
        dp_inblock<false>(best, XS, smin, j0, ein, Q, T, Cc, lane);
        CEL_TSTAMP(tq1);
        CEL_TADD(18, tq0, tq1);
        CEL_TCOUNT(19);
      }
      const int64_t G = best >> kIdxBits;
      if (j >= 1 && j <= n) P[j] = (int32_t)(best & kIdxMask) + base;
      if (j < n) s_h[rmod<RING>(j)] = G - Nt;
      if (j == n) st->s0 = PO[n] + G;
    } else if (more) {
      // stage block b + 1 (a dense one is not staged: it reads global memory)
      const int nbuf = buf ^ 1;
      const int x = tid - 64;
      const int32_t c1 = o2 - o1 <= kEC ? o2 - o1 : 0;
#pragma unroll
      for (int r = 0; r < kPF; r++) {
        const int32_t k = x + r * NT;
        if (k < c1) {
          s_eq[nbuf][k] = pq[r];
          s_et[nbuf][k] = pt[r];
          s_ec[nbuf][k] = pc[r];
          s_eE[nbuf][k] = pE[r];
          if (k == c1 - 1) s_eE[nbuf][c1] = pE[r] + pc[r];
        }
      }
      for (int32_t k = x + kPF * NT; k < c1; k += NT) {
        const int32_t e = o1 + k;
        s_eq[nbuf][k] = eq[e];
        s_et[nbuf][k] = et[e];
        s_ec[nbuf][k] = ec[e];
        s_eE[nbuf][k] = eE[e];
        if (k == c1 - 1) s_eE[nbuf][c1] = eE[e] + ec[e];
      }
      if (x == 0 && c1 == 0) s_eE[nbuf][0] = 0;
      if (x < 64) s_lo[nbuf][x] = plo;
    }
#ifdef CEL_PHASE_TIMERS
    {
      const unsigned long long t = wall_clock64();
      if (tid == 0) atomicAdd(&g_cel_phase[2], t - tp_b);
      if (tid == 64) atomicAdd(&g_cel_phase[5], t - tp_b);
      tp_prev = t;
    }
#endif
    o0 = o1;
    o1 = o2;
    o2 = o3;
  }
}

// Cluster starts by following a chain of positions: the DP's backtrack from
// n down through P (P[j] < j, at least j - R), or the greedy walk from 0 up
// through gend (gend[s] > s, at most s + R), flagging every start.  The chain
// is sequential, so one thread walks it, but through LDS: the table is staged
// in windows of kWalkWin positions, the next window loaded by waves 1-15 (all
// their loads in flight at once) while thread 0 walks the current one (a
// step moves at most R <= 4096 positions, so it never skips a window).
constexpr int kWalkWin = 16384;
constexpr int kWalkB = 1024;
constexpr int kWalkPer = (kWalkWin + kWalkB - 64 - 1) / (kWalkB - 64);  // loads per loading thread
static_assert(kWalkWin > 4096, "a step of at most R = 4096 positions stays in the next window");
template <bool DOWN>
__global__ void __launch_bounds__(kWalkB) k_walk(int32_t n, const int32_t *next, int32_t *flag,
                                                 Status *st) {
  __shared__ int32_t s_w[2][kWalkWin];
  __shared__ int32_t s_done[2];  // by window parity: a slow wave may still read the last one
  if (failed(st)) return;
  const int tid = threadIdx.x;
  // entries of the table: DOWN: next[0..n] (next[0] unused), UP: next[0..n-1]
  const int32_t ne = DOWN ? n + 1 : n;
  // window w covers [wlo, wlo + kWalkWin) clipped to [0, ne)
  auto wstart = [&](int32_t w) -> int32_t {
    return DOWN ? ne - (w + 1) * kWalkWin : w * kWalkWin;  // may be negative when DOWN
  };
  auto load = [&](int buf, int32_t w, int t0, int nt) {
    const int32_t lo = wstart(w);
    for (int32_t i0 = t0; i0 < kWalkWin; i0 += nt * kWalkPer) {
      int32_t v[kWalkPer];
#pragma unroll
      for (int u = 0; u < kWalkPer; u++) {
        const int32_t x = lo + i0 + u * nt;
        v[u] = (x >= 0 && x < ne && i0 + u * nt < kWalkWin) ? next[x] : 0;
      }
#pragma unroll
      for (int u = 0; u < kWalkPer; u++)
        if (i0 + u * nt < kWalkWin) s_w[buf][i0 + u * nt] = v[u];
    }
  };
  if (tid == 0) s_done[0] = s_done[1] = 0;
  load(0, 0, tid, kWalkB);
  __syncthreads();
  int32_t b = DOWN ? n : 0, C = 0;  // thread 0's walk
  for (int32_t w = 0;; w++) {
    const int buf = w & 1;
    int32_t &done = s_done[buf];
    if (tid >= 64) load(buf ^ 1, w + 1, tid - 64, kWalkB - 64);
    if (tid == 0) {
      const int32_t lo = wstart(w);
      bool moved = false;
      if (DOWN) {
        while (b > 0 && b >= lo) {
          const int32_t a = s_w[buf][b - lo];
          if (a < 0 || a >= b) {  // cannot happen: every step has a feasible predecessor
            raise_err(st, EB_ORDER);
            done = 1;
            break;
          }
          b = a;
          flag[b] = 1;
          C++;
          moved = true;
        }
        if (b == 0) done = 1;
      } else {
        while (b < n && b < lo + kWalkWin) {
          flag[b] = 1;
          C++;
          const int32_t e = s_w[buf][b - lo];
          if (e <= b || e > n) {
            raise_err(st, EB_ORDER);
            done = 1;
            break;
          }
          b = e;
          moved = true;
        }
        if (b >= n) done = 1;
      }
      // a chain that neither ends nor reaches this window (a corrupt table)
      if (!moved && !done) {
        raise_err(st, EB_ORDER);
        done = 1;
      }
      if (done) st->i0 = C;
    }
    __syncthreads();
    if (done) break;
  }
}

// cluster_id[order[p]] = (number of cluster starts at or before p) - 1
__global__ void k_label(int32_t n, const int32_t *order, const int32_t *incl, int32_t *cid,
                        const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x)
    cid[order[p]] = incl[p + 1] - 1;
}

// sum of c[u] over edges u -> v in different clusters (edge-balanced blocks)
__global__ void k_cut_cost(cel_graph g, int64_t bw, int64_t lat, const int32_t *cid, Status *st) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  __shared__ int64_t red[4];
  if (failed(st)) return;
  int64_t acc = 0;
  for_edges_balanced(g.out_ptr, g.n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    if (cid[u] != cid[g.out_idx[e]]) acc += comm_of(g.ob[u], bw, lat);
  });
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int64_t t = red[0] + red[1] + red[2] + red[3];
    atomicAdd((unsigned long long *)&st->s0, (unsigned long long)t);
  }
}

template <int SL>
static void launch_dp(int32_t n, int32_t R, const int32_t *lo, const int32_t *pptr,
                      const int32_t *pidx, const int64_t *cq, const int64_t *PO, int32_t *P,
                      Status *st, hipStream_t s) {
  KTimer kt(s, "k_cluster_dp_step");
  k_cluster_dp_step<SL><<<1, 64, 0, s>>>(n, R, lo, pptr, pidx, cq, PO, P, st);
}

// Blocked DP when every block fits the staging sizes (sets *done), else
// leaves the step-wise kernel to the caller.
static int dp_blocked(int32_t n, int32_t m, int32_t R, const int32_t *lo, const int32_t *pptr,
                      const int32_t *pidx, const int64_t *cq, const int64_t *PO, int32_t *P,
                      Status *st, Scratch &sc, hipStream_t s, bool *done) {
  *done = false;
  const int32_t nb = n / 64 + 1;
  int32_t *bcnt, *boff, *mx;
  CEL_TRY(sc.get(&bcnt, nb));
  CEL_TRY(sc.get(&boff, (int64_t)nb + 1));
  CEL_TRY(sc.get(&mx, 1));
  CEL_HIP(hipMemsetAsync(mx, 0, sizeof(int32_t), s));
  {
    k_dp_count<<<grid_for((int64_t)nb * 64, 256, 4096), 256, 0, s>>>(n, nb, pptr, pidx, lo, bcnt,
                                                                     mx, st);
  }
  CEL_TRY(exclusive_scan_i32(bcnt, boff, nb, sc, s));
  int64_t total = 0;
  CEL_HIP(hipMemcpyAsync(&total, PO + n, sizeof total, hipMemcpyDeviceToHost, s));
  CEL_HIP(hipStreamSynchronize(s));
  if (total >= kPackLim) return CEL_OK;  // step-wise kernel (keys need values below 2^48)
  int32_t *eq, *et;
  int64_t *ec, *eE;
  CEL_TRY(sc.get(&eq, m));
  CEL_TRY(sc.get(&et, m));
  CEL_TRY(sc.get(&ec, m));
  CEL_TRY(sc.get(&eE, m));
  {
    k_dp_fill<<<nb < 65535 ? nb : 65535, 256, 0, s>>>(n, nb, pptr, pidx, lo, cq, boff, eq, et, ec,
                                                      eE, st);
  }
  const int32_t K = (R + 15) / 16;  // about 16 candidates per wave
  const int NW = 1 + (K < kMaxW ? K : kMaxW);
  {
    KTimer kt(s, "k_cluster_dp");
    if (R + 64 <= kRingSmall)
      k_cluster_dp<true><<<1, 64 * NW, 0, s>>>(n, nb, lo, boff, eq, et, ec, eE, PO, pptr, pidx, cq,
                                              P, st);
    else
      k_cluster_dp<false><<<1, 64 * NW, 0, s>>>(n, nb, lo, boff, eq, et, ec, eE, PO, pptr, pidx,
                                               cq, P, st);
  }
  CEL_HIP(hipGetLastError());
  *done = true;
  return CEL_OK;
}

CEL_PHASE_READER(cel_debug_phases_cluster)

}  // namespace cel

using namespace cel;

constexpr int32_t kDpPolicyN = 16384;  // smaller graphs take the blocked DP directly

// How the calling thread's last cel_cluster call ran its DP.
struct ClInfo {
  int32_t path, iters;
};
static thread_local ClInfo t_cl_info{1, 0};

extern "C" int cel_cluster_info(int32_t *info) {
  if (!info) return set_error(CEL_E_ARG, "cel_cluster_info: NULL argument");
  info[0] = t_cl_info.path;
  info[1] = t_cl_info.iters;
  return CEL_OK;
}

extern "C" int cel_cluster(const cel_graph *g, const cel_devices *d, const int32_t *order,
                           int32_t R, int64_t M, int32_t mode, int32_t *cluster_id,
                           int32_t *n_clusters, int64_t *cut_cost, hipStream_t s) {
  const char *fn = "cel_cluster";
  CEL_TRY(check_host_graph(g, fn));
  CEL_TRY(check_host_devices(d, fn));
  const int32_t n = g->n;
  if (!n_clusters || !cut_cost || (n > 0 && (!order || !cluster_id)))
    return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  if (R < 1 || R > 4096) return set_error(CEL_E_ARG, "%s: R = %d not in [1, 4096]", fn, R);
  if (M < -1) return set_error(CEL_E_ARG, "%s: M < -1", fn);
  if (mode != CEL_CLUSTER_DP && mode != CEL_CLUSTER_GREEDY)
    return set_error(CEL_E_ARG, "%s: unknown mode", fn);
  if (M == -1) {
    int64_t mc = d->cap[0];
    for (int i = 1; i < d->D; i++) mc = d->cap[i] < mc ? d->cap[i] : mc;
    M = mc / 4;
  }
  Scratch sc(s);
  Status *st;
  int32_t *tmp, *pos;
  CEL_TRY(sc.get(&st, 1));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(sc.get(&tmp, n));
  CEL_TRY(sc.get(&pos, n));
  CEL_TRY(check_graph(g, d->bw, d->lat, true, st, tmp, sc, s));
  CEL_TRY(check_topo_order(g, order, pos, st, s));
  if (n == 0) {
    Status h;
    CEL_TRY(read_status(st, &h, s));
    if (h.err) return status_error(h, fn);
    *n_clusters = 0;
    *cut_cost = 0;
    return CEL_OK;
  }
  int64_t *memp, *cq, *outc, *PM, *PO;
  int32_t *lo, *gend, *flag, *incl;
  CEL_TRY(sc.get(&memp, n));
  CEL_TRY(sc.get(&cq, n));
  CEL_TRY(sc.get(&outc, n));
  CEL_TRY(sc.get(&PM, (int64_t)n + 1));
  CEL_TRY(sc.get(&PO, (int64_t)n + 1));
  CEL_TRY(sc.get(&lo, (int64_t)n + 1));
  CEL_TRY(sc.get(&gend, n));
  CEL_TRY(sc.get(&flag, n));
  CEL_TRY(sc.get(&incl, (int64_t)n + 1));
  k_cluster_pos<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, g->out_ptr, g->mem, g->ob, d->bw,
                                                      d->lat, memp, cq, outc, st);
  CEL_TRY(exclusive_scan_i64(memp, PM, n, sc, s));
  CEL_HIP(hipMemsetAsync(flag, 0, sizeof(int32_t) * (size_t)n, s));
  k_cluster_bounds<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, R, M, PM, lo, gend, st);
  if (mode == CEL_CLUSTER_DP) {
    int32_t *pptr, *pidx, *P;
    CEL_TRY(sc.get(&pptr, (int64_t)n + 1));
    CEL_TRY(sc.get(&pidx, g->m));
    CEL_TRY(sc.get(&P, (int64_t)n + 1));
    CEL_TRY(exclusive_scan_i64(outc, PO, n, sc, s));
    // policy iteration first (graphs of kDpPolicyN nodes and more)
    bool solved = false;
    t_cl_info = {1, 0};
    if (n >= kDpPolicyN && policy_iteration_on()) {
      int32_t *sptr, *sidx;
      CEL_TRY(sc.get(&sptr, (int64_t)n + 1));
      CEL_TRY(sc.get(&sidx, g->m));
      CEL_TRY(relabel_csr(n, g->m, order, pos, g->out_ptr, g->out_idx, sptr, sidx, sc, s, st));
      bool launched = false;
      CEL_TRY(dp_policy(n, g->m, R, lo, PO, cq, sptr, sidx, P, sc, s, st, &launched));
      if (launched) {
        Status h;
        CEL_TRY(read_status(st, &h, s));
        if (h.err) return status_error(h, fn);
        solved = h.i2 != 0;
        t_cl_info = {solved ? 0 : 1, h.i3};
      }
    }
    bool blocked = false;
    if (!solved) {
      CEL_TRY(relabel_csr(n, g->m, order, pos, g->in_ptr, g->in_idx, pptr, pidx, sc, s, st));
      CEL_TRY(dp_blocked(n, g->m, R, lo, pptr, pidx, cq, PO, P, st, sc, s, &blocked));
    }
    if (solved || blocked) {
    } else if (R <= 64) launch_dp<1>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 128) launch_dp<2>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 256) launch_dp<4>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 512) launch_dp<8>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 1024) launch_dp<16>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else if (R <= 2048) launch_dp<32>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    else launch_dp<64>(n, R, lo, pptr, pidx, cq, PO, P, st, s);
    bool marked = false;
    if (policy_iteration_on()) CEL_TRY(chain_marks(n, P, flag, sc, s, st, &marked));
    if (!marked) k_walk<true><<<1, kWalkB, 0, s>>>(n, P, flag, st);
  } else {
    k_walk<false><<<1, kWalkB, 0, s>>>(n, gend, flag, st);
  }
  CEL_TRY(exclusive_scan_i32(flag, incl, n, sc, s));
  k_label<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, incl, cluster_id, st);
  if (mode == CEL_CLUSTER_GREEDY)
    k_cut_cost<<<edge_blocks(g->m), 256, 0, s>>>(*g, d->bw, d->lat, cluster_id, st);
  CEL_HIP(hipGetLastError());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, fn);
  *n_clusters = h.i0;
  *cut_cost = h.s0;
  return CEL_OK;
}
