// The clustering DP (Section 5.1.3, eq. 4-6) by policy iteration.
//
// In position space, with PO the prefix sum of each node's out-going comm and
// Int(i, j) the comm of the edges with both ends in [i, j):
//   S(0) = 0,  S(j) = min over lo(j) <= i < j of S(i) + cost(i, j),
//   cost(i, j) = PO[j] - PO[i] - Int(i, j),
// a shortest path from 0 to every j over the breakpoint graph.  A policy is a
// back pointer P(j) in [lo(j), j) for every j; its values S_P(j) = S_P(P(j)) +
// cost(P(j), j) are sums along the pointers, found by pointer jumping.  Each
// j then switches to the candidate i of smallest S_P(i) + cost(i, j) when that
// is strictly below S_P(j).  Every policy's values are costs of real
// clusterings, a switch never raises a value, and when no j can switch the
// values satisfy the recurrence, whose solution is unique: S is exact.  The
// back pointers are then set to the smallest minimising i (the tie rule), so
// the breakpoints are those of the sequential DP.  Transformer-96 needs 9
// iterations where the blocked DP runs 16,728 dependent blocks.
//
// Improvement: one thread per target j sweeps its candidates i = j - 1 down to
// lo(j), keeping Int(i, j) = Int(i + 1, j) + c(i) * #{successors of i at
// offsets below j - i}.  The offsets below R of each position's successors
// are packed four to a 64-bit word (14 bits each), or, for a position with
// more, kept as a table of counts below every d: every count is one load.
// Neighbouring threads read neighbouring candidates, so the window's data is
// read from the L1 cache; S - PO of the candidates is published behind a grid
// barrier with agent-scope fences (the plain, cached loads need them), every
// other value crossing workgroups goes through agent-scope atomics.
#include <map>
#include <mutex>

#include "cel_internal.h"

namespace cel {

constexpr int kDpB = 1024;
constexpr int kDpU = 4;          // nodes per thread with loads in flight together
constexpr uint32_t kDpOffMask = 0x3FFF;

// near successors: count per position (edge-balanced over the position CSR)
__global__ void k_dpn_count(int32_t n, int32_t m, int32_t R, const int32_t *sptr,
                            const int32_t *sidx, int32_t *ncnt, const Status *st) {
  __shared__ int32_t rp[kRowsPB + 1], su[2];
  if (failed(st)) return;
  for_edges_balanced(sptr, n, m, rp, su, [&](int32_t i, int32_t e) {
    const int32_t o = sidx[e] - i;
    if (o > 0 && o < R) atomicAdd(&ncnt[i], 1);
  });
}

__global__ void k_dpn_fill(int32_t n, int32_t m, int32_t R, const int32_t *sptr,
                           const int32_t *sidx, const int32_t *nptr, int32_t *ncnt,
                           uint16_t *noff, const Status *st) {
  __shared__ int32_t rp[kRowsPB + 1], su[2];
  if (failed(st)) return;
  for_edges_balanced(sptr, n, m, rp, su, [&](int32_t i, int32_t e) {
    const int32_t o = sidx[e] - i;
    if (o > 0 && o < R) noff[nptr[i] + atomicSub(&ncnt[i], 1) - 1] = (uint16_t)o;
  });
}

// Each position's offsets below R: up to four packed in a 64-bit word (14
// bits each, the unused ones kDpOffMask, above any offset); a position with
// more gets kDpHeavy | h, h its index among such positions, whose counts of
// offsets below d (d = 0..R, parallel edges counted each) form a table of
// R + 1 entries.
constexpr uint64_t kDpHeavy = uint64_t(1) << 62;

__global__ void k_dpn_heavy(int32_t n, const int32_t *nptr, int32_t *hflag, const Status *st) {
  if (failed(st)) return;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    hflag[i] = nptr[i + 1] - nptr[i] > 4 ? 1 : 0;
}

__global__ void k_dpn_pack(int32_t n, int32_t R, const int32_t *nptr, const uint16_t *noff,
                           const int32_t *hoff, uint64_t *nearw, uint32_t *hcnt,
                           const Status *st) {
  if (failed(st)) return;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t b = nptr[i], e = nptr[i + 1];
    if (e - b > 4) {
      const int64_t h = hoff[i];
      uint32_t *t = hcnt + h * (R + 1);
      for (int32_t d = 0; d <= R; d++) t[d] = 0;
      for (int32_t x = b; x < e; x++) t[noff[x] + 1]++;  // offsets < R: index <= R
      for (int32_t d = 1; d <= R; d++) t[d] += t[d - 1];  // t[d] = offsets below d
      nearw[i] = kDpHeavy | (uint64_t)h;
      continue;
    }
    uint16_t o[4] = {kDpOffMask, kDpOffMask, kDpOffMask, kDpOffMask};
    for (int32_t x = b; x < e; x++) o[x - b] = noff[x];
    uint64_t w = 0;
    for (int k = 0; k < 4; k++) w |= (uint64_t)o[k] << (16 * k);
    nearw[i] = w;
  }
}

struct DpArgs {
  int32_t n, R, cap, max_rounds;
  int32_t packed;             // packed entries allowed where the values fit
  const int32_t *lo;          // [n + 1] first feasible i of a cluster ending at j
  const int64_t *PO;          // [n + 1]
  const int64_t *cq;          // [n] comm by position
  const uint64_t *nearw;      // [n] packed successor offsets below R, or a bitmask's index
  const uint32_t *hcnt;       // [H][R + 1] offsets below d of the positions with many
  int32_t *P;                 // [n + 1] back pointers (the output)
  int32_t *Parg;              // [n + 1] the smallest minimising i of the last improvement
  int64_t *cost;              // [n + 1] cost(P(j), j)
  int64_t *SP;                // [n + 1] S(i) - PO[i]
  LpE *e0, *e1;               // [n + 1] pointer-jumping entries
  int32_t *bar;
  Status *st;
};

// successors of a position at offsets below d (1 <= d <= R)
// (SWAR over the four 16-bit fields: a field b, an offset below 2^12 or the
// unused 0x3FFF, has bits 14-15 clear, so (0x8000 | d) - (b + 1) neither
// borrows nor carries across fields and keeps bit 15 exactly when b < d.)
__device__ inline int32_t dp_near_below(const DpArgs &a, uint64_t w, uint32_t d) {
  if (w & kDpHeavy) return (int32_t)a.hcnt[(int64_t)(uint32_t)w * (a.R + 1) + d];
  constexpr uint64_t kOnes = 0x0001000100010001ull, kHigh = 0x8000800080008000ull;
  const uint64_t t = (((uint64_t)d * kOnes) | kHigh) - (w + kOnes);
  return __popcll(t & kHigh);
}

template <bool PK>
__device__ inline void dp_run(const DpArgs &a, int32_t *s_okp, int32_t *s_bitp) {
  int32_t &s_ok = *s_okp, &s_bit = *s_bitp;
  Status *st = a.st;
  const int32_t n = a.n;
  uint64_t *E = reinterpret_cast<uint64_t *>(a.e0);  // PK: one packed entry per position
  const int64_t gsz = (int64_t)gridDim.x * kDpB;
  const int64_t gid = (int64_t)blockIdx.x * kDpB + threadIdx.x;
  int32_t bar = 0, bit;
  // The first policy: clusters of half the window, R / 2 positions (fewer
  // where lo(j) binds), cost(P(j), j) from one scan of each window.  Chains
  // of n / (R / 2) pointers instead of the n of singleton clusters: on the
  // transformer graphs a third fewer pointer-jumping passes in all, with no
  // more iterations (any policy is a valid start; only the fixed point ends
  // the iteration).
  const int32_t h = a.R / 2 > 1 ? a.R / 2 : 1;
  for (int64_t j = gid; j <= n; j += gsz) {
    if (j == 0) {
      st32(&a.P[0], -1);
      st_coherent(&a.cost[0], 0);
      continue;
    }
    const int32_t lj = a.lo[j];
    const int32_t p = (int32_t)j - h > lj ? (int32_t)j - h : lj;
    int64_t Int = 0;
    for (int32_t i = (int32_t)j - 1; i >= p; i--)
      Int += a.cq[i] * dp_near_below(a, a.nearw[i], (uint32_t)(j - i));
    st32(&a.P[j], p);
    st_coherent(&a.cost[j], a.PO[j] - a.PO[p] - Int);
  }
  if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
  LpE *cur = a.e0, *oth = a.e1;
  int32_t it = 0;
  bool done = false;
  for (; it < a.cap; it++) {
    if (PK) {
      // ---- evaluation, packed entries (see pk_make): one hop folded in,
      // a grid barrier, then asynchronous jumps; position 0 ends a chain
      for (int64_t j0 = gid; j0 <= n; j0 += kDpU * gsz) {
        int32_t q[kDpU];
#pragma unroll
        for (int u = 0; u < kDpU; u++) {
          const int64_t j = j0 + u * gsz;
          q[u] = j <= n ? ld32(&a.P[j]) : -1;
        }
        int64_t cq_[kDpU];
        int32_t nq[kDpU];
#pragma unroll
        for (int u = 0; u < kDpU; u++) {
          cq_[u] = q[u] > 0 ? ld_coherent(&a.cost[q[u]]) : 0;
          nq[u] = q[u] > 0 ? ld32(&a.P[q[u]]) : -1;
        }
#pragma unroll
        for (int u = 0; u < kDpU; u++) {
          const int64_t j = j0 + u * gsz;
          if (j <= n)
            pk_st(E + j, pk_make(ld_coherent(&a.cost[j]) + cq_[u], nq[u] > 0 ? (uint32_t)nq[u] : kPkEnd));
        }
      }
      if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
      for (int64_t j0 = gid; j0 <= n; j0 += kPkU * gsz) {
        uint64_t e[kPkU];
#pragma unroll
        for (int u = 0; u < kPkU; u++) {
          const int64_t j = j0 + u * gsz;
          e[u] = j <= n ? pk_ld(E + j) : pk_make(0, kPkEnd);
        }
        for (int32_t k = 0;; k++) {  // back pointers decrease: every chain ends
          uint64_t f[kPkU];
          bool any = false;
#pragma unroll
          for (int u = 0; u < kPkU; u++) {
            const uint32_t x = pk_next(e[u]);
            f[u] = x != kPkEnd ? pk_ld(E + x) : 0;
          }
#pragma unroll
          for (int u = 0; u < kPkU; u++) {
            if (pk_next(e[u]) == kPkEnd) continue;
            e[u] = pk_make(pk_val(e[u]) + pk_val(f[u]), pk_next(f[u]));
            pk_st(E + j0 + u * gsz, e[u]);
            any |= pk_next(e[u]) != kPkEnd;
          }
          if (!any) break;
          if (k > n) {  // cannot happen (P(j) < j); bounded all the same
            raise_err(st, EB_ORDER);
            break;
          }
        }
      }
      if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
      if (ld32(reinterpret_cast<const int32_t *>(&st->err))) return;  // uniform after the barrier
    } else {
  // ---- evaluation: S(j) = sum of cost along the back pointers (P(j) = 0 ends a chain)
      int32_t more = 0;
      for (int64_t j0 = gid; j0 <= n; j0 += kDpU * gsz) {
        int32_t q[kDpU];
#pragma unroll
        for (int u = 0; u < kDpU; u++) {
          const int64_t j = j0 + u * gsz;
          q[u] = j <= n ? ld32(&a.P[j]) : -1;
        }
        int64_t cq_[kDpU];
        int32_t nq[kDpU];
#pragma unroll
        for (int u = 0; u < kDpU; u++) {
          cq_[u] = q[u] > 0 ? ld_coherent(&a.cost[q[u]]) : 0;
          nq[u] = q[u] > 0 ? ld32(&a.P[q[u]]) : -1;
        }
#pragma unroll
        for (int u = 0; u < kDpU; u++) {
          const int64_t j = j0 + u * gsz;
          if (j > n) continue;
          const int32_t nx = nq[u] > 0 ? nq[u] : -1;
          more |= nx >= 0;
          lpe_st(&cur[j], LpE{ld_coherent(&a.cost[j]) + cq_[u], nx, 0});
        }
      }
      more = __syncthreads_or(more);
      if (!grid_sync(a.bar, ++bar, more, &s_ok, &s_bit, st, &bit)) return;
      int32_t r = 1;
      while (bit) {
        if (r == a.max_rounds) {  // a pointer cycle: cannot happen (P(j) < j)
          raise_err(st, EB_ORDER);
          return;  // uniform: bit and r are the same in every workgroup
        }
        more = 0;
        for (int64_t j0 = gid; j0 <= n; j0 += kDpU * gsz) {
          LpE x[kDpU];
#pragma unroll
          for (int u = 0; u < kDpU; u++) {
            const int64_t j = j0 + u * gsz;
            x[u] = j <= n ? lpe_ld(&cur[j]) : LpE{0, -1, 1};
          }
          LpE y[kDpU];
#pragma unroll
          for (int u = 0; u < kDpU; u++) y[u] = x[u].nxt >= 0 ? lpe_ld(&cur[x[u].nxt]) : LpE{0, -1, 0};
#pragma unroll
          for (int u = 0; u < kDpU; u++) {
            const int64_t j = j0 + u * gsz;
            if (j > n || x[u].both) continue;
            if (x[u].nxt < 0) {
              lpe_st(&oth[j], LpE{x[u].v, -1, 1});
              st32(&cur[j].both, 1);
            } else {
              const LpE z{x[u].v + y[u].v, y[u].nxt, 0};
              more |= z.nxt >= 0;
              lpe_st(&oth[j], z);
            }
          }
        }
        more = __syncthreads_or(more);
        if (!grid_sync(a.bar, ++bar, more, &s_ok, &s_bit, st, &bit)) return;
        LpE *t = cur;
        cur = oth;
        oth = t;
        r++;
      }
    }
    // S - PO for the candidates (plain stores, published by a fenced barrier)
    for (int64_t j = gid; j <= n; j += gsz)
      a.SP[j] = (PK ? pk_val(pk_ld(E + j)) : ld_coherent(&cur[j].v)) - a.PO[j];
    if (!grid_sync_fenced(a.bar, ++bar, &s_ok, &s_bit, st)) return;
    // ---- improvement: the best candidate of every target
    int32_t chg = 0;
    for (int64_t j = gid + 1; j <= n; j += gsz) {
      const int32_t lj = a.lo[j];
      int64_t Int = 0, best = kInf, ib = 0;
      int32_t arg = (int32_t)j - 1;
      int32_t i = (int32_t)j - 1;
      for (; i >= lj + 3; i -= 4) {  // four candidates with their loads in flight
        uint64_t nw[4];
        int64_t ci[4], sp[4];
#pragma unroll
        for (int u = 0; u < 4; u++) {
          nw[u] = a.nearw[i - u];
          ci[u] = a.cq[i - u];
          sp[u] = a.SP[i - u];
        }
        int32_t k[4];
#pragma unroll
        for (int u = 0; u < 4; u++) k[u] = dp_near_below(a, nw[u], (uint32_t)(j - (i - u)));
#pragma unroll
        for (int u = 0; u < 4; u++) {
          Int += ci[u] * k[u];
          const int64_t v = sp[u] - Int;
          if (v <= best) {
            best = v;
            arg = i - u;
            ib = Int;
          }
        }
      }
      for (; i >= lj; i--) {
        Int += a.cq[i] * dp_near_below(a, a.nearw[i], (uint32_t)(j - i));
        const int64_t v = a.SP[i] - Int;
        if (v <= best) {
          best = v;
          arg = i;
          ib = Int;
        }
      }
      st32(&a.Parg[j], arg);
      if (best < a.SP[j]) {  // PO[j] + best < S(j): strictly better
        st32(&a.P[j], arg);
        st_coherent(&a.cost[j], a.PO[j] - a.PO[arg] - ib);
        chg = 1;
      }
    }
    chg = __syncthreads_or(chg);
    if (!grid_sync(a.bar, ++bar, chg, &s_ok, &s_bit, st, &bit)) return;
    if (!bit) {
      done = true;
      break;
    }
  }
  if (!done) {
    if (gid == 0) {
      st->i2 = 0;
      st->i3 = it;
    }
    return;
  }
  // converged: the smallest minimising i of every target, and S(n)
  for (int64_t j = gid + 1; j <= n; j += gsz) a.P[j] = ld32(&a.Parg[j]);
  if (gid == 0) {
    st->s0 = a.SP[n] + a.PO[n];
    st->i2 = 1;
    st->i3 = it + 1;
  }
}

// Packed entries when every value fits: S is at most PO[n], the comm of all
// edges (every node a cluster of its own), below 2^40, and positions below
// 2^24 - 1.
__global__ void __launch_bounds__(kDpB) k_dp_policy(DpArgs a) {
  __shared__ int32_t s_ok, s_bit;
  if (failed(a.st)) return;
  if (a.packed && a.n < (int32_t)kPkEnd - 1 && a.PO[a.n] < (int64_t(1) << 40))
    dp_run<true>(a, &s_ok, &s_bit);
  else
    dp_run<false>(a, &s_ok, &s_bit);
}

// ------------------------------------------------------ cluster starts

// The cluster starts are the chain from n through the final back pointers P
// (each P(j) < j).  Doubling tables J_0 = P (J_0(0) = 0), J_{k+1} = J_k(J_k)
// are built until the 2^k-th ancestor of n is position 0; then M = {n}, and
// for l = k down to 0 every marked position marks J_l of itself: after level
// l the marks cover every distance along the chain from n that is a sum of
// distinct powers 2^l .. 2^k, so at the end every chain node is marked and
// nothing else (a mark another thread sets during a pass only adds ancestors).
// About 2 log2(C) whole-GPU passes where one thread would follow C pointers.
struct CmArgs {
  int32_t n, K;               // K levels allocated in J
  const int32_t *P;           // [n + 1]
  int32_t *J;                 // [K][n + 1]
  int32_t *M;                 // [n + 1]
  int32_t *flag;              // [n] 1 at the cluster starts
  int32_t *bar;
  Status *st;
};

__global__ void __launch_bounds__(kDpB) k_chain_marks(CmArgs a) {
  __shared__ int32_t s_ok, s_bit, s_red[kDpB / 64];
  Status *st = a.st;
  if (failed(st)) return;
  const int64_t n1 = (int64_t)a.n + 1;
  const int64_t gsz = (int64_t)gridDim.x * kDpB;
  const int64_t gid = (int64_t)blockIdx.x * kDpB + threadIdx.x;
  int32_t bar = 0, bit;
  for (int64_t j = gid; j < n1; j += gsz) {
    const int32_t pj = j > 0 ? a.P[j] : 0;
    if (j > 0 && (pj < 0 || pj >= j)) raise_err(st, EB_ORDER);  // not a back pointer
    st32(&a.J[j], j > 0 && pj >= 0 && pj < j ? pj : 0);
    st32(&a.M[j], j == a.n ? 1 : 0);
  }
  if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
  int32_t k = 0;
  while (ld32(&a.J[(int64_t)k * n1 + a.n]) != 0 && k + 1 < a.K) {  // uniform after the barrier
    const int32_t *Jk = a.J + (int64_t)k * n1;
    int32_t *Jn = a.J + (int64_t)(k + 1) * n1;
    for (int64_t j = gid; j < n1; j += gsz) st32(&Jn[j], ld32(&Jk[ld32(&Jk[j])]));
    if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
    k++;
  }
  for (int32_t l = k; l >= 0; l--) {
    const int32_t *Jl = a.J + (int64_t)l * n1;
    for (int64_t j = gid; j < n1; j += gsz)
      if (ld32(&a.M[j])) st32(&a.M[ld32(&Jl[j])], 1);
    if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
  }
  int32_t c = 0;
  for (int64_t j = gid; j < a.n; j += gsz) {
    const int32_t m = ld32(&a.M[j]);
    a.flag[j] = m;
    c += m;
  }
  for (int o = 32; o > 0; o >>= 1) c += __shfl_xor(c, o);
  if ((threadIdx.x & 63) == 0) s_red[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t t = 0;
    for (int i = 0; i < kDpB / 64; i++) t += s_red[i];
    atomicAdd(&st->i0, t);
  }
}

// ------------------------------------------------------------------- host

namespace {
std::mutex g_dp_mu;
std::map<int, int> g_dp_groups;  // device -> co-resident workgroups (one per CU at most)
std::map<int, int> g_cm_groups;  // the same for k_chain_marks
}  // namespace

int dp_policy(int32_t n, int32_t m, int32_t R, const int32_t *lo, const int64_t *PO,
              const int64_t *cq, const int32_t *sptr, const int32_t *sidx, int32_t *P,
              Scratch &sc, hipStream_t s, Status *st, bool *launched) {
  *launched = false;
  if (n <= 0) return CEL_OK;
  int gmax = 0;
  {
    int dev = 0;
    CEL_HIP(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lk(g_dp_mu);
    auto it = g_dp_groups.find(dev);
    if (it == g_dp_groups.end()) {
      int cus = 0, nb = 0;
      CEL_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
      CEL_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, (const void *)k_dp_policy, kDpB,
                                                           0));
      it = g_dp_groups.emplace(dev, cus * (nb < 1 ? nb : 1)).first;
    }
    gmax = it->second;
  }
  if (gmax < 1) return CEL_OK;
  const int64_t need = ((int64_t)n + 1 + kDpB - 1) / kDpB;
  const int G = (int)(need < gmax ? need : gmax);
  int32_t max_rounds = 2;
  while ((int64_t(1) << (max_rounds - 2)) < (int64_t)n + 1) max_rounds++;
  // Iterations allowed before the blocked DP is cheaper: an iteration costs
  // its pointer-jumping passes (a few us of barrier plus 48 bytes per node at
  // a few TB/s each) and a sweep of R candidates per target (about 0.5 ps per
  // candidate and target over the whole GPU); the blocked DP about 64 ns per
  // target after 0.5 ms of preparation.
  const double it_us = max_rounds * (5.0 + 48.0 * n / 4.0e6) + 10.0 + 0.5e-6 * R * (double)n;
  const double blocked_us = 500.0 + 0.064 * n;
  int32_t cap = (int32_t)(blocked_us / it_us);
  if (cap < 4) cap = 4;
  int32_t *ncnt, *nptr, *Parg, *bar, *hflag, *hoff;
  uint16_t *noff;
  uint64_t *nearw;
  uint32_t *hcnt;
  int64_t *cost, *SP;
  LpE *e0, *e1;
  CEL_TRY(sc.get(&ncnt, n));
  CEL_TRY(sc.get(&nptr, (int64_t)n + 1));
  CEL_TRY(sc.get(&noff, m));
  CEL_TRY(sc.get(&nearw, n));
  CEL_TRY(sc.get(&hflag, n));
  CEL_TRY(sc.get(&hoff, (int64_t)n + 1));
  CEL_TRY(sc.get(&Parg, (int64_t)n + 1));
  CEL_TRY(sc.get(&cost, (int64_t)n + 1));
  CEL_TRY(sc.get(&SP, (int64_t)n + 1));
  CEL_TRY(sc.get(&e0, (int64_t)n + 1));
  CEL_TRY(sc.get(&e1, (int64_t)n + 1));
  CEL_TRY(sc.get(&bar, 2 + (int64_t)G));
  k_fill_i32<<<grid_for(n, 256, 4096), 256, 0, s>>>(ncnt, n, 0);
  k_dpn_count<<<edge_blocks(m), 256, 0, s>>>(n, m, R, sptr, sidx, ncnt, st);
  CEL_TRY(exclusive_scan_i32(ncnt, nptr, n, sc, s));
  k_dpn_fill<<<edge_blocks(m), 256, 0, s>>>(n, m, R, sptr, sidx, nptr, ncnt, noff, st);
  k_dpn_heavy<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, nptr, hflag, st);
  CEL_TRY(exclusive_scan_i32(hflag, hoff, n, sc, s));
  int32_t H = 0;  // positions with more than four offsets below R
  CEL_HIP(hipMemcpyAsync(&H, hoff + n, sizeof H, hipMemcpyDeviceToHost, s));
  CEL_HIP(hipStreamSynchronize(s));
  if ((int64_t)H * (R + 1) * 4 > (int64_t(1) << 30)) return CEL_OK;  // tables too large: blocked DP
  CEL_TRY(sc.get(&hcnt, (int64_t)H * (R + 1)));
  k_dpn_pack<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, R, nptr, noff, hoff, nearw, hcnt, st);
  k_fill_i32<<<1, 256, 0, s>>>(bar, 2 + (int64_t)G, 0);
  CEL_HIP(hipGetLastError());
  DpArgs a{};
  a.n = n;
  a.R = R;
  a.cap = cap;
  a.max_rounds = max_rounds;
  a.packed = policy_iteration_packed() ? 1 : 0;
  a.lo = lo;
  a.PO = PO;
  a.cq = cq;
  a.nearw = nearw;
  a.hcnt = hcnt;
  a.P = P;
  a.Parg = Parg;
  a.cost = cost;
  a.SP = SP;
  a.e0 = e0;
  a.e1 = e1;
  a.bar = bar;
  a.st = st;
  {
    // at most one workgroup per CU, within the occupancy calculator's limit:
    // resident all at once on an idle GPU; the barriers' waits are bounded
    KTimer kt(s, "k_cluster_policy");
    k_dp_policy<<<G, kDpB, 0, s>>>(a);
  }
  CEL_HIP(hipGetLastError());
  *launched = true;
  return CEL_OK;
}

int chain_marks(int32_t n, const int32_t *P, int32_t *flag, Scratch &sc, hipStream_t s, Status *st,
                bool *launched) {
  *launched = false;
  if (n <= 0) return CEL_OK;
  int gmax = 0;
  {
    int dev = 0;
    CEL_HIP(hipGetDevice(&dev));
    std::lock_guard<std::mutex> lk(g_dp_mu);
    auto it = g_cm_groups.find(dev);
    if (it == g_cm_groups.end()) {
      int cus = 0, nb = 0;
      CEL_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
      CEL_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, (const void *)k_chain_marks, kDpB,
                                                           0));
      it = g_cm_groups.emplace(dev, cus * (nb < 1 ? nb : 1)).first;
    }
    gmax = it->second;
  }
  if (gmax < 1) return CEL_OK;
  const int64_t need = ((int64_t)n + 1 + kDpB - 1) / kDpB;
  const int G = (int)(need < gmax ? need : gmax);
  int32_t K = 2;  // 2^(K - 1) > n: enough levels for a chain through every position
  while ((int64_t(1) << (K - 1)) <= (int64_t)n) K++;
  int32_t *J, *M, *bar;
  CEL_TRY(sc.get(&J, (int64_t)K * ((int64_t)n + 1)));
  CEL_TRY(sc.get(&M, (int64_t)n + 1));
  CEL_TRY(sc.get(&bar, 2 + (int64_t)G));
  k_fill_i32<<<1, 256, 0, s>>>(bar, 2 + (int64_t)G, 0);
  CmArgs a{};
  a.n = n;
  a.K = K;
  a.P = P;
  a.J = J;
  a.M = M;
  a.flag = flag;
  a.bar = bar;
  a.st = st;
  {
    // at most one workgroup per CU (bounded grid-barrier waits, as k_dp_policy)
    KTimer kt(s, "k_chain_marks");
    k_chain_marks<<<G, kDpB, 0, s>>>(a);
  }
  CEL_HIP(hipGetLastError());
  *launched = true;
  return CEL_OK;
}

}  // namespace cel
