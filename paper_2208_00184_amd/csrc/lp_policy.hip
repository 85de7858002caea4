// Longest paths of a DAG by policy iteration: the b-level (eq. 3) over
// successors and the t-level (eq. 2) over predecessors, both of the form
//   val(p) = wv(p) + max over q in adj(p) of val(q)   (wv(p) when adj(p) is empty)
// with wv(p) = w(p) + c(p) for a node with successors, w(p) for a sink
// (b-level: val = b-level; t-level: val = t-level + wv).
//
// A policy picks one neighbour per node, or none.  Its values are the sums of
// wv along the chosen pointers until a node without one; pointer jumping finds
// them all in ceil(log2(longest pointer chain)) + 1 parallel rounds.  Then
// every node switches to a neighbour of strictly larger value, if it has one,
// and the next policy is evaluated.  Each policy's values are lengths of real
// paths, so no value exceeds the longest path; a switch never lowers a value;
// when no node can switch, every value equals wv plus the largest neighbour
// value, the recurrence whose solution on a DAG is unique: the values are
// exact.  A node h hops above the sinks (b-level) is exact after at most h + 1
// iterations, and on the transformer graphs about ten suffice where the level
// sweeps need one dependent step per level (10,565 on transformer-96).
//
// One persistent kernel runs everything; grid barriers (grid_sync) separate
// the phases.  Neighbour lists of more than kLpLight entries are split into
// chunks of kLpChunk, each taken by one wave, and combined after a barrier.
#include <map>
#include <mutex>

#include "cel_internal.h"

namespace cel {

constexpr int kLpB = 1024;        // threads per workgroup
constexpr int kLpLight = 8;       // longer neighbour lists are split into chunks (one wave each)
constexpr int kLpChunk = 256;     // entries of a chunk (one wave, four per lane in flight)
constexpr int kLpU = 4;           // nodes per thread with loads in flight together



struct LpArgs {
  int32_t n, cap, max_rounds;
  int32_t packed;                 // packed entries allowed where the values fit
  const int32_t *aptr, *aidx;     // adjacency (positions)
  const int64_t *wv;              // [n]
  const int32_t *hoff;            // [n + 1] first chunk of each node (chunks only for long lists)
  const int32_t *hnode;           // [H] node of each chunk
  int32_t *pol;                   // [n] the policy
  LpE *e0, *e1;                   // [n] each
  int64_t *hval;                  // [H] best value of each chunk
  int32_t *hidx;                  // [H] ... and its neighbour
  int32_t *bar;                   // grid barrier words [2 + gridDim]
  int64_t *out;                   // [n] results
  Status *st;
  int32_t *res;                   // [0] converged, [1] iterations
};

// Entries, policy pointers and chunk results are written and read by
// different workgroups inside the kernel: agent-scope atomic accesses (see
// grid_sync, and lpe_ld / lpe_st).

// larger value first, then the smaller neighbour index
__device__ inline bool lp_better(int64_t v, int32_t q, int64_t bv, int32_t bq) {
  return v > bv || (v == bv && q < bq);
}

__global__ void k_lp_heavy_count(int32_t n, const int32_t *aptr, int32_t *hcnt, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const int32_t d = aptr[p + 1] - aptr[p];
    hcnt[p] = d > kLpLight ? (d + kLpChunk - 1) / kLpChunk : 0;
  }
}

__global__ void k_lp_heavy_fill(int32_t n, const int32_t *hoff, int32_t *hnode, const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x)
    for (int32_t c = hoff[p]; c < hoff[p + 1]; c++) hnode[c] = (int32_t)p;
}

// KIND: 0 the b-level, 1 the t-level (out = val - wv), 2 the levels of Kahn's
// ordering; a template parameter so that profiles tell the three apart
template <int KIND, bool PK>
__device__ inline void lp_run(const LpArgs &a, int32_t *s_okp, int32_t *s_bitp) {
  int32_t &s_ok = *s_okp, &s_bit = *s_bitp;
  Status *st = a.st;
  const int32_t n = a.n;
  // PK: packed entries in two buffers; the improvement reads E and writes
  // each node's entry for the next policy (wv, new pointer) into En, where
  // the jumps then run; the buffers swap after every evaluation
  uint64_t *E = reinterpret_cast<uint64_t *>(a.e0), *En = reinterpret_cast<uint64_t *>(a.e1);
  const int64_t gsz = (int64_t)gridDim.x * kLpB;
  const int64_t gid = (int64_t)blockIdx.x * kLpB + threadIdx.x;
  const int lane = threadIdx.x & 63;
  const int32_t H = a.hoff[n];
  int32_t bar = 0, bit;
  // the empty policy: every node alone
  for (int64_t p = gid; p < n; p += gsz) {
    if (PK) pk_st(E + p, pk_make(a.wv[p], kPkEnd));
    else lpe_st(&a.e0[p], LpE{a.wv[p], -1, 0});
    st32(&a.pol[p], -1);
  }
  if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
  LpE *cur = a.e0, *oth = a.e1;
  int32_t it = 0;
  bool done = false;
  for (; it < a.cap; it++) {
    // ---- improvement: the best neighbour under the current values
    // chunks of long lists, one wave each
    const int64_t wid = gid >> 6, nw = gsz >> 6;
    for (int64_t c = wid; c < H; c += nw) {
      const int32_t p = a.hnode[c];
      const int32_t e0 = a.aptr[p] + (int32_t)(c - a.hoff[p]) * kLpChunk;
      const int32_t e1 = min(a.aptr[p + 1], e0 + kLpChunk);
      int64_t bv = -1;
      int32_t bq = INT32_MAX;
      int32_t q[kLpChunk / 64];
      int64_t v[kLpChunk / 64];
#pragma unroll
      for (int k = 0; k < kLpChunk / 64; k++) q[k] = e0 + 64 * k + lane < e1 ? a.aidx[e0 + 64 * k + lane] : -1;
#pragma unroll
      for (int k = 0; k < kLpChunk / 64; k++)
        v[k] = q[k] < 0 ? -1 : (PK ? pk_val(pk_ld(E + q[k])) : ld_coherent(&cur[q[k]].v));
#pragma unroll
      for (int k = 0; k < kLpChunk / 64; k++)
        if (q[k] >= 0 && lp_better(v[k], q[k], bv, bq)) {
          bv = v[k];
          bq = q[k];
        }
      for (int o = 32; o > 0; o >>= 1) {
        const int64_t v = __shfl_xor((long long)bv, o);
        const int32_t q = __shfl_xor(bq, o);
        if (lp_better(v, q, bv, bq)) {
          bv = v;
          bq = q;
        }
      }
      if (lane == 0) {
        st_coherent(&a.hval[c], bv);
        st32(&a.hidx[c], bq);
      }
    }
    int32_t chg = 0;
    // short lists, one thread per node, kLpU nodes with loads in flight
    for (int64_t p0 = gid; p0 < n; p0 += kLpU * gsz) {
      int32_t b0[kLpU], b1[kLpU], pq[kLpU];
#pragma unroll
      for (int u = 0; u < kLpU; u++) {
        const int64_t p = p0 + u * gsz;
        b0[u] = b1[u] = 0;
        pq[u] = -1;
        if (p < n) {
          b0[u] = a.aptr[p];
          b1[u] = a.aptr[p + 1];
          pq[u] = ld32(&a.pol[p]);
        }
      }
#pragma unroll
      for (int u = 0; u < kLpU; u++) {
        const int64_t p = p0 + u * gsz;
        const int32_t d = b1[u] - b0[u];
        if (PK && p < n && d == 0) pk_st(En + p, pk_make(a.wv[p], kPkEnd));
        if (p >= n || d == 0 || d > kLpLight) continue;
        int64_t bv = -1;
        int32_t bq = INT32_MAX;
        for (int32_t e0 = b0[u]; e0 < b1[u]; e0 += 4) {  // four neighbours' loads in flight
          int32_t q[4];
          int64_t v[4];
#pragma unroll
          for (int k = 0; k < 4; k++) q[k] = e0 + k < b1[u] ? a.aidx[e0 + k] : -1;
#pragma unroll
          for (int k = 0; k < 4; k++)
            v[k] = q[k] < 0 ? -1 : (PK ? pk_val(pk_ld(E + q[k])) : ld_coherent(&cur[q[k]].v));
#pragma unroll
          for (int k = 0; k < 4; k++)
            if (q[k] >= 0 && lp_better(v[k], q[k], bv, bq)) {
              bv = v[k];
              bq = q[k];
            }
        }
        const int64_t cv = pq[u] >= 0 ? (PK ? pk_val(pk_ld(E + pq[u])) : ld_coherent(&cur[pq[u]].v)) : -1;
        if (bv > cv) {
          st32(&a.pol[p], bq);
          chg = 1;
        }
        if (PK) pk_st(En + p, pk_make(a.wv[p], bv > cv ? (uint32_t)bq : pq[u] >= 0 ? (uint32_t)pq[u] : kPkEnd));
      }
    }
    if (H > 0) {  // combine the chunks of each long list: one wave per node
      if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
      const int64_t wid = gid >> 6, nw = gsz >> 6;
      for (int64_t c = wid; c < H; c += nw) {
        const int32_t p = a.hnode[c];
        if (c != a.hoff[p]) continue;  // uniform: the wave of the node's first chunk combines
        int64_t bv = -1;
        int32_t bq = INT32_MAX;
        for (int32_t k = (int32_t)c + lane; k < a.hoff[p + 1]; k += 64) {
          const int64_t v = ld_coherent(&a.hval[k]);
          const int32_t q = ld32(&a.hidx[k]);
          if (lp_better(v, q, bv, bq)) {
            bv = v;
            bq = q;
          }
        }
        for (int o = 32; o > 0; o >>= 1) {
          const int64_t v = __shfl_xor((long long)bv, o);
          const int32_t q = __shfl_xor(bq, o);
          if (lp_better(v, q, bv, bq)) {
            bv = v;
            bq = q;
          }
        }
        if (lane == 0) {
          const int32_t pq = ld32(&a.pol[p]);
          const int64_t cv = pq >= 0 ? (PK ? pk_val(pk_ld(E + pq)) : ld_coherent(&cur[pq].v)) : -1;
          if (bv > cv) {
            st32(&a.pol[p], bq);
            chg = 1;
          }
          if (PK) pk_st(En + p, pk_make(a.wv[p], bv > cv ? (uint32_t)bq : pq >= 0 ? (uint32_t)pq : kPkEnd));
        }
      }
    }
    chg = __syncthreads_or(chg);
    if (!grid_sync(a.bar, ++bar, chg, &s_ok, &s_bit, st, &bit)) return;
    if (KIND == 0 && it == 1) bit = 1;  // values of iteration 0 were cut short: evaluate
    if (!bit) {
      done = true;
      break;
    }
    if (PK) {
      // ---- evaluation, packed entries: the jumps start from the entries the
      // improvement wrote (wv, pointer) into En, asynchronously (see pk_make);
      // the b-level's first policy instead keeps one-hop values (wv(p) +
      // wv(pol(p)), next pol(pol(p))), folded in one pass
      if (KIND == 0 && it == 0) {
        for (int64_t p0 = gid; p0 < n; p0 += kLpU * gsz) {
          int32_t q[kLpU];
#pragma unroll
          for (int u = 0; u < kLpU; u++) {
            const int64_t p = p0 + u * gsz;
            q[u] = p < n ? ld32(&a.pol[p]) : -1;
          }
          int64_t wq[kLpU];
          int32_t nq[kLpU];
#pragma unroll
          for (int u = 0; u < kLpU; u++) {
            wq[u] = q[u] >= 0 ? a.wv[q[u]] : 0;
            nq[u] = q[u] >= 0 ? ld32(&a.pol[q[u]]) : -1;
          }
#pragma unroll
          for (int u = 0; u < kLpU; u++) {
            const int64_t p = p0 + u * gsz;
            if (p < n) pk_st(En + p, pk_make(a.wv[p] + wq[u], nq[u] >= 0 ? nq[u] : kPkEnd));
          }
        }
      } else {
        for (int64_t p0 = gid; p0 < n; p0 += kPkU * gsz) {
          uint64_t e[kPkU];
#pragma unroll
          for (int u = 0; u < kPkU; u++) {
            const int64_t p = p0 + u * gsz;
            e[u] = p < n ? pk_ld(En + p) : pk_make(0, kPkEnd);
          }
          // each jump moves a chain's end strictly forward, so a chain of a
          // DAG ends within n jumps; more means a pointer cycle
          for (int32_t k = 0;; k++) {
            uint64_t f[kPkU];
            bool any = false;
#pragma unroll
            for (int u = 0; u < kPkU; u++) {
              const uint32_t x = pk_next(e[u]);
              f[u] = x != kPkEnd ? pk_ld(En + x) : 0;
            }
#pragma unroll
            for (int u = 0; u < kPkU; u++) {
              if (pk_next(e[u]) == kPkEnd) continue;
              e[u] = pk_make(pk_val(e[u]) + pk_val(f[u]), pk_next(f[u]));
              pk_st(En + p0 + u * gsz, e[u]);
              any |= pk_next(e[u]) != kPkEnd;
            }
            if (!any) break;
            if (k > n) {
              raise_err(st, EB_CYCLE);
              break;
            }
          }
        }
      }
      if (!grid_sync(a.bar, ++bar, 0, &s_ok, &s_bit, st, &bit)) return;
      if (ld32(reinterpret_cast<const int32_t *>(&st->err))) return;  // uniform after the barrier
      uint64_t *t = E;
      E = En;
      En = t;
      continue;
    }
    // ---- evaluation of the new policy by pointer jumping; the first round
    // reads the policy itself (cur is free: nothing reads it any more)
    int32_t more = 0;
    for (int64_t p0 = gid; p0 < n; p0 += kLpU * gsz) {
      int32_t q[kLpU];
#pragma unroll
      for (int u = 0; u < kLpU; u++) {
        const int64_t p = p0 + u * gsz;
        q[u] = p < n ? ld32(&a.pol[p]) : -1;
      }
      int64_t wq[kLpU];
      int32_t nq[kLpU];
#pragma unroll
      for (int u = 0; u < kLpU; u++) {
        wq[u] = q[u] >= 0 ? a.wv[q[u]] : 0;
        nq[u] = q[u] >= 0 ? ld32(&a.pol[q[u]]) : -1;
      }
#pragma unroll
      for (int u = 0; u < kLpU; u++) {
        const int64_t p = p0 + u * gsz;
        if (p >= n) continue;
        more |= nq[u] >= 0;
        lpe_st(&cur[p], LpE{a.wv[p] + wq[u], nq[u], 0});
      }
    }
    more = __syncthreads_or(more);
    if (!grid_sync(a.bar, ++bar, more, &s_ok, &s_bit, st, &bit)) return;
    // b-level: the first policy's evaluation stops after this round, so the
    // next improvement compares wv(q) + wv(pol(q)), the longest paths of two
    // nodes, instead of the full chains of the greedy first policy; that
    // start saves iterations on the transformer and layered graphs (113 -> 80
    // pointer-jumping rounds on transformer-96).  Any policy is a valid start:
    // the next iteration evaluates its policy fully whatever the improvement
    // changes, and only exact values end the iteration.
    if (KIND == 0 && it == 0) bit = 0;
    int32_t r = 1;
    while (bit) {
      if (r == a.max_rounds) {  // a pointer cycle: the input is not a DAG
        raise_err(st, EB_CYCLE);
        return;  // every workgroup takes this branch: bit and r are uniform
      }
      more = 0;
      for (int64_t p0 = gid; p0 < n; p0 += kLpU * gsz) {
        LpE x[kLpU];
#pragma unroll
        for (int u = 0; u < kLpU; u++) {
          const int64_t p = p0 + u * gsz;
          x[u] = p < n ? lpe_ld(&cur[p]) : LpE{0, -1, 1};
        }
        LpE y[kLpU];
#pragma unroll
        for (int u = 0; u < kLpU; u++) y[u] = x[u].nxt >= 0 ? lpe_ld(&cur[x[u].nxt]) : LpE{0, -1, 0};
#pragma unroll
        for (int u = 0; u < kLpU; u++) {
          const int64_t p = p0 + u * gsz;
          if (p >= n || x[u].both) continue;  // ended, and final in both buffers
          if (x[u].nxt < 0) {
            // ended last round: the other buffer gets the final entry too
            // (readers of cur[p] see v and nxt unchanged)
            lpe_st(&oth[p], LpE{x[u].v, -1, 1});
            st32(&cur[p].both, 1);
          } else {
            const LpE z{x[u].v + y[u].v, y[u].nxt, 0};
            more |= z.nxt >= 0;
            lpe_st(&oth[p], z);
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
  // The values of the last policy evaluated, exact when converged; otherwise
  // lengths of real paths (never above the exact values, so levels stay
  // below n), which callers may use before they read res and replace.
  for (int64_t p = gid; p < n; p += gsz)
    a.out[p] = (PK ? pk_val(pk_ld(E + p)) : ld_coherent(&cur[p].v)) - (KIND == 1 ? a.wv[p] : 0);
  if (gid == 0) {
    a.res[0] = done ? 1 : 0;  // not converged: the caller runs the level-synchronous kernel
    a.res[1] = done ? it + 1 : it;
  }
}

// KIND: 0 the b-level, 1 the t-level (out = val - wv), 2 the levels of Kahn's
// ordering; a template parameter so that profiles tell the three apart.
// Packed entries when every value fits: positions below 2^24 - 1, and for
// the b-level and t-level the validation's total of w and c below 2^40 (the
// levels are at most n).  A pointer cycle (the levels of a graph that is not
// a DAG) keeps some chain from ending: its node gives up after n jumps with
// EB_CYCLE.
template <int KIND>
__global__ void __launch_bounds__(kLpB) k_lp_policy(LpArgs a) {
  __shared__ int32_t s_ok, s_bit;
  if (failed(a.st)) return;
  if (a.packed && a.n < (int32_t)kPkEnd && (KIND == 2 || a.st->total < (uint64_t(1) << 40)))
    lp_run<KIND, true>(a, &s_ok, &s_bit);
  else
    lp_run<KIND, false>(a, &s_ok, &s_bit);
}

// ------------------------------------------------------------------- host

namespace {
std::mutex g_lp_mu;
std::map<int, int> g_lp_cus;  // device -> co-resident workgroups of k_lp_policy (one per CU at most)

int lp_groups(int *out) {
  int dev = 0;
  CEL_HIP(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_lp_mu);
  auto it = g_lp_cus.find(dev);
  if (it == g_lp_cus.end()) {
    int cus = 0, nb = 0;
    CEL_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    CEL_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, (const void *)k_lp_policy<0>, kLpB, 0));
    it = g_lp_cus.emplace(dev, cus * (nb < 1 ? nb : 1)).first;
  }
  *out = it->second;
  return CEL_OK;
}
}  // namespace

int lp_policy(int32_t n, int32_t m, int32_t L, int32_t cap, const int32_t *aptr,
              const int32_t *aidx, const int64_t *wv, int kind, int64_t *out, int32_t *res,
              const char *timer, Scratch &sc, hipStream_t s, Status *st, bool *launched) {
  *launched = false;
  if (n <= 0) return CEL_OK;
  int gmax = 0;
  CEL_TRY(lp_groups(&gmax));
  if (gmax < 1) return CEL_OK;
  const int G = (int)((int64_t)n + kLpB - 1) / kLpB < gmax ? (int)(((int64_t)n + kLpB - 1) / kLpB)
                                                          : gmax;
  // pointer chains are at most L nodes long (one per level)
  int32_t max_rounds = 2;
  while ((int64_t(1) << (max_rounds - 2)) < L) max_rounds++;
  // Iterations allowed (cap <= 0: before the level sweep is cheaper): an
  // iteration costs about max_rounds barriers and passes over 48 bytes per
  // node, plus one pass over the neighbour lists; the sweep about 0.6 us per
  // level after 0.5 ms.
  if (cap <= 0) {
    const double it_us = max_rounds * (5.0 + 48.0 * n / 4.0e6) + 12.0 * m / 4.0e6;
    const double sweep_us = 500.0 + 0.6 * L;
    cap = (int32_t)(sweep_us / it_us);
    if (cap < 2) cap = 2;
  }
  int32_t *hcnt, *hoff, *hnode, *pol, *hidx, *bar;
  LpE *e0, *e1;
  int64_t *hval;
  CEL_TRY(sc.get(&hcnt, n));
  CEL_TRY(sc.get(&hoff, (int64_t)n + 1));
  k_lp_heavy_count<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, aptr, hcnt, st);
  CEL_TRY(exclusive_scan_i32(hcnt, hoff, n, sc, s));
  // chunks: at most m / kLpChunk + (nodes with long lists) <= m / kLpChunk + m / kLpLight
  const int64_t hmax = (int64_t)m / kLpChunk + (int64_t)m / kLpLight + 1;
  CEL_TRY(sc.get(&hnode, hmax));
  CEL_TRY(sc.get(&hval, hmax));
  CEL_TRY(sc.get(&hidx, hmax));
  CEL_TRY(sc.get(&pol, n));
  CEL_TRY(sc.get(&e0, n));
  CEL_TRY(sc.get(&e1, n));
  CEL_TRY(sc.get(&bar, 2 + (int64_t)G));
  k_lp_heavy_fill<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, hoff, hnode, st);
  k_fill_i32<<<1, 256, 0, s>>>(bar, 2 + (int64_t)G, 0);
  k_fill_i32<<<1, 64, 0, s>>>(res, 2, 0);
  CEL_HIP(hipGetLastError());
  LpArgs a{};
  a.n = n;
  a.cap = cap;
  a.max_rounds = max_rounds;
  a.packed = policy_iteration_packed() ? 1 : 0;
  a.aptr = aptr;
  a.aidx = aidx;
  a.wv = wv;
  a.hoff = hoff;
  a.hnode = hnode;
  a.pol = pol;
  a.e0 = e0;
  a.e1 = e1;
  a.hval = hval;
  a.hidx = hidx;
  a.bar = bar;
  a.out = out;
  a.st = st;
  a.res = res;
  {
    // at most one workgroup per CU, within the occupancy calculator's limit:
    // resident all at once on an idle GPU; the grid barriers' waits are
    // bounded (kGridSpin), so anything else ends in an error, not a hang
    KTimer kt(s, timer);
    if (kind == 1) k_lp_policy<1><<<G, kLpB, 0, s>>>(a);
    else if (kind == 2) k_lp_policy<2><<<G, kLpB, 0, s>>>(a);
    else k_lp_policy<0><<<G, kLpB, 0, s>>>(a);
  }
  CEL_HIP(hipGetLastError());
  *launched = true;
  return CEL_OK;
}

}  // namespace cel
