// cel_topo_levels: the levels of Kahn's ordering (Section 4.2.2).
//
// The level of a node is the length (in edges) of the longest path into it,
// 0 for a source: the level at which Kahn's algorithm frees it.  On graphs of
// at least kTopoPolicyN nodes the levels are first found by policy iteration
// (lp_policy.hip; each node follows one predecessor, pointer jumping counts the
// chains, nodes switch to a deeper predecessor until none can), which takes
// about ten whole-GPU iterations where the levels are many; the nodes are then
// sorted by (level, id) and the level starts read off the sorted levels.  Within kTopoPolicyIt
// iterations or not at all, the level-synchronous Kahn kernel runs instead:
//
// One workgroup runs all levels: a level costs dependent L2 round trips, so
// keeping the whole loop in one workgroup with workgroup barriers is far
// cheaper than one launch or one grid-wide barrier per level.  Frontier
// entries carry their node's adjacency, which leaves one round trip (the
// in-degree atomics) per level for nodes of small degree.  Frontiers are appended to the caller's
// order_id buffer; each level's slice is then sorted by id.
#include "cel_internal.h"

namespace cel {

constexpr int kKahnB = 1024;
constexpr int kKahnNW = kKahnB / 64;
constexpr int kKahnA = 4;         // successors carried with a frontier entry
constexpr int kKahnCap = 1024;    // frontier entries mirrored in LDS
constexpr int kKahnE = 4;         // edges per thread whose loads and atomics go out together
constexpr int kKahnCW = 16384;    // LDS words of packed in-degree counters (64 KB)

// Remaining in-edges of every node from non-sources (a source is removed in
// the first round and nothing waits on it: an edge from a source never needs
// its decrement), and the largest such count.
__global__ void k_kahn_cnt(int32_t n, const int32_t *in_ptr, const int32_t *in_idx, int32_t *cnt,
                           int32_t *cmax, const Status *st) {
  if (failed(st)) return;
  int32_t mx = 0;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    int32_t c = 0;
    for (int32_t e = in_ptr[v]; e < in_ptr[v + 1]; e++) {
      const int32_t u = in_idx[e];
      c += in_ptr[u + 1] > in_ptr[u] ? 1 : 0;
    }
    cnt[v] = c;
    mx = c > mx ? c : mx;
  }
  for (int off = 32; off > 0; off >>= 1) {
    const int32_t o = __shfl_xor(mx, off);
    mx = o > mx ? o : mx;
  }
  if ((threadIdx.x & 63) == 0 && mx > 0) atomicMax(cmax, mx);
}

// A successor entry of a node's record: the id, bit 31 set when that
// successor has exactly one in-edge from a non-source (this one: it becomes
// ready without a counter).
constexpr int32_t kOneBit = int32_t(0x80000000u);
__device__ inline int32_t succ_id(int32_t e) { return e & 0x7FFFFFFF; }
__device__ inline bool succ_one(int32_t e) { return e < 0; }

// Per node: first out-edge and out-degree, and its first kKahnA successors
// (-1 past the end; count-one successors flagged), so that a node that
// becomes ready brings its adjacency along with it.
__global__ void k_kahn_prep(int32_t n, const int32_t *out_ptr, const int32_t *out_idx,
                            const int32_t *cnt, int2 *deg, int4 *adj, const Status *st) {
  if (failed(st)) return;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t e0 = out_ptr[v], d = out_ptr[v + 1] - e0;
    deg[v] = make_int2(e0, d);
    int32_t s[kKahnA];
#pragma unroll
    for (int q = 0; q < kKahnA; q++) {
      s[q] = -1;
      if (q < d) {
        const int32_t t = out_idx[e0 + q];
        s[q] = cnt[t] == 1 ? (t | kOneBit) : t;
      }
    }
    adj[v] = make_int4(s[0], s[1], s[2], s[3]);
  }
}

__device__ inline int32_t int4_at(const int4 &a, int q) {
  return q == 0 ? a.x : (q == 1 ? a.y : (q == 2 ? a.z : a.w));
}

// Appends v (with its degree and first successors) to the frontier being
// built, for the lanes with want set: one LDS atomic per wave reserves the
// wave's slots.  F holds every frontier in order; the LDS mirror holds the
// first kKahnCap entries of the one being built (fe: its first index).
__device__ inline void kahn_append(bool want, int32_t v, const int2 &d, const int4 &a, int32_t *F,
                                   int32_t *s_tail, int32_t fe, int32_t *s_fv, int2 *s_fd,
                                   int4 *s_fa, int32_t *s_hv) {
  const uint64_t m = __ballot(want);
  if (m == 0) return;
  if (__ballot(want && d.y > kKahnA) != 0 && (int)(threadIdx.x & 63) == 0) *s_hv = 1;
  const int leader = __builtin_ctzll(m);
  int32_t base = 0;
  if ((int)(threadIdx.x & 63) == leader) base = atomicAdd(s_tail, __popcll(m));
  base = __shfl(base, leader);
  if (!want) return;
  const int32_t k =
      base + (int32_t)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                 __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
  F[k] = v;
  if (k - fe < kKahnCap) {
    s_fv[k - fe] = v;
    s_fd[k - fe] = d;
    s_fa[k - fe] = a;
  }
}

// The same for N candidates per lane (want[q], v[q], ...): one LDS atomic
// reserves the slots of all N ballots of the wave at once.
template <int N>
__device__ inline void kahn_append_n(const bool (&want)[N], const int32_t (&v)[N],
                                     const int2 (&d)[N], const int4 (&a)[N], int32_t *F,
                                     int32_t *s_tail, int32_t fe, int32_t *s_fv, int2 *s_fd,
                                     int4 *s_fa, int32_t *s_hv) {
  uint64_t m[N];
  int32_t off[N], tot = 0;
  bool hv = false;
#pragma unroll
  for (int q = 0; q < N; q++) {
    m[q] = __ballot(want[q]);
    off[q] = tot;
    tot += __popcll(m[q]);
    hv = hv || __ballot(want[q] && d[q].y > kKahnA) != 0;
  }
  if (tot == 0) return;
  const int lane = (int)(threadIdx.x & 63);
  if (hv && lane == 0) *s_hv = 1;
  int32_t base = 0;
  if (lane == 0) base = atomicAdd(s_tail, tot);
  base = __builtin_amdgcn_readfirstlane(base);
#pragma unroll
  for (int q = 0; q < N; q++) {
    if (!want[q]) continue;
    const int32_t k = base + off[q] +
                      (int32_t)__builtin_amdgcn_mbcnt_hi(
                          (uint32_t)(m[q] >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m[q], 0u));
    F[k] = v[q];
    if (k - fe < kKahnCap) {
      s_fv[k - fe] = v[q];
      s_fd[k - fe] = d[q];
      s_fa[k - fe] = a[q];
    }
  }
}

// Level-synchronous Kahn in one workgroup.  The sources form level 0 and
// their out-edges are never counted (k_kahn_cnt); the nodes whose in-edges
// all come from sources form level 1.  From there a frontier node of degree
// at most kKahnA removes its in-edge from each successor; the successor's
// degree and first successors are loaded in the same round, so the node that
// the last removal makes ready joins the next frontier with its adjacency.
// Nodes of higher degree are listed and their edges then spread over the
// whole block (flattened by a prefix sum of the degrees).
// In-degree counters live in LDS when they fit: b-bit fields (b = 2, 4 or 8,
// the smallest that holds the largest count) packed 32 / b to a word, each
// removal one LDS atomic subtract of 1 << field offset that returns the old
// word (a field only ever counts down to zero, so no borrow crosses fields).
// Otherwise they stay in global memory (one returning atomic per removal).
__global__ void __launch_bounds__(kKahnB) k_kahn(cel_graph g, int32_t *cnt, const int32_t *cmax,
                                                 const int2 *deg, const int4 *adj, int32_t *F,
                                                 int32_t *level, int32_t *lstart, Status *st) {
  __shared__ int32_t s_tail, s_nh[3];  // s_nh: listed nodes, counters used by passes in turn
  __shared__ int32_t s_fv[2][kKahnCap];
  __shared__ int2 s_fd[2][kKahnCap];  // first out-edge, out-degree
  __shared__ int4 s_fa[2][kKahnCap];
  __shared__ int32_t s_hd[kKahnB], s_he[kKahnB], s_hp[kKahnB + 1];
  __shared__ int32_t s_wt[kKahnNW];
  // per mirror: the frontier holds a node of more than kKahnA successors;
  // the state wave 0 leaves after a run of narrow levels
  __shared__ int32_t s_hv[2], s_state[4];
  __shared__ uint32_t s_cnt[kKahnCW];
  if (failed(st)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t n = g.n;
  // counter layout: b bits per node, 32 / b nodes per word
  const int32_t cm = *cmax;
  const int32_t cb = cm < 4 ? 2 : (cm < 16 ? 4 : 8);
  const int32_t lper = cb == 2 ? 4 : (cb == 4 ? 3 : 2);  // log2(32 / b)
  const uint32_t fmask = (1u << cb) - 1u;
  const bool ldsc = cm < 256 && (((int64_t)n << 5 >> lper) <= (int64_t)kKahnCW * 32);
  if (tid == 0) {
    s_tail = 0;
    s_nh[0] = s_nh[1] = s_nh[2] = 0;
    s_hv[0] = s_hv[1] = 0;
  }
  if (ldsc) {
    const int32_t per = 1 << lper, nw = (n + per - 1) >> lper;
    for (int32_t wd = tid; wd < nw; wd += kKahnB) {
      uint32_t x = 0;
      for (int32_t j = 0; j < per; j++) {
        const int32_t v = (wd << lper) + j;
        if (v < n) x |= (uint32_t)cnt[v] << (j * cb);
      }
      s_cnt[wd] = x;
    }
  }
  __syncthreads();
  // the count of t before this removal
  auto remove_edge = [&](int32_t t) -> int32_t {
    if (ldsc) {
      const int32_t sh = (t & ((1 << lper) - 1)) * cb;
      const uint32_t old = atomicSub(&s_cnt[t >> lper], 1u << sh);
      return (int32_t)((old >> sh) & fmask);
    }
    return atomicSub(&cnt[t], 1);
  };
  for (int32_t v0 = 0; v0 < n; v0 += kKahnB) {  // level 0: the sources
    const int32_t v = v0 + tid;
    const bool src = v < n && g.in_ptr[v + 1] == g.in_ptr[v];
    kahn_append(src, v, make_int2(0, 0), make_int4(-1, -1, -1, -1), F, &s_tail, 0, s_fv[0],
                s_fd[0], s_fa[0], &s_hv[0]);
  }
  __syncthreads();
  const int32_t nsrc = s_tail;
  if (tid == 0) lstart[0] = 0;
  __syncthreads();
  for (int32_t v0 = 0; v0 < n; v0 += kKahnB) {  // level 1: every in-edge from a source
    const int32_t v = v0 + tid;
    const bool one = v < n && g.in_ptr[v + 1] > g.in_ptr[v] && cnt[v] == 0;
    const int2 d = one ? deg[v] : make_int2(0, 0);
    const int4 a = one ? adj[v] : make_int4(-1, -1, -1, -1);
    kahn_append(one, v, d, a, F, &s_tail, nsrc, s_fv[1], s_fd[1], s_fa[1], &s_hv[1]);
  }
  for (int32_t i = tid; i < nsrc; i += kKahnB) level[F[i]] = 0;
  __syncthreads();
  int32_t fb = nsrc, fe = s_tail, lvl = nsrc > 0 ? 1 : 0, cur = 1, pp = 0;
  while (fb < fe) {
    if (fe - fb <= 64 && s_hv[cur] == 0) {
      // Narrow levels (at most 64 nodes, none of more than kKahnA
      // successors): wave 0 runs them alone, one node per lane, with no
      // workgroup barrier; the other waves wait for the next wide level.
      if (wave == 0) {
        int32_t tail = fe, cu = cur, lv = lvl;
        bool hv = false;
        while (true) {
          if (lane == 0) lstart[lv] = fb;
          const int32_t i = fb + lane;
          const bool act = i < fe;
          int32_t u = 0;
          int2 d = make_int2(0, 0);
          int4 a = make_int4(-1, -1, -1, -1);
          if (act) {
            u = s_fv[cu][i - fb];
            d = s_fd[cu][i - fb];
            a = s_fa[cu][i - fb];
            level[u] = lv;
          }
          int32_t c[kKahnA];
          int2 td[kKahnA];
          int4 ta[kKahnA];
#pragma unroll
          for (int q = 0; q < kKahnA; q++) {
            const int32_t e = int4_at(a, q), t = succ_id(e);
            c[q] = 0;
            td[q] = make_int2(0, 0);
            ta[q] = make_int4(-1, -1, -1, -1);
            if (act && q < d.y) {
              td[q] = deg[t];
              ta[q] = adj[t];
              c[q] = succ_one(e) ? 1 : remove_edge(t);
            }
          }
          // appends: slots by ballot, the tail in a scalar register
          int32_t *nv = s_fv[cu ^ 1];
          int2 *nd = s_fd[cu ^ 1];
          int4 *na = s_fa[cu ^ 1];
          hv = false;
#pragma unroll
          for (int q = 0; q < kKahnA; q++) {
            const bool want = c[q] == 1;
            const uint64_t m = __ballot(want);
            if (want) {
              const int32_t k = tail + (int32_t)__builtin_amdgcn_mbcnt_hi(
                                           (uint32_t)(m >> 32),
                                           __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
              const int32_t t = succ_id(int4_at(a, q));
              F[k] = t;
              nv[k - fe] = t;  // at most 4 * 64 entries: all in the mirror
              nd[k - fe] = td[q];
              na[k - fe] = ta[q];
            }
            tail += __popcll(m);
            hv = hv || __ballot(want && td[q].y > kKahnA) != 0;
          }
          lv++;
          cu ^= 1;
          fb = fe;
          fe = tail;
          if (fe == fb || fe - fb > 64 || hv) break;
        }
        if (lane == 0) {
          s_state[0] = fb;
          s_state[1] = fe;
          s_state[2] = lv;
          s_state[3] = cu;
          s_tail = tail;
          s_hv[cu] = hv ? 1 : 0;
          s_hv[cu ^ 1] = 0;
        }
      }
      __syncthreads();
      fb = s_state[0];
      fe = s_state[1];
      lvl = s_state[2];
      cur = s_state[3];
      __syncthreads();  // everyone has read the state before it can change again
      continue;
    }
    if (tid == 0) lstart[lvl] = fb;
    int32_t *nv = s_fv[cur ^ 1];
    int2 *nd = s_fd[cur ^ 1];
    int4 *na = s_fa[cur ^ 1];
    for (int32_t base = fb; base < fe; base += kKahnB, pp = pp == 2 ? 0 : pp + 1) {
      const int32_t i = base + tid;
      bool light = false;
      int2 d = make_int2(0, 0);
      int4 a = make_int4(-1, -1, -1, -1);
      if (i < fe) {
        int32_t u;
        if (i - fb < kKahnCap) {
          u = s_fv[cur][i - fb];
          d = s_fd[cur][i - fb];
          a = s_fa[cur][i - fb];
        } else {
          u = F[i];
          d = deg[u];
          a = adj[u];
        }
        level[u] = lvl;
        light = d.y <= kKahnA;
        if (!light) {
          const int32_t j = atomicAdd(&s_nh[pp], 1);
          s_hd[j] = d.y;
          s_he[j] = d.x;
        }
      }
      {  // light nodes: every removal and the successors' adjacency in one round
        int32_t c[kKahnA];
        int2 td[kKahnA];
        int4 ta[kKahnA];
#pragma unroll
        for (int q = 0; q < kKahnA; q++) {
          const int32_t e = int4_at(a, q), t = succ_id(e);
          c[q] = 0;
          td[q] = make_int2(0, 0);
          ta[q] = make_int4(-1, -1, -1, -1);
          if (light && q < d.y) {
            td[q] = deg[t];
            ta[q] = adj[t];
            c[q] = succ_one(e) ? 1 : remove_edge(t);
          }
        }
        bool want[kKahnA];
        int32_t tv[kKahnA];
#pragma unroll
        for (int q = 0; q < kKahnA; q++) {
          want[q] = c[q] == 1;
          tv[q] = succ_id(int4_at(a, q));
        }
        kahn_append_n<kKahnA>(want, tv, td, ta, F, &s_tail, fe, nv, nd, na, &s_hv[cur ^ 1]);
      }
      __syncthreads();
      const int32_t nh = s_nh[pp];
      // the counter of the pass after next: last read in the previous pass,
      // before this pass's barrier, and next counted after the next pass's
      if (tid == 0) {
        s_nh[pp == 0 ? 2 : pp - 1] = 0;
        s_hv[cur] = 0;  // read by every wave at the top of this level; the next frontier but one
      }
      if (nh > 0) {
        // exclusive prefix of the listed nodes' degrees (by wave 0 alone when
        // they fit one wave)
        const int32_t dj = tid < nh ? s_hd[tid] : 0;
        int32_t x = dj;
        if (nh > 64 || wave == 0)
          for (int o = 1; o < 64; o <<= 1) {
            const int32_t y = __shfl_up(x, o);
            if (lane >= o) x += y;
          }
        int32_t off = 0;
        if (nh > 64) {
          if (lane == 63) s_wt[wave] = x;
          __syncthreads();
          for (int w = 0; w < wave; w++) off += s_wt[w];
        }
        if (tid < nh) s_hp[tid] = off + x - dj;
        if (tid == nh - 1) s_hp[nh] = off + x;
        __syncthreads();
        const int32_t tot = s_hp[nh];
        int32_t h = 0;  // listed node of the thread's current edge (edges only move forward)
        for (int32_t t0 = tid; t0 < tot; t0 += kKahnE * kKahnB) {
          int32_t v[kKahnE];
#pragma unroll
          for (int q = 0; q < kKahnE; q++) {
            const int32_t t = t0 + q * kKahnB;
            v[q] = -1;
            if (t < tot) {
              int32_t lo = h, hi = nh - 1;  // last listed node whose edges start at or before t
              while (lo < hi) {
                const int32_t mid = (lo + hi + 1) >> 1;
                if (s_hp[mid] <= t) lo = mid;
                else hi = mid - 1;
              }
              h = lo;
              v[q] = g.out_idx[s_he[h] + (t - s_hp[h])];
            }
          }
          int32_t c[kKahnE];
          int2 td[kKahnE];
          int4 ta[kKahnE];
#pragma unroll
          for (int q = 0; q < kKahnE; q++) {
            c[q] = 0;
            td[q] = make_int2(0, 0);
            ta[q] = make_int4(-1, -1, -1, -1);
            if (v[q] >= 0) {
              td[q] = deg[v[q]];
              ta[q] = adj[v[q]];
              c[q] = remove_edge(v[q]);
            }
          }
          bool want[kKahnE];
#pragma unroll
          for (int q = 0; q < kKahnE; q++) want[q] = c[q] == 1;
          kahn_append_n<kKahnE>(want, v, td, ta, F, &s_tail, fe, nv, nd, na, &s_hv[cur ^ 1]);
        }
        __syncthreads();
      }
    }
    fb = fe;
    fe = s_tail;
    lvl++;
    cur ^= 1;
    __syncthreads();  // everyone has read s_tail before the next level appends
  }
  if (tid == 0) {
    st->i0 = lvl;     // number of levels
    st->i1 = s_tail;  // nodes taken; < n means a cycle
    lstart[lvl] = s_tail;
  }
}

constexpr int32_t kTopoPolicyN = 16384;  // smaller graphs take Kahn's kernel directly
constexpr int32_t kTopoPolicyIt = 12;    // policy iterations before Kahn's kernel takes over

// wv = 1 for a node with predecessors, 0 for a source
__global__ void k_topo_wv(int32_t n, const int32_t *in_ptr, int64_t *wv, const Status *st) {
  if (failed(st)) return;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x)
    wv[v] = in_ptr[v + 1] > in_ptr[v] ? 1 : 0;
}

// level[v] = val[v], sort keys (level) and ids (v) in node order, and the
// single segment [0, n) for the sort
__global__ void k_topo_keys(int32_t n, const int64_t *val, int32_t *level, uint64_t *keys,
                            uint32_t *ids, int32_t *seg, Status *st) {
  if (failed(st)) return;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t l = (int32_t)val[v];
    level[v] = l;
    keys[v] = (uint64_t)l;
    ids[v] = (uint32_t)v;
  }
  if (blockIdx.x == 0 && threadIdx.x < 2) seg[threadIdx.x] = threadIdx.x ? n : 0;
}

// level_ptr from the levels sorted ascending: every level up to the largest
// holds a node (a node of level l has a predecessor of level l - 1); the
// number of levels is the last key + 1
__global__ void k_topo_ptr(int32_t n, const uint64_t *keys, int32_t *level_ptr, Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t k = keys[p];
    if (p == 0 || keys[p - 1] != k) level_ptr[k] = (int32_t)p;
    if (p == n - 1) {
      level_ptr[k + 1] = n;
      st->i0 = (int32_t)k + 1;
    }
  }
}

__global__ void k_zero_u64(uint64_t *p, int64_t n) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

}  // namespace cel

using namespace cel;

// How the calling thread's last cel_topo_levels call found the levels.
struct TopoInfo {
  int32_t path, iters;
};
static thread_local TopoInfo t_topo_info{1, 0};

extern "C" int cel_topo_levels_info(int32_t *info) {
  if (!info) return set_error(CEL_E_ARG, "cel_topo_levels_info: NULL argument");
  info[0] = t_topo_info.path;
  info[1] = t_topo_info.iters;
  return CEL_OK;
}

extern "C" int cel_topo_levels(const cel_graph *g, int32_t *level, int32_t *order_id,
                               int32_t *level_ptr, int32_t *n_levels, hipStream_t s) {
  if (!g || !n_levels || !level_ptr) return set_error(CEL_E_ARG, "cel_topo_levels: NULL argument");
  if (g->n < 0 || g->m < 0) return set_error(CEL_E_ARG, "cel_topo_levels: negative size");
  if (!g->out_ptr || !g->in_ptr || (g->m > 0 && (!g->out_idx || !g->in_idx)) ||
      (g->n > 0 && (!g->w || !g->mem || !g->ob || !level || !order_id)))
    return set_error(CEL_E_ARG, "cel_topo_levels: NULL array");
  const int32_t n = g->n;
  Scratch sc(s);
  Status *st;
  int32_t *cnt;
  CEL_TRY(sc.get(&st, 1));
  CEL_TRY(sc.get(&cnt, n));
  CEL_HIP(hipMemsetAsync(st, 0, sizeof(Status), s));
  CEL_TRY(check_graph(g, 1, 0, /*bound=*/false, st, cnt, sc, s));
  if (n >= kTopoPolicyN && policy_iteration_on()) {
    // levels by policy iteration over the predecessors
    int64_t *wv, *val;
    CEL_TRY(sc.get(&wv, n));
    CEL_TRY(sc.get(&val, n));
    k_topo_wv<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, g->in_ptr, wv, st);
    bool launched = false;
    CEL_TRY(lp_policy(n, g->m, n, kTopoPolicyIt, g->in_ptr, g->in_idx, wv, 2, val, &st->i2,
                      "k_levels_policy", sc, s, st, &launched));
    if (launched) {
      // order_id: the nodes sorted by (level, id), one segment, queued before
      // the status is read (one host round trip when the iteration
      // converged; otherwise Kahn's kernel below rewrites every output, and
      // these values, lengths of real paths, stay below n meanwhile)
      uint64_t *keys;
      int32_t *seg;
      CEL_TRY(sc.get(&keys, n));
      CEL_TRY(sc.get(&seg, 2));
      uint32_t *ids = reinterpret_cast<uint32_t *>(order_id);
      k_topo_keys<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, val, level, keys, ids, seg, st);
      CEL_TRY(segmented_sort(keys, ids, seg, 1, n, sc, s, st));
      k_topo_ptr<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, keys, level_ptr, st);
      CEL_HIP(hipGetLastError());
      Status h;
      CEL_TRY(read_status(st, &h, s));
      if (h.err) return status_error(h, "cel_topo_levels");
      t_topo_info = {h.i2 ? 0 : 1, h.i3};
      if (h.i2) {
        *n_levels = h.i0;
        return CEL_OK;
      }
    } else {
      t_topo_info = {1, 0};
    }
  } else {
    t_topo_info = {1, 0};
  }
  int2 *deg;
  int4 *adj;
  int32_t *cmax;
  CEL_TRY(sc.get(&deg, n));
  CEL_TRY(sc.get(&adj, n));
  CEL_TRY(sc.get(&cmax, 1));
  CEL_HIP(hipMemsetAsync(cmax, 0, sizeof(int32_t), s));
  if (n > 0) {
    k_kahn_cnt<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, g->in_ptr, g->in_idx, cnt, cmax, st);
    k_kahn_prep<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, g->out_ptr, g->out_idx, cnt, deg, adj,
                                                      st);
  }
  {
    KTimer kt(s, "k_kahn");
    k_kahn<<<1, kKahnB, 0, s>>>(*g, cnt, cmax, deg, adj, order_id, level, level_ptr, st);
  }
  CEL_HIP(hipGetLastError());
  Status h;
  CEL_TRY(read_status(st, &h, s));
  if (h.err) return status_error(h, "cel_topo_levels");
  if (h.i1 != n) return set_error(CEL_E_CYCLE, "cel_topo_levels: the graph has a cycle (%d of %d nodes ordered)", h.i1, n);
  const int32_t L = h.i0;
  *n_levels = L;
  if (n == 0) return CEL_OK;
  // sort each level's frontier slice by id
  uint64_t *keys;
  CEL_TRY(sc.get(&keys, n));
  k_zero_u64<<<grid_for(n, 256, 4096), 256, 0, s>>>(keys, n);
  CEL_TRY(segmented_sort(keys, reinterpret_cast<uint32_t *>(order_id), level_ptr, L, n, sc, s, st));
  CEL_HIP(hipStreamSynchronize(s));
  return CEL_OK;
}
