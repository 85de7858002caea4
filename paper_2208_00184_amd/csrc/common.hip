// Shared pieces of libcel: error state, scratch memory, input validation,
// prefix scans, CSR relabelling into position space and a segmented sort.
#include <cstdarg>
#include <cstring>
#include <map>
#include <mutex>
#include <utility>
#include <vector>

#include "cel_internal.h"

namespace cel {

// ------------------------------------------------------------------ errors

static thread_local char g_msg[512] = "";

int set_error(int code, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof g_msg, fmt, ap);
  va_end(ap);
  return code;
}

const char *last_error_text() { return g_msg; }

int status_error(const Status &h, const char *fn) {
  if (h.err & EB_ARG) return set_error(CEL_E_ARG, "%s: malformed graph or argument arrays", fn);
  if (h.err & EB_CYCLE) return set_error(CEL_E_CYCLE, "%s: the graph has a cycle", fn);
  if (h.err & EB_OVERFLOW)
    return set_error(CEL_E_OVERFLOW, "%s: sum(w) + sum over edges of c[src] reaches 2^62", fn);
  if (h.err & EB_ORDER)
    return set_error(CEL_E_ORDER, "%s: order/level/cluster arrays inconsistent with the graph", fn);
  if (h.err & EB_WAIT)
    return set_error(CEL_E_HIP, "%s: a bounded wait between waves of a sweep timed out", fn);
  return CEL_OK;
}

int check_host_graph(const cel_graph *g, const char *fn) {
  if (!g) return set_error(CEL_E_ARG, "%s: graph is NULL", fn);
  if (g->n < 0 || g->m < 0) return set_error(CEL_E_ARG, "%s: negative n or m", fn);
  if (!g->out_ptr || !g->in_ptr || (g->m > 0 && (!g->out_idx || !g->in_idx)) ||
      (g->n > 0 && (!g->w || !g->mem || !g->ob)))
    return set_error(CEL_E_ARG, "%s: NULL graph array", fn);
  return CEL_OK;
}

int check_host_devices(const cel_devices *d, const char *fn) {
  if (!d || !d->cap) return set_error(CEL_E_ARG, "%s: devices or caps NULL", fn);
  if (d->D < 1 || d->D > kMaxD) return set_error(CEL_E_ARG, "%s: D = %d not in [1, 255]", fn, d->D);
  if (d->bw <= 0 || d->lat < 0 || d->lat >= kLim)
    return set_error(CEL_E_ARG, "%s: need bw > 0 and 0 <= lat < 2^62", fn);
  for (int i = 0; i < d->D; i++)
    if (d->cap[i] < 0) return set_error(CEL_E_ARG, "%s: negative memory cap", fn);
  return CEL_OK;
}

// ----------------------------------------------------------------- scratch

struct Arena {
  std::mutex mu;  // held by the Scratch object of the running call
  std::vector<std::pair<char *, size_t>> blocks;
  size_t blk = 0, off = 0;  // bump position of the running call
  size_t need = 0;          // bytes the running call asked for in total
  size_t grow_to = 0;       // one block of this size replaces the chain at the next call
};

static std::mutex g_arenas_mu;
static std::map<std::pair<int, hipStream_t>, Arena *> g_arenas;
constexpr size_t kAlign = 256;
constexpr size_t kMinBlock = size_t(8) << 20;

Scratch::Scratch(hipStream_t s) : s_(s) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    err_ = set_error(CEL_E_HIP, "hipGetDevice failed");
    return;
  }
  {
    std::lock_guard<std::mutex> lk(g_arenas_mu);
    Arena *&a = g_arenas[{dev, s}];
    if (!a) a = new Arena();  // kept until the process ends
    a_ = a;
  }
  a_->mu.lock();
  a_->blk = a_->off = a_->need = 0;
  if (a_->grow_to > 0) {
    // the last call spilled into several blocks: replace them by one that
    // fits it, once the stream has drained (earlier kernels may use them)
    if (hipStreamSynchronize(s_) != hipSuccess) {
      err_ = set_error(CEL_E_HIP, "hipStreamSynchronize failed");
      return;
    }
    for (auto &b : a_->blocks) (void)hipFree(b.first);
    a_->blocks.clear();
    void *p = nullptr;
    if (hipMalloc(&p, a_->grow_to) != hipSuccess || !p) {
      err_ = set_error(CEL_E_NOMEM, "scratch arena of %zu bytes: allocation failed", a_->grow_to);
      a_->grow_to = 0;
      return;
    }
    a_->blocks.push_back({(char *)p, a_->grow_to});
    a_->grow_to = 0;
  }
}

int Scratch::raw(void **out, size_t bytes) {
  if (err_ != CEL_OK) return err_;
  const size_t sz = (bytes + kAlign - 1) / kAlign * kAlign;
  if (base_) {  // fixed range: bump, never allocate
    if (sz > cap_ - off_)
      return err_ = set_error(CEL_E_ARG, "the call needs more than the %zu bytes of fixed scratch",
                              cap_);
    *out = base_ + off_;
    off_ += sz;
    return CEL_OK;
  }
  a_->need += sz;
  while (a_->blk < a_->blocks.size() && a_->off + sz > a_->blocks[a_->blk].second) {
    a_->blk++;
    a_->off = 0;
  }
  if (a_->blk == a_->blocks.size()) {  // grow: a new block at the end of the chain
    const size_t bsz = sz > kMinBlock ? sz : kMinBlock;
    void *p = nullptr;
    if (hipMalloc(&p, bsz) != hipSuccess || !p)
      return err_ = set_error(CEL_E_NOMEM, "scratch allocation of %zu bytes failed", bytes);
    a_->blocks.push_back({(char *)p, bsz});
    a_->off = 0;
  }
  *out = a_->blocks[a_->blk].first + a_->off;
  a_->off += sz;
  return CEL_OK;
}

Scratch::Mark Scratch::mark() const {
  if (base_ || !a_) return Mark{0, off_};
  return Mark{a_->blk, a_->off};
}

void Scratch::release(const Mark &m) {
  if (err_ != CEL_OK) return;
  if (base_ || !a_) {
    off_ = m.off;
    return;
  }
  // `need` keeps counting every request: it sizes the single block that
  // replaces a spilled chain, and a bound from above is enough there
  a_->blk = m.blk;
  a_->off = m.off;
}

Scratch::~Scratch() {
  if (!a_) return;
  if (a_->blocks.size() > 1) a_->grow_to = a_->need;
  a_->mu.unlock();
}

int read_status(const Status *dst, Status *host, hipStream_t s) {
  CEL_HIP(hipMemcpyAsync(host, dst, sizeof(Status), hipMemcpyDeviceToHost, s));
  CEL_HIP(hipStreamSynchronize(s));
  return CEL_OK;
}

// ------------------------------------------------------------ side stream

static std::mutex g_side_mu;
static std::map<int, hipStream_t> g_side;

int SideFork::start(hipStream_t s) {
  int dev = 0;
  CEL_HIP(hipGetDevice(&dev));
  {
    std::lock_guard<std::mutex> lk(g_side_mu);
    hipStream_t &t = g_side[dev];
    if (!t) CEL_HIP(hipStreamCreateWithFlags(&t, hipStreamNonBlocking));
    side_ = t;
  }
  CEL_HIP(hipEventCreateWithFlags(&fork_, hipEventDisableTiming));
  CEL_HIP(hipEventCreateWithFlags(&join_, hipEventDisableTiming));
  CEL_HIP(hipEventRecord(fork_, s));
  CEL_HIP(hipStreamWaitEvent(side_, fork_, 0));
  s_ = s;
  joined_ = false;
  return CEL_OK;
}

int SideFork::join() {
  if (joined_) return CEL_OK;
  joined_ = true;
  CEL_HIP(hipEventRecord(join_, side_));
  CEL_HIP(hipStreamWaitEvent(s_, join_, 0));
  return CEL_OK;
}

SideFork::~SideFork() {
  if (!joined_ && join() != CEL_OK) (void)hipStreamSynchronize(side_);
  if (join_) {
    (void)hipEventSynchronize(join_);
    (void)hipEventDestroy(join_);
  }
  if (fork_) (void)hipEventDestroy(fork_);
}

// ------------------------------------------------------------- validation

// saturating add for the overflow bound
__device__ inline uint64_t sat_add(uint64_t a, uint64_t b) {
  uint64_t r = a + b;
  return (r < a || r > (uint64_t)kLim) ? (uint64_t)kLim : r;
}

__global__ void k_check_nodes(cel_graph g, int64_t bw, int64_t lat, Status *st, uint64_t *part_out) {
  __shared__ uint64_t part[4];
  const int32_t n = g.n, m = g.m;
  uint64_t acc = 0;
  uint32_t bad = 0;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v <= n;
       v += (int64_t)gridDim.x * blockDim.x) {
    if (v == 0 && (g.out_ptr[0] != 0 || g.in_ptr[0] != 0)) bad |= EB_ARG;
    if (v == n) {
      if (g.out_ptr[n] != m || g.in_ptr[n] != m) bad |= EB_ARG;
      continue;
    }
    int32_t o0 = g.out_ptr[v], o1 = g.out_ptr[v + 1], i0 = g.in_ptr[v], i1 = g.in_ptr[v + 1];
    if (o1 < o0 || i1 < i0) bad |= EB_ARG;
    int64_t w = g.w[v], mem = g.mem[v], ob = g.ob[v];
    if (w < 0 || mem < 0 || ob < 0) {
      bad |= EB_ARG;
      continue;
    }
    int64_t deg = o1 > o0 ? (int64_t)o1 - o0 : 0;
    int64_t c = comm_of(ob, bw, lat);  // ob >= 0, bw >= 1, lat < 2^62: no overflow
    uint64_t t = (uint64_t)w;
    if (deg > 0) t = (c >= kLim / deg) ? (uint64_t)kLim : sat_add(t, (uint64_t)(c * deg));
    acc = sat_add(acc, t);
  }
  // wave reduce (saturating) then block
  for (int off = 32; off > 0; off >>= 1) {
    uint64_t o = __shfl_down(acc, off);
    acc = sat_add(acc, o);
  }
  int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) part[wv] = acc;
  if (bad) raise_err(st, bad);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t tot = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); i++) tot = sat_add(tot, part[i]);
    part_out[blockIdx.x] = tot;
  }
}

__device__ inline uint64_t mix64(uint64_t x) {  // SplitMix64 finaliser
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

// CSR and CSC must hold the same edge multiset.  Each side adds a 64-bit hash
// of every (source, target) pair into one total (block sums, one atomic per
// block); equal multisets give equal totals, and any difference is caught with
// overwhelming probability.  The CSC pass also writes each node's in-degree.
__device__ inline uint64_t pair_hash(int32_t u, int32_t v) {
  return mix64(((uint64_t)(uint32_t)u << 32) | (uint32_t)v);
}

// failed(st) read once per block, so that every thread of the block returns
// or none does (the kernels below reach block-wide barriers)
__device__ inline bool block_failed(const Status *st, int *flag) {
  if (threadIdx.x == 0) *flag = failed(st) ? 1 : 0;
  __syncthreads();
  return *flag != 0;
}

// the block's sum of x into *dst (one plain store per block: blocks write
// their own partials, which one small kernel adds up, so no address takes
// thousands of atomics)
__device__ inline void block_sum_u64(unsigned long long *dst, uint64_t x, uint64_t *red) {
  for (int off = 32; off > 0; off >>= 1) x += __shfl_down(x, off);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t t = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); i++) t += red[i];
    *dst = (unsigned long long)t;
  }
}

// CSR pass over edge-balanced blocks: target ranges and the pair-hash total
// (hs[block]: the block's part).
__global__ void k_check_csr(cel_graph g, Status *st, unsigned long long *hs) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  __shared__ uint64_t red[16];
  __shared__ int s_f;
  if (block_failed(st, &s_f)) return;  // row pointers not validated
  const int32_t n = g.n;
  uint32_t bad = 0;
  uint64_t acc = 0;
  for_edges_balanced(g.out_ptr, n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    const int32_t t = g.out_idx[e];
    if (t < 0 || t >= n) {
      bad |= EB_ARG;
      return;
    }
    acc += pair_hash(u, t);
  });
  if (bad) raise_err(st, bad);
  block_sum_u64(&hs[blockIdx.x], acc, red);
}

// CSC pass: source ranges, in-degrees and the pair-hash total (hs[block]).
__global__ void k_check_csc(cel_graph g, Status *st, int32_t *indeg, unsigned long long *hs) {
  __shared__ uint64_t red[16];
  __shared__ int s_f;
  if (block_failed(st, &s_f)) return;
  uint32_t bad = 0;
  uint64_t acc = 0;
  for (int64_t v = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; v < g.n;
       v += (int64_t)gridDim.x * blockDim.x) {
    const int32_t k0 = g.in_ptr[v], k1 = g.in_ptr[v + 1];
    indeg[v] = k1 - k0;
    for (int32_t k = k0; k < k1; k++) {
      const int32_t s = g.in_idx[k];
      if (s < 0 || s >= g.n) {
        bad |= EB_ARG;
        break;
      }
      acc += pair_hash(s, (int32_t)v);
    }
  }
  if (bad) raise_err(st, bad);
  block_sum_u64(&hs[blockIdx.x], acc, red);
}

// the two totals from the blocks' parts: [0, na) for the CSR side, then nb
// for the CSC side (a failed earlier check leaves parts unwritten: skipped)
__global__ void k_check_pairs(const unsigned long long *hs, int na, int nb, Status *st) {
  __shared__ uint64_t red[2][4];
  if (failed(st)) return;
  uint64_t a = 0, b = 0;
  for (int i = threadIdx.x; i < na; i += blockDim.x) a += hs[i];
  for (int i = threadIdx.x; i < nb; i += blockDim.x) b += hs[na + i];
  for (int off = 32; off > 0; off >>= 1) {
    a += __shfl_down(a, off);
    b += __shfl_down(b, off);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = a;
    red[1][threadIdx.x >> 6] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t ta = 0, tb = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); i++) {
      ta += red[0][i];
      tb += red[1][i];
    }
    if (ta != tb) raise_err(st, EB_ARG);
  }
}

// one block: saturating sum of the per-block partials
__global__ void k_finish_overflow(const uint64_t *part, int np, Status *st) {
  __shared__ uint64_t red[4];
  uint64_t acc = 0;
  for (int i = threadIdx.x; i < np; i += blockDim.x) acc = sat_add(acc, part[i]);
  for (int off = 32; off > 0; off >>= 1) acc = sat_add(acc, __shfl_down(acc, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t t = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); i++) t = sat_add(t, red[i]);
    st->total = t;
    if (t >= (uint64_t)kLim) raise_err(st, EB_OVERFLOW);
  }
}

int check_graph(const cel_graph *g, int64_t bw, int64_t lat, bool bound, Status *st,
                int32_t *indeg, Scratch &sc, hipStream_t s) {
  const int B = 256;
  const int nbk = grid_for((int64_t)g->n + 1, B, 2048);
  uint64_t *part;
  CEL_TRY(sc.get(&part, nbk));
  k_check_nodes<<<nbk, B, 0, s>>>(*g, bw, lat, st, part);
  if (g->n > 0) {
    const int na = (int)edge_blocks(g->m), nc = grid_for(g->n, B, 4096);
    unsigned long long *hs;
    CEL_TRY(sc.get(&hs, (int64_t)na + nc));
    k_check_csr<<<na, B, 0, s>>>(*g, st, hs);
    k_check_csc<<<nc, B, 0, s>>>(*g, st, indeg, hs + na);
    k_check_pairs<<<1, B, 0, s>>>(hs, na, nc, st);
  }
  if (bound) k_finish_overflow<<<1, B, 0, s>>>(part, nbk, st);
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

// pos[order[p]] = p; out-of-range ids raise EB_ORDER.  Duplicates are found
// by k_perm_verify: two positions naming one id leave pos[id] at one of them,
// and the other no longer reads itself back.
__global__ void k_inverse_perm(int32_t n, const int32_t *order, int32_t *pos, Status *st) {
  uint32_t bad = 0;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    int32_t v = order[p];
    if (v < 0 || v >= n) {
      bad |= EB_ORDER;
      continue;
    }
    pos[v] = (int32_t)p;
  }
  if (bad) raise_err(st, bad);
}

__global__ void k_perm_verify(int32_t n, const int32_t *order, const int32_t *pos, Status *st) {
  if (failed(st)) return;  // ids not in range
  uint32_t bad = 0;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x)
    if (pos[order[p]] != (int32_t)p) bad |= EB_ORDER;
  if (bad) raise_err(st, bad);
}

__global__ void k_check_levels_nodes(int32_t n, const int32_t *order, const int32_t *level,
                                     const int32_t *lp, int32_t L, Status *st) {
  uint32_t bad = 0;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p <= n;
       p += (int64_t)gridDim.x * blockDim.x) {
    if (p <= L) {  // level_ptr: 0 at the front, n at the back, non-decreasing
      int32_t a = lp[p];
      if (p == 0 && a != 0) bad |= EB_ORDER;
      if (p == L && a != n) bad |= EB_ORDER;
      if (p < L && lp[p + 1] < a) bad |= EB_ORDER;
    }
    if (p == n) continue;
    int32_t v = order[p];
    if (v < 0 || v >= n) {
      bad |= EB_ORDER;
      continue;
    }
    int32_t l = level[v];
    if (l < 0 || l >= L) {
      bad |= EB_ORDER;
      continue;
    }
    if (p < lp[l] || p >= lp[l + 1]) bad |= EB_ORDER;
  }
  if (bad) raise_err(st, bad);
}

// level[u] < level[v] on every edge (needs level values in range: checked above)
__global__ void k_check_levels_edges(cel_graph g, const int32_t *level, int32_t L, Status *st) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  if (failed(st)) return;  // edge indices or level values not validated
  uint32_t bad = 0;
  for_edges_balanced(g.out_ptr, g.n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    if (level[g.out_idx[e]] <= level[u]) bad |= EB_ORDER;
  });
  if (bad) raise_err(st, bad);
}

// pos[u] < pos[v] on every edge (pos must be a complete permutation: checked)
__global__ void k_check_topo_edges(cel_graph g, const int32_t *pos, Status *st) {
  __shared__ int32_t ptr[kRowsPB + 1], su[2];
  if (failed(st)) return;
  uint32_t bad = 0;
  for_edges_balanced(g.out_ptr, g.n, g.m, ptr, su, [&](int32_t u, int32_t e) {
    if (pos[g.out_idx[e]] <= pos[u]) bad |= EB_ORDER;
  });
  if (bad) raise_err(st, bad);
}

int check_level_order(const cel_graph *g, const int32_t *order, const int32_t *level,
                      const int32_t *level_ptr, int32_t L, int32_t *pos, Status *st,
                      hipStream_t s) {
  const int B = 256;
  const int32_t n = g->n;
  if (n > 0) {
    k_fill_i32<<<grid_for(n, B, 4096), B, 0, s>>>(pos, n, -1);
    k_inverse_perm<<<grid_for(n, B, 4096), B, 0, s>>>(n, order, pos, st);
    k_perm_verify<<<grid_for(n, B, 4096), B, 0, s>>>(n, order, pos, st);
  }
  k_check_levels_nodes<<<grid_for((int64_t)n + 1, B, 4096), B, 0, s>>>(n, order, level, level_ptr,
                                                                       L, st);
  if (n > 0) k_check_levels_edges<<<edge_blocks(g->m), B, 0, s>>>(*g, level, L, st);
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

int check_topo_order(const cel_graph *g, const int32_t *order, int32_t *pos, Status *st,
                     hipStream_t s) {
  const int B = 256;
  const int32_t n = g->n;
  if (n > 0) {
    k_fill_i32<<<grid_for(n, B, 4096), B, 0, s>>>(pos, n, -1);
    k_inverse_perm<<<grid_for(n, B, 4096), B, 0, s>>>(n, order, pos, st);
    k_perm_verify<<<grid_for(n, B, 4096), B, 0, s>>>(n, order, pos, st);
    k_check_topo_edges<<<edge_blocks(g->m), B, 0, s>>>(*g, pos, st);
  }
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

// ------------------------------------------------------------------- scans

constexpr int kScanB = 256, kScanItems = 16, kScanTile = kScanB * kScanItems;

template <class T>
__device__ T block_exclusive_scan(T x, T *wsum, T *total) {
  // 256 threads = 4 waves of 64
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  T inc = x;
  for (int off = 1; off < 64; off <<= 1) {
    T y = __shfl_up(inc, off);
    if (lane >= off) inc += y;
  }
  if (lane == 63) wsum[wv] = inc;
  __syncthreads();
  T base = 0, tot = 0;
  for (int i = 0; i < kScanB / 64; i++) {
    if (i < wv) base += wsum[i];
    tot += wsum[i];
  }
  __syncthreads();
  *total = tot;
  return base + inc - x;
}

template <class T>
__global__ void k_scan_reduce(const T *in, int64_t n, T *bsum) {
  __shared__ T wsum[kScanB / 64];
  int64_t base = (int64_t)blockIdx.x * kScanTile;
  T acc = 0;
  for (int i = threadIdx.x; i < kScanTile; i += kScanB) {
    int64_t k = base + i;
    if (k < n) acc += in[k];
  }
  T tot;
  (void)block_exclusive_scan<T>(acc, wsum, &tot);
  if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

template <class T>
__global__ void k_scan_apply(const T *in, T *out, int64_t n, const T *boff) {
  __shared__ T buf[kScanTile];
  __shared__ T wsum[kScanB / 64];
  int64_t base = (int64_t)blockIdx.x * kScanTile;
  for (int i = threadIdx.x; i < kScanTile; i += kScanB) {
    int64_t k = base + i;
    buf[i] = k < n ? in[k] : (T)0;
  }
  __syncthreads();
  T loc = 0;
  for (int k = 0; k < kScanItems; k++) loc += buf[threadIdx.x * kScanItems + k];
  T tot;
  T run = block_exclusive_scan<T>(loc, wsum, &tot) + (boff ? boff[blockIdx.x] : (T)0);
  for (int k = 0; k < kScanItems; k++) {
    run += buf[threadIdx.x * kScanItems + k];
    buf[threadIdx.x * kScanItems + k] = run;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < kScanTile; i += kScanB) {
    int64_t k = base + i;
    if (k < n) out[k + 1] = buf[i];
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) out[0] = 0;
}

template <class T>
static int exclusive_scan(const T *in, T *out, int64_t n, Scratch &sc, hipStream_t s) {
  if (n <= 0) {
    CEL_HIP(hipMemsetAsync(out, 0, sizeof(T), s));
    return CEL_OK;
  }
  int64_t nb = (n + kScanTile - 1) / kScanTile;
  if (nb == 1) {
    k_scan_apply<T><<<1, kScanB, 0, s>>>(in, out, n, nullptr);
    CEL_HIP(hipGetLastError());
    return CEL_OK;
  }
  T *bsum, *boff;
  CEL_TRY(sc.get(&bsum, nb));
  CEL_TRY(sc.get(&boff, nb + 1));
  k_scan_reduce<T><<<(unsigned)nb, kScanB, 0, s>>>(in, n, bsum);
  CEL_TRY(exclusive_scan<T>(bsum, boff, nb, sc, s));
  k_scan_apply<T><<<(unsigned)nb, kScanB, 0, s>>>(in, out, n, boff);
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

int exclusive_scan_i32(const int32_t *in, int32_t *out, int64_t n, Scratch &sc, hipStream_t s) {
  return exclusive_scan<int32_t>(in, out, n, sc, s);
}
int exclusive_scan_i64(const int64_t *in, int64_t *out, int64_t n, Scratch &sc, hipStream_t s) {
  return exclusive_scan<int64_t>(in, out, n, sc, s);
}

// ---------------------------------------------------------------- relabel

__global__ void k_row_deg(int32_t n, const int32_t *order, const int32_t *ptr, int32_t *deg,
                          const Status *st) {
  if (failed(st)) return;
  for (int64_t p = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; p < n;
       p += (int64_t)gridDim.x * blockDim.x) {
    int32_t v = order[p];
    deg[p] = ptr[v + 1] - ptr[v];
  }
}

// Output edges in edge-balanced blocks: slot k of row p (position p) takes
// edge k - pptr[p] of node order[p], so a row of huge degree is spread over
// many blocks.
__global__ void k_relabel_rows(int32_t n, int32_t m, const int32_t *order, const int32_t *pos,
                               const int32_t *ptr, const int32_t *idx, const int32_t *pptr,
                               int32_t *pidx, const Status *st) {
  __shared__ int32_t rp[kRowsPB + 1], su[2];
  if (failed(st)) return;
  for_edges_balanced(pptr, n, m, rp, su, [&](int32_t p, int32_t k) {
    pidx[k] = pos[idx[ptr[order[p]] + (k - pptr[p])]];
  });
}

int relabel_csr(int32_t n, int32_t m, const int32_t *order, const int32_t *pos,
                const int32_t *ptr, const int32_t *idx, int32_t *pptr, int32_t *pidx, Scratch &sc,
                hipStream_t s, const Status *st) {
  if (n <= 0) {
    CEL_HIP(hipMemsetAsync(pptr, 0, sizeof(int32_t), s));
    return CEL_OK;
  }
  int32_t *deg;
  CEL_TRY(sc.get(&deg, n));
  k_row_deg<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, order, ptr, deg, st);
  CEL_TRY(exclusive_scan_i32(deg, pptr, n, sc, s));
  k_relabel_rows<<<edge_blocks(m), 256, 0, s>>>(n, m, order, pos, ptr, idx, pptr, pidx, st);
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

// ------------------------------------------------------- segmented sort
//
// Device-only: tiles of at most kSortTile elements are bitonic-sorted in LDS,
// then segments longer than a tile are merged in passes of doubling run
// width.  Tile lists and pass counts come from device data and host-known
// upper bounds, so no host synchronisation is needed.

constexpr int kSortTile = 2048;

struct Tile {
  int32_t start, len;
};

__device__ inline bool kless(uint64_t ka, uint32_t ia, uint64_t kb, uint32_t ib) {
  return ka < kb || (ka == kb && ia < ib);
}

__global__ void k_tile_count(const int32_t *seg, int32_t nseg, int32_t *tcnt, const Status *st) {
  if (failed(st)) return;  // offsets not validated
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nseg;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t len = seg[i + 1] - seg[i];
    tcnt[i] = len > 1 ? (len + kSortTile - 1) / kSortTile : 0;
  }
}

__global__ void k_tile_fill(const int32_t *seg, int32_t nseg, const int32_t *toff, Tile *tiles,
                            const Status *st) {
  if (failed(st)) return;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < nseg;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int32_t a = seg[i], len = seg[i + 1] - a;
    if (len <= 1) continue;
    int32_t t = toff[i];
    for (int32_t o = 0; o < len; o += kSortTile, t++)
      tiles[t] = Tile{a + o, len - o < kSortTile ? len - o : kSortTile};
  }
}

// Bitonic sort of one tile (<= kSortTile elements) in LDS; blocks past the
// tile count (ntiles, on the device) exit.
__global__ void __launch_bounds__(256) k_sort_tiles(uint64_t *keys, uint32_t *ids,
                                                    const Tile *tiles, const int32_t *ntiles,
                                                    const Status *st) {
  __shared__ uint64_t sk[kSortTile];
  __shared__ uint32_t si[kSortTile];
  if (failed(st) || (int32_t)blockIdx.x >= *ntiles) return;
  const Tile t = tiles[blockIdx.x];
  int P = 2;
  while (P < t.len) P <<= 1;
  for (int i = threadIdx.x; i < P; i += blockDim.x) {
    if (i < t.len) {
      sk[i] = keys[t.start + i];
      si[i] = ids[t.start + i];
    } else {
      sk[i] = ~0ull;
      si[i] = ~0u;
    }
  }
  __syncthreads();
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = threadIdx.x; i < (P >> 1); i += blockDim.x) {
        int lo = 2 * stride * (i / stride) + (i % stride), hi = lo + stride;
        bool up = (lo & size) == 0;
        uint64_t ka = sk[lo], kb = sk[hi];
        uint32_t ia = si[lo], ib = si[hi];
        if (kless(kb, ib, ka, ia) == up) {
          sk[lo] = kb; sk[hi] = ka;
          si[lo] = ib; si[hi] = ia;
        }
      }
      __syncthreads();
    }
  }
  for (int i = threadIdx.x; i < t.len; i += blockDim.x) {
    keys[t.start + i] = sk[i];
    ids[t.start + i] = si[i];
  }
}

// segment of every element: last s with seg[s] <= i
__global__ void k_seg_of(const int32_t *seg, int32_t nseg, int64_t n, int32_t *sid,
                         const Status *st) {
  if (failed(st)) return;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    int32_t lo = 0, hi = nseg - 1;
    while (lo < hi) {
      const int32_t mid = (lo + hi + 1) >> 1;
      if (seg[mid] <= i) lo = mid;
      else hi = mid - 1;
    }
    sid[i] = lo;
  }
}

// One merge round over the segments longer than a tile: runs of `width` are
// merged in pairs (each element finds its slot by counting the smaller
// elements of the partner run); segments already one run are copied.
__global__ void k_merge_pass(const uint64_t *kin, const uint32_t *iin, uint64_t *kout,
                             uint32_t *iout, const int32_t *seg, const int32_t *sid, int64_t n,
                             int64_t width, const Status *st) {
  if (failed(st)) return;
  for (int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; g < n;
       g += (int64_t)gridDim.x * blockDim.x) {
    const int32_t s = sid[g];
    const int64_t base = seg[s], len = seg[s + 1] - base;
    if (len <= kSortTile) continue;  // sorted by its tile, never moves
    const uint64_t k = kin[g];
    const uint32_t id = iin[g];
    if (len <= width) {
      kout[g] = k;
      iout[g] = id;
      continue;
    }
    const int64_t off = g - base;
    const int64_t a0 = (off / (2 * width)) * (2 * width);
    const int64_t a1 = a0 + width < len ? a0 + width : len;
    const int64_t b1 = a0 + 2 * width < len ? a0 + 2 * width : len;
    int64_t r0, r1, own;
    if (off < a1) {
      r0 = a1; r1 = b1; own = off - a0;
    } else {
      r0 = a0; r1 = a1; own = off - a1;
    }
    int64_t l = r0, h = r1;  // partner elements smaller than (k, id)
    while (l < h) {
      const int64_t mid = (l + h) >> 1;
      if (kless(kin[base + mid], iin[base + mid], k, id)) l = mid + 1;
      else h = mid;
    }
    const int64_t dst = a0 + own + (l - r0);
    kout[base + dst] = k;
    iout[base + dst] = id;
  }
}

// elements of segments longer than a tile: copy back from the scratch copy
__global__ void k_copy_big(const uint64_t *kin, const uint32_t *iin, uint64_t *kout,
                           uint32_t *iout, const int32_t *seg, const int32_t *sid, int64_t n,
                           const Status *st) {
  if (failed(st)) return;
  for (int64_t g = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; g < n;
       g += (int64_t)gridDim.x * blockDim.x) {
    const int32_t s = sid[g];
    if (seg[s + 1] - seg[s] <= kSortTile) continue;
    kout[g] = kin[g];
    iout[g] = iin[g];
  }
}

int segmented_sort(uint64_t *keys, uint32_t *ids, const int32_t *seg, int32_t nseg, int64_t n,
                   Scratch &sc, hipStream_t s, const Status *st) {
  if (nseg <= 0 || n <= 1) return CEL_OK;
  int32_t *tcnt, *toff;
  Tile *tiles;
  const int64_t maxtiles = (int64_t)nseg + n / kSortTile + 1;
  CEL_TRY(sc.get(&tcnt, nseg));
  CEL_TRY(sc.get(&toff, (int64_t)nseg + 1));
  CEL_TRY(sc.get(&tiles, maxtiles));
  k_tile_count<<<grid_for(nseg, 256, 4096), 256, 0, s>>>(seg, nseg, tcnt, st);
  CEL_TRY(exclusive_scan_i32(tcnt, toff, nseg, sc, s));
  k_tile_fill<<<grid_for(nseg, 256, 4096), 256, 0, s>>>(seg, nseg, toff, tiles, st);
  {
    k_sort_tiles<<<(unsigned)maxtiles, 256, 0, s>>>(keys, ids, tiles, toff + nseg, st);
  }
  int passes = 0;  // enough for the longest possible segment (n)
  while (((int64_t)kSortTile << passes) < n) passes++;
  if (passes > 0) {
    int32_t *sid;
    uint64_t *k2;
    uint32_t *i2;
    CEL_TRY(sc.get(&sid, n));
    CEL_TRY(sc.get(&k2, n));
    CEL_TRY(sc.get(&i2, n));
    k_seg_of<<<grid_for(n, 256, 8192), 256, 0, s>>>(seg, nseg, n, sid, st);
    uint64_t *ka = keys, *kb = k2;
    uint32_t *ia = ids, *ib = i2;
    for (int p = 0; p < passes; p++) {
      k_merge_pass<<<grid_for(n, 256, 8192), 256, 0, s>>>(ka, ia, kb, ib, seg, sid, n,
                                                           (int64_t)kSortTile << p, st);
      std::swap(ka, kb);
      std::swap(ia, ib);
    }
    if (passes & 1)
      k_copy_big<<<grid_for(n, 256, 8192), 256, 0, s>>>(k2, i2, keys, ids, seg, sid, n, st);
  }
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

}  // namespace cel
