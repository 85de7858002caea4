// Internal declarations shared by the libcel translation units.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <vector>

#include "cel.h"

namespace cel {

constexpr int64_t kLim = int64_t(1) << 62;  // every sum the path forms stays below this
constexpr int64_t kInf = INT64_MAX;         // comparison sentinel only
constexpr int kMaxD = 255;
constexpr uint64_t kNoAllocScratchBytes = CEL_NOALLOC_SCRATCH_BYTES;  // cel_makespan_noalloc's array

// error bits raised by device-side checks (Status::err)
enum : uint32_t { EB_ARG = 1u, EB_CYCLE = 2u, EB_OVERFLOW = 4u, EB_ORDER = 8u, EB_WAIT = 16u };

// Per-call device status block.  Kernels after a failed check read `err` and
// return without touching data addressed by unchecked indices.
struct Status {
  uint32_t err;
  uint32_t pad;
  uint64_t total;      // saturating sum(w) + sum over edges c[src]
  int64_t s0, s1, s2;  // call-specific scalar results
  int32_t i0, i1, i2, i3;
};

__host__ __device__ inline int64_t comm_of(int64_t ob, int64_t bw, int64_t lat) {
  return ob / bw + (ob % bw != 0 ? 1 : 0) + lat;
}

__device__ inline void raise_err(Status *st, uint32_t bits) { atomicOr(&st->err, bits); }

__device__ inline bool failed(const Status *st) {
  return __atomic_load_n(&st->err, __ATOMIC_RELAXED) != 0u;
}

// Orders a wave's own LDS accesses: every LDS write or atomic issued before it
// by any lane of this wave is visible to every lane after it.  (Compiler
// fence plus a wait for the wave's outstanding LDS operations.)
__device__ inline void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0), vmcnt/expcnt untouched
  __builtin_amdgcn_wave_barrier();
}

// Compiler-only ordering of LDS accesses inside one wave.  A wave's LDS
// operations complete in issue order, so a lane reads what another lane of
// the same wave wrote earlier without a wait; the compiler must merely keep
// the accesses in program order.
__device__ inline void lds_order() { asm volatile("" ::: "memory"); }
// A workgroup barrier that orders LDS only: global loads issued before it
// stay in flight (a full __syncthreads() waits for them too).  Use it where
// no wave reads another wave's global stores across the barrier.
__device__ inline void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// ------------------------------------------------ wave-level scans with DPP
// DPP moves read another lane's register inside the VALU (no LDS round trip).
// Lanes whose source is outside the allowed rows keep `old`.
template <int CTRL, int ROWMASK>
__device__ inline int32_t dpp32(int32_t src, int32_t old) {
  return __builtin_amdgcn_update_dpp(old, src, CTRL, ROWMASK, 0xF, false);
}
template <int CTRL, int ROWMASK>
__device__ inline int64_t dpp64(int64_t src, int64_t old) {
  const int32_t lo = dpp32<CTRL, ROWMASK>((int32_t)src, (int32_t)old);
  const int32_t hi = dpp32<CTRL, ROWMASK>((int32_t)(src >> 32), (int32_t)(old >> 32));
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// One Hillis-Steele step of the segmented scan of max-plus maps x -> max(a,
// x + b): combine with the lane selected by CTRL unless this lane already
// starts its segment; the identity (kNeg, 0, no start) fills missing lanes.
constexpr int64_t kNeg = -(int64_t(1) << 62);
template <int CTRL, int ROWMASK>
__device__ inline void seg_step(int64_t &a, int64_t &b, int32_t &f) {
  const int64_t ua = dpp64<CTRL, ROWMASK>(a, kNeg);
  const int64_t ub = dpp64<CTRL, ROWMASK>(b, 0);
  const int32_t uf = dpp32<CTRL, ROWMASK>(f, 0);
  if (!f) {
    const int64_t c = ua + b;
    a = c > a ? c : a;
    b = ub + b;
    f = uf;
  }
}

// Inclusive segmented scan over the 64 lanes of a wave: rows of 16 by right
// shifts 1, 2, 4, 8, then row 0 -> 1 and 2 -> 3 (broadcast of lane 15 of the
// row below), then rows 0-1 -> 2-3 (broadcast of lane 31).  f = 1 marks a
// segment start and, on return, whether the segment began at or before the
// lane.  a values must lie in [kNeg, 2^62), b in [0, 2^62).
__device__ inline void wave_seg_scan_dpp(int64_t &a, int64_t &b, int32_t &f) {
  seg_step<0x111, 0xF>(a, b, f);  // row_shr:1
  seg_step<0x112, 0xF>(a, b, f);  // row_shr:2
  seg_step<0x114, 0xF>(a, b, f);  // row_shr:4
  seg_step<0x118, 0xF>(a, b, f);  // row_shr:8
  seg_step<0x142, 0xA>(a, b, f);  // row_bcast:15 into rows 1 and 3
  seg_step<0x143, 0xC>(a, b, f);  // row_bcast:31 into rows 2 and 3
}

// Level loops of the window sweeps: only wave 0 runs narrow levels, so the
// other waves jump from one level the whole block must visit to the next.
// Bit (k & 63) of m[k >> 6] marks level k; returns the first marked level at
// or after k, or 256 when there is none.
__device__ inline int32_t next_marked(const uint64_t (&m)[4], int32_t k) {
  while (k < 256) {
    const int u = k >> 6;
    const uint64_t r = m[u] >> (k & 63);
    if (r) return k + (int32_t)__builtin_ctzll(r);
    k = (u + 1) << 6;
  }
  return 256;
}

// Lane l's value of a 64-bit register, for a uniform l.
__device__ inline int64_t readlane64(int64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int32_t)(v >> 32), l);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Window staging records the owner slot of each edge for the first kOwnFill
// edges of every row (one thread per row); an edge past that (rows of very
// high degree only) finds its owner by binary search over the row starts:
// the last row i in [0, nrows) with rp[i] <= e.
constexpr int kOwnFill = 32;
__device__ inline int32_t owner_of(const int32_t *rp, int32_t nrows, int32_t recorded, int32_t e) {
  if (recorded >= 0) return recorded;
  int32_t lo = 0, hi = nrows - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (rp[mid] <= e) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

// Maximum of value(index(e)) over the edges [e0, e1) of a node with too many
// neighbours for a sweep window, taken by the whole block: thread tid takes
// every B-th edge, keeping U index loads and then U value loads in flight
// (the next group's indices are requested before this group's values), and
// the lanes of each wave then combine theirs.  Values are >= 0; the result
// (-1 when the wave saw no edge) is the same in every lane of a wave.
constexpr int kHeavyU = 8;
template <int U, int B, class IndexF, class ValueF>
__device__ inline int64_t heavy_max(int32_t e0, int32_t e1, int tid, IndexF index, ValueF value) {
  int64_t mx = -1;
  int32_t rn[U];
#pragma unroll
  for (int u = 0; u < U; u++) {
    const int64_t e = (int64_t)e0 + tid + (int64_t)u * B;
    rn[u] = e < e1 ? index((int32_t)e) : -1;
  }
  for (int64_t base = e0; base < e1; base += (int64_t)U * B) {
    int32_t r[U];
#pragma unroll
    for (int u = 0; u < U; u++) {
      r[u] = rn[u];
      const int64_t e = base + (int64_t)U * B + tid + (int64_t)u * B;
      rn[u] = e < e1 ? index((int32_t)e) : -1;
    }
    int64_t x[U];
#pragma unroll
    for (int u = 0; u < U; u++) x[u] = r[u] >= 0 ? value(r[u]) : -1;
#pragma unroll
    for (int u = 0; u < U; u++) mx = x[u] > mx ? x[u] : mx;
  }
  for (int off = 32; off > 0; off >>= 1) {
    const int64_t o = __shfl_xor((long long)mx, off);
    mx = o > mx ? o : mx;
  }
  return mx;
}

// Edge-balanced CSR traversal: block b takes edges [b * kEdgesPB, +kEdgesPB)
// whatever their sources, so a node of huge out-degree is spread over many
// blocks.  Wave 0 finds the rows of the slice's first and last edge by a
// 64-way search over out_ptr; the slice's row pointers are staged in LDS
// (kRowsPB at most, else the per-edge search reads out_ptr).  Row pointers must
// already be validated (non-decreasing, out_ptr[0] = 0, out_ptr[n] = m).
constexpr int kEdgesPB = 2048;
constexpr int kRowsPB = 1024;

inline unsigned edge_blocks(int32_t m) {
  return m > 0 ? (unsigned)((m + kEdgesPB - 1) / kEdgesPB) : 1u;
}

// last u in [0, n) with out_ptr[u] <= x, for 0 <= x < m; wave-uniform result
__device__ inline int32_t wave_row_of(const int32_t *out_ptr, int32_t n, int32_t x, int lane) {
  int32_t lo = 0, hi = n - 1;  // out_ptr[lo] <= x; the answer lies in [lo, hi]
  while (lo < hi) {
    const int64_t span = (int64_t)hi - lo;
    const int32_t probe = lo + (int32_t)((span * (lane + 1) + 63) / 64);  // lane 63 probes hi
    const uint64_t le = __ballot(out_ptr[probe] <= x);  // a prefix of the lanes
    if (le == 0) {
      hi = __builtin_amdgcn_readlane(probe, 0) - 1;
    } else {
      const int k = 63 - __builtin_clzll(le);
      const int32_t pk = __builtin_amdgcn_readlane(probe, k);
      if (k < 63) hi = __builtin_amdgcn_readlane(probe, k + 1) - 1;
      lo = pk;
    }
  }
  return lo;
}

// Calls f(u, e) for every edge e of the block's slice, u its source.  s_ptr
// holds kRowsPB + 1 ints, s_u two.
template <class F>
__device__ inline void for_edges_balanced(const int32_t *out_ptr, int32_t n, int32_t m,
                                          int32_t *s_ptr, int32_t *s_u, F f) {
  const int64_t e0 = (int64_t)blockIdx.x * kEdgesPB;
  if (e0 >= m) return;  // uniform over the block
  const int32_t e1 = e0 + kEdgesPB < m ? (int32_t)(e0 + kEdgesPB) : m;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int32_t u0 = wave_row_of(out_ptr, n, (int32_t)e0, lane);
    const int32_t u1 = wave_row_of(out_ptr, n, e1 - 1, lane);
    if (lane == 0) {
      s_u[0] = u0;
      s_u[1] = u1;
    }
  }
  __syncthreads();
  const int32_t u0 = s_u[0], nr = s_u[1] - u0 + 1;
  const bool staged = nr <= kRowsPB;
  if (staged)
    for (int t = threadIdx.x; t <= nr; t += blockDim.x) s_ptr[t] = out_ptr[u0 + t];
  __syncthreads();
  for (int32_t e = (int32_t)e0 + threadIdx.x; e < e1; e += blockDim.x) {
    int32_t lo = 0, hi = nr - 1;  // last row r with ptr[u0 + r] <= e
    while (lo < hi) {
      const int32_t mid = (lo + hi + 1) >> 1;
      if ((staged ? s_ptr[mid] : out_ptr[u0 + mid]) <= e) lo = mid;
      else hi = mid - 1;
    }
    f(u0 + lo, e);
  }
}

// Phase timers for tuning builds (-DCEL_PHASE_TIMERS): thread 0 of each
// workgroup adds wall-clock intervals (100 MHz ticks) to a device array that
// cel_debug_phases() reads back.  Compiled out otherwise.
#ifdef CEL_PHASE_TIMERS
static __device__ unsigned long long g_cel_phase[32];  // one copy per translation unit
#define CEL_PHASE_READER(name)                                                          \
  extern "C" int name(unsigned long long *out) {                                       \
    unsigned long long z[32] = {};                                                     \
    if (hipMemcpyFromSymbol(out, HIP_SYMBOL(cel::g_cel_phase), sizeof z) != hipSuccess) \
      return -1;                                                                       \
    return hipMemcpyToSymbol(HIP_SYMBOL(cel::g_cel_phase), z, sizeof z) == hipSuccess ? 0 : -1; \
  }
#define CEL_TSTAMP(v) const unsigned long long v = wall_clock64()
#define CEL_TADD(i, a, b) \
  do { if (threadIdx.x == 0) atomicAdd(&g_cel_phase[i], (b) - (a)); } while (0)
#define CEL_TCOUNT(i) \
  do { if (threadIdx.x == 0) atomicAdd(&g_cel_phase[i], 1ull); } while (0)
#else
#define CEL_PHASE_READER(name)
#define CEL_TSTAMP(v) ((void)0)
#define CEL_TADD(i, a, b) ((void)0)
#define CEL_TCOUNT(i) ((void)0)
#endif

// ---------------------------------------------------------------- host side

int set_error(int code, const char *fmt, ...);

#define CEL_HIP(call)                                                              \
  do {                                                                             \
    hipError_t e_ = (call);                                                        \
    if (e_ != hipSuccess)                                                          \
      return ::cel::set_error(CEL_E_HIP, "%s failed: %s", #call, hipGetErrorString(e_)); \
  } while (0)

#define CEL_TRY(expr)          \
  do {                         \
    int rc_ = (expr);          \
    if (rc_ != CEL_OK) return rc_; \
  } while (0)

// Scratch memory of one call: sub-allocations from a per-(device, stream)
// arena of device blocks that persist across calls, so a call costs no
// allocator round trip once the arena has grown to its working size.  The
// arena is held for the object's lifetime, so calls on one stream from
// several host threads take turns; calls on different streams use different
// arenas.  Pointers stay valid until the object dies.
// The second form bumps through a fixed device range [base, base + cap) that
// the caller owns and never allocates: a request beyond `cap` fails with
// CEL_E_ARG.
struct Arena;
class Scratch {
 public:
  explicit Scratch(hipStream_t s);
  Scratch(hipStream_t s, char *base, size_t cap) : s_(s), base_(base), cap_(cap) {}
  ~Scratch();
  size_t used() const { return off_; }
  Scratch(const Scratch &) = delete;
  Scratch &operator=(const Scratch &) = delete;
  // allocate `count` elements of T (count may be 0: a 1-element block is taken)
  template <class T>
  int get(T **out, int64_t count) {
    return raw(reinterpret_cast<void **>(out), sizeof(T) * (size_t)(count > 0 ? count : 1));
  }
  int raw(void **out, size_t bytes);
  // A bump position, and a return to it: the space handed out since the mark
  // is taken again by later requests (for work queued after the work that
  // used it, on the same stream).
  struct Mark {
    size_t blk, off;
  };
  Mark mark() const;
  void release(const Mark &m);

 private:
  hipStream_t s_;
  Arena *a_ = nullptr;
  int err_ = CEL_OK;
  char *base_ = nullptr;  // fixed range (second form), else null
  size_t cap_ = 0, off_ = 0;
};

// Launch-configuration helpers
inline int grid_for(int64_t work, int block, int cap = 65535 * 4) {
  int64_t g = (work + block - 1) / block;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (int)g;
}

// Optional per-kernel timing: records HIP events around one launch when
// cel_timing(1) is on.  Pending pairs are resolved lazily, by
// cel_kernel_stats() or once many are pending.
class KTimer {
 public:
  KTimer(hipStream_t s, const char *name);
  ~KTimer();
  KTimer(const KTimer &) = delete;
  KTimer &operator=(const KTimer &) = delete;

 private:
  hipStream_t s_;
  const char *name_;
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

// Host-side argument checks (NULLs, sizes, device parameters).
int check_host_graph(const cel_graph *g, const char *fn);
int check_host_devices(const cel_devices *d, const char *fn);

// ----------------------------------------------------------- common kernels
// (launchers; defined in common.hip)

// Validates the graph arrays and, when `bound` is set, the overflow bound
// sum(w) + sum over edges of c[src] < 2^62.  CSR and CSC must hold the same
// edge multiset (compared by a hash total of the (source, target) pairs).
// Fills indeg_scratch (n ints) with the in-degrees.  Raises EB_ARG /
// EB_OVERFLOW in st.
int check_graph(const cel_graph *g, int64_t bw, int64_t lat, bool bound, Status *st,
                int32_t *indeg_scratch, Scratch &sc, hipStream_t s);

// Checks that `order` is a permutation of 0..n-1 consistent with level /
// level_ptr (level-monotone) and that level[u] < level[v] on every edge.
// Fills pos (inverse permutation).  Raises EB_ORDER.
int check_level_order(const cel_graph *g, const int32_t *order, const int32_t *level,
                      const int32_t *level_ptr, int32_t L, int32_t *pos, Status *st,
                      hipStream_t s);

// Checks that `order` is a permutation with pos[u] < pos[v] on every edge.
int check_topo_order(const cel_graph *g, const int32_t *order, int32_t *pos, Status *st,
                     hipStream_t s);

// out[0] = 0, out[i+1] = out[i] + in[i] for i < n (n+1 outputs).
int exclusive_scan_i32(const int32_t *in, int32_t *out, int64_t n, Scratch &sc, hipStream_t s);
int exclusive_scan_i64(const int64_t *in, int64_t *out, int64_t n, Scratch &sc, hipStream_t s);

// Relabels a CSR (ptr/idx over node ids, m edges, validated) into position
// space of `order`: row p lists pos[idx[k]] for the edges of node order[p].
int relabel_csr(int32_t n, int32_t m, const int32_t *order, const int32_t *pos,
                const int32_t *ptr, const int32_t *idx, int32_t *pptr, int32_t *pidx, Scratch &sc,
                hipStream_t s, const Status *st);

// Sorts each segment [seg[i], seg[i+1]) of (key, id) pairs by (key, id), both
// ascending; (key, id) pairs must be distinct.  seg is a device array of
// nseg + 1 offsets covering [0, n), trusted only while st holds no error (the
// kernels return early otherwise).  Stream-ordered: no host synchronisation.
int segmented_sort(uint64_t *keys, uint32_t *ids, const int32_t *seg, int32_t nseg, int64_t n,
                   Scratch &sc, hipStream_t s, const Status *st);

// Makespan helpers (makespan.hip), shared with the device-model variant.
// devp[k][p] = node_dev[k][order[p]] (EB_ARG when >= D); wp/cq = w and c by
// position; k_makespan_out scatters finish (and start = finish - w) by
// position back to node ids; k_fill_i64 sets n values.
__global__ void k_dev_gather(int32_t K, int32_t n, const int32_t *order, const uint8_t *node_dev,
                             int32_t D, uint8_t *devp, Status *st);
__global__ void k_pos_costs(int32_t n, const int32_t *order, const int64_t *w, const int64_t *ob,
                            int64_t bw, int64_t lat, int64_t *wp, int64_t *cq, const Status *st);
__global__ void k_makespan_out(int32_t K, int32_t n, const int32_t *order, const int64_t *finp,
                               const int64_t *wp, int64_t *start, int64_t *finish,
                               const Status *st);
__global__ void k_fill_i64(int64_t *p, int64_t n, int64_t v);
__global__ void k_fill_i32(int32_t *p, int64_t n, int32_t v);  // common.hip
// Maximum of two non-negative int64 values below 2^62 with one v_max_f64:
// read as IEEE doubles, such bit patterns are finite, non-negative numbers
// (subnormal below 2^52, which the kernels' f64 denormal mode keeps) whose
// order is the integers' order, and the maximum returns one operand's bits
// unchanged.  Every finish time, b-level and t-level is below 2^62 (the
// overflow check of the inputs).
__device__ inline int64_t max_nonneg(int64_t a, int64_t b) {
  int64_t r;
  asm volatile("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// Segmented prefix maximum over a wave (makespan.hip, ms_ring.hip).
// One step of the segmented prefix max: take the value of the lane selected
// by CTRL when `ok` (that lane lies in the same run); lanes the DPP move does
// not reach read the identity.
template <int CTRL, int ROWMASK>
__device__ inline void pmax_step(int64_t &y, bool ok) {
  const int32_t lo = __builtin_amdgcn_update_dpp((int32_t)kNeg, (int32_t)y, CTRL, ROWMASK, 0xF, false);
  const int32_t hi =
      __builtin_amdgcn_update_dpp((int32_t)(kNeg >> 32), (int32_t)(y >> 32), CTRL, ROWMASK, 0xF, false);
  const int64_t u = (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
  y = (ok && u > y) ? u : y;
}

// Inclusive prefix max over the run of every lane inside the wave's 64 lanes;
// hd = distance from the lane's slot to its run's first slot.
__device__ inline int64_t wave_seg_pmax(int64_t y, int32_t hd, int lane) {
  pmax_step<0x111, 0xF>(y, hd >= 1);               // row_shr:1
  pmax_step<0x112, 0xF>(y, hd >= 2);               // row_shr:2
  pmax_step<0x114, 0xF>(y, hd >= 4);               // row_shr:4
  pmax_step<0x118, 0xF>(y, hd >= 8);               // row_shr:8
  pmax_step<0x142, 0xA>(y, hd >= (lane & 15) + 1);  // row_bcast:15 into rows 1 and 3
  pmax_step<0x143, 0xC>(y, hd >= lane - 31);        // row_bcast:31 into rows 2 and 3
  return y;
}

// Device-coherent access to values that waves of other workgroups, or of
// this one, write during the same kernel (sweep.hip, ms_ring.hip).
__device__ inline int64_t ld_coherent(const int64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st_coherent(int64_t *p, int64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
constexpr int32_t kSpin = 1 << 21;  // polls before a wait gives up (far longer than any real wait)

// A pull value written earlier by this kernel, read again until it is
// visible.  A wait that outlasts kSpin polls raises EB_WAIT and sets the
// workgroup's abort flag (a broken invariant, never a slow run); the value
// returned then is 0 and the results are discarded by the error.
__device__ inline int64_t ld_final(const int64_t *p, int32_t *s_abort, Status *st) {
  int64_t v = ld_coherent(p);
  for (int32_t i = 0; v < 0; i++) {
    if (i == kSpin || __hip_atomic_load(s_abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) {
      raise_err(st, EB_WAIT);
      __hip_atomic_store(s_abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      return 0;
    }
    __builtin_amdgcn_s_sleep(1);
    v = ld_coherent(p);
  }
  return v;
}

// Values of the positions q[j] (q < 0: 0), every load issued before the first
// use; one not yet visible is read again by ld_final (rare).
template <int N>
__device__ inline void ld_many(int64_t (&x)[N], const int32_t (&q)[N], const int64_t *gx,
                               int32_t *s_abort, Status *st) {
#pragma unroll
  for (int j = 0; j < N; j++) x[j] = q[j] >= 0 ? ld_coherent(&gx[q[j]]) : 0;
#pragma unroll
  for (int j = 0; j < N; j++)
    if (x[j] < 0) x[j] = ld_final(&gx[q[j]], s_abort, st);
}

// ------------------------------------------------------- grid-wide barrier
// bar: [0] the released barrier (k << 1 | OR of the bits), [1] abort flag,
// [2 + b] workgroup b's arrival (k << 1 | its bit); zero before the launch.
constexpr int32_t kGridSpin = 1 << 20;  // polls of a grid barrier wait before it gives up
__device__ inline int32_t ld32(const int32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st32(int32_t *p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Grid barrier number k (1, 2, ...; the grid is no larger than what the GPU
// holds at once) that also ORs one bit over the workgroups.  Every value that
// one workgroup writes and another reads inside the kernel goes through
// agent-scope atomic stores and loads (st_coherent / ld_coherent, st32 /
// ld32): those are written through to, and read from, the level where all
// XCDs meet, so they need no L2 write-back or invalidation (an agent-scope
// fence performs both for the whole XCD's L2, in every workgroup: three
// quarters of a barrier's time at 256 workgroups).  What the barrier orders
// is completion: each wave waits for its own stores (vmcnt(0)) before its
// workgroup arrives, and the loads after the barrier are issued only once the
// release word has been seen.  Thread 0 of workgroup b publishes (k << 1 |
// bit) in its own arrival word; workgroup 0 waits until every arrival
// carries k, ORs the bits and publishes the release word; the others wait
// for it.  No two workgroups write one word.  Every wait is bounded: one that
// gives up, or an abort raised anywhere, returns false in every thread of
// every workgroup.  *bit_out = the OR.
__device__ inline bool grid_sync(int32_t *bar, int32_t k, int32_t bit, int32_t *s_ok, int32_t *s_bit,
                                 Status *st, int32_t *bit_out) {
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's stores are complete
  const int32_t G = (int32_t)gridDim.x;
  const int32_t mine = (k << 1) | bit;
  if (blockIdx.x == 0) {
    __syncthreads();
    int32_t ok = 1, orb = bit;
    for (int32_t i = threadIdx.x + 1; i < G; i += (int32_t)blockDim.x) {
      int32_t v = ld32(&bar[2 + i]);
      for (int32_t t = 0; (v >> 1) < k; t++) {
        if (t == kGridSpin || ld32(&bar[1]) != 0) {
          ok = 0;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
        v = ld32(&bar[2 + i]);
      }
      if (!ok) break;
      orb |= v & 1;
    }
    ok = __syncthreads_and(ok);
    orb = __syncthreads_or(orb);
    if (threadIdx.x == 0) {
      if (ok) {
        st32(&bar[0], (k << 1) | orb);
      } else {
        raise_err(st, EB_WAIT);
        st32(&bar[1], 1);
      }
      *s_ok = ok;
      *s_bit = orb;
    }
  } else {
    __syncthreads();
    if (threadIdx.x == 0) {
      st32(&bar[2 + blockIdx.x], mine);
      int32_t ok = 1;
      int32_t v = ld32(&bar[0]);
      for (int32_t t = 0; (v >> 1) < k; t++) {
        if (t == kGridSpin || ld32(&bar[1]) != 0) {
          raise_err(st, EB_WAIT);
          st32(&bar[1], 1);
          ok = 0;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
        v = ld32(&bar[0]);
      }
      *s_ok = ok;
      *s_bit = v & 1;
    }
  }
  __syncthreads();
  *bit_out = *s_bit;
  return *s_ok != 0;
}

// One node's state during pointer jumping (lp_policy.hip, dp_policy.hip):
// v the sum along the node's chain up to (not including) nxt, nxt the next
// node on the chain (-1 at its end), both = 1 once the chain has ended and
// both buffers hold the final entry.  Read and written by different
// workgroups of one kernel as two agent-scope 64-bit words.
struct LpE {
  int64_t v;       // sum of wv from the node up to (not including) nxt
  int32_t nxt;     // next node on the pointer chain, -1 at its end
  int32_t both;    // 1: the chain has ended and both buffers hold the final entry
};
__device__ inline LpE lpe_ld(const LpE *p) {
  const int64_t w = ld_coherent(reinterpret_cast<const int64_t *>(&p->nxt));
  return LpE{ld_coherent(&p->v), (int32_t)(uint32_t)w, (int32_t)(w >> 32)};
}
__device__ inline void lpe_st(LpE *p, const LpE &x) {
  st_coherent(&p->v, x.v);
  st_coherent(reinterpret_cast<int64_t *>(&p->nxt),
              (int64_t)(((uint64_t)(uint32_t)x.both << 32) | (uint32_t)x.nxt));
}

// Packed entries (policy iteration): value in the high 40 bits, next node
// in the low 24 (kPkEnd: the chain has ended), read and written whole by
// 64-bit agent-scope atomics.  Every version of an entry a reader can see is
// a true (sum of wv from the node up to next, next) pair, so a node may jump
// through whatever entry its next node holds at that moment: the result is
// again a true pair, further along the chain.  Pointer jumping then needs no
// barrier between rounds; a node's owner keeps its entry in registers and
// jumps until its chain ends.
constexpr uint32_t kPkEnd = 0xFFFFFFu;
__device__ inline uint64_t pk_make(int64_t v, uint32_t nx) { return ((uint64_t)v << 24) | nx; }
__device__ inline int64_t pk_val(uint64_t e) { return (int64_t)(e >> 24); }
__device__ inline uint32_t pk_next(uint64_t e) { return (uint32_t)e & kPkEnd; }
__device__ inline uint64_t pk_ld(const uint64_t *p) {
  return (uint64_t)ld_coherent(reinterpret_cast<const int64_t *>(p));
}
__device__ inline void pk_st(uint64_t *p, uint64_t e) {
  st_coherent(reinterpret_cast<int64_t *>(p), (int64_t)e);
}

// Nodes per thread in the asynchronous jumps: all of a thread's nodes jump
// together, so that no node starts late (a node that lags holds back every
// chain through it) as long as n <= kPkU times the grid's threads (2.1 million
// nodes on 256 workgroups of 1024); larger graphs take several groups.
constexpr int kPkU = 8;

// Grid barrier with agent-scope fences around the arrival and the release:
// plain stores before it are visible to plain loads after it, in every
// workgroup (thread 0's release writes back, and its acquire invalidates, the
// L2 of its XCD and its CU's L1, shared by the workgroup's waves).
__device__ inline bool grid_sync_fenced(int32_t *bar, int32_t k, int32_t *s_ok, int32_t *s_bit,
                                        Status *st) {
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();
  if (threadIdx.x == 0) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  int32_t bit;
  const bool ok = grid_sync(bar, k, 0, s_ok, s_bit, st, &bit);
  if (threadIdx.x == 0) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  __syncthreads();
  return ok;
}

// sweep.hip: level sweeps of eq. 3 (rev: b-level over successors) or eq. 2
// (t-level over predecessors) in position space; out[p] = the value at p.
struct SweepArgs {
  int32_t n, L;
  const int32_t *lp;              // [L + 1] level starts (positions)
  const int32_t *rptr, *ridx;     // neighbours (positions): successors (rev) or predecessors
  const int64_t *cst;             // [n] w (sink) / w + c
  const uint4 *rec;               // [n] pull records
  const int32_t *fptr, *fidx;     // far neighbours
  const int32_t *hptr, *hidx;     // slot lists of positions with many near neighbours
  const int32_t *seg;             // [segments + 1] first level of each segment
  const int32_t *wide;            // [L] levels out of ring mode
  int64_t *gx;                    // [n] pull values, -1 until written
  int64_t *out;                   // [n] results (== gx for rev)
};
constexpr int kPlanHead = 2, kPlanRec = 3, kPlanFirst = 64;  // plan table layout (ints)
struct SweepPlan {
  bool rev = false;
  SweepArgs a{};
  const int32_t *gkp = nullptr;   // [n + 1] chunk offsets of split rows in grid levels
  int32_t *tab = nullptr;         // the plan table on the device
};
// sweep_prepare queues the preparation on s; sweep_run reads the plan table
// back (synchronising s) and queues the sweep's kernels on s.
int sweep_prepare(SweepPlan &pl, bool rev, int32_t n, int32_t m, int32_t L, const int32_t *lp,
                  const int32_t *order, const int32_t *level, const int32_t *rptr,
                  const int32_t *ridx, const int64_t *wp, const int64_t *wcp, int64_t *out,
                  class Scratch &sc, hipStream_t s, Status *st);
int sweep_run(SweepPlan &pl, hipStream_t s, Status *st, const char *timer);
// segment starts of the level sweeps (sweep.hip), also used by ms_ring.hip
__global__ void k_sw_segflag(int32_t L, const int32_t *wide, int32_t *flag, const Status *st);
__global__ void k_sw_segfill(int32_t L, const int32_t *flag, const int32_t *pre, int32_t *seg,
                             int32_t *segid, int32_t *nseg, const Status *st);
// ms_batch.hip: makespans of K placements over the priority order (positions:
// lp, pptr/pidx, wp, cq by position; devp [K][n]); fin and fc [K][n] each
// (fin, fin + c), makespan [K]
int mb_ring(int32_t K, int32_t n, int32_t m, int32_t L, const int32_t *lp, const int32_t *order,
            const int32_t *level, const int32_t *pptr, const int32_t *pidx, const int64_t *wp,
            const int64_t *cq, const uint8_t *devp, int64_t *fin, int64_t *fc, int64_t *makespan,
            class Scratch &sc, hipStream_t s, Status *st);
// ms_wide.hip: makespans of K placements over a level-grouped priority order
// whose levels are wide (positions as for mb_ring; 1 <= D <= kWDev,
// n <= kWMaxN); fin [K][n], makespan [K]
constexpr int kWDev = 16;
constexpr int32_t kWMaxN = 1 << 27;
int mw_batch(int32_t K, int32_t n, int32_t L, int32_t D, const int32_t *lp, const int32_t *pptr,
             const int32_t *pidx, const int64_t *wp, const int64_t *cq, const uint8_t *devp,
             int64_t *fin, int64_t *makespan, class Scratch &sc, hipStream_t s, Status *st);
// ms_ring.hip: finish times of one placement over the device-grouped order
// (slots), levels run by one wave from an LDS ring; finp holds 2n int64 (the
// finish times, then finish + c), makespan one
int ms_ring(int32_t n, int32_t m, int32_t L, const int32_t *lp, const int32_t *gorder,
            const int32_t *level, const int32_t *pptr, const int32_t *pidx, const int64_t *wp,
            const int64_t *cq, const uint8_t *devp, const int64_t *sxp, const int32_t *metap,
            int64_t *finp, int64_t *makespan, class Scratch &sc, hipStream_t s, Status *st);
// lp_policy.hip: val(p) = wv(p) + max over q in aptr/aidx rows of val(q) by
// policy iteration on a persistent grid; out = val (- wv for kind 1, the
// t-level; kind 0 is the b-level, 2 the levels: they differ only there).  L
// bounds the pointer chains (nodes); at most cap iterations (cap <= 0: as
// many as are cheaper than a level sweep of L levels).  res[0] = 1 once
// converged (out written), res[1] = iterations; *launched false when the
// grid cannot be launched (the caller runs the level sweep).
int lp_policy(int32_t n, int32_t m, int32_t L, int32_t cap, const int32_t *aptr,
              const int32_t *aidx, const int64_t *wv, int kind, int64_t *out, int32_t *res,
              const char *timer, class Scratch &sc, hipStream_t s, Status *st, bool *launched);
// whether the calling thread's cel_topo_levels and cel_blevel calls try
// policy iteration first (cel_policy_iteration)
bool policy_iteration_on();
bool policy_iteration_packed();  // packed entries allowed (mode 1), else 16-byte rounds
// dp_policy.hip: the clustering DP's back pointers P[1..n] (smallest
// minimising i) and st->s0 = S(n) by policy iteration, given lo, PO, the comm
// by position and the successors in positions (sptr / sidx).  st->i2 = 1 once
// converged, st->i3 = iterations; *launched false when not launched.
// cluster starts from the DP's back pointers by doubling tables (flag[j] = 1
// at every start, st->i0 = their number); *launched false: nothing queued
int chain_marks(int32_t n, const int32_t *P, int32_t *flag, Scratch &sc, hipStream_t s, Status *st,
                bool *launched);
int dp_policy(int32_t n, int32_t m, int32_t R, const int32_t *lo, const int64_t *PO,
              const int64_t *cq, const int32_t *sptr, const int32_t *sidx, int32_t *P,
              class Scratch &sc, hipStream_t s, Status *st, bool *launched);
// ms_relax.hip: finish times of one placement by relaxation over the
// cross-device edges (devp = devices by position).  Queues the preparation
// and one persistent kernel on s and sets *launched; st->i3 = 1 once the
// kernel has converged (start, finish and makespan[0] are then written) and
// st->i2 = the rounds it ran.  *launched stays false when the grid cannot be
// co-resident (the caller runs the level sweep).  max_groups > 0 caps the
// workgroups (more tiles per thread).
int ms_relax(const cel_graph *g, const cel_devices *d, int32_t L, const int32_t *order,
             const uint8_t *node_dev, const uint8_t *devp, int64_t *start, int64_t *finish,
             int64_t *makespan, int max_groups, class Scratch &sc, hipStream_t s, Status *st,
             bool *launched);
// makespan_model.hip: a heterogeneous descriptor's ranges, its slowest
// multiplier, smallest bandwidth and largest latency; lead[g] = smallest
// pos[v] over the members v of group g (INT32_MAX before)
int check_hetero(const cel_hetero *h, const cel_devices *d, const char *fn, int64_t *bwmin,
                 int64_t *latmax, int64_t *tmax);
__global__ void k_colo_lead(int32_t n, int32_t G, const int32_t *group, const int32_t *pos,
                            int32_t *lead, Status *st);

// Copies the status block to the host (synchronising the stream).
int read_status(const Status *dst, Status *host, hipStream_t s);

// Fork/join onto a second stream of the current device (created once, at the
// default priority, non-blocking, kept until the process ends), for two
// independent single-workgroup kernels that would each leave the chip idle.
// start() orders the side stream after the work already on `s`; join()
// orders `s` after the work put on the side stream since.  The destructor
// joins if join() was not called, so an early error return still leaves
// every later use of `s` (scratch reuse included) behind the side work, and
// it waits for the join before releasing its events.
class SideFork {
 public:
  SideFork() = default;
  ~SideFork();
  SideFork(const SideFork &) = delete;
  SideFork &operator=(const SideFork &) = delete;
  int start(hipStream_t s);
  int join();
  hipStream_t side() const { return side_; }

 private:
  hipStream_t s_ = nullptr, side_ = nullptr;
  hipEvent_t fork_ = nullptr, join_ = nullptr;
  bool joined_ = true;
};

// Translates device error bits into an API error code with a message.
int status_error(const Status &h, const char *fn);

}  // namespace cel
