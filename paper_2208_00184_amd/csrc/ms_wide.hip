// Batched makespans (Algorithm 3's scoring, Section 3.3's list schedule) over
// graphs with wide levels: one workgroup of kWB threads per placement walks
// the level-grouped priority order in chunks of at most kWB positions of one
// level.  A node's finish time is max(ready, free time of its device) + w,
// ready = max over its predecessors q of fin(q) + c(q) when q runs on another
// device; within a level the nodes of one device follow each other in order.
//
// Layout for this regime (hundreds to thousands of nodes per level, few
// devices):
//  * a ring in LDS holds the finish time and device of the last kWR positions
//    of the placement, so most predecessors are read from LDS; older ones
//    ("far") come from the placement's finish times in global memory, loaded
//    one chunk ahead (they were final two chunks earlier);
//  * the placement-independent part of every node (first kWPre predecessor
//    positions, their comm costs, w) is one record built once per call and
//    loaded two chunks ahead, so a chunk's critical path holds LDS work only;
//  * each wave orders its 64 nodes by device with ballots (stable, bit by bit
//    of the device id) and ds_permute, scans them as max-plus maps per device
//    run, and publishes one map per device; after one barrier every node
//    composes the free time of its device with the maps of the earlier waves.
//    Two workgroup barriers per chunk.
#include "cel_internal.h"

namespace cel {
namespace {

constexpr int kWB = 512;        // threads per placement
constexpr int kWW = kWB / 64;   // waves
constexpr int kWR = 8192;       // ring positions (finish time and device of each)
constexpr int kWPre = 3;        // in-edges held in a node's record
static_assert(kWR > 2 * kWB + 64, "far predecessors must be final two chunks ahead");
static_assert(kWDev <= 16 && kWMaxN <= (1 << 27), "4-bit device keys, 32-bit byte offsets");

// One chunk: positions [cb, cb + cnt) of level l, whose positions end at he;
// cnt == 0 marks the end of the walk.
struct WChunk {
  int32_t cb, cnt, he, l;
};

// level ends are read through the constant address space: scalar loads,
// which do not wait behind the vector loads in flight
typedef __attribute__((address_space(4))) const int32_t cint32_t;

// the first chunk at position nb of level l or of a later level (levels may
// be empty)
__device__ inline WChunk wstart(int32_t nb, int32_t l, const int32_t *lp, int32_t L) {
  for (; l < L; l++) {
    const int32_t he = ((const cint32_t *)lp)[l + 1];
    if (he > nb) return {nb, he - nb < kWB ? he - nb : kWB, he, l};
  }
  return {0, 0, 0, L};
}

__device__ inline WChunk wnext(const WChunk &c, const int32_t *lp, int32_t L) {
  if (c.cnt == 0) return c;
  const int32_t nb = c.cb + c.cnt;
  if (nb < c.he) return {nb, c.he - nb < kWB ? c.he - nb : kWB, c.he, c.l};
  return wstart(nb, c.l + 1, lp, L);
}

// What one thread loads for one chunk ahead of time.
struct WSet {
  int32_t q0, q1, q2, deg;  // first predecessors (-1: none), in-degree
  int64_t c0, c1, c2, w;    // their comm costs, the node's weight
  uint8_t dv;               // the node's device
  int64_t f0, f1, f2;       // far predecessors' finish times (unused when near)
  uint8_t d0, d1, d2;       // and devices
};

struct WArgs {
  int32_t n, L, D, dbits;  // dbits: bits of the largest device id
  const int32_t *lp, *pptr, *pidx;
  const int4 *rec;
  const longlong2 *cw;
  const int64_t *cq;
  const uint8_t *devp;
  int64_t *fin, *makespan;
};

// Loads and stores at 32-bit byte offsets from a base held in scalar
// registers (n * 32 bytes stay below 4 GiB: at most kWMaxN positions).
template <class T>
__device__ inline T ldo(const T *base, uint32_t i) {
  return *(const T *)((const char *)base + i * (uint32_t)sizeof(T));
}
template <class T>
__device__ inline void sto(T *base, uint32_t i, T v) {
  *(T *)((char *)base + i * (uint32_t)sizeof(T)) = v;
}

// the record part; idle lanes and finished walks load position cb (or 0)
__device__ inline void load_rec(WSet &S, const WChunk &c, const WArgs &a, const uint8_t *dk,
                                int tid) {
  const uint32_t ps = (uint32_t)(c.cb + (tid < c.cnt ? tid : 0));
  const int4 r = ldo(a.rec, ps);
  const longlong2 u = ldo(a.cw, 2 * ps), v = ldo(a.cw, 2 * ps + 1);
  S.q0 = r.x;
  S.q1 = r.y;
  S.q2 = r.z;
  S.deg = r.w;
  S.c0 = u.x;
  S.c1 = u.y;
  S.c2 = v.x;
  S.w = v.y;
  S.dv = ldo(dk, ps);
}

// far predecessors: positions below lo = max(0, chunk end - kWR); the others
// load position 0 (any valid address; the value is not used)
__device__ inline void load_far(WSet &S, const WChunk &c, const int64_t *fk, const uint8_t *dk) {
  const int32_t e = c.cb + c.cnt - kWR;
  const uint32_t lo = e > 0 ? (uint32_t)e : 0u;
  const uint32_t a0 = (uint32_t)S.q0 < lo ? (uint32_t)S.q0 : 0u;
  const uint32_t a1 = (uint32_t)S.q1 < lo ? (uint32_t)S.q1 : 0u;
  const uint32_t a2 = (uint32_t)S.q2 < lo ? (uint32_t)S.q2 : 0u;
  S.f0 = ldo(fk, a0);
  S.f1 = ldo(fk, a1);
  S.f2 = ldo(fk, a2);
  S.d0 = ldo(dk, a0);
  S.d1 = ldo(dk, a1);
  S.d2 = ldo(dk, a2);
}

struct WLds {
  uint8_t rd[kWR];              // device of position p at p % kWR
  int64_t rf[kWR];              // its finish time
  longlong2 t[kWW][kWDev];      // per wave and device: the run's map (a, b); absent: (kNeg, 0)
  int64_t avail[kWDev];         // free time of every device
};

// a predecessor's contribution to ready: from the ring unless far (q below
// lo), then the prefetched values.  q = -1 (no predecessor) reads a ring slot
// whose value the caller discards.
__device__ inline int64_t pred_val(int32_t q, int64_t c, int64_t ff, int32_t fd, uint32_t lo,
                                   int dv, const WLds &L) {
  const int32_t sl = q & (kWR - 1);
  const int64_t lf = L.rf[sl];
  const int32_t ld = L.rd[sl];
  const bool far = (uint32_t)q < lo;
  const int64_t f = far ? ff : lf;
  const int32_t d = far ? fd : ld;
  return f + (d != dv ? c : 0);
}

// DPP move of a 64-bit value; lanes whose source lies outside the row read 0
template <int CTRL>
__device__ inline int64_t shr64(int64_t v) {
  const int32_t lo = __builtin_amdgcn_mov_dpp((int32_t)v, CTRL, 0xF, 0xF, true);
  const int32_t hi = __builtin_amdgcn_mov_dpp((int32_t)(v >> 32), CTRL, 0xF, 0xF, true);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// One step of the inclusive scan of maps x -> max(a, x + b) over runs of equal
// devices: combine with the map the DPP move brings when `take` (its lane lies
// in the same run).  A real lane has a >= b >= 0, so the zeros that lanes
// without a source read act as the identity.
__device__ inline void map_step(int64_t &a, int64_t &b, int64_t ua, int64_t ub, bool take) {
  const int64_t na = max_nonneg(ua + b, a), nb = ub + b;
  a = take ? na : a;
  b = take ? nb : b;
}

__device__ inline int64_t join64(int32_t lo, int32_t hi) {
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Processes chunk cx with the loads in X; starts the loads of the chunk after
// next (into Z, descriptor cz) and the far loads of the next chunk (Y, cy).
__device__ __forceinline__ bool wbody(WSet &X, WSet &Y, WSet &Z, const WChunk &cx,
                                      const WChunk &cy, WChunk &cz, const WArgs &a,
                                      const uint8_t *dk, int64_t *fk, WLds &L, int tid) {
  if (cx.cnt == 0) return false;
  cz = wnext(cy, a.lp, a.L);
  load_rec(Z, cz, a, dk, tid);
  load_far(Y, cy, fk, dk);
  const int lane = tid & 63, wv = tid >> 6;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  lds_barrier();  // the previous chunk's ring, table and free-time writes are visible

  // ---- ready time of this thread's node
  const int32_t e = cx.cb + cx.cnt - kWR;
  const uint32_t lo = e > 0 ? (uint32_t)e : 0u;
  const bool act = tid < cx.cnt;
  const int dv = X.dv & (kWDev - 1);
  int64_t rdy = max_nonneg(max_nonneg(pred_val(X.q0, X.c0, X.f0, X.d0, lo, dv, L),
                                      pred_val(X.q1, X.c1, X.f1, X.d1, lo, dv, L)),
                           pred_val(X.q2, X.c2, X.f2, X.d2, lo, dv, L));
  rdy = X.deg > 0 ? rdy : 0;
  if (act && X.deg > kWPre) {  // in-edges past the record: read one by one
    const int32_t p = cx.cb + tid;
    const int32_t e1 = a.pptr[p + 1];
    for (int32_t k = a.pptr[p] + kWPre; k < e1; k++) {
      const int32_t q = a.pidx[k];
      int64_t f;
      int32_t d;
      if ((uint32_t)q >= lo) {
        f = L.rf[q & (kWR - 1)];
        d = L.rd[q & (kWR - 1)];
      } else {
        f = fk[q];
        d = dk[q];
      }
      rdy = max_nonneg(rdy, f + (d != dv ? a.cq[q] : 0));
    }
  }

  // ---- stable order of the wave's nodes by device.  Idle lanes (the highest
  // ones) take the last device with the map (kNeg, 0): they follow its real
  // lanes and leave the run's map unchanged.
  const int key = act ? dv : a.D - 1;
  uint64_t eq = ~0ull, lt = 0;
  for (int bit = a.dbits - 1; bit >= 0; bit--) {
    const uint64_t bb = __ballot((key >> bit) & 1);
    const uint64_t m = 0ull - (uint64_t)((key >> bit) & 1);  // all ones where the bit is set
    lt |= eq & ~bb & m;
    eq &= ~(bb ^ m);
  }
  const uint64_t below = eq & lt_mask;
  const int hd = __popcll(below);  // lanes of the run before this one
  const int slot = __popcll(lt) + hd;
  const int32_t meta = key | (lane << 4) | (hd << 10) | (((eq >> lane) == 1ull) << 16) |
                       ((int)act << 17);
  const int64_t a0 = act ? rdy + X.w : kNeg, b0 = act ? X.w : 0;
  const int sa4 = slot * 4;
  const int32_t pa_lo = __builtin_amdgcn_ds_permute(sa4, (int32_t)a0);
  const int32_t pa_hi = __builtin_amdgcn_ds_permute(sa4, (int32_t)(a0 >> 32));
  const int32_t pb_lo = __builtin_amdgcn_ds_permute(sa4, (int32_t)b0);
  const int32_t pb_hi = __builtin_amdgcn_ds_permute(sa4, (int32_t)(b0 >> 32));
  const int32_t pm = __builtin_amdgcn_ds_permute(sa4, meta);
  int64_t sa = join64(pa_lo, pa_hi), sb = join64(pb_lo, pb_hi);
  const int skey = pm & 15, shd = (pm >> 10) & 63;
  const int64_t av = L.avail[skey];  // read before wave 0 updates it

  // ---- scan of the maps over each run of the wave
  map_step(sa, sb, shr64<0x111>(sa), shr64<0x111>(sb), shd >= 1);  // row_shr:1
  map_step(sa, sb, shr64<0x112>(sa), shr64<0x112>(sb), shd >= 2);  // row_shr:2
  map_step(sa, sb, shr64<0x114>(sa), shr64<0x114>(sb), shd >= 4);  // row_shr:4
  map_step(sa, sb, shr64<0x118>(sa), shr64<0x118>(sb), shd >= 8);  // row_shr:8
  map_step(sa, sb, dpp64<0x142, 0xA>(sa, 0), dpp64<0x142, 0xA>(sb, 0),
           shd >= (lane & 15) + 1);  // row_bcast:15 into rows 1 and 3
  map_step(sa, sb, dpp64<0x143, 0xC>(sa, 0), dpp64<0x143, 0xC>(sb, 0),
           shd >= lane - 31);  // row_bcast:31 into rows 2 and 3

  // ---- publish the map of every device's run in this wave (absent: identity)
  if (lane < a.D) L.t[wv][lane] = make_longlong2(kNeg, 0);
  if ((pm >> 16) & 1) L.t[wv][skey] = make_longlong2(sa, sb);
  lds_barrier();  // every wave's maps are published

  // ---- compose: free time, then the earlier waves' maps of the device
  if ((pm >> 17) & 1) {
    int64_t x = av;
    for (int w2 = 0; w2 < wv; w2++) {
      const longlong2 t = L.t[w2][skey];
      x = max_nonneg(x + t.y, t.x);
    }
    const int64_t fin = max_nonneg(x + sb, sa);
    const uint32_t pos = (uint32_t)(cx.cb + wv * 64 + ((pm >> 4) & 63));
    L.rf[pos & (kWR - 1)] = fin;
    L.rd[pos & (kWR - 1)] = (uint8_t)skey;
    sto(fk, pos, fin);
  }
  if (wv == 0 && lane < a.D) {  // free times after the chunk: every wave's map in order
    int64_t x = L.avail[lane];
#pragma unroll
    for (int w2 = 0; w2 < kWW; w2++) {
      const longlong2 t = L.t[w2][lane];
      x = max_nonneg(x + t.y, t.x);
    }
    L.avail[lane] = x;
  }
  return true;
}

// two placements share a CU: 4 waves per SIMD, at most 128 VGPRs each
__global__ void __launch_bounds__(kWB, 4) k_mw_batch(WArgs a, const Status *st) {
  __shared__ WLds L;
  if (failed(st)) return;
  const int tid = threadIdx.x;
  const int64_t koff = (int64_t)blockIdx.x * a.n;
  const uint8_t *dk = a.devp + koff;
  int64_t *fk = a.fin + koff;
  if (tid < kWDev) L.avail[tid] = 0;
  WChunk c0 = wstart(0, 0, a.lp, a.L), c1 = wnext(c0, a.lp, a.L), c2;
  WSet A, B, C;
  load_rec(A, c0, a, dk, tid);
  load_rec(B, c1, a, dk, tid);
  load_far(A, c0, fk, dk);
  while (true) {
    if (!wbody(A, B, C, c0, c1, c2, a, dk, fk, L, tid)) break;
    if (!wbody(B, C, A, c1, c2, c0, a, dk, fk, L, tid)) break;
    if (!wbody(C, A, B, c2, c0, c1, a, dk, fk, L, tid)) break;
  }
  lds_barrier();
  if (tid < 64) {  // makespan: the latest free time (runs end at their device's last node)
    int64_t v = tid < a.D ? L.avail[tid] : 0;
    for (int off = 32; off > 0; off >>= 1) v = max_nonneg(v, __shfl_xor(v, off));
    if (tid == 0) a.makespan[blockIdx.x] = v;
  }
}

// records: first kWPre predecessor positions and in-degree; their comm costs
// and the node's weight
__global__ void k_mw_prep(int32_t n, const int32_t *pptr, const int32_t *pidx, const int64_t *cq,
                          const int64_t *wp, int4 *rec, longlong2 *cw, const Status *st) {
  if (failed(st)) return;
  for (int32_t p = blockIdx.x * blockDim.x + threadIdx.x; p < n; p += gridDim.x * blockDim.x) {
    const int32_t e0 = pptr[p], deg = pptr[p + 1] - e0;
    // a missing second or third predecessor repeats the first (the maximum
    // does not change); a source keeps -1 and the kernel sets its ready to 0
    const int32_t q0 = deg > 0 ? pidx[e0] : -1;
    const int32_t q1 = deg > 1 ? pidx[e0 + 1] : q0;
    const int32_t q2 = deg > 2 ? pidx[e0 + 2] : q0;
    rec[p] = make_int4(q0, q1, q2, deg);
    longlong2 u, v;
    u.x = q0 >= 0 ? cq[q0] : 0;
    u.y = q1 >= 0 ? cq[q1] : 0;
    v.x = q2 >= 0 ? cq[q2] : 0;
    v.y = wp[p];
    cw[2 * (int64_t)p] = u;
    cw[2 * (int64_t)p + 1] = v;
  }
}

}  // namespace

int mw_batch(int32_t K, int32_t n, int32_t L, int32_t D, const int32_t *lp, const int32_t *pptr,
             const int32_t *pidx, const int64_t *wp, const int64_t *cq, const uint8_t *devp,
             int64_t *fin, int64_t *makespan, Scratch &sc, hipStream_t s, Status *st) {
  if (D < 1 || D > kWDev || n < 1 || n > kWMaxN || L < 1) return CEL_E_ARG;
  int4 *rec;
  longlong2 *cw;
  CEL_TRY(sc.get(&rec, n));
  CEL_TRY(sc.get(&cw, 2 * (int64_t)n));
  k_mw_prep<<<grid_for(n, 256, 4096), 256, 0, s>>>(n, pptr, pidx, cq, wp, rec, cw, st);
  WArgs a{};
  a.n = n;
  a.L = L;
  a.D = D;
  while ((1 << a.dbits) < D) a.dbits++;
  a.lp = lp;
  a.pptr = pptr;
  a.pidx = pidx;
  a.rec = rec;
  a.cw = cw;
  a.cq = cq;
  a.devp = devp;
  a.fin = fin;
  a.makespan = makespan;
  {
    KTimer kt(s, "k_makespan_batch");
    k_mw_batch<<<(unsigned)K, kWB, 0, s>>>(a, st);
  }
  CEL_HIP(hipGetLastError());
  return CEL_OK;
}

}  // namespace cel
