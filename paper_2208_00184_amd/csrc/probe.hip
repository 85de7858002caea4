// cel_step_latency: the dependent step below which a level of a
// level-synchronous sweep cannot go on this GPU.
//
// Every level of the b-level and makespan sweeps is a chain: gather the
// predecessors' values, combine them across the level with a wave scan,
// write the results where the next level gathers them.  The probe runs that
// chain with no other work: each iteration's gather index depends on the
// previous iteration's scan result, so iterations cannot overlap.  Three
// variants:
//   0  one wave: gather from LDS, 64-bit segmented max-plus scan (DPP), LDS
//      write (a narrow level run by one wave from a staged window);
//   1  the same in a workgroup of 1024 threads with a barrier after the
//      write (a level that needs the whole block);
//   2  one wave, the gather from a global array resident in L2 (a level whose
//      predecessors lie outside the staged window).
// The host times two launches of different lengths with HIP events and takes
// the difference per iteration, so launch overhead cancels.
#include "cel_internal.h"

namespace cel {

constexpr int kProbeTab = 4096;  // int64 entries: 32 KB of LDS or L2

template <int MODE>
__global__ void __launch_bounds__(1024)
    k_step_probe(int32_t steps, const int64_t *tab, int64_t *out) {
  __shared__ int64_t s_tab[kProbeTab];
  const int tid = threadIdx.x, lane = tid & 63;
  for (int i = tid; i < kProbeTab; i += blockDim.x) s_tab[i] = tab[i];
  __syncthreads();
  int64_t x = lane;
  for (int32_t it = 0; it < steps; it++) {
    const int32_t idx = (int32_t)((x + tid * 7) & (kProbeTab - 1));
    int64_t a = (MODE == 2) ? __builtin_nontemporal_load(&tab[idx]) : s_tab[idx];
    int64_t b = (a & 1023) + 1;
    int32_t f = (lane == 0) ? 1 : 0;
    wave_seg_scan_dpp(a, b, f);
    x = a + b;
    if (MODE == 1) {
      s_tab[(tid * 3 + it) & (kProbeTab - 1)] = x & 0xFFFF;
      __syncthreads();
    } else {
      s_tab[(lane * 5 + it) & (kProbeTab - 1)] = x & 0xFFFF;
      wave_lds_sync();
    }
  }
  out[blockIdx.x * blockDim.x + tid] = x;
}

}  // namespace cel

using namespace cel;

extern "C" int cel_step_latency(int32_t variant, int32_t steps, double *ns_per_step,
                                hipStream_t s) {
  const char *fn = "cel_step_latency";
  if (!ns_per_step || variant < 0 || variant > 2 || steps < 1 || steps > (1 << 24))
    return set_error(CEL_E_ARG, "%s: variant must be 0..2, steps in [1, 2^24]", fn);
  Scratch sc(s);
  int64_t *tab, *out;
  CEL_TRY(sc.get(&tab, kProbeTab));
  CEL_TRY(sc.get(&out, 1024));
  CEL_HIP(hipMemsetAsync(tab, 0, sizeof(int64_t) * kProbeTab, s));
  const int threads = variant == 1 ? 1024 : 64;
  hipEvent_t ev[4];
  for (auto &e : ev) CEL_HIP(hipEventCreate(&e));
  const int32_t lens[2] = {steps / 8 > 0 ? steps / 8 : 1, steps};
  int rc = CEL_OK;
  float ms[2] = {0.f, 0.f};
  for (int r = 0; r < 2 && rc == CEL_OK; r++) {
    if (hipEventRecord(ev[2 * r], s) != hipSuccess) rc = CEL_E_HIP;
    if (variant == 0)
      k_step_probe<0><<<1, threads, 0, s>>>(lens[r], tab, out);
    else if (variant == 1)
      k_step_probe<1><<<1, threads, 0, s>>>(lens[r], tab, out);
    else
      k_step_probe<2><<<1, threads, 0, s>>>(lens[r], tab, out);
    if (hipGetLastError() != hipSuccess || hipEventRecord(ev[2 * r + 1], s) != hipSuccess ||
        hipEventSynchronize(ev[2 * r + 1]) != hipSuccess ||
        hipEventElapsedTime(&ms[r], ev[2 * r], ev[2 * r + 1]) != hipSuccess)
      rc = CEL_E_HIP;
  }
  for (auto &e : ev) (void)hipEventDestroy(e);
  if (rc != CEL_OK) return set_error(rc, "%s: launch or event failed", fn);
  const double dn = (double)(lens[1] - lens[0]);
  *ns_per_step = dn > 0 ? (ms[1] - ms[0]) * 1e6 / dn : ms[1] * 1e6 / lens[1];
  return CEL_OK;
}
