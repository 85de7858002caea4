// cel_cpd_order: the CPD-TOPO order (Section 5.1.3, Algorithm 1).
//
// The b-level and t-level that rank the nodes come from the GPU (cel_blevel).
// The walk itself pops one node at a time from a stack whose next top depends
// on what the previous pop freed: a chain of n dependent steps, each a few
// irregular memory reads.  On the GPU each step would wait on global-memory
// round trips (microseconds per node); the host walks a copy of the
// successor lists out of its caches in a fraction of that, so this entry
// point copies the CSR and cpath down, walks, and copies the order back.
#include <algorithm>
#include <vector>

#include "cel_internal.h"

using namespace cel;

extern "C" int cel_cpd_order(const cel_graph *g, const int64_t *blevel, const int64_t *tlevel,
                             int32_t *cpd_order, hipStream_t s) {
  const char *fn = "cel_cpd_order";
  CEL_TRY(check_host_graph(g, fn));
  const int32_t n = g->n;
  if (n == 0) return CEL_OK;
  if (!blevel || !tlevel || !cpd_order) return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  const int32_t m = g->m;
  std::vector<int32_t> rp((size_t)n + 1), ri((size_t)m);
  std::vector<int64_t> bl((size_t)n), tl((size_t)n);
  CEL_HIP(hipMemcpyAsync(rp.data(), g->out_ptr, sizeof(int32_t) * ((size_t)n + 1),
                         hipMemcpyDeviceToHost, s));
  if (m > 0)
    CEL_HIP(hipMemcpyAsync(ri.data(), g->out_idx, sizeof(int32_t) * (size_t)m,
                           hipMemcpyDeviceToHost, s));
  CEL_HIP(hipMemcpyAsync(bl.data(), blevel, sizeof(int64_t) * (size_t)n, hipMemcpyDeviceToHost, s));
  CEL_HIP(hipMemcpyAsync(tl.data(), tlevel, sizeof(int64_t) * (size_t)n, hipMemcpyDeviceToHost, s));
  CEL_HIP(hipStreamSynchronize(s));
  if (rp[0] != 0 || rp[n] != m) return set_error(CEL_E_ARG, "%s: out_ptr does not span m", fn);
  std::vector<int32_t> indeg((size_t)n, 0);
  for (int32_t v = 0; v < n; v++)
    if (rp[v + 1] < rp[v]) return set_error(CEL_E_ARG, "%s: out_ptr decreases at %d", fn, v);
  for (int32_t e = 0; e < m; e++) {
    const int32_t t = ri[e];
    if (t < 0 || t >= n) return set_error(CEL_E_ARG, "%s: out_idx[%d] = %d out of range", fn, e, t);
    indeg[t]++;
  }
  std::vector<int64_t> cpath((size_t)n);
  for (int32_t v = 0; v < n; v++) cpath[v] = tl[v] + bl[v];
  // push order: increasing cpath, equal cpath by decreasing id, so the top
  // of the stack is the largest cpath with the lowest id
  auto before = [&](int32_t a, int32_t b) {
    return cpath[a] != cpath[b] ? cpath[a] < cpath[b] : a > b;
  };
  std::vector<int32_t> stack, freed, out;
  stack.reserve((size_t)n);
  out.reserve((size_t)n);
  for (int32_t v = 0; v < n; v++)
    if (indeg[v] == 0) stack.push_back(v);
  std::sort(stack.begin(), stack.end(), before);
  while (!stack.empty()) {
    const int32_t v = stack.back();
    stack.pop_back();
    out.push_back(v);
    freed.clear();
    for (int32_t e = rp[v]; e < rp[v + 1]; e++)
      if (--indeg[ri[e]] == 0) freed.push_back(ri[e]);  // a child freed by its last in-edge
    if (freed.size() > 1) std::sort(freed.begin(), freed.end(), before);
    stack.insert(stack.end(), freed.begin(), freed.end());
  }
  if ((int32_t)out.size() != n)
    return set_error(CEL_E_CYCLE, "%s: the graph has a cycle (%zu of %d nodes ordered)", fn,
                     out.size(), n);
  CEL_HIP(hipMemcpyAsync(cpd_order, out.data(), sizeof(int32_t) * (size_t)n,
                         hipMemcpyHostToDevice, s));
  CEL_HIP(hipStreamSynchronize(s));
  return CEL_OK;
}
