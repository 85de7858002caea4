// cel_cpd_order: the CPD-TOPO order (Section 5.1.3, Algorithm 1), and
// cel_dfs_order: the DFS-TOPO order it refines (Section 4.2.2).
//
// CPD-TOPO ranks the nodes by b-level + t-level, which come from the GPU
// (cel_blevel); DFS-TOPO ranks the nodes freed together by id alone.
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

namespace {

// Copies the CSR (and, for CPD-TOPO, b-level and t-level) down, walks, and
// copies the order back.  The stack's top is the head of the paper's queue:
// the nodes freed by one pop go on top together, so the next pop takes one of
// them before anything older.  Among nodes pushed together the largest cpath
// (CPD-TOPO) comes first, then the lowest id.
int host_walk(const char *fn, const cel_graph *g, const int64_t *blevel, const int64_t *tlevel,
              int32_t *order, hipStream_t s) {
  const int32_t n = g->n;
  const int32_t m = g->m;
  const bool cpd = blevel != nullptr;
  std::vector<int32_t> rp((size_t)n + 1), ri((size_t)m);
  std::vector<int64_t> bl(cpd ? (size_t)n : 0), tl(cpd ? (size_t)n : 0);
  CEL_HIP(hipMemcpyAsync(rp.data(), g->out_ptr, sizeof(int32_t) * ((size_t)n + 1),
                         hipMemcpyDeviceToHost, s));
  if (m > 0)
    CEL_HIP(hipMemcpyAsync(ri.data(), g->out_idx, sizeof(int32_t) * (size_t)m,
                           hipMemcpyDeviceToHost, s));
  if (cpd) {
    CEL_HIP(hipMemcpyAsync(bl.data(), blevel, sizeof(int64_t) * (size_t)n, hipMemcpyDeviceToHost, s));
    CEL_HIP(hipMemcpyAsync(tl.data(), tlevel, sizeof(int64_t) * (size_t)n, hipMemcpyDeviceToHost, s));
  }
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
  std::vector<int64_t> cpath(cpd ? (size_t)n : 0);
  for (int32_t v = 0; cpd && v < n; v++) cpath[v] = tl[v] + bl[v];
  // push order: increasing cpath, equal cpath by decreasing id, so the top
  // of the stack is the largest cpath with the lowest id
  auto before = [&](int32_t a, int32_t b) {
    return (cpd && cpath[a] != cpath[b]) ? cpath[a] < cpath[b] : a > b;
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
  CEL_HIP(hipMemcpyAsync(order, out.data(), sizeof(int32_t) * (size_t)n, hipMemcpyHostToDevice, s));
  CEL_HIP(hipStreamSynchronize(s));
  return CEL_OK;
}

}  // namespace

extern "C" int cel_cpd_order(const cel_graph *g, const int64_t *blevel, const int64_t *tlevel,
                             int32_t *cpd_order, hipStream_t s) {
  const char *fn = "cel_cpd_order";
  CEL_TRY(check_host_graph(g, fn));
  if (g->n == 0) return CEL_OK;
  if (!blevel || !tlevel || !cpd_order) return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  return host_walk(fn, g, blevel, tlevel, cpd_order, s);
}

extern "C" int cel_dfs_order(const cel_graph *g, int32_t *dfs_order, hipStream_t s) {
  const char *fn = "cel_dfs_order";
  CEL_TRY(check_host_graph(g, fn));
  if (g->n == 0) return CEL_OK;
  if (!dfs_order) return set_error(CEL_E_ARG, "%s: NULL argument", fn);
  return host_walk(fn, g, nullptr, nullptr, dfs_order, s);
}
