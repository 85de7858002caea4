/*
 * CPU oracle for the Celeritas placement hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain single-threaded C, written from the definitions of Xu et al.,
 * "Celeritas: Fast Optimizer for Large Dataflow Graphs" (arXiv 2208.00184).
 * It is slow on purpose: every function evaluates the paper's definition (or
 * walks the paper's algorithm) in the most direct way, so it can be checked
 * against the text by eye.  Readings of passages where the paper is silent or
 * garbled are stated at each use.
 *
 * Only the tests, the package smoke check and the benchmark's CPU-baseline leg
 * call this code.  It shares nothing with the GPU library.
 */
#include "cel_oracle.h"

#include <stdlib.h>
#include <string.h>

#define INF INT64_MAX /* comparison sentinel only, never used in arithmetic */
#define LIM (((int64_t)1) << 62)

/* ---------------------------------------------------------------- helpers */

/* Communication time of node v's output: the linear fit t = k*d + b of
 * Section 4.2.1 with k = 1/bw rounded up to whole ns and b = lat. */
static int64_t comm_of(int64_t ob, int64_t bw, int64_t lat) {
  return ob / bw + (ob % bw != 0) + lat;
}

static int cmp_i64(const void *a, const void *b) {
  int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
  return (x > y) - (x < y);
}

/* Structural checks shared by every entry point of the oracle. */
static int check_graph(const orc_graph *g) {
  if (!g || g->n < 0 || g->m < 0) return ORC_E_ARG;
  int32_t n = g->n, m = g->m;
  if (!g->out_ptr || !g->in_ptr) return ORC_E_ARG;
  if (m > 0 && (!g->out_idx || !g->in_idx)) return ORC_E_ARG;
  if (n > 0 && (!g->w || !g->mem || !g->ob)) return ORC_E_ARG;
  if (g->out_ptr[0] != 0 || g->in_ptr[0] != 0 || g->out_ptr[n] != m || g->in_ptr[n] != m)
    return ORC_E_ARG;
  for (int32_t v = 0; v < n; v++) {
    if (g->out_ptr[v + 1] < g->out_ptr[v] || g->in_ptr[v + 1] < g->in_ptr[v]) return ORC_E_ARG;
    if (g->w[v] < 0 || g->mem[v] < 0 || g->ob[v] < 0) return ORC_E_ARG;
  }
  for (int32_t e = 0; e < m; e++)
    if (g->out_idx[e] < 0 || g->out_idx[e] >= n || g->in_idx[e] < 0 || g->in_idx[e] >= n)
      return ORC_E_ARG;
  /* CSR and CSC must hold the same multiset of edges. */
  if (m > 0) {
    int64_t *a = malloc(sizeof(int64_t) * (size_t)m), *b = malloc(sizeof(int64_t) * (size_t)m);
    if (!a || !b) { free(a); free(b); return ORC_E_ARG; }
    for (int32_t u = 0; u < n; u++)
      for (int32_t e = g->out_ptr[u]; e < g->out_ptr[u + 1]; e++)
        a[e] = ((int64_t)u << 32) | g->out_idx[e];
    for (int32_t v = 0; v < n; v++)
      for (int32_t e = g->in_ptr[v]; e < g->in_ptr[v + 1]; e++)
        b[e] = ((int64_t)g->in_idx[e] << 32) | v;
    qsort(a, (size_t)m, sizeof(int64_t), cmp_i64);
    qsort(b, (size_t)m, sizeof(int64_t), cmp_i64);
    int same = memcmp(a, b, sizeof(int64_t) * (size_t)m) == 0;
    free(a); free(b);
    if (!same) return ORC_E_ARG;
  }
  return ORC_OK;
}

static int check_devices(const orc_devices *d) {
  if (!d || d->D < 1 || d->D > 255 || !d->cap || d->bw <= 0 || d->lat < 0) return ORC_E_ARG;
  for (int32_t i = 0; i < d->D; i++)
    if (d->cap[i] < 0) return ORC_E_ARG;
  return ORC_OK;
}

/* Every time the path can produce is bounded by sum w + sum over edges of
 * c[src]; rejecting inputs where that reaches 2^62 keeps all sums exact. */
static int check_overflow(const orc_graph *g, const orc_devices *d) {
  int64_t tot = 0;
  for (int32_t v = 0; v < g->n; v++) {
    if (g->w[v] >= LIM - tot) return ORC_E_OVERFLOW;
    tot += g->w[v];
    int64_t c = comm_of(g->ob[v], d->bw, d->lat);
    int64_t k = g->out_ptr[v + 1] - g->out_ptr[v];
    if (k > 0) {
      if (c >= LIM / k) return ORC_E_OVERFLOW;
      if (c * k >= LIM - tot) return ORC_E_OVERFLOW;
      tot += c * k;
    }
  }
  return ORC_OK;
}

/* order must be a permutation of 0..n-1 with pos[u] < pos[v] on every edge;
 * fills pos (inverse permutation). */
static int check_order(const orc_graph *g, const int32_t *order, int32_t *pos) {
  int32_t n = g->n;
  if (n > 0 && !order) return ORC_E_ARG;
  for (int32_t v = 0; v < n; v++) pos[v] = -1;
  for (int32_t p = 0; p < n; p++) {
    int32_t v = order[p];
    if (v < 0 || v >= n || pos[v] != -1) return ORC_E_ORDER;
    pos[v] = p;
  }
  for (int32_t u = 0; u < n; u++)
    for (int32_t e = g->out_ptr[u]; e < g->out_ptr[u + 1]; e++)
      if (pos[u] >= pos[g->out_idx[e]]) return ORC_E_ORDER;
  return ORC_OK;
}

/* ------------------------------------------------------- topological levels */

/* Kahn's method (Section 4.2.2): repeatedly take a node of indegree 0 and
 * delete its out-edges; the FIFO queue is M-TOPO's.  A node's level is one more
 * than the largest level among its predecessors (0 for a source), which is the
 * round of a level-by-level Kahn in which it becomes free.  Fewer than n nodes
 * taken means a cycle. */
int orc_topo_levels(const orc_graph *g, int32_t *level, int32_t *order_id,
                    int32_t *level_ptr, int32_t *n_levels) {
  int rc = check_graph(g);
  if (rc) return rc;
  int32_t n = g->n;
  if (!level_ptr || !n_levels || (n > 0 && (!level || !order_id))) return ORC_E_ARG;
  int32_t *indeg = malloc(sizeof(int32_t) * (size_t)(n + 1));
  int32_t *queue = malloc(sizeof(int32_t) * (size_t)(n + 1));
  int32_t head = 0, tail = 0;
  for (int32_t v = 0; v < n; v++) {
    indeg[v] = g->in_ptr[v + 1] - g->in_ptr[v];
    level[v] = 0;
    if (indeg[v] == 0) queue[tail++] = v;
  }
  while (head < tail) {
    int32_t u = queue[head++];
    for (int32_t e = g->out_ptr[u]; e < g->out_ptr[u + 1]; e++) {
      int32_t v = g->out_idx[e];
      if (level[u] + 1 > level[v]) level[v] = level[u] + 1;
      if (--indeg[v] == 0) queue[tail++] = v;
    }
  }
  free(indeg);
  free(queue);
  if (tail != n) return ORC_E_CYCLE;
  int32_t L = 0;
  for (int32_t v = 0; v < n; v++)
    if (level[v] + 1 > L) L = level[v] + 1;
  /* stable counting sort of the ids by level */
  for (int32_t l = 0; l <= L; l++) level_ptr[l] = 0;
  for (int32_t v = 0; v < n; v++) level_ptr[level[v] + 1]++;
  for (int32_t l = 0; l < L; l++) level_ptr[l + 1] += level_ptr[l];
  int32_t *fill = malloc(sizeof(int32_t) * (size_t)(L + 1));
  memcpy(fill, level_ptr, sizeof(int32_t) * (size_t)(L + 1));
  for (int32_t v = 0; v < n; v++) order_id[fill[level[v]]++] = v;
  free(fill);
  *n_levels = L;
  return ORC_OK;
}

/* ------------------------------------------------------ b-level and t-level */

typedef struct {
  int32_t level;
  int64_t bl;
  int32_t id;
} prio_key;

static int cmp_prio(const void *a, const void *b) {
  const prio_key *x = a, *y = b;
  if (x->level != y->level) return x->level < y->level ? -1 : 1;
  if (x->bl != y->bl) return x->bl > y->bl ? -1 : 1; /* larger b-level first */
  return (x->id > y->id) - (x->id < y->id);
}

/* eq. 3: blevel(v) = w_v for a sink, else max over successors s of
 * (blevel(s) + c_{v,s}) + w_v; eq. 2: tlevel(v) = 0 for a source, else max over
 * predecessors p of (tlevel(p) + w_p + c_{p,v}).  c_{v,s} is the source's comm
 * time c[v] (before placement it is always paid), or 0 with ORC_COMM_OFF.  The
 * critical path is the largest b-level (Section 5.1.3).  The priority order
 * sorts by level, then larger b-level, then id (a topological order that
 * visits longer critical paths first inside each level). */
int orc_blevel(const orc_graph *g, const orc_devices *d, const int32_t *level,
               const int32_t *order_id, int32_t flags, int64_t *blevel,
               int64_t *tlevel, int32_t *prio_order, int64_t *cp) {
  int rc = check_graph(g);
  if (rc) return rc;
  if ((rc = check_devices(d))) return rc;
  if ((rc = check_overflow(g, d))) return rc;
  int32_t n = g->n;
  if (!cp || (n > 0 && (!level || !order_id || !blevel))) return ORC_E_ARG;
  int32_t *pos = malloc(sizeof(int32_t) * (size_t)(n + 1));
  rc = check_order(g, order_id, pos);
  free(pos);
  if (rc) return rc;
  int64_t *c = malloc(sizeof(int64_t) * (size_t)(n + 1));
  for (int32_t v = 0; v < n; v++)
    c[v] = (flags & ORC_COMM_OFF) ? 0 : comm_of(g->ob[v], d->bw, d->lat);
  for (int32_t p = n - 1; p >= 0; p--) {
    int32_t v = order_id[p];
    if (g->out_ptr[v + 1] == g->out_ptr[v]) {
      blevel[v] = g->w[v];
    } else {
      int64_t best = 0;
      for (int32_t e = g->out_ptr[v]; e < g->out_ptr[v + 1]; e++) {
        int64_t t = blevel[g->out_idx[e]] + c[v];
        if (e == g->out_ptr[v] || t > best) best = t;
      }
      blevel[v] = best + g->w[v];
    }
  }
  if (tlevel) {
    for (int32_t p = 0; p < n; p++) {
      int32_t v = order_id[p];
      int64_t best = 0;
      for (int32_t e = g->in_ptr[v]; e < g->in_ptr[v + 1]; e++) {
        int32_t u = g->in_idx[e];
        int64_t t = tlevel[u] + g->w[u] + c[u];
        if (t > best) best = t;
      }
      tlevel[v] = best;
    }
  }
  int64_t best = 0;
  for (int32_t v = 0; v < n; v++)
    if (blevel[v] > best) best = blevel[v];
  *cp = best;
  if (prio_order) {
    prio_key *k = malloc(sizeof(prio_key) * (size_t)(n + 1));
    for (int32_t v = 0; v < n; v++) {
      k[v].level = level[v];
      k[v].bl = blevel[v];
      k[v].id = v;
    }
    qsort(k, (size_t)n, sizeof(prio_key), cmp_prio);
    for (int32_t p = 0; p < n; p++) prio_order[p] = k[p].id;
    free(k);
  }
  free(c);
  return ORC_OK;
}

/* ---------------------------------------------------------------- CPD-TOPO */

typedef struct {
  int64_t cpath;
  int32_t id;
} cp_key;

/* increasing cpath, and among equal cpath the higher id first: pushed in this
 * order, the top of the stack is the largest cpath with the lowest id */
static int cmp_push(const void *a, const void *b) {
  const cp_key *x = a, *y = b;
  if (x->cpath != y->cpath) return x->cpath < y->cpath ? -1 : 1;
  return (y->id > x->id) - (y->id < x->id);
}

/* Algorithm 1 (CPD_Topo), Section 5.1.3: the queue Q has the sources in
 * decreasing cpath order; the head node is dequeued and numbered, its
 * children sorted by increasing cpath, its out-edges deleted, and each child
 * left with in-degree 0 is put at the head of Q.  Q is a stack here (the head
 * is the top).  A child reached by several edges from the node is counted
 * once: it becomes free when its last in-edge goes. */
int orc_cpd_topo(const orc_graph *g, const int64_t *blevel, const int64_t *tlevel,
                 int32_t *cpd_order) {
  int rc = check_graph(g);
  if (rc) return rc;
  int32_t n = g->n;
  if (n > 0 && (!blevel || !tlevel || !cpd_order)) return ORC_E_ARG;
  int32_t *indeg = calloc((size_t)n + 1, sizeof(int32_t));
  int32_t *stack = malloc(sizeof(int32_t) * ((size_t)n + 1));
  cp_key *tmp = malloc(sizeof(cp_key) * ((size_t)n + 1));
  for (int32_t e = 0; e < g->m; e++) indeg[g->out_idx[e]]++;
  /* sources, pushed so that the largest cpath (lowest id on ties) is on top */
  int32_t ns = 0;
  for (int32_t v = 0; v < n; v++)
    if (indeg[v] == 0) {
      tmp[ns].cpath = tlevel[v] + blevel[v];
      tmp[ns].id = v;
      ns++;
    }
  qsort(tmp, (size_t)ns, sizeof(cp_key), cmp_push);
  int32_t top = 0;
  for (int32_t k = 0; k < ns; k++) stack[top++] = tmp[k].id;
  int32_t out = 0;
  while (top > 0) {
    int32_t v = stack[--top];
    cpd_order[out++] = v;
    int32_t nr = 0;
    for (int32_t e = g->out_ptr[v]; e < g->out_ptr[v + 1]; e++) {
      int32_t s = g->out_idx[e];
      if (--indeg[s] == 0) {
        tmp[nr].cpath = tlevel[s] + blevel[s];
        tmp[nr].id = s;
        nr++;
      }
    }
    qsort(tmp, (size_t)nr, sizeof(cp_key), cmp_push);
    for (int32_t k = 0; k < nr; k++) stack[top++] = tmp[k].id;
  }
  free(indeg);
  free(stack);
  free(tmp);
  return out == n ? ORC_OK : ORC_E_CYCLE;
}

/* DFS-TOPO order (Section 4.2.2): a queue Q holds every node with no
 * remaining in-edge, sources first in increasing id; the head of Q is removed
 * and output, its out-edges removed, and the successors that this leaves with
 * no in-edge go to the head of Q, the lowest id in front.  Q is held as an
 * array whose end is the head. */
int orc_dfs_topo(const orc_graph *g, int32_t *dfs_order) {
  int rc = check_graph(g);
  if (rc) return rc;
  int32_t n = g->n;
  if (n > 0 && !dfs_order) return ORC_E_ARG;
  int32_t *indeg = calloc((size_t)n + 1, sizeof(int32_t));
  int32_t *q = malloc(sizeof(int32_t) * ((size_t)n + 1));
  for (int32_t e = 0; e < g->m; e++) indeg[g->out_idx[e]]++;
  int32_t head = 0; /* q[0 .. head-1]; q[head-1] is the head of Q */
  for (int32_t v = n - 1; v >= 0; v--)
    if (indeg[v] == 0) q[head++] = v;
  int32_t out = 0;
  while (head > 0) {
    int32_t v = q[--head];
    dfs_order[out++] = v;
    /* the successors freed now, in decreasing id, so the lowest ends in front */
    int32_t first = head;
    for (int32_t e = g->out_ptr[v]; e < g->out_ptr[v + 1]; e++) {
      int32_t s = g->out_idx[e];
      if (--indeg[s] == 0) {
        int32_t k = head++;
        while (k > first && q[k - 1] < s) {
          q[k] = q[k - 1];
          k--;
        }
        q[k] = s;
      }
    }
  }
  free(indeg);
  free(q);
  return out == n ? ORC_OK : ORC_E_CYCLE;
}

/* ------------------------------------------------- CCR and Order-Place */

/* eq. 1: CCR = sum over edges of c_{i,j} / sum over nodes of w_i; fusion keeps
 * the total compute and drops the edges inside clusters (Section 5.1.1). */
int orc_comm_sums(const orc_graph *g, const orc_devices *d, const int32_t *cluster_id,
                  int64_t *edge_comm, int64_t *w_sum) {
  int rc = check_graph(g);
  if (rc) return rc;
  if ((rc = check_devices(d))) return rc;
  if ((rc = check_overflow(g, d))) return rc;
  if (!edge_comm || !w_sum) return ORC_E_ARG;
  int64_t ec = 0, ws = 0;
  for (int32_t u = 0; u < g->n; u++) {
    ws += g->w[u];
    int64_t cu = comm_of(g->ob[u], d->bw, d->lat);
    for (int32_t e = g->out_ptr[u]; e < g->out_ptr[u + 1]; e++)
      if (!cluster_id || cluster_id[u] != cluster_id[g->out_idx[e]]) ec += cu;
  }
  *edge_comm = ec;
  *w_sum = ws;
  return ORC_OK;
}

/* Order-Place, Section 6: the coarse nodes in order, one device until its
 * memory is used up, then the next. */
int orc_order_place(const orc_graph *g, const orc_devices *d, const int32_t *cluster_id,
                    int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
                    int32_t *best_effort_count) {
  int rc = check_graph(g);
  if (rc) return rc;
  if ((rc = check_devices(d))) return rc;
  int32_t n = g->n, C = n_clusters;
  if (C < 0 || !best_effort_count) return ORC_E_ARG;
  if ((n > 0 && (!cluster_id || !node_dev || C < 1)) || (C > 0 && !cluster_dev)) return ORC_E_ARG;
  for (int32_t v = 0; v < n; v++)
    if (cluster_id[v] < 0 || cluster_id[v] >= C) return ORC_E_ARG;
  int64_t *MEM = calloc((size_t)C + 1, sizeof(int64_t));
  for (int32_t v = 0; v < n; v++) MEM[cluster_id[v]] += g->mem[v];
  int32_t dev = 0, be = 0;
  int64_t used = 0;
  for (int32_t t = 0; t < C; t++) {
    while (used + MEM[t] > d->cap[dev] && dev + 1 < d->D) {  /* full: the next device */
      dev++;
      used = 0;
    }
    if (used + MEM[t] > d->cap[dev]) be++;  /* the last device, over its cap */
    cluster_dev[t] = (uint8_t)dev;
    used += MEM[t];
  }
  for (int32_t v = 0; v < n; v++) node_dev[v] = cluster_dev[cluster_id[v]];
  *best_effort_count = be;
  free(MEM);
  return ORC_OK;
}

/* ------------------------------------------------------------- clustering */

/* eq. 4 evaluated literally: the comm time of every edge that leaves the node
 * set {v_i .. v_{j-1}} towards a node at position >= j. */
static int64_t cost_direct(const orc_graph *g, const int32_t *pos, const int64_t *c,
                           int32_t i, int32_t j) {
  int64_t s = 0;
  for (int32_t u = 0; u < g->n; u++)
    for (int32_t e = g->out_ptr[u]; e < g->out_ptr[u + 1]; e++) {
      int32_t pu = pos[u], pv = pos[g->out_idx[e]];
      if (i <= pu && pu < j && j <= pv) s += c[u];
    }
  return s;
}

/* Section 5.1.3.  The given topological order v_1..v_n is cut at breakpoints;
 * the nodes between consecutive breakpoints form one cluster.  With S(0) = 0,
 *   S(j) = min over i of S(i) + cost(i, j)                       (eq. 6)
 * over i = j-1, j-2, ... subject to j - i <= R (exploration range) and the
 * cluster's memory sum <= M, where cost(i, j) (eq. 4) is the comm leaving
 * {v_i..v_{j-1}} for nodes at or after v_j.  cost is kept incrementally with
 * eq. 5: adding v_{j-1} adds all its out-edges and removes its in-edges from
 * nodes already inside the interval (the garbled lower summation limit is read
 * as i).  Readings: a single node is always a feasible cluster, even above M;
 * among equal S the smallest i wins (the longest cluster: merging never raises
 * the cut, and Table 2's cluster counts sit near n/R); P(j)
 * records the chosen i and breakpoints are recovered by following P from n
 * down to 0.  Greedy mode extends the current cluster while both limits hold.
 * Positions are 0-based here: cluster [i, j) holds order[i..j-1]. */
int orc_cluster(const orc_graph *g, const orc_devices *d, const int32_t *order,
                int32_t R, int64_t M, int32_t mode, int32_t *cluster_id,
                int32_t *n_clusters, int64_t *cut_cost) {
  int rc = check_graph(g);
  if (rc) return rc;
  if ((rc = check_devices(d))) return rc;
  if ((rc = check_overflow(g, d))) return rc;
  int32_t n = g->n;
  if (R < 1 || M < -1 || !n_clusters || !cut_cost || (n > 0 && !cluster_id)) return ORC_E_ARG;
  if (mode != ORC_DP && mode != ORC_GREEDY && mode != ORC_DP_DIRECT) return ORC_E_ARG;
  if (M == -1) {
    int64_t mc = d->cap[0];
    for (int32_t i = 1; i < d->D; i++)
      if (d->cap[i] < mc) mc = d->cap[i];
    M = mc / 4;
  }
  int32_t *pos = malloc(sizeof(int32_t) * (size_t)(n + 1));
  if ((rc = check_order(g, order, pos))) { free(pos); return rc; }
  int64_t *c = malloc(sizeof(int64_t) * (size_t)(n + 1));
  int64_t *PM = malloc(sizeof(int64_t) * (size_t)(n + 1)); /* memory prefix sums */
  int32_t *bp = malloc(sizeof(int32_t) * (size_t)(n + 1)); /* breakpoints */
  for (int32_t v = 0; v < n; v++) c[v] = comm_of(g->ob[v], d->bw, d->lat);
  PM[0] = 0;
  for (int32_t p = 0; p < n; p++) PM[p + 1] = PM[p] + g->mem[order[p]];
  int32_t nb = 0; /* breakpoints bp[0] = 0 < bp[1] < ... < bp[nb] = n */

  if (mode == ORC_GREEDY) {
    int32_t start = 0;
    bp[nb] = 0;
    while (start < n) {
      int32_t end = start + 1;
      while (end < n && end + 1 - start <= R && PM[end + 1] - PM[start] <= M) end++;
      bp[++nb] = end;
      start = end;
    }
    int64_t cut = 0;
    for (int32_t t = 0; t < nb; t++)
      for (int32_t p = bp[t]; p < bp[t + 1]; p++) cluster_id[order[p]] = t;
    for (int32_t u = 0; u < n; u++)
      for (int32_t e = g->out_ptr[u]; e < g->out_ptr[u + 1]; e++)
        if (cluster_id[u] != cluster_id[g->out_idx[e]]) cut += c[u];
    *n_clusters = nb;
    *cut_cost = cut;
  } else {
    int64_t *S = malloc(sizeof(int64_t) * (size_t)(n + 1));
    int32_t *P = malloc(sizeof(int32_t) * (size_t)(n + 1));
    int64_t *cost = malloc(sizeof(int64_t) * (size_t)(n + 1)); /* cost[i] = cost(i, j) */
    S[0] = 0;
    P[0] = 0;
    for (int32_t j = 1; j <= n; j++) {
      int32_t lo = j - R > 0 ? j - R : 0;
      int32_t v = order[j - 1];
      if (mode == ORC_DP) {
        /* eq. 5: cost(i,j) = cost(i,j-1) + out-comm of v_{j-1}
         *                    - comm of edges v_s -> v_{j-1} with i <= s < j-1 */
        int64_t oc = c[v] * (int64_t)(g->out_ptr[v + 1] - g->out_ptr[v]);
        cost[j - 1] = 0; /* cost(j-1, j-1): the empty interval */
        for (int32_t i = lo; i <= j - 1; i++) cost[i] += oc;
        for (int32_t e = g->in_ptr[v]; e < g->in_ptr[v + 1]; e++) {
          int32_t u = g->in_idx[e], s = pos[u];
          for (int32_t i = lo; i <= s && i < j - 1; i++) cost[i] -= c[u];
        }
      }
      int64_t best = INF;
      int32_t arg = -1;
      for (int32_t i = j - 1; i >= lo; i--) {
        if (j - i > 1 && PM[j] - PM[i] > M) break; /* memory only grows as i drops */
        int64_t cij = mode == ORC_DP ? cost[i] : cost_direct(g, pos, c, i, j);
        if (S[i] + cij <= best) { /* scanning i downwards: ties -> smallest i */
          best = S[i] + cij;
          arg = i;
        }
      }
      S[j] = best;
      P[j] = arg;
    }
    /* follow P from n back to 0 */
    int32_t cnt = 0;
    for (int32_t b = n; b > 0; b = P[b]) cnt++;
    nb = cnt;
    bp[0] = 0;
    for (int32_t b = n, t = cnt; b > 0; b = P[b]) bp[t--] = b;
    for (int32_t t = 0; t < nb; t++)
      for (int32_t p = bp[t]; p < bp[t + 1]; p++) cluster_id[order[p]] = t;
    *n_clusters = nb;
    *cut_cost = S[n];
    free(S); free(P); free(cost);
  }
  free(pos); free(c); free(PM); free(bp);
  return ORC_OK;
}

/* ---------------------------------------------------------------- placement */

typedef struct {
  int64_t key; /* (a << 32) | b */
  int64_t c;
} cedge;

static int cmp_cedge(const void *x, const void *y) {
  int64_t a = ((const cedge *)x)->key, b = ((const cedge *)y)->key;
  return (a > b) - (a < b);
}

/* Section 5.2.  Clusters become the nodes of a coarse DAG: a cluster's compute
 * time is the sum of its members' (Section 5.1.1), its memory the sum of their
 * memory, and the comm time of the coarse edge a -> b the sum of c[u] over the
 * fine edges u -> v with u in a and v in b (eq. 1's sum of edge comm times).
 * Algorithm 2 then visits the clusters in index order (a topological order,
 * since clusters are intervals of one):
 *   back_cost = max comm time to a successor (eq. 8; 0 for a sink);
 *   for every device d: pre_t = max over predecessors p of Fin[p] + I(d_p)c
 *     (eq. 7, I = 1 when p sits on another device), then the earliest start
 *     >= pre_t at which the cluster fits between the device's busy intervals
 *     (first fit), and EST(d) = that start, or infinity when the device's
 *     remaining memory is below the cluster's;
 *   d_k = device of the previous cluster (device 0 for the first);
 *   d_1 = device of smallest EST (lowest id on ties);
 *   move to d_1 when EST(d_k) - EST(d_1) > back_cost (eq. 9), else stay on d_k;
 *   if every EST is infinite, take the device with the most remaining memory
 *   ("lowest memory usage", lowest id on ties) -- best effort.
 * The chosen device's memory drops by the cluster's, the cluster occupies
 * [start, start + W) there, and Fin = start + W.  Nodes inherit their
 * cluster's device. */
int orc_place(const orc_graph *g, const orc_devices *d, const int32_t *cluster_id,
              int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
              int64_t *cluster_fin, int64_t *coarse_makespan, int32_t *best_effort_count) {
  int rc = check_graph(g);
  if (rc) return rc;
  if ((rc = check_devices(d))) return rc;
  if ((rc = check_overflow(g, d))) return rc;
  int32_t n = g->n, C = n_clusters, D = d->D;
  if (C < 0 || !coarse_makespan || !best_effort_count) return ORC_E_ARG;
  if ((n > 0 && (!cluster_id || !node_dev || C < 1)) || (C > 0 && !cluster_dev)) return ORC_E_ARG;
  for (int32_t v = 0; v < n; v++)
    if (cluster_id[v] < 0 || cluster_id[v] >= C) return ORC_E_ARG;
  /* coarse nodes */
  int64_t *W = calloc((size_t)C + 1, sizeof(int64_t));
  int64_t *MEM = calloc((size_t)C + 1, sizeof(int64_t));
  for (int32_t v = 0; v < n; v++) {
    W[cluster_id[v]] += g->w[v];
    MEM[cluster_id[v]] += g->mem[v];
  }
  /* coarse edges: one per distinct (a, b), comm summed */
  cedge *ce = malloc(sizeof(cedge) * (size_t)(g->m + 1));
  int32_t ne = 0;
  for (int32_t u = 0; u < n; u++) {
    int64_t cu = comm_of(g->ob[u], d->bw, d->lat);
    for (int32_t e = g->out_ptr[u]; e < g->out_ptr[u + 1]; e++) {
      int32_t a = cluster_id[u], b = cluster_id[g->out_idx[e]];
      if (a == b) continue;
      if (a > b) { free(W); free(MEM); free(ce); return ORC_E_ORDER; }
      ce[ne].key = ((int64_t)a << 32) | b;
      ce[ne].c = cu;
      ne++;
    }
  }
  qsort(ce, (size_t)ne, sizeof(cedge), cmp_cedge);
  int32_t k = 0;
  for (int32_t i = 0; i < ne; i++) {
    if (k > 0 && ce[k - 1].key == ce[i].key) ce[k - 1].c += ce[i].c;
    else ce[k++] = ce[i];
  }
  ne = k;
  /* successors' max comm (eq. 8) and predecessor lists (CSC of the coarse DAG) */
  int64_t *back = calloc((size_t)C + 1, sizeof(int64_t));
  int32_t *pp = calloc((size_t)C + 2, sizeof(int32_t));
  int32_t *pa = malloc(sizeof(int32_t) * (size_t)(ne + 1));
  int64_t *pc = malloc(sizeof(int64_t) * (size_t)(ne + 1));
  for (int32_t i = 0; i < ne; i++) {
    int32_t a = (int32_t)(ce[i].key >> 32), b = (int32_t)(ce[i].key & 0xffffffff);
    if (ce[i].c > back[a]) back[a] = ce[i].c;
    pp[b + 1]++;
  }
  for (int32_t t = 0; t < C; t++) pp[t + 1] += pp[t];
  int32_t *fill = malloc(sizeof(int32_t) * (size_t)(C + 1));
  memcpy(fill, pp, sizeof(int32_t) * (size_t)(C + 1));
  for (int32_t i = 0; i < ne; i++) {
    int32_t a = (int32_t)(ce[i].key >> 32), b = (int32_t)(ce[i].key & 0xffffffff);
    pa[fill[b]] = a;
    pc[fill[b]] = ce[i].c;
    fill[b]++;
  }
  free(fill);
  free(ce);
  /* device state */
  int64_t *Ava = malloc(sizeof(int64_t) * (size_t)D);
  int32_t *nbusy = calloc((size_t)D, sizeof(int32_t));
  int64_t **bs = malloc(sizeof(int64_t *) * (size_t)D), **bf = malloc(sizeof(int64_t *) * (size_t)D);
  for (int32_t i = 0; i < D; i++) {
    Ava[i] = d->cap[i];
    bs[i] = malloc(sizeof(int64_t) * (size_t)(C + 1));
    bf[i] = malloc(sizeof(int64_t) * (size_t)(C + 1));
  }
  int64_t *Fin = malloc(sizeof(int64_t) * (size_t)(C + 1));
  int64_t *EST = malloc(sizeof(int64_t) * (size_t)D), *slot = malloc(sizeof(int64_t) * (size_t)D);
  int32_t be = 0;
  int64_t span = 0;
  for (int32_t t = 0; t < C; t++) {
    for (int32_t x = 0; x < D; x++) {
      int64_t pre = 0;
      for (int32_t e = pp[t]; e < pp[t + 1]; e++) {
        int32_t a = pa[e];
        int64_t r = Fin[a] + (cluster_dev[a] != x ? pc[e] : 0);
        if (r > pre) pre = r;
      }
      int64_t s = pre;
      if (W[t] > 0) {
        for (int32_t q = 0; q < nbusy[x]; q++) {
          if (bf[x][q] <= s) continue;
          if (bs[x][q] < s + W[t]) s = bf[x][q];
          else break;
        }
      }
      slot[x] = s;
      EST[x] = Ava[x] < MEM[t] ? INF : s;
    }
    int32_t dk = t == 0 ? 0 : cluster_dev[t - 1];
    int32_t d1 = 0;
    for (int32_t x = 1; x < D; x++)
      if (EST[x] < EST[d1]) d1 = x;
    int32_t pick;
    if (EST[d1] == INF) {
      pick = 0;
      for (int32_t x = 1; x < D; x++)
        if (Ava[x] > Ava[pick]) pick = x;
      be++;
    } else if (EST[dk] == INF || EST[dk] - EST[d1] > back[t]) {
      pick = d1;
    } else {
      pick = dk;
    }
    cluster_dev[t] = (uint8_t)pick;
    Fin[t] = slot[pick] + W[t];
    if (Fin[t] > span) span = Fin[t];
    Ava[pick] -= MEM[t];
    if (W[t] > 0) { /* keep the busy list sorted by start */
      int32_t q = nbusy[pick];
      while (q > 0 && bs[pick][q - 1] > slot[pick]) {
        bs[pick][q] = bs[pick][q - 1];
        bf[pick][q] = bf[pick][q - 1];
        q--;
      }
      bs[pick][q] = slot[pick];
      bf[pick][q] = Fin[t];
      nbusy[pick]++;
    }
  }
  for (int32_t v = 0; v < n; v++) node_dev[v] = cluster_dev[cluster_id[v]];
  if (cluster_fin)
    for (int32_t t = 0; t < C; t++) cluster_fin[t] = Fin[t];
  *coarse_makespan = span;
  *best_effort_count = be;
  for (int32_t i = 0; i < D; i++) { free(bs[i]); free(bf[i]); }
  free(bs); free(bf); free(nbusy); free(Ava); free(Fin); free(EST); free(slot);
  free(W); free(MEM); free(back); free(pp); free(pa); free(pc);
  return ORC_OK;
}

/* ----------------------------------------------------------------- makespan */

/* Schedule of a placement: nodes are started in the given topological order;
 * each device runs its nodes one at a time in that order; a node is ready once
 * every predecessor has finished and, if it sits on another device, its output
 * has arrived (eq. 7's pre_t with the indicator I); it starts at the later of
 * ready and its device's previous finish (eq. 7's EST without insertion), and
 * runs for w.  The makespan is the latest finish (0 for an empty graph). */
int orc_makespan(const orc_graph *g, const orc_devices *d, const int32_t *order,
                 int32_t K, const uint8_t *node_dev, int64_t *start, int64_t *finish,
                 int64_t *makespan) {
  int rc = check_graph(g);
  if (rc) return rc;
  if ((rc = check_devices(d))) return rc;
  if ((rc = check_overflow(g, d))) return rc;
  int32_t n = g->n;
  if (K < 1 || !makespan || (n > 0 && !node_dev)) return ORC_E_ARG;
  for (int64_t i = 0; i < (int64_t)K * n; i++)
    if (node_dev[i] >= d->D) return ORC_E_ARG;
  int32_t *pos = malloc(sizeof(int32_t) * (size_t)(n + 1));
  rc = check_order(g, order, pos);
  free(pos);
  if (rc) return rc;
  int64_t *c = malloc(sizeof(int64_t) * (size_t)(n + 1));
  for (int32_t v = 0; v < n; v++) c[v] = comm_of(g->ob[v], d->bw, d->lat);
  int64_t *fin = malloc(sizeof(int64_t) * (size_t)(n + 1));
  int64_t *avail = malloc(sizeof(int64_t) * (size_t)d->D);
  for (int32_t k = 0; k < K; k++) {
    const uint8_t *dev = node_dev + (int64_t)k * n;
    for (int32_t x = 0; x < d->D; x++) avail[x] = 0;
    int64_t span = 0;
    for (int32_t p = 0; p < n; p++) {
      int32_t v = order[p];
      int64_t ready = 0;
      for (int32_t e = g->in_ptr[v]; e < g->in_ptr[v + 1]; e++) {
        int32_t u = g->in_idx[e];
        int64_t r = fin[u] + (dev[u] != dev[v] ? c[u] : 0);
        if (r > ready) ready = r;
      }
      int64_t s = ready > avail[dev[v]] ? ready : avail[dev[v]];
      fin[v] = s + g->w[v];
      avail[dev[v]] = fin[v];
      if (fin[v] > span) span = fin[v];
      if (start) start[(int64_t)k * n + v] = s;
    }
    if (finish) memcpy(finish + (int64_t)k * n, fin, sizeof(int64_t) * (size_t)n);
    makespan[k] = span;
  }
  free(c); free(fin); free(avail);
  return ORC_OK;
}

/* Makespan under the richer device models (node_dev is [K][n], model a set of
 * ORC_MODEL_* bits; model 0 is orc_makespan's schedule).
 *
 * ORC_MODEL_INSERT: the device slot rule of eq. 7 applied to single nodes.  A
 *   node starts at the earliest time >= ready at which it fits between the
 *   tasks already placed on its device (first fit over that device's busy
 *   intervals), instead of after the device's last task.  A node with w = 0
 *   starts at ready and occupies nothing.
 * ORC_MODEL_COMM_TASKS: a transfer is a task of its own (the runtime model of
 *   Section 6.1).  After node u finishes on device a, one transfer of its
 *   output goes to each other device b that holds a successor of u, in
 *   increasing b; it takes c[u] and occupies a's send channel and b's receive
 *   channel together, each channel serving its transfers one at a time in the
 *   order they are issued: start = max(fin[u], send free[a], receive free[b]).
 *   A successor on b is ready for u's output when that transfer ends; outputs
 *   consumed on their own device need no transfer.  Compute never waits for a
 *   channel other than through its inputs.
 * ORC_MODEL_COMM_BLOCK (alone; FIFO devices): the same transfers, one per
 *   (producer, other device holding a successor) in increasing device order,
 *   are operations on the devices themselves (Section 6.1 places a transfer
 *   node on every device that sends or receives).  Each enters the compute
 *   queue of both its sending and its receiving device right after its
 *   producer, starts when both devices are free and holds both for c[u]:
 *   start = max(free[a], free[b]), then free[a] = free[b] = start + c[u].
 *   A successor on b is ready for u's output when that transfer ends. */
/* Heterogeneous devices: node v takes ceil(w[v] * tmul[x] / 1024) on device x,
 * and its output takes ceil(ob[v] / bw[a][b]) + lat[a][b] from device a to b.
 * h == NULL, or a NULL member, means the homogeneous value (1024, d->bw,
 * d->lat). */
static int64_t dur_on(const orc_hetero *h, int64_t w, int32_t x) {
  if (!h || !h->tmul) return w;
  __int128 t = (__int128)w * h->tmul[x];
  return (int64_t)((t + 1023) / 1024);
}

static int64_t link_comm(const orc_hetero *h, const orc_devices *d, int64_t ob, int32_t a,
                         int32_t b) {
  int64_t bw = h && h->bw ? h->bw[a * d->D + b] : d->bw;
  int64_t lat = h && h->lat ? h->lat[a * d->D + b] : d->lat;
  return comm_of(ob, bw, lat);
}

/* The overflow bound with the slowest device and the worst link. */
static int check_hetero(const orc_graph *g, const orc_devices *d, const orc_hetero *h) {
  if (!h) return check_overflow(g, d);
  int32_t D = d->D;
  int64_t tmax = 1024, bwmin = d->bw, latmax = d->lat;
  if (h->tmul) {
    tmax = 0;
    for (int32_t x = 0; x < D; x++) {
      if (h->tmul[x] < 1 || h->tmul[x] > 65536) return ORC_E_ARG;
      if (h->tmul[x] > tmax) tmax = h->tmul[x];
    }
  }
  if (h->bw) {
    bwmin = INT64_MAX;
    for (int32_t i = 0; i < D * D; i++) {
      if (i / D == i % D) continue;
      if (h->bw[i] < 1) return ORC_E_ARG;
      if (h->bw[i] < bwmin) bwmin = h->bw[i];
    }
    if (D == 1) bwmin = 1;
  }
  if (h->lat) {
    latmax = 0;
    for (int32_t i = 0; i < D * D; i++) {
      if (i / D == i % D) continue;
      if (h->lat[i] < 0 || h->lat[i] >= ((int64_t)1 << 62)) return ORC_E_ARG;
      if (h->lat[i] > latmax) latmax = h->lat[i];
    }
  }
  orc_devices worst = *d;
  worst.bw = bwmin;
  worst.lat = latmax;
  int rc = check_overflow(g, &worst);
  if (rc) return rc;
  /* every duration at most ceil(tmax / 1024) times w */
  __int128 tot = 0, f = (tmax + 1023) / 1024;
  for (int32_t v = 0; v < g->n; v++) {
    tot += (__int128)g->w[v] * f;
    int64_t c = comm_of(g->ob[v], bwmin, latmax);
    tot += (__int128)c * (g->out_ptr[v + 1] - g->out_ptr[v]);
  }
  return tot >= ((__int128)1 << 62) ? ORC_E_OVERFLOW : ORC_OK;
}

int orc_makespan_model(const orc_graph *g, const orc_devices *d, const orc_hetero *h,
                       const int32_t *order, int32_t K, const uint8_t *node_dev, int32_t model,
                       int64_t *start, int64_t *finish, int64_t *makespan) {
  int rc = check_graph(g);
  if (rc) return rc;
  if ((rc = check_devices(d))) return rc;
  if ((rc = check_hetero(g, d, h))) return rc;
  int32_t n = g->n, D = d->D;
  /* COMM_BLOCK replaces both other bits: transfers on the compute queues */
  if (K < 1 || !makespan || (n > 0 && !node_dev) || (model & ~7) || ((model & 4) && (model & 3)))
    return ORC_E_ARG;
  for (int64_t i = 0; i < (int64_t)K * n; i++)
    if (node_dev[i] >= D) return ORC_E_ARG;
  int32_t *pos = malloc(sizeof(int32_t) * (size_t)(n + 1));
  rc = check_order(g, order, pos);
  free(pos);
  if (rc) return rc;
  const int insert = model & ORC_MODEL_INSERT, tasks = model & ORC_MODEL_COMM_TASKS;
  const int block = model & ORC_MODEL_COMM_BLOCK;
  int64_t *c = malloc(sizeof(int64_t) * (size_t)(n + 1));
  for (int32_t v = 0; v < n; v++) c[v] = comm_of(g->ob[v], d->bw, d->lat);
  int64_t *fin = malloc(sizeof(int64_t) * (size_t)(n + 1));
  int64_t *avail = malloc(sizeof(int64_t) * (size_t)D);
  int64_t *snd = malloc(sizeof(int64_t) * (size_t)D), *rcv = malloc(sizeof(int64_t) * (size_t)D);
  /* arrival of u's output on device b (transfers only) */
  int64_t *arr = tasks || block ? malloc(sizeof(int64_t) * ((size_t)n * D + 1)) : NULL;
  char *wants = malloc((size_t)D);
  /* busy intervals per device, sorted by start (insertion only) */
  int64_t *bs = insert ? malloc(sizeof(int64_t) * ((size_t)n + 1)) : NULL;
  int64_t *bf = insert ? malloc(sizeof(int64_t) * ((size_t)n + 1)) : NULL;
  int32_t *boff = malloc(sizeof(int32_t) * (size_t)(D + 1)), *nb = malloc(sizeof(int32_t) * (size_t)D);
  for (int32_t k = 0; k < K; k++) {
    const uint8_t *dev = node_dev + (int64_t)k * n;
    for (int32_t x = 0; x < D; x++) avail[x] = snd[x] = rcv[x] = 0, nb[x] = 0;
    /* device x's busy list lives in bs/bf[boff[x] .. boff[x] + its node count) */
    for (int32_t x = 0; x <= D; x++) boff[x] = 0;
    for (int32_t v = 0; v < n; v++) boff[dev[v] + 1]++;
    for (int32_t x = 0; x < D; x++) boff[x + 1] += boff[x];
    int64_t span = 0;
    for (int32_t p = 0; p < n; p++) {
      int32_t v = order[p], dv = dev[v];
      int64_t ready = 0;
      for (int32_t e = g->in_ptr[v]; e < g->in_ptr[v + 1]; e++) {
        int32_t u = g->in_idx[e];
        int64_t r;
        if (dev[u] == dv) r = fin[u];
        else if (tasks || block) r = arr[(int64_t)u * D + dv];
        else r = fin[u] + (h ? link_comm(h, d, g->ob[u], dev[u], dv) : c[u]);
        if (r > ready) ready = r;
      }
      int64_t s, w = dur_on(h, g->w[v], dv);
      if (!insert) {
        s = ready > avail[dv] ? ready : avail[dv];
        avail[dv] = s + w;
      } else {
        int64_t *xs = bs + boff[dv], *xf = bf + boff[dv];
        int32_t cnt = nb[dv];
        s = ready;
        if (w > 0) {
          /* intervals ending at or before ready cannot overlap [s, s + w):
           * skip them by bisection (the intervals are disjoint, so their ends
           * are sorted too), then take the first gap that holds w */
          int32_t lo = 0, hi = cnt;
          while (lo < hi) {
            int32_t mid = lo + (hi - lo) / 2;
            if (xf[mid] <= s) lo = mid + 1; else hi = mid;
          }
          int32_t q = lo;
          for (; q < cnt; q++) {
            if (xs[q] < s + w) s = xf[q];
            else break;
          }
          for (int32_t i = cnt; i > q; i--) xs[i] = xs[i - 1], xf[i] = xf[i - 1];
          xs[q] = s;
          xf[q] = s + w;
          nb[dv] = cnt + 1;
        }
      }
      fin[v] = s + w;
      if (fin[v] > span) span = fin[v];
      if (start) start[(int64_t)k * n + v] = s;
      if (tasks) {
        for (int32_t x = 0; x < D; x++) wants[x] = 0;
        for (int32_t e = g->out_ptr[v]; e < g->out_ptr[v + 1]; e++) wants[dev[g->out_idx[e]]] = 1;
        for (int32_t b = 0; b < D; b++) {
          if (b == dv || !wants[b]) continue;
          int64_t t0 = fin[v];
          if (snd[dv] > t0) t0 = snd[dv];
          if (rcv[b] > t0) t0 = rcv[b];
          int64_t cv = h ? link_comm(h, d, g->ob[v], dv, b) : c[v];
          arr[(int64_t)v * D + b] = t0 + cv;
          snd[dv] = rcv[b] = t0 + cv;
        }
      }
      if (block) {
        /* each transfer is a task on both devices' compute queues, entered
         * right after its producer: it starts when both devices are free
         * (the sender's queue already ends at or after fin[v]) and holds
         * both until it ends */
        for (int32_t x = 0; x < D; x++) wants[x] = 0;
        for (int32_t e = g->out_ptr[v]; e < g->out_ptr[v + 1]; e++) wants[dev[g->out_idx[e]]] = 1;
        for (int32_t b = 0; b < D; b++) {
          if (b == dv || !wants[b]) continue;
          int64_t t0 = avail[dv] > avail[b] ? avail[dv] : avail[b];
          int64_t cv = h ? link_comm(h, d, g->ob[v], dv, b) : c[v];
          arr[(int64_t)v * D + b] = t0 + cv;
          avail[dv] = avail[b] = t0 + cv;
        }
      }
    }
    if (finish) memcpy(finish + (int64_t)k * n, fin, sizeof(int64_t) * (size_t)n);
    makespan[k] = span;
  }
  free(c); free(fin); free(avail); free(snd); free(rcv); free(arr); free(wants);
  free(bs); free(bf); free(boff); free(nb);
  return ORC_OK;
}

typedef struct {
  int64_t key; /* (a << 32) | b */
  int64_t c, ob, cnt;
} xedge;

static int cmp_xedge(const void *x, const void *y) {
  int64_t a = ((const xedge *)x)->key, b = ((const xedge *)y)->key;
  return (a > b) - (a < b);
}

/* Adjusting Placement with heterogeneous devices and links and with
 * co-location groups inside the algorithm (Section 5.2's Algorithm 2 with the
 * generality of Sections 4.1 and 6.1).  The steps are orc_place's, with:
 *  - Device speeds: cluster t takes W_x[t] = sum over its members v of
 *    ceil(w[v] * tmul[x] / 1024) on device x (each member at device x's
 *    speed, as in orc_makespan_model), both for its first-fit slot and for
 *    its finish time.  Devices are compared, and the move test of eq. 9 is
 *    made, on the earliest finish time, slot + W_x[t]: with identical
 *    devices W_x[t] is the same on every device, so the ordering and the
 *    differences are those of eq. 7's start times.
 *  - Links: with per-link tables, the coarse edge a -> b is charged, on the
 *    link from device y to device x, ceil(OB / bw[y][x]) + N * lat[y][x],
 *    where OB is the sum of ob[u] over its N member edges u -> v: the
 *    members' tensors cross the link together, each edge paying the link's
 *    latency.  pre_t on device x (eq. 7) uses the link from each
 *    predecessor's device to x.  back_cost (eq. 8) is the largest charge of
 *    t's outgoing coarse edges on the link from the best device d_1 back to
 *    the previous cluster's device d_k, the link t's outputs would take if t
 *    moved away from d_k.  Without link tables every coarse edge costs the sum
 *    of c[u] exactly as in orc_place.
 *  - Co-location: a group's leading cluster is the smallest cluster id among
 *    its members (the first of them Algorithm 2 places); every member runs on
 *    that cluster's device.  A member outside the leading cluster (a
 *    follower) is charged to that device's memory when its own cluster is
 *    placed, before the devices are compared; the cluster's memory test and
 *    its own device's charge count only its other members (MEM_own).  The
 *    coarse schedule keeps every member's compute in its cluster.
 * h == NULL and group == NULL give orc_place's result. */
int orc_place_ext(const orc_graph *g, const orc_devices *d, const orc_hetero *h,
                  const int32_t *group, int32_t n_groups, const int32_t *cluster_id,
                  int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
                  int64_t *cluster_fin, int64_t *coarse_makespan, int32_t *best_effort_count) {
  int rc = check_graph(g);
  if (rc) return rc;
  if ((rc = check_devices(d))) return rc;
  if ((rc = check_hetero(g, d, h))) return rc;
  int32_t n = g->n, C = n_clusters, D = d->D;
  if (C < 0 || !coarse_makespan || !best_effort_count || n_groups < 0) return ORC_E_ARG;
  if ((n > 0 && (!cluster_id || !node_dev || C < 1)) || (C > 0 && !cluster_dev)) return ORC_E_ARG;
  if (n_groups > 0 && !group) return ORC_E_ARG;
  for (int32_t v = 0; v < n; v++) {
    if (cluster_id[v] < 0 || cluster_id[v] >= C) return ORC_E_ARG;
    if (group && (group[v] < -1 || group[v] >= n_groups)) return ORC_E_ARG;
  }
  const int links = h && (h->bw || h->lat);
  /* leading cluster of each group */
  int32_t *lead = malloc(sizeof(int32_t) * ((size_t)n_groups + 1));
  for (int32_t x = 0; x < n_groups; x++) lead[x] = INT32_MAX;
  for (int32_t v = 0; v < n; v++)
    if (group && group[v] >= 0 && cluster_id[v] < lead[group[v]]) lead[group[v]] = cluster_id[v];
  /* coarse nodes: duration per device, own memory; followers by cluster */
  int64_t *Wx = calloc((size_t)C * D + 1, sizeof(int64_t));
  int64_t *MEM = calloc((size_t)C + 1, sizeof(int64_t));
  int32_t *fp = calloc((size_t)C + 2, sizeof(int32_t)), *fv = malloc(sizeof(int32_t) * ((size_t)n + 1));
  for (int32_t v = 0; v < n; v++) {
    int32_t t = cluster_id[v];
    for (int32_t x = 0; x < D; x++) Wx[(int64_t)t * D + x] += dur_on(h, g->w[v], x);
    int follower = group && group[v] >= 0 && lead[group[v]] < t;
    if (follower) fp[t + 1]++;
    else MEM[t] += g->mem[v];
  }
  for (int32_t t = 0; t < C; t++) fp[t + 1] += fp[t];
  {
    int32_t *fill = malloc(sizeof(int32_t) * ((size_t)C + 1));
    memcpy(fill, fp, sizeof(int32_t) * (size_t)(C + 1));
    for (int32_t v = 0; v < n; v++)
      if (group && group[v] >= 0 && lead[group[v]] < cluster_id[v]) fv[fill[cluster_id[v]]++] = v;
    free(fill);
  }
  /* coarse edges, one per distinct (a, b): sum of c[u], sum of ob[u], count */
  xedge *xe = malloc(sizeof(xedge) * ((size_t)g->m + 1));
  int32_t ne = 0;
  for (int32_t u = 0; u < n; u++) {
    int64_t cu = comm_of(g->ob[u], d->bw, d->lat);
    for (int32_t e = g->out_ptr[u]; e < g->out_ptr[u + 1]; e++) {
      int32_t a = cluster_id[u], b = cluster_id[g->out_idx[e]];
      if (a == b) continue;
      if (a > b) {
        free(lead); free(Wx); free(MEM); free(fp); free(fv); free(xe);
        return ORC_E_ORDER;
      }
      xe[ne].key = ((int64_t)a << 32) | b;
      xe[ne].c = cu;
      xe[ne].ob = g->ob[u];
      xe[ne].cnt = 1;
      ne++;
    }
  }
  qsort(xe, (size_t)ne, sizeof(xedge), cmp_xedge);
  int32_t k = 0;
  for (int32_t i = 0; i < ne; i++) {
    if (k > 0 && xe[k - 1].key == xe[i].key) {
      xe[k - 1].c += xe[i].c;
      xe[k - 1].ob += xe[i].ob;
      xe[k - 1].cnt += xe[i].cnt;
    } else {
      xe[k++] = xe[i];
    }
  }
  ne = k;
  /* predecessor lists (by target) and successor lists (by source) */
  int32_t *pp = calloc((size_t)C + 2, sizeof(int32_t)), *sp = calloc((size_t)C + 2, sizeof(int32_t));
  int32_t *pe = malloc(sizeof(int32_t) * ((size_t)ne + 1)), *se = malloc(sizeof(int32_t) * ((size_t)ne + 1));
  for (int32_t i = 0; i < ne; i++) {
    pp[(xe[i].key & 0xffffffff) + 1]++;
    sp[(xe[i].key >> 32) + 1]++;
  }
  for (int32_t t = 0; t < C; t++) pp[t + 1] += pp[t], sp[t + 1] += sp[t];
  {
    int32_t *fa = malloc(sizeof(int32_t) * ((size_t)C + 1)), *fb = malloc(sizeof(int32_t) * ((size_t)C + 1));
    memcpy(fa, pp, sizeof(int32_t) * (size_t)(C + 1));
    memcpy(fb, sp, sizeof(int32_t) * (size_t)(C + 1));
    for (int32_t i = 0; i < ne; i++) {
      pe[fa[xe[i].key & 0xffffffff]++] = i;
      se[fb[xe[i].key >> 32]++] = i;
    }
    free(fa); free(fb);
  }
  /* device state */
  int64_t *Ava = malloc(sizeof(int64_t) * (size_t)D);
  int32_t *nbusy = calloc((size_t)D, sizeof(int32_t));
  int64_t **bs = malloc(sizeof(int64_t *) * (size_t)D), **bf = malloc(sizeof(int64_t *) * (size_t)D);
  for (int32_t i = 0; i < D; i++) {
    Ava[i] = d->cap[i];
    bs[i] = malloc(sizeof(int64_t) * (size_t)(C + 1));
    bf[i] = malloc(sizeof(int64_t) * (size_t)(C + 1));
  }
  int64_t *Fin = malloc(sizeof(int64_t) * (size_t)(C + 1));
  int64_t *EST = malloc(sizeof(int64_t) * (size_t)D), *slot = malloc(sizeof(int64_t) * (size_t)D);
  int32_t be = 0;
  int64_t span = 0;
  for (int32_t t = 0; t < C; t++) {
    /* followers take memory on their leading cluster's device */
    for (int32_t i = fp[t]; i < fp[t + 1]; i++) {
      int32_t v = fv[i];
      Ava[cluster_dev[lead[group[v]]]] -= g->mem[v];
    }
    for (int32_t x = 0; x < D; x++) {
      int64_t pre = 0;
      for (int32_t q = pp[t]; q < pp[t + 1]; q++) {
        const xedge *ed = &xe[pe[q]];
        int32_t a = (int32_t)(ed->key >> 32), y = cluster_dev[a];
        int64_t cost = 0;
        if (y != x) {
          if (links) {
            int64_t bw = h->bw ? h->bw[y * D + x] : d->bw, lat = h->lat ? h->lat[y * D + x] : d->lat;
            cost = (ed->ob + bw - 1) / bw + ed->cnt * lat;
          } else {
            cost = ed->c;
          }
        }
        if (Fin[a] + cost > pre) pre = Fin[a] + cost;
      }
      int64_t s = pre, wx = Wx[(int64_t)t * D + x];
      if (wx > 0) {
        for (int32_t q = 0; q < nbusy[x]; q++) {
          if (bf[x][q] <= s) continue;
          if (bs[x][q] < s + wx) s = bf[x][q];
          else break;
        }
      }
      slot[x] = s;
      EST[x] = Ava[x] < MEM[t] ? INF : s + wx; /* the earliest finish time */
    }
    int32_t dk = t == 0 ? 0 : cluster_dev[t - 1];
    int32_t d1 = 0;
    for (int32_t x = 1; x < D; x++)
      if (EST[x] < EST[d1]) d1 = x;
    int32_t pick;
    if (EST[d1] == INF) {
      pick = 0;
      for (int32_t x = 1; x < D; x++)
        if (Ava[x] > Ava[pick]) pick = x;
      be++;
    } else if (EST[dk] == INF) {
      pick = d1;
    } else {
      /* back_cost (eq. 8): largest charge of t's outgoing coarse edges, on the
       * link d_1 -> d_k under link tables */
      int64_t back = 0;
      for (int32_t q = sp[t]; q < sp[t + 1]; q++) {
        const xedge *ed = &xe[se[q]];
        int64_t cost = ed->c;
        if (links && d1 != dk) {
          int64_t bw = h->bw ? h->bw[d1 * D + dk] : d->bw, lat = h->lat ? h->lat[d1 * D + dk] : d->lat;
          cost = (ed->ob + bw - 1) / bw + ed->cnt * lat;
        }
        if (cost > back) back = cost;
      }
      pick = EST[dk] - EST[d1] > back ? d1 : dk;
    }
    cluster_dev[t] = (uint8_t)pick;
    int64_t wp = Wx[(int64_t)t * D + pick];
    Fin[t] = slot[pick] + wp;
    if (Fin[t] > span) span = Fin[t];
    Ava[pick] -= MEM[t];
    if (wp > 0) {
      int32_t q = nbusy[pick];
      while (q > 0 && bs[pick][q - 1] > slot[pick]) {
        bs[pick][q] = bs[pick][q - 1];
        bf[pick][q] = bf[pick][q - 1];
        q--;
      }
      bs[pick][q] = slot[pick];
      bf[pick][q] = Fin[t];
      nbusy[pick]++;
    }
  }
  for (int32_t v = 0; v < n; v++)
    node_dev[v] = group && group[v] >= 0 ? cluster_dev[lead[group[v]]] : cluster_dev[cluster_id[v]];
  if (cluster_fin)
    for (int32_t t = 0; t < C; t++) cluster_fin[t] = Fin[t];
  *coarse_makespan = span;
  *best_effort_count = be;
  for (int32_t i = 0; i < D; i++) { free(bs[i]); free(bf[i]); }
  free(bs); free(bf); free(nbusy); free(Ava); free(Fin); free(EST); free(slot);
  free(lead); free(Wx); free(MEM); free(fp); free(fv); free(xe); free(pp); free(sp); free(pe); free(se);
  return ORC_OK;
}

/* Co-location groups (Section 6.1, as in Baechi): every node of a group runs
 * on the device of the group's first node in `order`; nodes with group -1
 * keep theirs.  node_dev is [K][n], rewritten in place. */
int orc_colocate(const orc_graph *g, const int32_t *order, const int32_t *group,
                 int32_t n_groups, int32_t K, uint8_t *node_dev) {
  int rc = check_graph(g);
  if (rc) return rc;
  int32_t n = g->n;
  if (K < 1 || n_groups < 0 || (n > 0 && (!order || !group || !node_dev))) return ORC_E_ARG;
  int32_t *pos = malloc(sizeof(int32_t) * (size_t)(n + 1));
  rc = check_order(g, order, pos);
  free(pos);
  if (rc) return rc;
  for (int32_t v = 0; v < n; v++)
    if (group[v] < -1 || group[v] >= n_groups) return ORC_E_ARG;
  int32_t *lead = malloc(sizeof(int32_t) * ((size_t)n_groups + 1));
  for (int32_t x = 0; x < n_groups; x++) lead[x] = -1;
  for (int32_t p = 0; p < n; p++) {  /* the first member in the order leads */
    int32_t v = order[p];
    if (group[v] >= 0 && lead[group[v]] < 0) lead[group[v]] = v;
  }
  for (int32_t k = 0; k < K; k++) {
    uint8_t *dev = node_dev + (int64_t)k * n;
    for (int32_t v = 0; v < n; v++)
      if (group[v] >= 0) dev[v] = dev[lead[group[v]]];
  }
  free(lead);
  return ORC_OK;
}
