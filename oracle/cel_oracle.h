/*
 * CPU oracle for the Celeritas placement hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded C implementation of what the GPU library
 * computes, written from the paper's definitions (Xu et al., "Celeritas: Fast
 * Optimizer for Large Dataflow Graphs", arXiv 2208.00184).  Only the tests, the
 * package's smoke check and the benchmark's CPU-baseline leg may call it.  It
 * shares no header, source, table or helper with the GPU library.
 *
 * Conventions: every pointer is host memory owned by the caller; all times are
 * int64 nanoseconds and all sizes int64 bytes; a node's communication cost is
 * c[v] = ceil(ob[v] / bw) + lat (the linear fit t = k d + b of Section 4.2.1 in
 * integer form), paid once per consumer edge.
 */
#ifndef CEL_ORACLE_H
#define CEL_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ORC_OK = 0,
  ORC_E_ARG = -1,      /* bad sizes, ranges or pointers */
  ORC_E_CYCLE = -2,    /* graph is not a DAG */
  ORC_E_OVERFLOW = -3, /* sum w + sum over edges c[src] >= 2^62 */
  ORC_E_ORDER = -6     /* order not a topological permutation / clusters not ordered */
};

enum { ORC_COMM_OFF = 1 };                 /* orc_blevel: comm costs treated as 0 */
enum { ORC_DP = 0, ORC_GREEDY = 1, ORC_DP_DIRECT = 2 }; /* orc_cluster modes */

typedef struct {
  int32_t n, m;
  const int32_t *out_ptr, *out_idx; /* successors, CSR  [n+1], [m] */
  const int32_t *in_ptr, *in_idx;   /* predecessors, CSC [n+1], [m] */
  const int64_t *w;                 /* compute time (ns), >= 0 */
  const int64_t *mem;               /* memory (bytes), >= 0 */
  const int64_t *ob;                /* output tensor bytes, >= 0 */
} orc_graph;

typedef struct {
  int32_t D;          /* 1..255 modelled devices */
  const int64_t *cap; /* [D] memory caps (bytes) */
  int64_t bw;         /* link bytes per ns, > 0 */
  int64_t lat;        /* link latency ns, >= 0 */
} orc_devices;

/* Kahn levels (Section 4.2.2): level[v] = 0 for sources, else 1 + max level of
 * predecessors.  order_id = ids sorted by (level, id); level_ptr[0..L] bucket
 * offsets (capacity n+1); *n_levels = L. */
int orc_topo_levels(const orc_graph *g, int32_t *level, int32_t *order_id,
                    int32_t *level_ptr, int32_t *n_levels);

/* b-level (eq. 3), t-level (eq. 2), critical path = max b-level, and the
 * priority order sorted by (level asc, b-level desc, id asc).  tlevel and
 * prio_order may be NULL. */
int orc_blevel(const orc_graph *g, const orc_devices *d, const int32_t *level,
               const int32_t *order_id, int32_t flags, int64_t *blevel,
               int64_t *tlevel, int32_t *prio_order, int64_t *cp);

/* CPD-TOPO order (Section 5.1.3, Algorithm 1): with cpath(v) = tlevel(v) +
 * blevel(v) (eq. 2-3, as given), a stack starts with the sources, the largest
 * cpath on top; repeatedly the top node is popped and output, its out-edges
 * are removed, and the successors left with no in-edge are pushed in
 * increasing cpath order, so the most critical one is popped next.  Equal
 * cpath: the lower id is output first.  cpd_order[k] = k-th node output. */
int orc_cpd_topo(const orc_graph *g, const int64_t *blevel, const int64_t *tlevel,
                 int32_t *cpd_order);

/* DFS-TOPO order (Section 4.2.2): a queue starts with the sources, lowest id
 * at the head; the head node is removed and output, its out-edges removed,
 * and the successors left with no in-edge are put at the head of the queue,
 * the lowest id in front, so a freed child is output before anything older.
 * dfs_order[k] = k-th node output. */
int orc_dfs_topo(const orc_graph *g, int32_t *dfs_order);

/* Contiguous clustering of a topological order (Section 5.1.3, eq. 4-6):
 * DP over breakpoints minimising inter-cluster comm with cluster length <= R
 * and cluster memory <= M (a single node may exceed M).  M = -1 selects
 * floor(min cap / 4). */
int orc_cluster(const orc_graph *g, const orc_devices *d, const int32_t *order,
                int32_t R, int64_t M, int32_t mode, int32_t *cluster_id,
                int32_t *n_clusters, int64_t *cut_cost);

/* Coarse graph + Adjusting Placement (Section 5.2, eq. 7-9, Algorithm 2).
 * cluster_fin ([C] finish time of each cluster) may be NULL. */
int orc_place(const orc_graph *g, const orc_devices *d, const int32_t *cluster_id,
              int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
              int64_t *cluster_fin, int64_t *coarse_makespan, int32_t *best_effort_count);

/* CCR (eq. 1) parts: *edge_comm = sum over edges u->v of c[u] (with a
 * cluster_id, only edges between different clusters: the coarse graph's
 * edges), *w_sum = sum of w (unchanged by fusion).  cluster_id may be NULL. */
int orc_comm_sums(const orc_graph *g, const orc_devices *d, const int32_t *cluster_id,
                  int64_t *edge_comm, int64_t *w_sum);

/* Order-Place (the baseline of Section 6, built on the coarse graph of
 * Section 5.2): clusters in index order fill device 0 and move on to the next
 * device when the next cluster does not fit the current one's remaining
 * memory; the last device takes whatever is left (best effort, counted). */
int orc_order_place(const orc_graph *g, const orc_devices *d, const int32_t *cluster_id,
                    int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
                    int32_t *best_effort_count);

/* Makespan of K placements (node_dev is [K][n]): nodes taken in `order`, each
 * device runs its nodes first-in first-out, comm (eq. 7's indicator) paid only
 * across devices.  start/finish ([K][n], by node id) may be NULL. */
int orc_makespan(const orc_graph *g, const orc_devices *d, const int32_t *order,
                 int32_t K, const uint8_t *node_dev, int64_t *start, int64_t *finish,
                 int64_t *makespan);

/* Makespan under richer device models: model is a set of ORC_MODEL_* bits
 * (0 gives orc_makespan's schedule).  INSERT: first-fit insertion of each
 * node into its device's busy intervals (eq. 7's slot rule at node level).
 * COMM_TASKS: transfers are tasks on per-device send and receive channels,
 * one per (producer, other device holding a successor), issued in increasing
 * device order (Section 6.1's runtime model).  COMM_BLOCK (alone, with FIFO
 * devices): each such transfer is instead a task on the compute queues of
 * both the sending and the receiving device (Section 6.1's transfer
 * operations on the devices that send or receive), entered into both queues
 * right after its producer and starting when both are free.  `order` is any
 * topological order; start/finish ([K][n], by node id) may be NULL. */
enum { ORC_MODEL_INSERT = 1, ORC_MODEL_COMM_TASKS = 2, ORC_MODEL_COMM_BLOCK = 4 };
/* Heterogeneous devices (NULL members: homogeneous): tmul[D] scales compute
 * time by tmul / 1024 (rounded up, 1 <= tmul <= 65536); bw[D*D], lat[D*D]
 * give the link from device a to b at [a * D + b] (diagonal unused). */
typedef struct {
  const int64_t *tmul;
  const int64_t *bw;
  const int64_t *lat;
} orc_hetero;
int orc_makespan_model(const orc_graph *g, const orc_devices *d, const orc_hetero *h,
                       const int32_t *order, int32_t K, const uint8_t *node_dev, int32_t model,
                       int64_t *start, int64_t *finish, int64_t *makespan);

/* Adjusting Placement with heterogeneous devices and links (h, or NULL) and
 * co-location groups decided inside the algorithm (group [n] in [-1,
 * n_groups), or NULL): clusters take W_x = sum of their members' durations on
 * device x, and devices are compared on the earliest finish time (the start
 * of eq. 7 plus W_x, the same ordering with identical devices); under link tables a coarse edge costs ceil(OB / bw) + N lat on
 * the link used (OB = its members' summed ob, N = their count), in eq. 7 from
 * each predecessor's device and in eq. 8 from the best device back to the
 * previous one; a group follows its smallest cluster, whose device is charged
 * with the followers' memory when their clusters are placed.  h == NULL and
 * group == NULL give orc_place's result. */
int orc_place_ext(const orc_graph *g, const orc_devices *d, const orc_hetero *h,
                  const int32_t *group, int32_t n_groups, const int32_t *cluster_id,
                  int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
                  int64_t *cluster_fin, int64_t *coarse_makespan, int32_t *best_effort_count);

/* Co-location groups: nodes with group[v] >= 0 take the device of their
 * group's first node in `order` (a topological order); node_dev [K][n] in
 * place. */
int orc_colocate(const orc_graph *g, const int32_t *order, const int32_t *group,
                 int32_t n_groups, int32_t K, uint8_t *node_dev);

#ifdef __cplusplus
}
#endif
#endif
