/*
 * libcel -- MI355X (gfx950) implementation of the data-parallel hot path of
 * Celeritas's placement optimiser (Xu, Liao, Xie, Zhou, "Celeritas: Fast
 * Optimizer for Large Dataflow Graphs", arXiv 2208.00184):
 *
 *   cel_topo_levels  level-synchronous topological ordering      (Section 4.2.2)
 *   cel_blevel       b-level / t-level / critical path, priority  (Section 5.1.3, eq. 2-3)
 *   cel_cpd_order    CPD-TOPO critical-path depth-first order    (Section 5.1.3, Algorithm 1)
 *   cel_dfs_order    DFS-TOPO depth-first topological order      (Section 4.2.2)
 *   cel_cluster      memory-capped contiguous clustering (DP)     (Section 5.1.3, eq. 4-6)
 *   cel_place        coarse graph + Adjusting Placement           (Section 5.2, eq. 7-9, Alg. 2)
 *   cel_makespan     makespan of one or K placements              (Section 5.2, eq. 7)
 *   cel_makespan_model  makespan with insertion / transfer tasks  (Section 5.2 eq. 7, 6.1)
 *   cel_colocate     co-location groups follow their first node  (Section 6.1)
 *   cel_order_place  Order-Place baseline placement               (Section 5.2, 6.2.2)
 *   cel_comm_sums    the parts of the comm/compute ratio CCR      (Section 5.1.1, eq. 1)
 *
 * Conventions (all entry points):
 *  - Arrays are DEVICE pointers owned by the caller unless marked (host).  The
 *    library never frees or keeps a caller pointer after it returns.
 *  - Work is enqueued on `stream`; every call returns after its results are
 *    complete (it synchronises `stream` once to read its status and scalar
 *    outputs).  Scratch memory comes from a library-owned arena per (device,
 *    stream): device blocks that grow to the largest call's needs and are
 *    kept until the process ends, so repeated calls allocate nothing.  Calls
 *    on one stream from several host threads take turns on its arena.
 *  - Times are int64 nanoseconds, sizes int64 bytes, indices int32.  A node's
 *    communication time is c[v] = ceil(ob[v] / bw) + lat (the paper's linear
 *    fit t = k*d + b, Section 4.2.1, in integer form), paid once per consumer
 *    edge: always in b-/t-levels, only between different devices in EST and
 *    makespan (eq. 7).  All results are exact integers, hence deterministic.
 *  - Return value: CEL_OK or a negative CEL_E_* code; cel_last_error() gives a
 *    message for the calling thread.  Outputs are unspecified after an error.
 *  - Calls on the same device may run concurrently on different streams.
 */
#ifndef CEL_H
#define CEL_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *hipStream_t; /* HIP's stream handle (NULL = default stream) */

enum {
  CEL_OK = 0,
  CEL_E_ARG = -1,      /* NULL pointer, bad size or range, malformed CSR/CSC, negative w/mem/ob */
  CEL_E_CYCLE = -2,    /* the graph has a cycle (self-loops included) */
  CEL_E_OVERFLOW = -3, /* sum(w) + sum over edges of c[src] >= 2^62 */
  CEL_E_HIP = -4,      /* a HIP runtime call failed */
  CEL_E_NOMEM = -5,    /* scratch allocation failed */
  CEL_E_ORDER = -6     /* an order/level/cluster argument is inconsistent with the graph */
};

/* cel_blevel flags */
enum { CEL_COMM_OFF = 1 /* treat every c[v] as 0 (compute-only critical path) */ };

/* cel_makespan_model model bits */
enum {
  CEL_MODEL_INSERT = 1,     /* first-fit insertion into each device's idle slots */
  CEL_MODEL_COMM_TASKS = 2, /* transfers as tasks on per-device send/receive channels */
  CEL_MODEL_COMM_BLOCK = 4  /* transfers as operations on both devices' compute queues */
};

/* cel_cluster modes */
enum { CEL_CLUSTER_DP = 0, CEL_CLUSTER_GREEDY = 1 };

/* Operator DAG, device pointers, read-only (Section 4.1: nodes are operations,
 * edges are data transfers).  Multi-edges are allowed and counted separately. */
typedef struct {
  int32_t n, m;                       /* nodes, edges (both >= 0) */
  const int32_t *out_ptr, *out_idx;   /* successors (CSR): [n+1], [m] */
  const int32_t *in_ptr, *in_idx;     /* predecessors (CSC): [n+1], [m], same edges */
  const int64_t *w;                   /* [n] compute time, ns, >= 0 */
  const int64_t *mem;                 /* [n] memory, bytes, >= 0 */
  const int64_t *ob;                  /* [n] output tensor bytes, >= 0 */
} cel_graph;

/* Modelled target devices (Section 4.1: devices with memory limits). */
typedef struct {
  int32_t D;                          /* 1..255 */
  const int64_t *cap;                 /* (host) [D] memory caps, bytes, >= 0 */
  int64_t bw;                         /* link bytes per ns, > 0 */
  int64_t lat;                        /* link latency, ns, >= 0 */
} cel_devices;

/* Level-synchronous Kahn ordering (Section 4.2.2: repeatedly remove the nodes
 * of indegree 0; one level = one round).  level[v] = 0 for a source, else
 * 1 + max level of its predecessors.  order_id lists the ids sorted by
 * (level, id); level_ptr[l] is the first position of level l in order_id
 * (capacity n+1; entries 0..L are written, level_ptr[L] = n).
 * Outputs: level [n], order_id [n], level_ptr [n+1], n_levels (host) = L.
 * Errors: CEL_E_ARG, CEL_E_CYCLE, CEL_E_HIP, CEL_E_NOMEM. */
int cel_topo_levels(const cel_graph *g, int32_t *level, int32_t *order_id,
                    int32_t *level_ptr, int32_t *n_levels, hipStream_t stream);

/* b-level (eq. 3): blevel[v] = w[v] for a sink, else w[v] + c[v] + max over
 * successors s of blevel[s]; t-level (eq. 2): tlevel[v] = 0 for a source,
 * else max over predecessors p of tlevel[p] + w[p] + c[p]; cp (host) = the
 * critical path = max blevel (Section 5.1.3).  prio_order lists the ids sorted
 * by (level ascending, blevel descending, id ascending): a level-monotone
 * topological order that visits longer critical paths first.
 * Inputs: level, level_ptr, order_id, n_levels as produced by cel_topo_levels
 * (any order_id that lists each level's nodes contiguously is accepted).
 * Outputs: blevel [n]; tlevel [n] or NULL; prio_order [n] or NULL; cp (host).
 * flags: CEL_COMM_OFF.  Errors: CEL_E_ARG, CEL_E_ORDER, CEL_E_OVERFLOW,
 * CEL_E_HIP, CEL_E_NOMEM. */
int cel_blevel(const cel_graph *g, const cel_devices *d, const int32_t *level,
               const int32_t *level_ptr, const int32_t *order_id, int32_t n_levels,
               int32_t flags, int64_t *blevel, int64_t *tlevel, int32_t *prio_order,
               int64_t *cp, hipStream_t stream);

/* CPD-TOPO order (Section 5.1.3, Algorithm 1), the critical-path depth-first
 * topological order that the paper feeds to the clustering.  With cpath[v] =
 * tlevel[v] + blevel[v], a stack starts with the sources (largest cpath on
 * top); the top node is popped and output, its out-edges removed, and the
 * successors left with no in-edge are pushed in increasing cpath order, so
 * the most critical one comes next.  Equal cpath: the lower id first.
 * Inputs: blevel [n] and tlevel [n] as produced by cel_blevel (with or
 * without CEL_COMM_OFF); only the CSR half of the graph is read.
 * Output: cpd_order [n], the node ids in CPD-TOPO order (a topological order,
 * which cel_cluster accepts).  The walk is one dependent step per node, so
 * it runs on the host over a copy of the successor lists; the call
 * synchronises `stream` first.
 * Errors: CEL_E_ARG (NULL or a malformed CSR), CEL_E_CYCLE, CEL_E_HIP. */
int cel_cpd_order(const cel_graph *g, const int64_t *blevel, const int64_t *tlevel,
                  int32_t *cpd_order, hipStream_t stream);

/* DFS-TOPO order (Section 4.2.2), the depth-first topological order that
 * CPD-TOPO refines.  A queue starts with the sources, the lowest id at its
 * head; the head node is removed and output, its out-edges removed, and the
 * successors left with no in-edge are put at the head of the queue, the
 * lowest id in front, so a freed child comes before every older entry.
 * Only the CSR half of the graph is read.  Output: dfs_order [n], the node
 * ids in DFS-TOPO order (a topological order, which cel_cluster accepts).
 * Like cel_cpd_order it walks on the host over a copy of the successor
 * lists and synchronises `stream`.
 * Errors: CEL_E_ARG (NULL or a malformed CSR), CEL_E_CYCLE, CEL_E_HIP. */
int cel_dfs_order(const cel_graph *g, int32_t *dfs_order, hipStream_t stream);

/* Contiguous clustering of a topological order (Section 5.1.3, eq. 4-6;
 * clusters are runs of consecutive positions, which keeps the coarse graph
 * acyclic by Lemma 1).  DP mode minimises the total comm of edges between
 * clusters, S(j) = min over i of S(i) + cost(i, j), subject to j - i <= R and
 * the cluster's summed memory <= M (a single node may exceed M); among equal
 * totals the smaller i (longer cluster) wins.  GREEDY mode grows each cluster
 * while both limits hold.  M = -1 selects floor(min cap / 4).
 * Inputs: order [n] any topological order (permutation with pos[u] < pos[v]
 * on every edge); 1 <= R <= 4096; M >= -1.
 * Outputs: cluster_id [n] (cluster 0 holds order[0]); n_clusters (host);
 * cut_cost (host) = sum of c[u] over edges u->v in different clusters.
 * Errors: CEL_E_ARG, CEL_E_ORDER, CEL_E_OVERFLOW, CEL_E_HIP, CEL_E_NOMEM. */
int cel_cluster(const cel_graph *g, const cel_devices *d, const int32_t *order,
                int32_t R, int64_t M, int32_t mode, int32_t *cluster_id,
                int32_t *n_clusters, int64_t *cut_cost, hipStream_t stream);

/* Coarse graph and Adjusting Placement (Section 5.2, Algorithm 2).  Cluster t
 * has W = sum of its members' w, MEM = sum of their mem; the coarse edge a->b
 * carries the sum of c[u] over edges u->v with u in a, v in b.  Clusters are
 * visited in index order; for each device the start time is the earliest
 * first-fit slot at or after pre_t (eq. 7), or infinite when the device's
 * remaining memory is below MEM; the cluster stays on the previous cluster's
 * device (device 0 for the first) unless EST(prev) - EST(best) > back_cost,
 * the max comm to a successor (eq. 8-9); if every device is full it goes to the
 * device with the most remaining memory (best effort).  Ties go to the lowest
 * device id.  Nodes inherit their cluster's device.
 * Inputs: cluster_id [n] with values in [0, n_clusters) and cluster_id[u] <=
 * cluster_id[v] on every edge.
 * Outputs: cluster_dev [C] uint8; node_dev [n] uint8; cluster_fin [C] or NULL;
 * coarse_makespan (host) = max finish; best_effort_count (host).
 * Errors: CEL_E_ARG, CEL_E_ORDER, CEL_E_OVERFLOW, CEL_E_HIP, CEL_E_NOMEM. */
int cel_place(const cel_graph *g, const cel_devices *d, const int32_t *cluster_id,
              int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
              int64_t *cluster_fin, int64_t *coarse_makespan, int32_t *best_effort_count,
              hipStream_t stream);

/* Adjusting Placement (Section 5.2, eq. 7-9, Algorithm 2) with the device
 * generality of Section 4.1 and the co-location groups of Section 6.1 decided
 * inside the algorithm.  As cel_place, except:
 *  - h (heterogeneous devices and links, or NULL): cluster t takes W_x = the
 *    sum of its members' durations ceil(w * tmul[x] / 1024) on device x, and
 *    devices are compared, and the move test of eq. 9 made, on the earliest
 *    finish time (first-fit start + W_x), which orders identical devices as
 *    eq. 7's start times do.  With link tables (h->bw or h->lat) a coarse edge
 *    whose N member edges carry OB output bytes in total costs
 *    ceil(OB / bw[y][x]) + N * lat[y][x] on the link y -> x: in pre_t from each
 *    predecessor's device y (eq. 7), and in back_cost on the link from the best
 *    device back to the previous cluster's (eq. 8); without them a coarse edge
 *    costs the sum of its members' c[u] as in cel_place.
 *  - group [n] (device, in [-1, n_groups), or NULL): a group's leading
 *    cluster is the smallest cluster id among its members and every member
 *    runs on that cluster's device; a member in a later cluster (a follower)
 *    is charged to that device's memory when its own cluster is placed, before
 *    the devices are compared, and its cluster's memory test and charge count
 *    only the other members.  The coarse schedule keeps every member's
 *    compute in its own cluster.
 * h == NULL and group == NULL give cel_place's results.
 * Inputs: as cel_place; D <= 64; tmul in [1, 65536], link bw in [1, 2^31) and
 * lat in [0, 2^31).  Outputs: cluster_dev [C]; node_dev [n] (group members on
 * their leading cluster's device); cluster_fin [C] or NULL; coarse_makespan
 * and best_effort_count (host).
 * Errors: CEL_E_ARG (also D > 64 or a bad group id), CEL_E_ORDER,
 * CEL_E_OVERFLOW, CEL_E_HIP, CEL_E_NOMEM. */
typedef struct cel_hetero cel_hetero;
int cel_place_ext(const cel_graph *g, const cel_devices *d, const cel_hetero *h,
                  const int32_t *group, int32_t n_groups, const int32_t *cluster_id,
                  int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
                  int64_t *cluster_fin, int64_t *coarse_makespan, int32_t *best_effort_count,
                  hipStream_t stream);

/* Order-Place, the baseline placement of Sections 5.2 and 6.2.2: clusters are taken in
 * index order and filled onto device 0 until the next cluster's MEM (sum of
 * its members' mem) no longer fits that device's remaining cap, then onto
 * device 1, and so on; once the last device is reached every remaining
 * cluster goes there, and each one that does not fit it counts as best
 * effort.  Nodes inherit their cluster's device.  Clusters may be empty.
 * Inputs: cluster_id [n] with values in [0, n_clusters); n_clusters >= 1
 * when n > 0; the total mem must stay below 2^63.
 * Outputs: cluster_dev [C] uint8; node_dev [n] uint8; best_effort_count
 * (host).
 * Errors: CEL_E_ARG, CEL_E_HIP, CEL_E_NOMEM. */
int cel_order_place(const cel_graph *g, const cel_devices *d, const int32_t *cluster_id,
                    int32_t n_clusters, uint8_t *cluster_dev, uint8_t *node_dev,
                    int32_t *best_effort_count, hipStream_t stream);

/* The two parts of the communication-to-computation ratio CCR (Section 5.1.1, eq. 1): edge_comm
 * = sum over edges u->v of c[u] (only the edges whose ends sit in different
 * clusters when cluster_id is given), w_sum = sum of w; CCR = edge_comm /
 * w_sum is left to the caller.
 * Inputs: cluster_id [n] or NULL for the whole graph.
 * Outputs: edge_comm, w_sum (host).
 * Errors: CEL_E_ARG, CEL_E_OVERFLOW, CEL_E_HIP, CEL_E_NOMEM. */
int cel_comm_sums(const cel_graph *g, const cel_devices *d, const int32_t *cluster_id,
                  int64_t *edge_comm, int64_t *w_sum, hipStream_t stream);

/* Makespan of K placements (eq. 7 without insertion): nodes are taken in
 * `order`; a node is ready when every predecessor p has finished, plus c[p]
 * when p sits on another device; it starts at the later of ready and the end
 * of the previous node placed on its device; makespan = latest finish.
 * Inputs: order [n] level-monotone (level[order[k]] non-decreasing and
 * level_ptr[l] <= k < level_ptr[l+1] for level l), e.g. prio_order from
 * cel_blevel with level/level_ptr/n_levels from cel_topo_levels; K >= 1;
 * node_dev [K][n] uint8 device per node id, each < D.
 * Outputs: start, finish [K][n] by node id, or NULL; makespan [K] (device).
 * Errors: CEL_E_ARG, CEL_E_ORDER, CEL_E_OVERFLOW, CEL_E_HIP, CEL_E_NOMEM. */
int cel_makespan(const cel_graph *g, const cel_devices *d, const int32_t *order,
                 const int32_t *level, const int32_t *level_ptr, int32_t n_levels,
                 int32_t K, const uint8_t *node_dev, int64_t *start, int64_t *finish,
                 int64_t *makespan, hipStream_t stream);

/* cel_makespan for callers that cannot allocate device memory: code being
 * captured into a HIP graph, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, outputs and results as cel_makespan; the call
 * makes no hipMalloc, hipFree or other allocating call.  Its scratch is one
 * fixed array of CEL_NOALLOC_SCRATCH_BYTES per GPU, created with the
 * library's code object on that GPU and held until the process ends; it keeps
 * the last call's contents (each call clears what it needs).  Inputs whose
 * scratch bound, 65536 + 200 (n + 1) + 16 m + 21 K n bytes, exceeds that size
 * are rejected with CEL_E_ARG before any work is queued (about 870k nodes
 * with m = 2n at K = 1; 32 placements of a 200k-node graph).  Calls
 * through this entry point take turns on a process-wide lock and return
 * after their results are complete, so they never overlap; anything else
 * that wrote the same array at the same time would race with them.
 * Errors: as cel_makespan. */
#define CEL_NOALLOC_SCRATCH_BYTES (128ull << 20)
int cel_makespan_noalloc(const cel_graph *g, const cel_devices *d, const int32_t *order,
                         const int32_t *level, const int32_t *level_ptr, int32_t n_levels,
                         int32_t K, const uint8_t *node_dev, int64_t *start, int64_t *finish,
                         int64_t *makespan, hipStream_t stream);

/* Heterogeneous devices for cel_makespan_model (host arrays; a NULL member
 * keeps the homogeneous value): device x runs a node of compute time w in
 * ceil(w * tmul[x] / 1024) (1024 = the reference speed, 1 <= tmul <= 65536);
 * node u's output takes ceil(ob[u] / bw[a*D + b]) + lat[a*D + b] from device
 * a to device b (1 <= bw < 2^31, 0 <= lat < 2^31; the diagonal is unused). */
struct cel_hetero {
  const int64_t *tmul; /* (host) [D] */
  const int64_t *bw;   /* (host) [D*D] bytes per ns */
  const int64_t *lat;  /* (host) [D*D] ns */
};

/* Makespan of K placements under richer device models (Section 5.2's slot
 * rule, eq. 7, at node level; Section 6.1's transfers as tasks).  Nodes are
 * taken in `order`; a node is ready when each input has arrived: a
 * predecessor p on the same device at its finish, on another device at
 * finish + c[p] or, with CEL_MODEL_COMM_TASKS, when p's transfer to this
 * device ends.  Start: model without CEL_MODEL_INSERT, the later of ready and
 * the end of the device's previous node (cel_makespan's FIFO schedule for
 * model 0); with it, the earliest time >= ready at which the node fits
 * between the nodes already placed on the device (w = 0: ready).
 * CEL_MODEL_COMM_TASKS: after p finishes, one transfer per other device
 * holding a successor of p, in increasing device order, each taking c[p] and
 * holding p's device's send channel and the target's receive channel:
 * start = max(finish of p, both channels' previous transfer end).
 * CEL_MODEL_COMM_BLOCK (alone, FIFO devices): the same transfers are
 * operations on the devices themselves (Section 6.1 adds a transfer node on
 * every device that sends or receives): each enters the compute queue of the
 * sending and of the receiving device right after its producer, starts when
 * both are free and holds both for its duration.
 * h: heterogeneous devices (cel_hetero; node durations and link costs follow
 * it), or NULL.
 * Inputs: order [n] any topological order (permutation with pos[u] < pos[v]
 * on every edge); K >= 1; node_dev [K][n] uint8, each < D; D <= 64; model a
 * combination of CEL_MODEL_INSERT and CEL_MODEL_COMM_TASKS, or
 * CEL_MODEL_COMM_BLOCK alone.
 * Outputs: start, finish [K][n] by node id, or NULL; makespan [K] (device).
 * Errors: CEL_E_ARG (also D > 64), CEL_E_ORDER, CEL_E_OVERFLOW, CEL_E_HIP,
 * CEL_E_NOMEM. */
int cel_makespan_model(const cel_graph *g, const cel_devices *d, const cel_hetero *h,
                       const int32_t *order, int32_t K, const uint8_t *node_dev, int32_t model,
                       int64_t *start, int64_t *finish, int64_t *makespan, hipStream_t stream);

/* Co-location groups (Section 6.1): every node with group[v] >= 0 moves to the
 * device of its group's first node in `order`; nodes with group -1 keep
 * theirs.  Memory caps are not rechecked (the group's leader decides).
 * Inputs: order [n] a topological order; group [n] in [-1, n_groups);
 * node_dev [K][n] uint8, rewritten in place.
 * Errors: CEL_E_ARG, CEL_E_ORDER, CEL_E_HIP, CEL_E_NOMEM. */
int cel_colocate(const cel_graph *g, const int32_t *order, const int32_t *group,
                 int32_t n_groups, int32_t K, uint8_t *node_dev, hipStream_t stream);

/* Diagnostics: per-kernel device time.  After cel_timing(1), every call
 * records a pair of HIP events on its stream around each of its main kernel
 * launches; the elapsed times are added to process-wide totals when the call
 * completes.  cel_kernel_stats writes one line per kernel, "name launches
 * total_ms\n", into buf (NUL-terminated, truncated to buflen), returns the
 * number of kernels listed, and clears the totals when reset != 0.
 * cel_timing returns the previous setting. */
int cel_timing(int enable);
int cel_kernel_stats(char *buf, int buflen, int reset);

/* Diagnostics: how the calling thread's last cel_makespan or
 * cel_makespan_noalloc call evaluated its schedule.  *path = 0: K = 1 by
 * relaxation over the edges between different devices (each device's FIFO
 * chain makes edges inside one device redundant), exact after *rounds rounds,
 * the last of which changed nothing; 1: K = 1 by the level sweep, after
 * *rounds rounds of relaxation that did not converge within their budget (0
 * when the relaxation could not be launched); 2: K > 1 (level sweeps of the
 * batch), *rounds = 0.
 * Outputs: path, rounds (host).
 * Errors: CEL_E_ARG (NULL argument). */
int cel_makespan_info(int32_t *path, int32_t *rounds);

/* Diagnostics: how the calling thread's last cel_blevel call found its
 * longest paths.  info[0] = 0: the b-level by policy iteration (each node
 * follows one successor; pointer jumping sums the chains; nodes switch to a
 * successor of larger value until none can), exact after info[1] iterations;
 * 1: by the level sweep (after info[1] iterations that did not converge
 * within their budget, or 0 when policy iteration was not tried).  info[2],
 * info[3]: the same for the t-level (info[2] = 2: not requested).
 * Outputs: info [4] (host).
 * Errors: CEL_E_ARG (NULL argument). */
int cel_blevel_info(int32_t *info);

/* Diagnostics: how the calling thread's last cel_topo_levels call found the
 * levels.  info[0] = 0: by policy iteration over the predecessors (graphs of
 * 16,384 nodes and more), exact after info[1] iterations; 1: by Kahn's
 * level-synchronous kernel (after info[1] iterations that did not converge
 * within their budget of 12, or 0 when policy iteration was not tried).
 * Outputs: info [2] (host).
 * Errors: CEL_E_ARG (NULL argument). */
int cel_topo_levels_info(int32_t *info);

/* Diagnostics: how the calling thread's last cel_cluster call ran the DP
 * (mode CEL_CLUSTER_DP).  info[0] = 0: by policy iteration over the back
 * pointers (graphs of 16,384 nodes and more), exact after info[1]
 * iterations; 1: by the blocked sequential DP (after info[1] iterations that
 * did not converge within their budget, or 0 when policy iteration was not
 * tried).
 * Outputs: info [2] (host).
 * Errors: CEL_E_ARG (NULL argument). */
int cel_cluster_info(int32_t *info);

/* Diagnostics: cel_policy_iteration(0) makes the calling thread's
 * cel_topo_levels, cel_blevel and cel_cluster calls take Kahn's kernel, the
 * level sweeps and the blocked DP directly; 1 (the default) tries policy
 * iteration first, with packed 64-bit entries and asynchronous pointer
 * jumping where the values fit; 2 tries policy iteration first with 16-byte
 * entries and synchronous rounds everywhere.  Every mode gives the same
 * results.  Returns the previous mode (CEL_E_ARG for a negative mode). */
int cel_policy_iteration(int mode);

/* Diagnostics: which K = 1 path the calling thread's cel_makespan and
 * cel_makespan_noalloc calls take.  mode 0: the level sweep directly (path 1
 * without relaxation rounds); 1 (the default): the relaxation first, on as
 * many workgroups as the GPU holds at once; m >= 2: the relaxation first, on
 * at most m workgroups (more slots per thread; for tests and tuning).  Every
 * mode gives the same results.  Returns the previous mode (CEL_E_ARG for a
 * negative mode). */
int cel_makespan_relax(int mode);

/* Diagnostics: the dependent step that bounds a level-synchronous sweep
 * (each level of the b-level recursion, eq. 3, and of the makespan, eq. 7,
 * waits for the previous one).  Runs `steps` dependent iterations of gather
 * -> 64-bit segmented max-plus wave scan -> write, each iteration's gather
 * index taken from the previous result, and returns the time per iteration
 * in *ns_per_step (host).  variant 0: one wave, gather from LDS; 1: a
 * workgroup of 1024 threads, gather from LDS and a barrier after the write;
 * 2: one wave, gather from a global array resident in L2.  Two launches of
 * steps/8 and steps iterations are timed with HIP events and differenced, so
 * launch overhead cancels.  1 <= steps <= 2^24.  Synchronises `stream`.
 * Errors: CEL_E_ARG, CEL_E_HIP, CEL_E_NOMEM. */
int cel_step_latency(int32_t variant, int32_t steps, double *ns_per_step, hipStream_t stream);

/* Message describing the calling thread's last error ("" if none). */
const char *cel_last_error(void);

/* Library version: major * 10000 + minor * 100 + patch. */
int cel_version(void);

#ifdef __cplusplus
}
#endif
#endif
