/*
 * pardnn.h -- C ABI of the MI355X (gfx950) placement-aware critical-path
 * evaluator: the data-parallel hot path of ParDNN's partitioner
 * (arXiv 2008.08636).
 *
 * The problem (paper Sec. 2 and 3): a computational DAG G = (V, E) whose node
 * n costs comp(n) time and holds mem(n) bytes (Table 2), whose edge e costs
 * comm(e) to transfer its tensor (Table 2) -- zero when both ends sit on the
 * same device label (Fig. 2 caption; Sec. 3.1.2, cluster criticality) -- and a
 * placement of every node on a label. The evaluator computes the quantities
 * the partitioner recomputes again and again (Alg. 1 compute_weighted_levels
 * and find_heaviest_path; Alg. 2; Memory Heuristic II of Sec. 3.2):
 *   - topological levels,
 *   - t-level tl(n) (costliest source-to-n path, excluding n) and b-level
 *     bl(n) (costliest n-to-sink path, including n), Table 2,
 *   - makespan M = max over n of tl(n) + bl(n), the critical nodes
 *     (tl + bl == M) and one canonical critical path (Table 2, CP),
 *   - memory per label and its overflow against a capacity (Sec. 3.2, Sec. 4).
 *
 * Conventions shared by every entry point
 *   - Array arguments are DEVICE pointers on the handle's device (e.g. the
 *     data_ptr() of a torch tensor), owned by the caller. Outputs are
 *     allocated by the caller. Work is enqueued on the handle's stream; the
 *     caller synchronises that stream before reading outputs on the host.
 *     Only arguments documented as "host" are host pointers.
 *   - Node ids are 0..n_nodes-1 in the caller's numbering; every per-node
 *     output is in that numbering.
 *   - Weights (comp, edge_cost, mem) are int64 and must be >= 0. All
 *     arithmetic is exact int64: results are bit-exact.
 *   - The artificial source and sink of Sec. 3 are implicit: a node without
 *     predecessors has tl = 0, a node without successors has bl = comp.
 *   - Multi-edges are allowed; each edge is relaxed on its own.
 *   - Every call returns PARDNN_OK or a negative status, never aborts and never
 *     throws. pardnn_last_error() gives a detail string for the calling thread.
 *   - A handle is used by one host thread at a time. Calls that report an
 *     error found on the device (marked "syncs") wait for the stream, unless
 *     the handle defers such errors (pardnn_set_deferred_errors): then those
 *     calls only enqueue, and pardnn_take_errors reports what they found.
 *     Either way the kernels bound every access by the sizes passed, so bad
 *     values give wrong results at worst, never an access out of bounds.
 *
 * Batched layout: arrays of several placements are PLACEMENT-MINOR, i.e.
 * element (node v, placement p) of a [V][n_place] array sits at
 * v * n_place + p.
 */
#ifndef PARDNN_H
#define PARDNN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pardnn_graph pardnn_graph;

enum pardnn_status {
    PARDNN_OK = 0,
    PARDNN_E_INVAL = -1,    /* bad argument: NULL pointer, id or label out of range, negative weight */
    PARDNN_E_CYCLE = -2,    /* the graph has a cycle or a self-loop */
    PARDNN_E_OVERFLOW = -3, /* sum(comp) + sum(edge_cost) or sum(mem) exceeds INT64_MAX */
    PARDNN_E_NOMEM = -4,    /* a device allocation failed */
    PARDNN_E_DEVICE = -5    /* no usable GPU, or a HIP runtime call failed */
};

/* Largest graph a handle accepts: 2^26 nodes and 2^27 edges (the evaluation
 * kernels address per-node and per-edge arrays with 32-bit byte offsets). */
#define PARDNN_MAX_NODES (1 << 26)
#define PARDNN_MAX_EDGES (1 << 27)

typedef struct pardnn_info {
    int32_t n_nodes;
    int64_t n_edges;
    int32_t n_levels;      /* valid once levelized, else -1 */
    int32_t max_width;     /* widest level, valid once levelized, else -1 */
    int32_t device;        /* HIP device ordinal the handle lives on */
} pardnn_info;

/*
 * Create a handle for G = (V, E) (Sec. 2; Table 2 comp, comm, mem).
 *   n_nodes        V, 0 <= V <= PARDNN_MAX_NODES.
 *   n_edges        |E|, 0 <= |E| <= PARDNN_MAX_EDGES.
 *   src, dst       int32[n_edges], edge e runs src[e] -> dst[e].
 *   comp           int64[n_nodes], node cost (comp(n)), >= 0.
 *   edge_cost      int64[n_edges], transfer cost of edge e when its ends carry
 *                  different labels (comm(e)), >= 0.
 *   mem            int64[n_nodes], output memory of node n (mem(n)), >= 0.
 *   stream         hipStream_t for all later work on the handle (NULL: the
 *                  default stream of the current device).
 *   out            host pointer receiving the new handle.
 * The handle copies what it needs; the caller may free the inputs afterwards.
 * Errors: E_INVAL (NULL pointer, id out of range, negative weight),
 * E_OVERFLOW, E_NOMEM, E_DEVICE. Syncs once (validation result).
 */
int pardnn_graph_create(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                        const int32_t *dst, const int64_t *comp,
                        const int64_t *edge_cost, const int64_t *mem,
                        void *stream, pardnn_graph **out);

/* Release a handle and its device memory (waits for its stream). NULL is a no-op. */
int pardnn_graph_destroy(pardnn_graph *g);

/* Rebind the handle to another stream of the same device. */
int pardnn_set_stream(pardnn_graph *g, void *stream);

/* Host query of sizes; levels are reported once pardnn_levelize has run. */
int pardnn_get_info(const pardnn_graph *g, pardnn_info *info);

/*
 * Topological levels by Kahn's algorithm (Sec. 3.1.1: weighted levels come
 * from one pass in topological order, O(|V| + |E|); the per-level work
 * tables of Sec. 3.1.2 are indexed by level). level(v) = 0 without
 * predecessors, else 1 + the largest level of its predecessors.
 *   level          int32[n_nodes] or NULL: level of each node.
 *   order          int32[n_nodes] or NULL: node ids sorted by (level, id).
 *   level_ptr      int32[n_nodes + 1] or NULL: order[level_ptr[l] ..
 *                  level_ptr[l+1]) is level l; entries past n_levels are
 *                  left untouched.
 *   n_levels_host  host int32* or NULL: number of levels.
 * The result depends on the structure only and is cached: later calls only
 * copy it out. Errors: E_CYCLE. Syncs (once per handle).
 */
int pardnn_levelize(pardnn_graph *g, int32_t *level, int32_t *order,
                    int32_t *level_ptr, int32_t *n_levels_host);

/*
 * t-levels, b-levels and makespan under one placement (Table 2: tl, bl,
 * w_lvl; Alg. 1 compute_weighted_levels).
 *   tl(v) = max over edges (u,v) of tl(u) + comp(u) + c(u,v), 0 if none;
 *   bl(v) = comp(v) + max over edges (v,s) of c(v,s) + bl(s), or comp(v);
 *   c(u,v) = 0 if placement[u] == placement[v] else edge_cost(u,v);
 *   M = max over v of tl(v) + bl(v) (0 for an empty graph).
 *   placement      int32[n_nodes], any int32 values: only equality matters,
 *                  so cluster ids work as labels (Sec. 3.1.2 criticality).
 *   tl, bl         int64[n_nodes] outputs.
 *   makespan       int64[1] output.
 * Levelizes first if needed (E_CYCLE). The first single or batched
 * evaluation on a handle also builds the per-graph edge split of the batched
 * sweep and syncs once; later calls do not sync. Labels all in [0, 2^16) take
 * the batched sweep with one placement (decided on the device), others the
 * single-placement sweep; the results are the same.
 */
int pardnn_tb_levels(pardnn_graph *g, const int32_t *placement, int64_t *tl,
                     int64_t *bl, int64_t *makespan);

/*
 * Critical nodes and the canonical critical path (Table 2 CP; Alg. 1
 * find_heaviest_path on freshly computed weighted levels).
 *   is_critical[v] = (tl[v] + bl[v] == *makespan).
 *   path           int32[n_nodes] output: starts at the smallest-id node
 *                  without predecessors that is critical, then repeatedly
 *                  steps to the smallest-id successor s of the current node u
 *                  with tl[u] + comp[u] + c(u,s) + bl[s] == *makespan, and
 *                  stops at a node without such a successor. For tl/bl/M from
 *                  pardnn_tb_levels this is the lexicographically smallest
 *                  node sequence among the maximum-length paths.
 *   path_len       int32[1] output, <= number of levels.
 *   placement, tl, bl, makespan  inputs as produced by pardnn_tb_levels.
 * No sync.
 */
int pardnn_critical_path(pardnn_graph *g, const int32_t *placement,
                         const int64_t *tl, const int64_t *bl,
                         const int64_t *makespan, uint8_t *is_critical,
                         int32_t *path, int32_t *path_len);

/*
 * Memory per label (Sec. 3.2, Memory Heuristic II per-partition totals,
 * without the residual/normal split; Sec. 4 capacity):
 *   label_mem[k] = sum of mem[v] over v with placement[v] == k;
 *   overflow[k]  = max(0, label_mem[k] - capacity[k]).
 *   placement      int32[n_nodes], every value in [0, n_labels).
 *   n_labels       K >= 1.
 *   capacity       int64[K] >= 0, or NULL (no limit: overflow = 0). The caller
 *                  applies the paper's 10 % reserve (Sec. 4) itself.
 *   label_mem      int64[K] output.
 *   overflow       int64[K] output or NULL.
 * Errors: E_INVAL if a label is outside [0, K) or a capacity is negative.
 * Syncs.
 */
int pardnn_label_memory(pardnn_graph *g, const int32_t *placement,
                        int32_t n_labels, const int64_t *capacity,
                        int64_t *label_mem, int64_t *overflow);

/*
 * Apply moves to a placement in place: placement[node[i]] = label[i] for
 * i = 0..n_moves-1 in order (a later move of the same node wins). This is the
 * node movement of Sec. 3.2 (overflow handling, Heuristic II) as the
 * refinement loop issues it.
 *   placement      int32[n_nodes], updated in place.
 *   node, label    int32[n_moves].
 * Errors: E_INVAL if a node id is out of range (no move is applied then).
 * Syncs.
 */
int pardnn_apply_moves(pardnn_graph *g, int32_t *placement, int32_t n_moves,
                       const int32_t *node, const int32_t *label);

/*
 * Materialise n_place successive placements of a refinement loop: placement
 * p is `base` with the moves of steps 0..p applied in order, where step p's
 * moves are node[step_ptr[p] .. step_ptr[p+1]) -> label[same range] (a later
 * move of a node wins, within and across steps).
 *   base           int32[n_nodes].
 *   step_ptr       int64[n_place + 1], non-decreasing, step_ptr[0] = 0,
 *                  step_ptr[n_place] = n_moves (checked on the device).
 *   n_moves        host value: the length of node and label, 0 <= n_moves
 *                  < 2^31.
 *   node, label    int32[n_moves].
 *   placements     int32[n_nodes][n_place] output (placement-minor).
 * Errors: E_INVAL if a node id is out of range or step_ptr does not match
 * n_moves. Syncs (unless errors are deferred).
 */
int pardnn_build_placements(pardnn_graph *g, const int32_t *base,
                            int32_t n_place, const int64_t *step_ptr,
                            int64_t n_moves, const int32_t *node,
                            const int32_t *label, int32_t *placements);

/*
 * Evaluate n_place placements at once: for every placement p the results of
 * pardnn_tb_levels, pardnn_critical_path and pardnn_label_memory. All arrays
 * are placement-minor.
 *   placements     int32[n_nodes][n_place].
 *   n_labels, capacity  as for pardnn_label_memory. When label_mem is NULL,
 *                  labels are not checked and only their equality matters;
 *                  n_labels in [1, 2^16] is then a hint that they lie in
 *                  [0, n_labels) (fewer bits to pack: faster when it holds,
 *                  the same results either way), and other values give none.
 *   tl, bl         int64[n_nodes][n_place] outputs, each or both NULL: the
 *                  levels are still computed (they decide everything else)
 *                  but not written out, for callers that keep only the
 *                  per-placement results.
 *   makespan       int64[n_place] output.
 *   is_critical    uint8[n_nodes][n_place] output or NULL.
 *   path           int32[n_place][path_stride] output or NULL: row p holds
 *                  placement p's canonical critical path in its first
 *                  path_len[p] entries; the rest of the row is scratch
 *                  (unspecified on return).
 *   path_stride    >= number of levels when path != NULL.
 *   path_len       int32[n_place] output (NULL iff path is NULL).
 *   label_mem      int64[n_place][n_labels] output or NULL.
 *   overflow       int64[n_place][n_labels] output or NULL.
 * Errors: E_INVAL (bad label when label_mem != NULL, short path_stride).
 * Syncs when label_mem != NULL (unless errors are deferred).
 */
int pardnn_evaluate_batch(pardnn_graph *g, int32_t n_place,
                          const int32_t *placements, int32_t n_labels,
                          const int64_t *capacity, int64_t *tl, int64_t *bl,
                          int64_t *makespan, uint8_t *is_critical,
                          int32_t *path, int32_t path_stride,
                          int32_t *path_len, int64_t *label_mem,
                          int64_t *overflow);

/*
 * pardnn_evaluate_batch for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same arguments and results, but its workspace is a fixed
 * array of 128 MiB compiled into the library (one per GPU, held until the
 * process ends) and the call allocates nothing.
 *   Limit: the batch must fit that workspace, about 42 bytes per node and
 *   placement (n_nodes * n_place <= ~3.2M, e.g. 10 placements of a
 *   300k-node graph); larger batches return E_INVAL with the bytes needed.
 *   The graph must already be levelized (pardnn_levelize); otherwise E_INVAL.
 *   All calls on one GPU share the array: calls that overlap in time on one
 *   GPU (from any handle or stream) race and give undefined results.
 * Errors and syncs as for pardnn_evaluate_batch.
 */
int pardnn_evaluate_batch_fixed(pardnn_graph *g, int32_t n_place,
                                const int32_t *placements, int32_t n_labels,
                                const int64_t *capacity, int64_t *tl,
                                int64_t *bl, int64_t *makespan,
                                uint8_t *is_critical, int32_t *path,
                                int32_t path_stride, int32_t *path_len,
                                int64_t *label_mem, int64_t *overflow);

/*
 * The refinement loop's successive placements evaluated in one call (the
 * partitioner re-evaluates after every batch of node moves: Sec. 3.2 memory
 * heuristics, Alg. 2 mapping). Placement p is `base` with the moves of steps
 * 0..p applied in order, exactly as pardnn_build_placements defines them;
 * every output is exactly that of pardnn_evaluate_batch on those placements,
 * but the [V][n_place] placement matrix is never materialised.
 *   base, step_ptr, n_moves, node, label   as for pardnn_build_placements.
 *   other arguments               as for pardnn_evaluate_batch.
 * Errors: E_INVAL (bad move node id, bad label when label_mem != NULL, short
 * path_stride, step_ptr not matching n_moves). Syncs (unless errors are
 * deferred); no other host round trip.
 */
int pardnn_evaluate_moves(pardnn_graph *g, const int32_t *base, int32_t n_place,
                          const int64_t *step_ptr, int64_t n_moves, const int32_t *node,
                          const int32_t *label, int32_t n_labels,
                          const int64_t *capacity, int64_t *tl, int64_t *bl,
                          int64_t *makespan, uint8_t *is_critical,
                          int32_t *path, int32_t path_stride,
                          int32_t *path_len, int64_t *label_mem,
                          int64_t *overflow);

/*
 * Memory Heuristic II (Sec. 3.2.2) evaluated for n_place placements: the
 * per-partition memory of residual and of normal nodes, the balance predicate
 * of Eq. 6 per partition, and the co-location of reference nodes with the
 * residual node they mutate (node kinds of Sec. 3.2.1).
 *   placements     int32[n_nodes][n_place], labels in [0, n_labels).
 *   node_type      int32[n_nodes]: 0 normal, 1 residual, 2 reference.
 *   ref_target     int32[n_nodes]: for a reference node the node it mutates,
 *                  or -1; ignored for other kinds.
 *   res_mem, nor_mem  int64[n_place][n_labels] outputs: sum of the graph's
 *                  mem over the residual / normal nodes of each label
 *                  (reference nodes reserve no memory).
 *   balanced       uint8[n_place][n_labels] output: Eq. 6, n_labels / 2 *
 *                  (res share + normal share) >= 1, decided exactly; a kind
 *                  with no memory at all counts as the fair share 1 / n_labels.
 *   ref_misplaced  int64[n_place] output: reference nodes whose target carries
 *                  another label.
 * Errors: E_INVAL (null pointers, n_labels < 1, a label, kind or target out of
 * range). Syncs.
 */
int pardnn_memory_balance(pardnn_graph *g, int32_t n_place,
                          const int32_t *placements, const int32_t *node_type,
                          const int32_t *ref_target, int32_t n_labels,
                          int64_t *res_mem, int64_t *nor_mem, uint8_t *balanced,
                          int64_t *ref_misplaced);

/*
 * Cluster criticality of the mapping stage (Sec. 3.1.2): with communication
 * inside every cluster set to zero (the cluster ids used as labels), the
 * weighted levels w(n) = tl(n) + bl(n) are recomputed and each cluster gets
 * the largest w of its nodes, the length of the longest path through it; the
 * clusters are then ordered by non-increasing criticality.
 *   cluster        int32[n_nodes], ids in [0, n_clusters).
 *   criticality    int64[n_clusters] output (-1 for a cluster without nodes).
 *   order          int32[n_clusters] output: cluster ids by criticality
 *                  descending, equal criticality by id ascending.
 * Errors: E_INVAL (null pointers, n_clusters < 1 on a non-empty graph, an id
 * out of range), E_CYCLE. Syncs.
 */
int pardnn_cluster_criticality(pardnn_graph *g, const int32_t *cluster,
                               int32_t n_clusters, int64_t *criticality,
                               int32_t *order);

/*
 * The terms of level-aware load balancing (Eq. 2, Sec. 3.1.2) for a batch of
 * clusters against the K partitions of a partial placement, all answered
 * against the same state (the sequential mapping loop that merges one cluster
 * at a time stays with the caller).
 *   label      int32[n_nodes]: partition of each mapped node, -1 unmapped.
 *   cluster    int32[n_nodes]: cluster id in [0, n_clusters), -1 for none.
 *   tl         int64[n_nodes]: the top levels the spans are measured in
 *              (for instance pardnn_tb_levels with cluster ids as labels).
 * With f the cluster's first node and l its last (smallest and largest
 * (hop level, id)), span = [lo, hi] with lo = max over parents p of f of
 * tl(p) + comp(p) (0 without parents) and hi = min over children c of l of
 * tl(c) (max over all nodes of tl + comp without children) -- Table 2's span.
 * Outputs (device, caller-allocated):
 *   span_lo, span_hi int64[n_clusters]  (0 and -1 for a cluster without nodes)
 *   work  int64[n_clusters][K]: sum of comp over nodes on partition k whose tl
 *         lies in [lo, hi] (the first sum of Eq. 2)
 *   comm  int64[n_clusters][K]: sum of edge costs between the cluster and
 *         nodes on partition k, edges inside one cluster excluded
 *   choice int32[n_clusters]: argmin over k of work + sum(comm) - comm[k]
 *         (Eq. 2), ties to the largest comm[k], then the smallest k; -1 for a
 *         cluster without nodes.
 * Errors: E_INVAL (K < 1, n_clusters < 0, null pointers, an id out of
 * range), E_CYCLE. Syncs.
 */
int pardnn_span_work(pardnn_graph *g, const int32_t *label, int32_t K, const int32_t *cluster,
                     int32_t n_clusters, const int64_t *tl, int64_t *span_lo, int64_t *span_hi,
                     int64_t *work, int64_t *comm, int32_t *choice);

/*
 * The primary clusters of graph slicing (Alg. 1, Sec. 3.1.1): K rounds, each
 * computing the weighted levels of the remaining graph, taking its heaviest
 * path -- a critical path, the canonical one of pardnn_critical_path -- as
 * primary cluster j, and removing that path's nodes and their edges. Before
 * any placement exists every edge carries its communication cost (every node
 * is its own cluster). A path starts at a node without remaining predecessors.
 *   primary        int32[n_nodes] output: the round that took each node, or -1.
 *   paths          int32[K][path_stride] output: round j's path in its first
 *                  path_len[j] entries (original ids, source to sink).
 *   path_stride    >= number of levels.
 *   path_len       int32[K] output (0 once no node remains).
 *   makespan       int64[K] output: the critical-path length of the graph
 *                  remaining before round j (0 when empty).
 * Errors: E_INVAL (K < 0, null pointers, short path_stride), E_CYCLE.
 * Syncs only when the graph is levelised first.
 */
int pardnn_slice_primaries(pardnn_graph *g, int32_t K, int32_t *primary,
                           int32_t *paths, int32_t path_stride,
                           int32_t *path_len, int64_t *makespan);

/*
 * Graph slicing in full (Alg. 1, Sec. 3.1.1): the K primary clusters exactly
 * as pardnn_slice_primaries finds them, then the secondary clusters. Past K
 * paths the weighted levels are no longer recomputed: with the priorities
 * w = tl + bl of the graph left after the K-th primary (every edge paying its
 * cost), each further path starts at the remaining node without a remaining
 * predecessor of largest w, steps to the remaining successor of largest w and
 * ends at a node without a remaining successor (a single node when the start
 * has none); ties in w go to the smaller node id. The path and its edges
 * leave the graph, and walks continue until no node remains.
 * Outputs (device, caller-allocated):
 *   cluster        int32[n_nodes]: cluster of each node; primaries 0..K-1,
 *                  secondaries K, K+1, ... in the order found.
 *   cluster_off    int32[n_nodes + K + 1]: cluster c holds
 *                  cluster_nodes[cluster_off[c] .. cluster_off[c+1]) (a
 *                  primary of an exhausted graph is empty).
 *   cluster_nodes  int32[n_nodes]: every cluster's nodes in path order.
 *   n_clusters     int32[1] (device): the number of clusters, K + secondaries.
 *   makespan       int64[K] or NULL: as for pardnn_slice_primaries.
 * The walk itself is sequential; it runs in one wave on the GPU (see the
 * design notes). Environment: PARDNN_PEEL_GLOBAL_MAPS=1 keeps the walk's bit
 * maps in device memory even when they fit in LDS (for testing).
 * Errors: E_INVAL (K < 0, null pointers), E_CYCLE, E_DEVICE. Syncs.
 */
int pardnn_slice_graph(pardnn_graph *g, int32_t K, int32_t *cluster, int32_t *cluster_off,
                       int32_t *cluster_nodes, int32_t *n_clusters, int64_t *makespan);

/* pardnn_evaluate_batch restricted to tl, bl and makespan. No sync. */
int pardnn_tb_levels_batch(pardnn_graph *g, int32_t n_place,
                           const int32_t *placements, int64_t *tl, int64_t *bl,
                           int64_t *makespan);

/*
 * Instrumentation (not part of the method): when enabled, the handle records
 * a pair of HIP events on its stream around the main kernel of each
 * pardnn_tb_levels, pardnn_evaluate_batch / pardnn_tb_levels_batch and
 * pardnn_levelize call. pardnn_get_timing waits for the last recorded pair and
 * returns its elapsed time in milliseconds and the kernel's name (a static
 * string). Errors: E_INVAL if nothing was recorded yet. Independently of
 * this switch, the same spots push roctx ranges named for those kernels, which
 * a profiler's marker trace shows.
 */
int pardnn_set_timing(pardnn_graph *g, int enable);
int pardnn_get_timing(pardnn_graph *g, const char **kernel, float *ms);

/*
 * Deferred errors, for callers that keep the GPU busy with back-to-back calls
 * (the refinement loop): with enable != 0, the calls that would wait for the
 * stream to report an argument error found on the device (label or node id
 * out of range, negative capacity, bad node kind or cluster id, step_ptr not
 * matching n_moves; those marked "syncs") return PARDNN_OK once their work
 * is enqueued, and the error flags accumulate on the device. Host-side checks
 * still fail at once. pardnn_take_errors waits for the handle's stream,
 * returns E_INVAL if a call made since the last take found such an error
 * (detail: the flags; results of those calls are unspecified) and clears
 * them; PARDNN_OK otherwise. With errors not deferred (the default) every
 * call reports its own, and pardnn_take_errors only waits for the stream.
 * Switching the mode clears the flags.
 */
int pardnn_set_deferred_errors(pardnn_graph *g, int enable);
int pardnn_take_errors(pardnn_graph *g);

/* Static text for a status code. */
const char *pardnn_status_string(int status);

/* Detail of the last failing call on this host thread ("" if none). */
const char *pardnn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PARDNN_H */
