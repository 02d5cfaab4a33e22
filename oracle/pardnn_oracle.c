/*
 * pardnn_oracle.c -- sequential CPU oracle for placement-aware critical-path
 * evaluation of a weighted DAG (ParDNN, arXiv 2008.08636).
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT. Only the tests, the smoke
 * check and the CPU-baseline leg of the benchmark load this library. The HIP
 * library never links, loads or calls it, and the two share no code, header,
 * table or helper.
 *
 * Every routine is the plain textbook definition, written for reading rather
 * than speed: one thread, one pass, no blocking and no reordering.
 *
 * Definitions (paper, Sec. 3 Table 2 "Terminology"):
 *   - G = (V, E) is the computational DAG (Sec. 2).
 *   - comp(n) is the node weight, mem(n) its output memory, comm(e) the cost
 *     of an edge.
 *   - The length of a path is the sum of comp over its nodes plus the sum of
 *     comm over its edges.
 *   - tl(n) is the length of the costliest path from a source to n,
 *     EXCLUDING n; bl(n) is the length of the costliest path from n to a sink,
 *     INCLUDING n; w_lvl(n) = tl(n) + bl(n).
 *   - CP is the costliest path of the graph; its length is the makespan M.
 *   - Communication between two nodes on the same device label counts as
 *     zero (Fig. 2 caption; Sec. 3.1.2, cluster criticality).
 *   - compute_weighted_levels is one pass in topological order, costing
 *     O(|V| + |E|) (Sec. 3.1.1, complexity of Alg. 1).
 *
 * Readings where the paper is silent (each is also listed in the design
 * notes of the repository):
 *   - The artificial source and sink of Sec. 3 are implicit: a node with no
 *     predecessor has tl = 0 and a node with no successor has bl = comp. This
 *     equals adding a zero-weight source and sink joined by zero-cost edges.
 *   - The level of a node is its hop depth: 0 without predecessors, else
 *     1 + the largest level among its predecessors (the Kahn frontier index).
 *   - Within a level, nodes are ordered by ascending id.
 *   - Among several critical paths the canonical one is the lexicographically
 *     smallest node-id sequence: start at the smallest-id critical source and
 *     repeatedly step to the smallest-id successor s with
 *     tl(u) + comp(u) + c(u,s) + bl(s) == M, until a node without successors.
 *   - Memory per label is the static sum of mem over the nodes carrying that
 *     label; overflow = max(0, sum - capacity). The caller applies the 10 %
 *     reserve of Sec. 4 to the capacity it passes.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "pardnn_oracle.h"

/* ------------------------------------------------------------------------ */
/* Argument checks (shared by every entry point of the oracle).             */
/* ------------------------------------------------------------------------ */

static int check_graph(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                       const int32_t *dst)
{
    if (n_nodes < 0 || n_edges < 0 || n_edges > (int64_t)INT32_MAX)
        return ORC_E_INVAL;
    if (n_edges > 0 && (src == NULL || dst == NULL))
        return ORC_E_INVAL;
    for (int64_t e = 0; e < n_edges; e++) {
        if (src[e] < 0 || src[e] >= n_nodes || dst[e] < 0 || dst[e] >= n_nodes)
            return ORC_E_INVAL;
    }
    return ORC_OK;
}

int orc_validate(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                 const int32_t *dst, const int64_t *comp,
                 const int64_t *edge_cost, const int64_t *mem)
{
    int st = check_graph(n_nodes, n_edges, src, dst);
    if (st != ORC_OK)
        return st;
    if (n_nodes > 0 && (comp == NULL || mem == NULL))
        return ORC_E_INVAL;
    if (n_edges > 0 && edge_cost == NULL)
        return ORC_E_INVAL;
    /* Weights are profiled times and sizes, hence never negative. */
    for (int32_t v = 0; v < n_nodes; v++)
        if (comp[v] < 0 || mem[v] < 0)
            return ORC_E_INVAL;
    for (int64_t e = 0; e < n_edges; e++)
        if (edge_cost[e] < 0)
            return ORC_E_INVAL;
    /* Every path length is bounded by sum(comp) + sum(cost); requiring that
     * bound to fit in int64 rules out overflow anywhere below. */
    int64_t total = 0;
    for (int32_t v = 0; v < n_nodes; v++) {
        if (comp[v] > INT64_MAX - total)
            return ORC_E_OVERFLOW;
        total += comp[v];
    }
    for (int64_t e = 0; e < n_edges; e++) {
        if (edge_cost[e] > INT64_MAX - total)
            return ORC_E_OVERFLOW;
        total += edge_cost[e];
    }
    int64_t mtotal = 0;
    for (int32_t v = 0; v < n_nodes; v++) {
        if (mem[v] > INT64_MAX - mtotal)
            return ORC_E_OVERFLOW;
        mtotal += mem[v];
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Adjacency lists by counting sort: row v of `off/eid` lists, in edge-id   */
/* order, the edges e with key[e] == v (key = src: out-edges; dst: in).     */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t *off; /* [n_nodes + 1] */
    int64_t *eid; /* [n_edges]     */
} adj_t;

static void adj_free(adj_t *a)
{
    free(a->off);
    free(a->eid);
    a->off = NULL;
    a->eid = NULL;
}

static int adj_build(int32_t n_nodes, int64_t n_edges, const int32_t *key,
                     adj_t *a)
{
    a->off = (int64_t *)calloc((size_t)n_nodes + 1, sizeof(int64_t));
    a->eid = (int64_t *)malloc(((size_t)n_edges + 1) * sizeof(int64_t));
    int64_t *cursor = (int64_t *)malloc(((size_t)n_nodes + 1) * sizeof(int64_t));
    if (a->off == NULL || a->eid == NULL || cursor == NULL) {
        free(cursor);
        adj_free(a);
        return ORC_E_NOMEM;
    }
    for (int64_t e = 0; e < n_edges; e++)
        a->off[key[e] + 1]++;
    for (int32_t v = 0; v < n_nodes; v++)
        a->off[v + 1] += a->off[v];
    memcpy(cursor, a->off, ((size_t)n_nodes + 1) * sizeof(int64_t));
    for (int64_t e = 0; e < n_edges; e++)
        a->eid[cursor[key[e]]++] = e;
    free(cursor);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Topological order by Kahn's algorithm with a FIFO queue seeded with the  */
/* sources in ascending id. Fails with ORC_E_CYCLE when some node is never  */
/* released (a cycle or a self-loop).                                       */
/* ------------------------------------------------------------------------ */

static int topo_order(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                      const int32_t *dst, const adj_t *out, int32_t *topo)
{
    int64_t *indeg = (int64_t *)calloc((size_t)n_nodes + 1, sizeof(int64_t));
    if (indeg == NULL)
        return ORC_E_NOMEM;
    for (int64_t e = 0; e < n_edges; e++)
        indeg[dst[e]]++;
    int64_t head = 0, tail = 0;
    for (int32_t v = 0; v < n_nodes; v++)
        if (indeg[v] == 0)
            topo[tail++] = v;
    while (head < tail) {
        int32_t u = topo[head++];
        for (int64_t i = out->off[u]; i < out->off[u + 1]; i++) {
            int32_t s = dst[out->eid[i]];
            if (--indeg[s] == 0)
                topo[tail++] = s;
        }
    }
    (void)src;
    free(indeg);
    return tail == n_nodes ? ORC_OK : ORC_E_CYCLE;
}

/* ------------------------------------------------------------------------ */
/* Levels: level(v) = 0 without predecessors, else 1 + max level of preds.  */
/* order = node ids sorted by (level, id); level_ptr[l] = first position of */
/* level l in order, level_ptr[n_levels] = n_nodes.                         */
/* ------------------------------------------------------------------------ */

int orc_levelize(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                 const int32_t *dst, int32_t *level, int32_t *order,
                 int32_t *level_ptr, int32_t *n_levels)
{
    int st = check_graph(n_nodes, n_edges, src, dst);
    if (st != ORC_OK)
        return st;
    adj_t out = {0, 0};
    st = adj_build(n_nodes, n_edges, src, &out);
    if (st != ORC_OK)
        return st;
    int32_t *topo = (int32_t *)malloc(((size_t)n_nodes + 1) * sizeof(int32_t));
    if (topo == NULL) {
        adj_free(&out);
        return ORC_E_NOMEM;
    }
    st = topo_order(n_nodes, n_edges, src, dst, &out, topo);
    if (st == ORC_OK) {
        for (int32_t v = 0; v < n_nodes; v++)
            level[v] = 0;
        /* Predecessors precede their successors in topo, so level(u) is
         * final when u is visited. */
        for (int32_t i = 0; i < n_nodes; i++) {
            int32_t u = topo[i];
            for (int64_t j = out.off[u]; j < out.off[u + 1]; j++) {
                int32_t s = dst[out.eid[j]];
                if (level[u] + 1 > level[s])
                    level[s] = level[u] + 1;
            }
        }
        int32_t nl = 0;
        for (int32_t v = 0; v < n_nodes; v++)
            if (level[v] + 1 > nl)
                nl = level[v] + 1;
        /* Stable counting sort by level keeps ascending id within a level. */
        for (int32_t l = 0; l <= nl; l++)
            level_ptr[l] = 0;
        for (int32_t v = 0; v < n_nodes; v++)
            level_ptr[level[v] + 1]++;
        for (int32_t l = 0; l < nl; l++)
            level_ptr[l + 1] += level_ptr[l];
        int32_t *cursor = (int32_t *)malloc(((size_t)nl + 1) * sizeof(int32_t));
        if (cursor == NULL) {
            st = ORC_E_NOMEM;
        } else {
            memcpy(cursor, level_ptr, ((size_t)nl + 1) * sizeof(int32_t));
            for (int32_t v = 0; v < n_nodes; v++)
                order[cursor[level[v]]++] = v;
            free(cursor);
            *n_levels = nl;
        }
    }
    free(topo);
    adj_free(&out);
    return st;
}

/* Communication cost of edge e under a placement: zero inside a label. */
static int64_t comm_cost(const int32_t *label, const int32_t *src,
                         const int32_t *dst, const int64_t *edge_cost,
                         int64_t e)
{
    return label[src[e]] == label[dst[e]] ? 0 : edge_cost[e];
}

/* ------------------------------------------------------------------------ */
/* t-level, b-level and makespan under a placement.                        */
/*   tl(v) = max over edges (u,v) of tl(u) + comp(u) + c(u,v); 0 if none.  */
/*   bl(v) = comp(v) + max over edges (v,s) of c(v,s) + bl(s); comp(v) if  */
/*           none.                                                         */
/*   M     = max over v of tl(v) + bl(v); 0 for an empty graph.            */
/* ------------------------------------------------------------------------ */

int orc_tb_levels(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                  const int32_t *dst, const int64_t *comp,
                  const int64_t *edge_cost, const int32_t *label, int64_t *tl,
                  int64_t *bl, int64_t *makespan)
{
    int st = check_graph(n_nodes, n_edges, src, dst);
    if (st != ORC_OK)
        return st;
    adj_t out = {0, 0}, in = {0, 0};
    st = adj_build(n_nodes, n_edges, src, &out);
    if (st == ORC_OK)
        st = adj_build(n_nodes, n_edges, dst, &in);
    int32_t *topo = (int32_t *)malloc(((size_t)n_nodes + 1) * sizeof(int32_t));
    if (topo == NULL && st == ORC_OK)
        st = ORC_E_NOMEM;
    if (st == ORC_OK)
        st = topo_order(n_nodes, n_edges, src, dst, &out, topo);
    if (st == ORC_OK) {
        for (int32_t i = 0; i < n_nodes; i++) {
            int32_t v = topo[i];
            int64_t best = 0;
            for (int64_t j = in.off[v]; j < in.off[v + 1]; j++) {
                int64_t e = in.eid[j];
                int32_t u = src[e];
                int64_t cand = tl[u] + comp[u] + comm_cost(label, src, dst, edge_cost, e);
                if (cand > best)
                    best = cand;
            }
            tl[v] = best;
        }
        for (int32_t i = n_nodes - 1; i >= 0; i--) {
            int32_t v = topo[i];
            int64_t best = 0;
            for (int64_t j = out.off[v]; j < out.off[v + 1]; j++) {
                int64_t e = out.eid[j];
                int32_t s = dst[e];
                int64_t cand = comm_cost(label, src, dst, edge_cost, e) + bl[s];
                if (cand > best)
                    best = cand;
            }
            bl[v] = comp[v] + best;
        }
        int64_t m = 0;
        for (int32_t v = 0; v < n_nodes; v++)
            if (tl[v] + bl[v] > m)
                m = tl[v] + bl[v];
        *makespan = m;
    }
    free(topo);
    adj_free(&out);
    adj_free(&in);
    return st;
}

/* ------------------------------------------------------------------------ */
/* Critical nodes and the canonical critical path.                          */
/*   crit(v) = (tl(v) + bl(v) == M).                                       */
/*   The path starts at the smallest-id node without predecessors that is  */
/*   critical, and from u steps to the smallest-id successor s with        */
/*   tl(u) + comp(u) + c(u,s) + bl(s) == M, stopping at a node without     */
/*   successors (or, for inconsistent inputs, without a tight successor).  */
/* ------------------------------------------------------------------------ */

int orc_critical_path(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                      const int32_t *dst, const int64_t *comp,
                      const int64_t *edge_cost, const int32_t *label,
                      const int64_t *tl, const int64_t *bl, int64_t makespan,
                      uint8_t *is_critical, int32_t *path, int32_t *path_len)
{
    int st = check_graph(n_nodes, n_edges, src, dst);
    if (st != ORC_OK)
        return st;
    adj_t out = {0, 0};
    st = adj_build(n_nodes, n_edges, src, &out);
    if (st != ORC_OK)
        return st;
    int32_t *topo = (int32_t *)malloc(((size_t)n_nodes + 1) * sizeof(int32_t));
    int64_t *indeg = (int64_t *)calloc((size_t)n_nodes + 1, sizeof(int64_t));
    if (topo == NULL || indeg == NULL)
        st = ORC_E_NOMEM;
    if (st == ORC_OK)
        st = topo_order(n_nodes, n_edges, src, dst, &out, topo);
    if (st == ORC_OK) {
        for (int64_t e = 0; e < n_edges; e++)
            indeg[dst[e]]++;
        for (int32_t v = 0; v < n_nodes; v++)
            is_critical[v] = (uint8_t)(tl[v] + bl[v] == makespan);
        int32_t start = -1;
        for (int32_t v = 0; v < n_nodes; v++) {
            if (indeg[v] == 0 && is_critical[v]) {
                start = v;
                break;
            }
        }
        int32_t len = 0;
        int32_t u = start;
        while (u >= 0) {
            path[len++] = u;
            int32_t next = -1;
            for (int64_t j = out.off[u]; j < out.off[u + 1]; j++) {
                int64_t e = out.eid[j];
                int32_t s = dst[e];
                int64_t through = tl[u] + comp[u] +
                                  comm_cost(label, src, dst, edge_cost, e) + bl[s];
                if (through == makespan && (next < 0 || s < next))
                    next = s;
            }
            u = next;
        }
        *path_len = len;
    }
    free(indeg);
    free(topo);
    adj_free(&out);
    return st;
}

/* ------------------------------------------------------------------------ */
/* Memory per device label (the per-partition totals of Memory Heuristic    */
/* II, Sec. 3.2, without the residual/normal split):                        */
/*   sum[k] = sum of mem(v) over v with label(v) == k                       */
/*   overflow[k] = max(0, sum[k] - capacity[k])                             */
/* ------------------------------------------------------------------------ */

int orc_label_memory(int32_t n_nodes, const int64_t *mem, const int32_t *label,
                     int32_t n_labels, const int64_t *capacity,
                     int64_t *label_mem, int64_t *overflow)
{
    if (n_nodes < 0 || n_labels < 0 || (n_nodes > 0 && n_labels == 0))
        return ORC_E_INVAL;
    for (int32_t v = 0; v < n_nodes; v++)
        if (label[v] < 0 || label[v] >= n_labels)
            return ORC_E_INVAL;
    if (capacity != NULL)
        for (int32_t k = 0; k < n_labels; k++)
            if (capacity[k] < 0)
                return ORC_E_INVAL;
    for (int32_t k = 0; k < n_labels; k++)
        label_mem[k] = 0;
    for (int32_t v = 0; v < n_nodes; v++)
        label_mem[label[v]] += mem[v];
    if (overflow != NULL) {
        for (int32_t k = 0; k < n_labels; k++) {
            int64_t cap = capacity != NULL ? capacity[k] : INT64_MAX;
            overflow[k] = label_mem[k] > cap ? label_mem[k] - cap : 0;
        }
    }
    return ORC_OK;
}
