// internal.h -- private declarations of the gfx950 evaluator library.
//
// Device data layout (all owned by the handle):
//   original numbering (caller's ids):
//     e_src, e_dst int32[E], e_cost int64[E]        edge list copy
//     comp, mem int64[V], indeg, outdeg int32[V]
//     o_off int32[V+1], o_nbr int32[E]              out-adjacency (Kahn)
//   level-major numbering ("lm": nodes sorted by (level, id)):
//     order int32[V] lm -> original id, rank int32[V + 1] original -> lm (rank[V] = -1)
//     level int32[V] (original ids), level_ptr int32[L+1]
//     linfo LevelInfo[L+1]: first node, first in-edge, first out-edge of
//       each level (entry L holds the totals)
//     CSC (in-edges, grouped by destination):  in_off[V+1], in_src, in_dst,
//       in_cost -- the in-edges of one level are one contiguous range
//     CSR (out-edges, grouped by source):      out_off[V+1], out_src,
//       out_dst, out_dst_orig (original id of the destination), out_cost
//     comp_lm, mem_lm int64[V]
//     in_rec, out_rec EdgeRec16[E] and node_rec NodeRec16[V]: the same data
//       as 16-byte records, so a sweep task loads its edge with one load
//     pl_t / pl_b PairLevel[L+2], nr_t / nr_b NearRec12[], fr_t / fr_b
//       FarRec16[]: the edges of each level split into span-1
//       ("near") and longer ("far") edges for the batched sweeps, per
//       direction; built on first use
//   linfo has L + 2 entries: entry L + 1 repeats entry L, so the pair
//   (linfo[x], linfo[x + 1]) of an empty level can be read at x = L.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "pardnn.h"
#include "records.h"

namespace pardnn {

struct ValidateAcc {
    unsigned long long flags;    // bit 0: id out of range, bit 1: negative weight
    unsigned long long w_lo, w_hi;  // sum(comp) + sum(edge_cost), split at bit 32
    unsigned long long m_lo, m_hi;  // sum(mem), split at bit 32
};

// Nodes in (tl, id) order for the span-work tables, with the tl they were
// sorted by (device arrays of the handle; valid once built).
struct SpanCache {
    int64_t *tl = nullptr;       // [V] the tl of the cached order
    int32_t *ids = nullptr;      // [V] node ids in (tl, id) order
    int32_t *changed = nullptr;  // [1] set on the device when a call's tl differs
    bool valid = false;
};

// One item of a segmented single-placement sweep, per direction: a run of
// chain steps [a, b) or one wide level a computed grid-wide (kind 1).
struct SegItem {
    int32_t kind, a, b;
};

struct Graph {
    int device = 0;
    size_t lds_max = 65536;   // LDS bytes a workgroup may use on the device
    hipStream_t stream = nullptr;
    int32_t V = 0;
    int64_t E = 0;
    int64_t weight_bound = 0;   // sum(comp) + sum(edge_cost): bounds every path length

    int32_t *e_src = nullptr, *e_dst = nullptr;
    int64_t *e_cost = nullptr;
    int64_t *comp = nullptr, *mem = nullptr;
    int32_t *indeg = nullptr, *outdeg = nullptr;
    int32_t *o_off = nullptr, *o_nbr = nullptr;

    bool levelized = false;
    int32_t L = -1, max_width = -1;
    int32_t *level = nullptr, *order = nullptr, *rank = nullptr, *level_ptr = nullptr;
    LevelInfo *linfo = nullptr;
    std::vector<int32_t> h_level_ptr;
    int32_t *in_off = nullptr, *in_src = nullptr, *in_dst = nullptr;
    int64_t *in_cost = nullptr;
    int32_t *out_off = nullptr, *out_src = nullptr, *out_dst = nullptr, *out_dst_orig = nullptr;
    int64_t *out_cost = nullptr;
    int64_t *comp_lm = nullptr, *mem_lm = nullptr;
    EdgeRec16 *in_rec = nullptr, *out_rec = nullptr;
    NodeRec16 *node_rec = nullptr;
    PairLevel *pl_t = nullptr, *pl_b = nullptr;   // built on first batched evaluation
    NearRec12 *nr_t = nullptr, *nr_b = nullptr;
    FarRec16 *fr_t = nullptr, *fr_b = nullptr;
    int32_t *lsrc_t = nullptr, *lsrc_b = nullptr;   // long edges' neighbours per block
    int32_t *preoff_t = nullptr, *preoff_b = nullptr;
    PreRec16 *pre_t = nullptr, *pre_b = nullptr;
    int32_t *pretie_b = nullptr;

    // single-placement scratch
    int32_t *lab_lm = nullptr, *next_lm = nullptr, *move_stamp = nullptr;
    // the path's list pass: flags, positions [V + 1], scan space, list [V], ok
    int32_t *cp_flag = nullptr, *cp_pos = nullptr, *cp_ws = nullptr, *cp_list = nullptr;
    int32_t *cp_ok = nullptr;
    uint8_t *crit_lm = nullptr;
    int64_t *ft_lm = nullptr, *bl_lm = nullptr;   // {value, label} pairs, 2 * V each
    // graph slicing scratch (allocated on first use): masked node weights,
    // remaining-node flags, an identity placement, tl / bl / flags, the start
    NodeRec16 *sl_node_rec = nullptr;
    int64_t *sl_comp = nullptr, *sl_tl = nullptr, *sl_bl = nullptr;
    uint8_t *sl_alive = nullptr, *sl_crit = nullptr;
    int32_t *sl_iota = nullptr, *sl_start = nullptr;
    int64_t *sl_m = nullptr;   // makespan of the evaluation after the last round
    // one placement through the batched pair sweep (two slots, one idle):
    // ftl, bll [V + pad][2] packed, labels [V][2]; allocated on first use
    int64_t *ps_ftl = nullptr, *ps_bll = nullptr;
    int32_t *ps_lab = nullptr, *ps_gate = nullptr;
    // segmented single sweeps: levels wider than seg_thresh nodes are computed
    // grid-wide; the plan per direction and the accumulators of one level
    int32_t seg_thresh = -1;
    std::vector<SegItem> seg_t, seg_b;
    std::vector<LevelInfo> h_linfo;   // host copy of linfo, taken with the first plan
    long long *ps_acc = nullptr;   // [2][max_width]
    SpanCache span_cache;
    // cluster criticality scratch: tl, bl, makespan
    int64_t *cl_tl = nullptr, *cl_bl = nullptr, *cl_m = nullptr;
    // sort and table scratch of the cluster and span calls (grown on demand)
    void *aux_scratch = nullptr;
    size_t aux_scratch_bytes = 0;
    int32_t *bt_fit = nullptr;       // device flag: a batch's labels fit the packed keys
    int32_t *err = nullptr;          // device error words [4]
    int32_t *h_err = nullptr;        // pinned host mirror [4]

    // batch workspace, grown on demand
    void *batch_ws = nullptr;
    size_t batch_ws_bytes = 0;

    // instrumentation: events around the main kernel of a call
    bool timing = false;
    bool defer_errors = false;   // argument errors found on the device: kept for pardnn_take_errors
    bool timed = false;
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    const char *timed_kernel = "";

    std::vector<void *> allocs;
};

// ---- status helpers (api.hip) ----
int fail(int status, const std::string &msg);

// ---- structure.hip ----
hipError_t launch_fill_i32(int32_t *p, int64_t n, int32_t value, hipStream_t s);
hipError_t launch_fill_i64(int64_t *p, int64_t n, int64_t value, hipStream_t s);
hipError_t launch_iota_i32(int32_t *p, int32_t n, hipStream_t s);   // p[i] = i
hipError_t launch_validate(const Graph &g, const int32_t *src, const int32_t *dst,
                           const int64_t *comp, const int64_t *cost, const int64_t *mem,
                           ValidateAcc *acc);
hipError_t launch_count_degrees(const Graph &g);
hipError_t launch_exclusive_scan(const int32_t *in, int32_t *out, int32_t n, int32_t *ws,
                                 hipStream_t s);
size_t scan_workspace_elems(int32_t n);
hipError_t launch_build_orig_csr(const Graph &g, int32_t *cursor);
hipError_t launch_build_lm(Graph &g, int32_t *deg_ws, int32_t *cursor_in, int32_t *cursor_out,
                           int32_t *scan_ws);

// ---- radix_sort.hip ----
// Stable LSD radix sort of (key, value) pairs on bits [begin_bit, end_bit) of
// the keys, 8 bits per pass; n < 2^31. The inputs are left unchanged. With
// `gate` given, every launch returns at once unless *gate != 0 (decided on the
// device). Scratch: sort_pairs_scratch_bytes(n, sizeof key) bytes.
size_t sort_pairs_scratch_bytes(int32_t n, int key_bytes);
hipError_t sort_pairs_u32(const uint32_t *keys_in, uint32_t *keys_out, const int32_t *vals_in,
                          int32_t *vals_out, int32_t n, int begin_bit, int end_bit,
                          void *scratch, hipStream_t s, const int32_t *gate = nullptr);
hipError_t sort_pairs_u64(const uint64_t *keys_in, uint64_t *keys_out, const int32_t *vals_in,
                          int32_t *vals_out, int32_t n, int begin_bit, int end_bit,
                          void *scratch, hipStream_t s, const int32_t *gate = nullptr);
// out[i] = in[0] + ... + in[i] (int64); scratch: inclusive_scan_i64_scratch_bytes(n)
size_t inclusive_scan_i64_scratch_bytes(int32_t n);
hipError_t inclusive_scan_i64(const int64_t *in, int64_t *out, int32_t n, void *scratch,
                              hipStream_t s);

// ---- levelize.hip ----
// levels, level_ptr and the release order (queue); result = {levels, released}
// rec_scratch: kahn_rec_bytes(V) bytes for the nodes' adjacency records
size_t kahn_rec_bytes(int32_t V);
hipError_t launch_kahn(const Graph &g, int32_t *indeg_work, int32_t *queue, int32_t *result,
                       void *rec_scratch);
// order = ids sorted by (level, id), levels below 2^bits
size_t level_order_scratch_bytes(int32_t V);
hipError_t launch_level_order(const Graph &g, int32_t bits, void *scratch);

// ---- sweep.hip ----
hipError_t launch_permute_labels(const Graph &g, const int32_t *placement, int32_t *lab_lm);
// K > 0: labels outside [0, K) set bit 0 of err. fit (if given): set to 0
// when a label lies outside [0, fit_limit). lab16 (S = 2): the labels are
// stored as 16 bits (lab_stride in 16-bit elements); the checks see the full
// values. gate (if given): the kernel returns at once unless *gate ==
// gate_want (read on the device).
hipError_t launch_permute_labels_batch(const Graph &g, const int32_t *placements, int32_t P,
                                       int32_t S, int32_t *lab_w, int64_t lab_stride,
                                       int32_t K = 0, int32_t *err = nullptr,
                                       int32_t *fit = nullptr, uint32_t fit_limit = kPackLabels,
                                       bool lab16 = false, const int32_t *gate = nullptr,
                                       int32_t gate_want = 0);
// flag = 1 if every label lies in [0, limit), else 0 (on the device)
hipError_t launch_label_fit(const Graph &g, const int32_t *labels, int32_t limit, int32_t *flag);
hipError_t launch_sweep(const SweepArgs &a, int32_t S, hipStream_t s);
// cbits: [P][ceil(V / 32)] bit words of the critical flags, scratch for the
// path walk (needed when path is given)
// alt (S = 2 only): a second, gated set of arguments whose emit pass is
// enqueued beside a's (the two sweeps of a device-side choice); the path pass
// runs once after both.
hipError_t launch_finish(const SweepArgs &a, int32_t S, uint8_t *crit, uint32_t *cbits,
                         int32_t *path, int32_t stride, int32_t *path_len, hipStream_t s,
                         const SweepArgs *alt = nullptr);

// ---- sweep_pair.hip ----
// flag[e] = 1 for the span-1 edges of the direction's level-major edge order
hipError_t launch_pair_flags(const Graph &g, bool fwd, int32_t *flag);
// near_rank = exclusive scan of flag (E + 1 entries); fills pl, nr, fr
hipError_t launch_pair_split(const Graph &g, bool fwd, const int32_t *near_rank, PairLevel *pl,
                             NearRec12 *nr, FarRec16 *fr);
// long edges of the pair sweep: fills lsrc (long_list_elems(L)) and points
// the far records of long edges at their LDS entries
hipError_t launch_long_blocks(const Graph &g, bool fwd, PairLevel *pl, FarRec16 *fr,
                              int32_t *lsrc);
// flag[e] = 1 for the edges a wide level folds early (neighbour-grouped order)
hipError_t launch_pre_flags(const Graph &g, bool fwd, int32_t *flag);
// rank = exclusive scan of those flags; fills preoff [L + 1], pre, pretie
hipError_t launch_pre_split(const Graph &g, bool fwd, const int32_t *rank, int32_t *preoff,
                            PreRec16 *pre, int32_t *pretie);
// Packed {value, label} only (a.lb > 0).
hipError_t launch_sweep_pair(const SweepArgs &a, hipStream_t s);
// The same with one placement per chain (workspace [P][V + pad], labels
// [P][V]), no label sums.
hipError_t launch_sweep_pair_one(const SweepArgs &a, hipStream_t s);
// One placement, segmented: the t level xt and the b level xb (-1: none)
// computed by grid-wide passes from the workspace (n_edges / n_nodes: their
// edges and nodes together; acc_t / acc_b: int64 per node of the level, all
// zero on entry, left zero); and the makespan over level 0 afterwards.
hipError_t launch_wide_level(const SweepArgs &a, int32_t xt, int32_t xb, int64_t n_edges,
                             int32_t n_nodes, long long *acc_t, long long *acc_b, hipStream_t s);
hipError_t launch_level0_makespan(const SweepArgs &a, hipStream_t s);

// ---- critpath.hip ----
// tight successors and critical flags of one placement (comp_lm: the node
// weights to use), then the walk from start_orig (device, INT32_MAX: none) or,
// when null, from the smallest-id critical node without predecessors
hipError_t launch_crit_next(const Graph &g, const int32_t *placement, const int64_t *comp_lm,
                            const int64_t *tl, const int64_t *bl, const int64_t *makespan,
                            uint8_t *is_critical);
hipError_t launch_chase_from(const Graph &g, const int32_t *start_orig, int32_t *path,
                             int32_t *path_len);
// ---- spanwork.hip ----
// Eq. 2 terms for C clusters against K partitions (see pardnn_span_work);
// err bit 0: cluster id outside [-1, C), bit 1: label outside [-1, K).
size_t span_work_scratch_bytes(int32_t V, int32_t C, int32_t K);
hipError_t launch_span_work(const Graph &g, const int32_t *label, int32_t K,
                            const int32_t *cluster, int32_t C, const int64_t *tl,
                            int64_t *span_lo, int64_t *span_hi, int64_t *work, int64_t *comm,
                            int32_t *choice, void *scratch, SpanCache *cache, int32_t *err);

// ---- clusters.hip ----
// scratch of launch_cluster_criticality for V nodes and n clusters
size_t cluster_sort_bytes(int32_t V, int32_t n);
// labels with the cluster ids' equality on every edge, in [0, L + n_multi):
// *lab (int32[V], original ids) and *n_multi (device) point into scratch
size_t cluster_relabel_bytes(int32_t V, int32_t C);
hipError_t launch_cluster_relabel(const Graph &g, const int32_t *cluster, int32_t C,
                                  int32_t *scratch, int32_t **lab, int32_t **n_multi);
// criticality[c] = tl(first) + sum of comp + bl(last) - comp(last) for a
// cluster whose nodes in (level, id) order form a path, else -1 (also when it
// has no node); order: cluster ids by (criticality desc, id asc); err bit 0:
// cluster id out of range
hipError_t launch_cluster_criticality(const Graph &g, const int32_t *cluster, int32_t n_clusters,
                                      const int64_t *tl, const int64_t *bl, int64_t *crit,
                                      int32_t *order, void *scratch, size_t scratch_bytes,
                                      int32_t *err);
// ---- slicing.hip ----
hipError_t launch_slice_init(const Graph &g, NodeRec16 *node_rec_s, int64_t *comp_lm_s,
                             uint8_t *alive_lm, int32_t *primary);
hipError_t launch_slice_makespan(const Graph &g, const uint8_t *alive_lm, const int64_t *tl,
                                const int64_t *bl, int64_t *makespan);
hipError_t launch_slice_start(const Graph &g, const uint8_t *alive_lm, int32_t *start);
hipError_t launch_slice_remove(const Graph &g, int32_t round, const int32_t *path,
                               const int32_t *path_len, int64_t big, NodeRec16 *node_rec_s,
                               int64_t *comp_lm_s, uint8_t *alive_lm, int32_t *primary);
// ---- peel.hip ----
size_t peel_scratch_bytes(int32_t V, int64_t E);
size_t peel_lds_bytes(int32_t V);
// The secondary clusters after K primaries (paths [K][stride], plen [K],
// device): with tl / bl of the remaining graph (original ids) and its
// remaining nodes alive_lm, fills cluster (secondaries K, K + 1, ...; the
// primaries' entries are already set), cl_off [n_clusters + 1], cl_nodes [V]
// (every cluster's nodes in path order) and n_clusters (device). lds_maps:
// the walk's bit maps in LDS (peel_lds_bytes(V) of it), else in scratch.
// err bit 0: the walk stopped early (inconsistent state; cannot happen).
hipError_t launch_slice_secondaries(const Graph &g, int32_t K, const int32_t *paths,
                                    int32_t stride, const int32_t *plen, const int64_t *tl,
                                    const int64_t *bl, const uint8_t *alive_lm, int32_t *cluster,
                                    int32_t *cl_off, int32_t *cl_nodes, int32_t *n_clusters,
                                    void *scratch, bool lds_maps, int32_t *err);
hipError_t launch_critical_path(const Graph &g, const int32_t *placement, const int64_t *tl,
                                const int64_t *bl, const int64_t *makespan,
                                uint8_t *is_critical, int32_t *path, int32_t *path_len);

// ---- labelmem.hip ----
hipError_t launch_label_memory(const Graph &g, const int32_t *placement, int32_t K,
                               const int64_t *capacity, int64_t *label_mem, int64_t *overflow,
                               int32_t *err);
hipError_t launch_overflow(int64_t n, int32_t K, const int64_t *capacity,
                           const int64_t *label_mem, int64_t *overflow, int32_t *err,
                           hipStream_t s);
hipError_t launch_apply_moves(const Graph &g, int32_t *placement, int32_t n, const int32_t *node,
                              const int32_t *label, int32_t *err);
hipError_t launch_build_placements(const Graph &g, const int32_t *base, int32_t P,
                                   const int64_t *step_ptr, int64_t M, const int32_t *node,
                                   const int32_t *label, int32_t *placements, int32_t *err);
// err bit of a step_ptr that does not start at 0, decreases somewhere or does
// not end at the number of moves the caller passed
constexpr int32_t kErrSteps = 8;
// checks step_ptr[0 .. P] against M moves (sets kErrSteps in *err)
hipError_t launch_check_steps(const int64_t *step_ptr, int32_t P, int64_t M, int32_t *err,
                              hipStream_t s);
// ---- heuristics.hip ----
// Memory Heuristic II sums, Eq. 6 and reference co-location for P placements
// [V][P]; err bits: 1 label out of range, 2 bad node kind, 4 bad reference target
hipError_t launch_mem_balance(const Graph &g, int32_t P, const int32_t *placements,
                              const int32_t *node_type, const int32_t *ref_target, int32_t K,
                              int64_t *res_mem, int64_t *nor_mem, uint8_t *balanced,
                              int64_t *misplaced, int32_t *err);

// int32 elements of the scratch launch_moves_to_slices needs for M moves
size_t moves_scratch_elems(int32_t V, int64_t M);
hipError_t launch_moves_to_slices(const Graph &g, const int32_t *base, int32_t P,
                                  const int64_t *step_ptr, int64_t M, const int32_t *node,
                                  const int32_t *label, int32_t S, int32_t *scratch,
                                  int32_t *lab_w, int64_t lab_stride, int32_t K, int32_t *err,
                                  int32_t *fit = nullptr, uint32_t fit_limit = kPackLabels,
                                  bool lab16 = false);
// The 32-bit labels again from the moves launch_moves_to_slices grouped in
// the same scratch (no checks), when *gate == gate_want on the device: the
// unpacked alternative of a call without label sums.
hipError_t launch_moves_write(const Graph &g, const int32_t *base, int32_t P, int64_t M,
                              int32_t S, int32_t *scratch, int32_t *lab_w, int64_t lab_stride,
                              const int32_t *gate, int32_t gate_want);

}  // namespace pardnn
