// records.h -- the records and argument block the sweep kernels read:
// per-level bounds, 16-byte edge and node records, the near / far split of
// the batched sweeps and the sweep arguments. Kept apart from the host-side
// declarations so that the kernels' sources change only when these do.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace pardnn {

struct LevelInfo {
    int32_t node_lo;   // first lm node of the level
    int32_t in_e_lo;   // first CSC edge of the level
    int32_t out_e_lo;  // first CSR edge of the level
    int32_t pad;
};

// Level-major edge record of one sweep direction: the neighbour whose value
// is gathered, the node the candidate is folded into, and the edge cost.
struct alignas(16) EdgeRec16 {
    int32_t nb;
    int32_t own;
    int64_t cost;
};

// Batched sweeps: per level and direction, the first node and the first
// near / far edge record (entries L and L + 1 hold the totals), and how many
// of the level's far records read the workspace (kNoRing); those come first
// among the level's far records.
struct alignas(16) PairLevel {
    int32_t node_lo, near_lo, far_lo, n_gather;
};
// The cost word of the batched sweeps' edge records: in the t direction the
// edge cost; in the b direction the cost with the successor tie-break below
// it, (cost << ob) | (2^ob - 1 - successor's original id), so that a b key
// is (value << ob) plus this word (labels differ) or its low ob bits (same
// label). It fits whenever the packed keys are used: their condition bounds
// every cost by 2^(62 - ob).
// A span-1 edge: the cost word (as two 32-bit halves, so that the records
// pack at a twelve-byte stride and a level's records span fewer cache lines;
// one load instruction reads a record) and the owner's and neighbour's index
// inside their levels (own | nb << 16).
struct NearRec12 {
    uint32_t ck_lo, ck_hi;
    uint32_t ol;
};
static_assert(sizeof(NearRec12) == 12, "twelve-byte span-1 records");
// A longer edge: the cost word, the owner's index inside its level and where
// the sweep finds the neighbour's value (own | ring << 16), and the neighbour
// (level-major id). The cost word comes first: a load of the first twelve
// bytes (the neighbour unused) keeps it in an aligned register pair. `ring` indexes the LDS entries of the chain: below
// kLongBase the ring of recent levels, from kLongBase on the bulk buffers of
// long edges (see kLongBlock); kNoRing: gathered from the workspace level by
// level; kPreFolded: folded by the general path of the neighbour's level,
// which is too wide for the ring.
struct alignas(16) FarRec16 {
    int64_t ck;
    uint32_t ol;
    int32_t nb;
};
constexpr uint32_t kNoRing = 0xffffu;
constexpr uint32_t kPreFolded = 0xfffeu;
// Long edges of the batched sweeps. The steps of a chain fall into blocks of
// kLongBlock; an edge whose neighbour finished at least kLongLead steps before
// its owner's block begins is long. Per block, the distinct neighbours of its
// long edges (at most kLongCap, in level-major order) are listed once; the
// chain gathers them in 64-lane chunks, one chunk per step, into one of two
// LDS buffers ahead of the block, so that neighbours shared by nearby levels
// cost one gather and neighbours on one cache line one line. The list holds
// kLongCap entries per block (0 past its distinct neighbours) and three
// blocks of padding past the last.
constexpr int kLongBlock = 8;
constexpr int kLongCap = 512;
constexpr int kLongLead = 12;
constexpr uint32_t kLongBase = 256;   // LDS ring entries before the bulk buffers
inline int64_t long_list_elems(int32_t L) {
    return ((int64_t)(L + kLongBlock - 1) / kLongBlock + 3) * kLongCap;
}
// An edge folded early by the general path of its neighbour's (wide) level:
// the neighbour, the owner's index in its level and the span (own | span << 16)
// and the cost; grouped by the neighbour's level (pre_off).
struct alignas(16) PreRec16 {
    int32_t nb;
    uint32_t os;
    int64_t cost;
};

// Bits that hold a node id in the b-direction keys: 2^bits > V.
inline int32_t succ_bits(int32_t V) {
    int32_t b = 1;
    while ((1ll << b) <= (int64_t)V) b++;
    return b;
}

// Per-node constants of the sweeps, level-major.
struct alignas(16) NodeRec16 {
    int64_t comp;
    int64_t mem;
};


// Sweep kernels: per-label memory bins live in LDS while labels x slots fit
// kBinsCap; level boundaries are staged in LDS kLevelWindow levels at a time.
constexpr int kBinsCap = 512;
constexpr int kLevelWindow = 128;
// Placements per chain of the batched evaluation (slice of the workspace),
// and padding nodes per slice of ftl / bll / nx_w.
constexpr int kBatchSlots = 2;
// labels below this bound fit the pair sweep's packed keys
constexpr uint32_t kPackLabels = 1u << 16;
constexpr int kSlicePad = 64;

struct SweepArgs {
    int32_t V, L, P, K;     // nodes, levels, placements, labels (K = 0: no label sums)
    int64_t E;
    int32_t lb;             // > 0: {value, label} packed as (value << lb) | label
    int32_t ob;             // with lb > 0: b keys are (value << ob) | (2^ob - 1 - successor id)
    const LevelInfo *linfo;
    const int32_t *in_off, *in_src, *in_dst;
    const int64_t *in_cost;
    const int32_t *out_off, *out_src, *out_dst, *out_dst_orig;
    const int64_t *out_cost;
    const int64_t *comp_lm, *mem_lm;
    const EdgeRec16 *in_rec, *out_rec;   // t: {src, dst, cost} by dst; b: {dst, src, cost} by src
    const NodeRec16 *node_rec;
    const int32_t *order;   // level-major -> original id
    const int32_t *level;   // original id -> level
    const int32_t *level_ptr;  // first level-major node of each level
    const int32_t *rank;    // original id -> level-major, [V + 1] with rank[V] = -1
    const int32_t *lab_w;   // [slice][V][S] labels in level-major order
    int64_t lab_stride;     // elements of lab_w per slice (>= V * S)
    int64_t *ftl, *bll;     // [slice][V][S] {value, label}: tl + comp, bl (packed or pairs)
    int32_t *nx_w;          // [slice][V][S] original id of the chosen successor (-1: none), or null
    int64_t ws_stride;      // elements of ftl / bll / nx_w per slice (>= V * S)
    const PairLevel *pl_t, *pl_b;         // batched sweeps: near / far split per level
    const NearRec12 *nr_t, *nr_b;
    const FarRec16 *fr_t, *fr_b;
    const int32_t *lsrc_t, *lsrc_b;       // long edges' neighbours per block (long_list_elems)
    const int32_t *preoff_t, *preoff_b;   // [L + 1] per neighbour level
    const PreRec16 *pre_t, *pre_b;
    const int32_t *pretie_b;
    int64_t *tl_out, *bl_out, *makespan;  // [V][P], [V][P], [P], caller's numbering
    int32_t *start;         // [P] level-major id where the critical path starts, or null
    int64_t *label_mem;     // [P][K], zeroed by the caller, or null
    int32_t *err;           // device error word
    // set: the launch runs only if *gate == gate_want (two alternative paths
    // enqueued together, chosen on the device without a host round trip)
    const int32_t *gate;
    int32_t gate_want;
    // Segmented chains (one placement per chain, seg_on = 1): the t chain
    // walks steps [seg_t0, seg_t1), the b chain [seg_b0, seg_b1); a segment
    // that does not start at step 0 takes the general path for its first
    // levels (its LDS state starts empty), and the makespan is left to a
    // separate pass. seg_on = 0: both chains walk every step.
    int32_t seg_on;
    int32_t seg_t0, seg_t1, seg_b0, seg_b1;
    // Batched pair sweep with successor links (nx_w given): 1 = the links
    // ride in the b values instead of nx_w, each b value being
    // (((bl << ob) | (2^ob - 1 - successor id, 0: none)) << lb) | label, which
    // needs values below 2^(62 - ob - lb); 0 = plain packed b values.
    int32_t nxf;
    // 1: lab_w holds 16-bit labels (unsigned; lab_stride counts 16-bit
    // elements), so a node's two labels of a slice are one 32-bit word. The
    // batched pair sweep takes them (labels checked below 2^lb <= 2^16 as
    // they were written); every other sweep reads 32-bit labels.
    int32_t lab16;
};

}  // namespace pardnn
