// Host-side plan lowering: a batch of queries (structure ids + the layout of
// the caller's anchor / relation arrays) -> the row layout and index lists
// that the device stages consume.
//
// The paper's Graph Capturer (Eq. 2) maps each query to a computation graph
// whose operator nodes are projections, intersections, unions and
// negations, and its Operator Fuser groups them horizontally (a projection
// chain on one path), vertically (an intersection or union across paths)
// or both. Here that grouping is fixed per structure and per batch:
//   - every branch of every query is one "chain" row; all chains of the batch
//     run in one stage (GQE / Query2Box: one kernel; BetaE: one MLP pass per
//     hop level across all chains that reach that level);
//   - every intersection of the batch runs in one stage (all groups at once),
//     with negation folded into the intersection inputs;
//   - a union keeps its two branches as separate scored rows and the scorer
//     takes the max (disjunctive normal form, Eq. 1);
//   - scoring and top-k run once over all scored rows of the batch.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

namespace kgq {

struct BranchDef {
    int anchor;      // anchor slot
    int n_hops;      // projections on this branch (1..3)
    int rel[3];      // relation slots in hop order
    bool negated;    // BetaE: negated before the intersection
};

enum MergeKind { MERGE_NONE = 0, MERGE_AND = 1, MERGE_OR = 2 };

struct StructureDef {
    const char* name;
    int n_anchors, n_relations;
    int n_branches;
    BranchDef br[3];
    int merge;
    int post_rel;    // relation slot projected after the intersection, or -1
    bool negation;   // uses negation (BetaE only)
};

const StructureDef* structure_def(int id);   // nullptr if out of range
constexpr int kNumStructures = 14;

struct Plan {
    int model = 0, B = 0;
    // chains (rows 0 .. n_chain-1 of the state buffer)
    int n_chain = 0;
    std::vector<int32_t> chain_anchor_ref;   // [n_chain]  index into anchors[]
    std::vector<int32_t> chain_rel_ref;      // [n_chain * 3], -1 = no hop
    // intersection groups; inputs are chain rows in_start .. in_start+n-1
    int n_groups = 0, n_int_in = 0;
    std::vector<int32_t> g_in_start, g_n, g_out, g_post, g_neg;
    // BetaE projection levels: 0,1,2 = hop levels, 3 = after the intersection
    std::vector<int32_t> lv_src[4], lv_anchor[4], lv_rel[4], lv_dst[4];
    // scoring: rows [0, n_union_rows) are union pairs, then single rows
    int n_score_rows = 0, n_union_rows = 0;
    std::vector<int32_t> score_src;          // state row of each scored row
    std::vector<int32_t> out_dest;           // query index of each output
    std::vector<int32_t> arity;              // [2B] (mixed batches)
    int n_state_rows = 0;

    // Flattened device image: every list above at a fixed offset.
    std::vector<int32_t> image;
    struct Off {
        int64_t chain_anchor, chain_rel, g_in_start, g_n, g_out, g_post, g_neg;
        int64_t lv_src[4], lv_anchor[4], lv_rel[4], lv_dst[4];
        int64_t score_src, out_dest, arity;
    } off{};
};

// Lower a batch. sid(q) gives query q's structure; anchors of query q sit at
// q * a_stride + slot, relations at q * r_stride + slot. Returns false (with
// a message) for an unknown structure or a negation structure on a model
// without negation.
bool lower(int model, int B, const int32_t* sid, int fixed_sid, int a_stride, int r_stride,
           bool mixed, Plan& out, std::string& err, int& err_status);

// Upper bound on the image size (int32 words) for a batch of B queries.
int64_t plan_image_words(int B);

// Rows of the state buffer needed per query, at most.
constexpr int kStateRowsPerQuery = 8;

// Number of kernel launches one execute of this plan makes (without the
// checked-mode validation).
int plan_launches(const Plan& p, bool topk);

}  // namespace kgq
