// Host-side compilation of query structures and lowering of batches.
//
// The paper's pipeline (Methodology, Fig. 2) maps a first-order query to a
// computation graph (Graph Capturer, Eq. 2), recognises the operator
// patterns in it (Pattern Recognizer) and fuses them (Operator Fuser,
// Algorithm 1: decide a strategy per operator, merge each group into one
// fused operator, rewrite the graph). Here:
//
//   capture     a structure is given as its graph (kgq_node list, or the
//               text form read by parse_graph); the 14 benchmark structures
//               are predefined graphs compiled the same way;
//   recognise   the graph is rewritten into disjunctive normal form (Eq. 1):
//               unions move to the top (projection and intersection
//               distribute over them; the negation of a union becomes the
//               intersection of the negations), and chains of negations
//               reduce to their parity;
//   fuse        each maximal run of projections on one path becomes one
//               chain (horizontal fusion); each intersection becomes one
//               group whose branches are combined in one pass (vertical
//               fusion); for GQE / Query2Box a projection run that follows
//               an intersection is folded into that intersection's combine
//               (hybrid fusion). Negations become flags on the edges that
//               read them (an intersection input, a projection source or
//               the answer).
//
// The result, a Program, is a list of fused operators with their schedule
// position: its intersection stage (one more than the deepest stage below
// it) and, for MLP projections (BetaE, ConE, LogicE), the position within the run of
// projections since the last stage. lower() then builds one plan for a
// whole batch, in which every fused operator kind at one schedule position
// runs as one launch across all queries, whatever their structures.
#pragma once

#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/kgq.h"

namespace kgq {

constexpr int kNumStructures = KGQ_NUM_STRUCTURES;   // built-in structure ids 0 .. 13
constexpr int kMaxTerms = KGQ_MAX_DISJUNCTS;          // conjunctive terms of a node's DNF
constexpr int kMaxBranches = 4;                       // inputs of one intersection
constexpr int kMaxSlots = KGQ_MAX_SLOTS;              // anchor slots, relation slots
constexpr int kMaxGraphNodes = KGQ_MAX_GRAPH_NODES;
constexpr int kMaxFusedOps = 256;                     // fused operators of one structure

enum OpKind { OP_CHAIN = 0, OP_PROJ = 1, OP_AND = 2 };

struct FusedOp {
    int kind = OP_CHAIN;
    // Schedule: CHAIN / PROJ take the stage of their source (0 for an
    // anchor); AND is stage 1 + the deepest stage among its inputs.
    int stage = 0;
    int hop = 0;                  // PROJ: 1 + hop of a PROJ source, else 1
    int src = -1;                 // CHAIN / PROJ: producing op, or -1 for an anchor
    int anchor = -1;              //   anchor slot when src < 0
    bool src_neg = false;         // PROJ: the source is read negated (BetaE, ConE, LogicE)
    std::vector<int> rels;        // CHAIN: relation slots in hop order; PROJ: one;
                                  // AND: relation slots of a folded post-chain (GQE / Query2Box)
    std::vector<int> in;          // AND: input ops, in the graph's order
    std::vector<char> in_neg;     // AND: inputs read negated (BetaE, ConE, LogicE)
};

struct Program {
    std::string name;
    int n_anchors = 0, n_relations = 0;
    bool negation = false;        // uses negation (BetaE, ConE, LogicE only)
    bool supported = true;        // false: a built-in structure this model cannot run
    std::vector<FusedOp> ops;     // every op after its inputs
    int n_terms = 1;              // conjunctive terms of the answer (1 .. 4)
    std::vector<int> answer;      // op of each scored row: 1, 2 or 4 rows (3 terms repeat the last)
    std::vector<char> answer_neg;
    int and_stages = 0;
    // per-query needs, for capacity checks
    int max_stage_level = 0;      // MLP models: largest projection level (rows at one stage and hop)
    int max_stage_inputs = 0;     // largest intersection-stage input count
    int max_stage_groups = 0;     // largest intersection-stage group count
    int image_words = 0;          // plan-image words per query (without per-stage padding)
};

// Read the text form of a graph (post-order nodes, the answer last):
//   e<k>                 anchor slot k
//   p(<x>, r<k>)         projection of x by relation slot k
//   i(<x>, <y>[, ...])   intersection of 2 to 4 subqueries
//   u(<x>, <y>[, ...])   union of 2 to 4 subqueries
//   n(<x>)               negation
// Whitespace is ignored.
bool parse_graph(const char* text, std::vector<kgq_node>& out, std::string& err);

// Compile a graph for one model. Fails with KGQ_E_INVALID_ARG for a
// malformed graph and KGQ_E_UNSUPPORTED for negation on GQE / Query2Box.
bool compile_graph(int model, const kgq_node* nodes, int n, const std::string& name, Program& out,
                   std::string& err, int& err_status);

// The built-in structures (ids 0 .. 13) compiled for a model.
const Program* builtin_program(int model, int id);
const char* builtin_text(int id);

// A stage of a lowered batch: one launch group.
enum StageKind { ST_CHAIN = 0, ST_LEVEL = 1, ST_AND = 2 };

struct Stage {
    int kind = ST_CHAIN;
    int count = 0;                // chains / projection rows / groups
    int stage = 0, hop = 0;       // schedule position
    int in_base = 0, n_in = 0;    // ST_AND: the stage's contiguous input rows
    bool table = false;           // ST_LEVEL: first hop from anchors (first-layer table path)
    // Image offsets of the stage's lists:
    //   ST_CHAIN: a anchor_ref, b rel_off (count + 1), c rel_ref, d dst
    //   ST_LEVEL: a src_row (-1: anchor), b anchor_ref, c rel_ref, d neg, e dst
    //   ST_AND:   a in_start (relative to in_base), b n_in, c out_row, d neg_mask,
    //             e post_off (count + 1), f post_ref
    int64_t a = 0, b = 0, c = 0, d = 0, e = 0, f = 0;
};

struct Plan {
    int model = 0, B = 0;
    std::vector<Stage> stages;    // in execution order
    int n_state_rows = 0;
    // Scored rows: groups of four (answers with 3 or 4 terms), then pairs,
    // then single rows, each region in query order; one output per group.
    int n_score_rows = 0, n_quad_rows = 0, n_pair_rows = 0;
    // summary counts
    int n_anchor_chains = 0, n_groups = 0, n_int_in = 0, n_and_stages = 0;
    int level_rows[4] = {0, 0, 0, 0};   // MLP models: stage-0 hops 1, 2, >= 3; later stages
    int max_level = 0, max_and_in = 0, max_and_groups = 0;
    // Flattened device image: every list at a fixed, 16-byte aligned offset.
    std::vector<int32_t> image;
    int64_t off_score_src = 0, off_score_neg = 0, off_out_dest = 0, off_arity = 0;
};

// Lower a batch. Query q has structure table[sid[q]] (mixed) or
// table[fixed_sid]; its anchors sit at q * a_stride + slot, its relations at
// q * r_stride + slot. Returns false with a message for an unknown
// structure, one the model cannot run, or one with more slots than the
// strides hold.
bool lower(int model, int B, const int32_t* sid, int fixed_sid, int a_stride, int r_stride, bool mixed,
           const std::vector<const Program*>& table, Plan& out, std::string& err, int& err_status);

// Image words a plan may need beyond the per-query words (list padding and
// CSR ends).
constexpr int64_t kPlanOverheadWords = 8192;

// Rows of the state buffer reserved per query of max_batch.
constexpr int kStateRowsPerQuery = 8;

// Kernel launches one execute of this plan makes (without the checked-mode
// validation and without the second pass of a split small-batch layer).
int plan_launches(const Plan& p, bool topk);
int program_launches(int model, const Program& prog, bool topk);

}  // namespace kgq
