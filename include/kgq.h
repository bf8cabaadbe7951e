/*
 * kgq.h -- C ABI of libkgq: batched complex logical query answering (CLQA)
 * over knowledge-graph embeddings on one AMD Instinct MI355X (gfx950).
 *
 * The calls follow the paper's query-plan formulation (Methodology, Fig. 2
 * and Eq. 2): a first-order query is identified by its structure, the
 * structure fixes a computation graph of projection, intersection, union
 * and negation operators over anchor entities and relations, and the
 * library executes that graph for a batch of queries, then scores every
 * entity against each query embedding (the entity-similarity step that the
 * Experiments section times together with the operators) and selects the
 * top k.
 *
 * Five embedding models are supported: GQE, Query2Box, BetaE, ConE and
 * LogicE (the paper names them in Related Work and Experiments/Baselines and
 * times them in Table 1; BetaE's Beta embedding is its Eq. 3 and BetaE's
 * projection the MLP of its Eq. 4; the operators of the others follow the
 * models' own definitions, as described at kgq_load_params).
 *
 * Conventions
 *  - Every function returns a kgq_status; no C++ exception crosses the ABI.
 *  - Pointers marked "device" must point to memory of the handle's GPU (for
 *    example torch.Tensor.data_ptr() of a CUDA tensor). Pointers marked
 *    "host" point to ordinary host memory.
 *  - The caller owns every buffer it passes in. The handle owns device
 *    copies of all parameters, the derived tables, and its scratch space,
 *    all freed by kgq_destroy.
 *  - kgq_execute / kgq_execute_mixed are asynchronous: work is enqueued on
 *    the caller's stream and the call returns. Outputs are valid after the
 *    caller synchronises that stream; inputs must stay alive until then.
 *    Calls on one handle must be issued from one host thread at a time.
 *  - A handle owns cfg.concurrency sets of scratch space, used round-robin
 *    by successive execute calls. Before a call reuses a set, its stream
 *    waits on the device for the set's previous call to finish, so calls on
 *    different streams may overlap (up to cfg.concurrency at once) and calls
 *    on one stream stay in order. The host never blocks for this.
 *  - Each set stages the lowered plan of a call through two pinned host
 *    slots, used alternately. A call whose slot is still being read by the
 *    execute that used it two calls earlier on the same set waits on the host
 *    for that execute to finish (backpressure): the host runs at most
 *    2 * cfg.concurrency execute calls ahead of the device. No other host
 *    wait occurs outside checked mode.
 *  - Host-checkable errors are reported before anything is enqueued.
 */
#ifndef KGQ_H
#define KGQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kgq_handle kgq_handle;

typedef enum {
    KGQ_OK = 0,
    KGQ_E_INVALID_ARG = -1,   /* null pointer, bad id/size/shape/dtype, k or batch out of range */
    KGQ_E_OUT_OF_RANGE = -2,  /* checked mode: an anchor or relation id in device memory is out of range */
    KGQ_E_NOT_LOADED = -3,    /* execute before every parameter of the model was loaded */
    KGQ_E_UNSUPPORTED = -4,   /* structure with negation on GQE or Query2Box */
    KGQ_E_NO_DEVICE = -5,     /* no usable GPU (or a validation-only handle, device = -1) */
    KGQ_E_OOM = -6,           /* device or pinned host allocation failed */
    KGQ_E_DEVICE = -7         /* a HIP runtime call failed */
} kgq_status;

typedef enum { KGQ_GQE = 0, KGQ_Q2B = 1, KGQ_BETAE = 2, KGQ_CONE = 3, KGQ_LOGICE = 4 } kgq_model;
typedef enum { KGQ_F32 = 0, KGQ_BF16 = 1 } kgq_dtype;
/* LogicE intersection t-norm: a * b, min(a, b), or max(0, a + b - 1). */
typedef enum { KGQ_TNORM_PRODUCT = 0, KGQ_TNORM_MIN = 1, KGQ_TNORM_LUKASIEWICZ = 2 } kgq_tnorm;

/* Query structures, in the column order of the paper's Table 1. The shapes
 * (the paper shows them only in its Fig. 1): "p" chains projections, "i"
 * intersects branches, "u" takes a union (evaluated in disjunctive normal
 * form, Eq. 1: the entity score is the max over the branch scores), "n"
 * negates one branch before the intersection. Anchor slots a0..a2 and
 * relation slots r0..r2 are consumed in the order written:
 *   1p  a0.r0                      2p  a0.r0.r1          3p  a0.r0.r1.r2
 *   2i  a0.r0 & a1.r1              3i  a0.r0 & a1.r1 & a2.r2
 *   pi  a0.r0.r1 & a1.r2           ip  (a0.r0 & a1.r1).r2
 *   2u  a0.r0 | a1.r1              up  (a0.r0 | a1.r1).r2 = a0.r0.r2 | a1.r1.r2
 *   2in a0.r0 & !a1.r1             3in a0.r0 & a1.r1 & !a2.r2
 *   inp (a0.r0 & !a1.r1).r2        pin a0.r0.r1 & !a1.r2      pni !(a0.r0.r1) & a1.r2
 * The five structures with negation (ids 9..13) exist for BetaE, ConE and
 * LogicE; GQE and Query2Box define no negation (Experiments, Baselines). */
typedef enum {
    KGQ_1P = 0, KGQ_2P, KGQ_3P, KGQ_2I, KGQ_3I, KGQ_PI, KGQ_IP, KGQ_2U, KGQ_UP,
    KGQ_2IN, KGQ_3IN, KGQ_INP, KGQ_PIN, KGQ_PNI, KGQ_NUM_STRUCTURES
} kgq_structure;

#define KGQ_MAX_K 1024

typedef struct {
    int32_t model;        /* kgq_model */
    int32_t dim;          /* embedding dimension d; a multiple of 4, at most 4096 */
    int64_t n_entities;   /* N >= 1, at most 2^31 - 1 */
    int32_t n_relations;  /* R >= 1 */
    int32_t entity_dtype; /* kgq_dtype of the entity table as passed to kgq_load_params */
    float gamma;          /* score margin: score = gamma - distance */
    float center_reg;     /* Query2Box and ConE: weight of the inside distance (0.02 in the standard
                             models); ignored otherwise */
    int32_t max_batch;    /* largest batch any execute call will pass; sizes the scratch space */
    int32_t device;       /* HIP device ordinal, or -1 for a validation-only handle with no GPU */
    int32_t concurrency;  /* scratch sets (1 if 0): executes issued on different streams can run
                             concurrently, up to this many at once */
    int32_t tnorm;        /* LogicE: kgq_tnorm of the intersection; ignored otherwise */
} kgq_config;

/* Create a handle for one embedding model on one GPU (GQE, Query2Box,
 * BetaE, ConE or LogicE: Related Work; Experiments, Baselines; Table 1).
 * Validates cfg, selects the
 * device, and allocates all scratch space for max_batch queries (execute
 * allocates nothing). The handle is the compiled form of the paper's
 * pipeline for that model (Methodology, Fig. 2): the 14 benchmark
 * structures are compiled into fused programs (once per process, at the
 * first create) and the handle refers to them; parameters arrive with
 * kgq_load_params.
 * Errors: INVALID_ARG (cfg or out null, bad field, tnorm outside kgq_tnorm
 * for LogicE), NO_DEVICE, OOM, DEVICE.
 * A handle with device = -1 validates arguments exactly like a real one;
 * its execute calls return NO_DEVICE once every argument has passed. */
kgq_status kgq_create(const kgq_config* cfg, kgq_handle** out);

/* Load one named parameter array (row-major; dense layers W are [out x in]
 * and compute y = W x + b).
 *   GQE:   "entity" [N x d], "relation" [R x d],
 *          "inter.w1" [d x d], "inter.b1" [d], "inter.w2" [d x d], "inter.b2" [d]
 *   Q2B:   "entity" [N x d], "relation.center" [R x d],
 *          "relation.offset_raw" [R x d] (the library applies softplus),
 *          "inter.center.{w1,b1,w2,b2}" and "inter.offset.{w1,b1,w2,b2}" ([d x d], [d])
 *   BetaE: "entity.alpha_beta" [N x 2d] (alpha in columns 0..d-1, beta in d..2d-1, all > 0),
 *          "relation" [R x 2d],
 *          "proj.w1" [4d x 2d], "proj.b1" [4d], "proj.w2" [4d x 4d], "proj.b2" [4d],
 *          "proj.w3" [2d x 4d], "proj.b3" [2d],
 *          "inter.w1" [2d x 2d], "inter.b1" [2d], "inter.w2" [d x 2d], "inter.b2" [d]
 *   ConE:  "entity.axis" [N x d] (entity cone axes in [-pi, pi); an entity is a
 *          cone of aperture 0), "relation" [R x 2d] (axis | half-aperture, added
 *          to the source cone before the projection MLP),
 *          "proj.w1" [4d x 2d], "proj.b1" [4d], "proj.w2" [4d x 4d], "proj.b2" [4d],
 *          "proj.w3" [2d x 4d], "proj.b3" [2d] (axis = pi tanh(y), half-aperture =
 *          pi/2 (tanh(2 y') + 1)),
 *          "inter.axis.{w1 [d x 2d], b1 [d], w2 [d x d], b2 [d]}" (attention over
 *          [axis - aperture; axis + aperture], softmax across branches, weighted
 *          mean of the axes' unit vectors),
 *          "inter.arg.{w1 [d x 2d], b1 [d], w2 [d x d], b2 [d]}" (sigmoid gate on
 *          the mean of the branches' features, times the minimum half-aperture),
 *          "modulus" [1] (score = gamma - modulus (outside + center_reg inside
 *          sector distance)); negation is the complementary cone
 *   LogicE: "entity.bounds" [N x 2d] (lower bounds in columns 0..d-1, upper in
 *          d..2d-1, 0 <= lower <= upper <= 1), "relation" [R x d] (concatenated
 *          to the source bounds before the projection MLP),
 *          "proj.w1" [4d x 3d], "proj.b1" [4d], "proj.w2" [4d x 4d], "proj.b2" [4d],
 *          "proj.w3" [2d x 4d], "proj.b3" [2d] (lower = sigmoid(y), upper = lower +
 *          sigmoid(y') (1 - lower)); intersection by cfg.tnorm, negation
 *          [l; u] -> [1 - u; 1 - l], score gamma - ||e - q||_1 / (2d)
 * dtype is KGQ_F32 for every array except the entity table, which takes
 * cfg.entity_dtype (KGQ_BF16: bfloat16 bit patterns, decoded to float32 on
 * the device). nbytes must equal the array's size. src is a host pointer,
 * or a device pointer if src_is_device is non-zero; it is read before the
 * call returns (the call synchronises). Loading a name again replaces it.
 * Derived tables are rebuilt here, not in execute: the blocked entity
 * layout for scoring, Query2Box's softplus offsets, BetaE's per-entity
 * digamma / log-Beta tables, ConE's per-entity half-angle sines and cosines,
 * ConE's stacked intersection first layer ([inter.axis.w1; inter.arg.w1]),
 * and the first-projection-layer tables of BetaE, ConE and LogicE (entity
 * state . W1^T [N x 4d] and relation . W1^T + b1 [R x 4d], where W1 is split
 * by columns for LogicE's concatenated input; the layer is linear in its
 * input, Eq. 4), rebuilt when the entity table, "relation", "proj.w1" or
 * "proj.b1" is loaded and all four are present.
 * Errors: INVALID_ARG (unknown name, wrong nbytes or dtype, null src), OOM, DEVICE. */
kgq_status kgq_load_params(kgq_handle* h, const char* name, const void* src, size_t nbytes,
                           int32_t dtype, int32_t src_is_device);

/* Number of anchor entities and relations a query of a built-in structure
 * takes (compiled structures: kgq_structure_info).
 * Errors: INVALID_ARG (unknown structure id or null outputs). */
kgq_status kgq_structure_arity(int32_t structure_id, int32_t* n_anchors, int32_t* n_relations);

/* Execute a batch of queries that all have the same structure (built-in,
 * or compiled on this handle): the structure's computation graph (Eq. 2;
 * unions in disjunctive normal form, Eq. 1) run through its fused plan
 * (Methodology, Operator Fuser, Algorithm 1), then the entity-similarity
 * query over all N entities and the top k (the two parts of the paper's
 * reasoning time; Experiments, Metrics).
 *   anchors   device int32 [batch x n_anchors(structure)]
 *   relations device int32 [batch x n_relations(structure)]
 *   k         1 <= k <= min(N, KGQ_MAX_K) when top-k outputs are requested
 *   out_scores      device float [batch x N] or NULL: score of every entity
 *   out_topk_idx    device int32 [batch x k] or NULL
 *   out_topk_score  device float [batch x k] or NULL
 *   stream          hipStream_t, or NULL for the null stream
 * At least one output must be requested; the two top-k outputs go together.
 * Top-k lists are ordered by score descending, equal scores by entity index
 * ascending.
 * Ids out of range never cause an out-of-bounds access: the device replaces
 * them and raises a flag. In checked mode (environment KGQ_CHECKED=1 at
 * create, or kgq_set_checked) execute then synchronises the stream and
 * returns OUT_OF_RANGE; otherwise the affected outputs are unspecified.
 * A structure larger than the built-in ones may bound the batch below
 * max_batch (kgq_structure_info); a larger batch is INVALID_ARG.
 * Errors: INVALID_ARG, UNSUPPORTED, NOT_LOADED, OUT_OF_RANGE (checked),
 * NO_DEVICE, DEVICE. */
kgq_status kgq_execute(kgq_handle* h, int32_t structure_id, int32_t batch,
                       const int32_t* anchors, const int32_t* relations, int32_t k,
                       float* out_scores, int32_t* out_topk_idx, float* out_topk_score,
                       void* stream);

/* Execute a batch whose queries have different structures, in one plan:
 * the fused operators of all structures (Methodology, Operator Fuser,
 * Algorithm 1) are grouped by kind and schedule position, so each kind runs
 * as one launch across the whole batch; then scoring and top-k as in
 * kgq_execute (Experiments, Metrics).
 *   structure_ids  HOST int32 [batch]: the plan is lowered on the host.
 *   anchors        device int32 [batch x 3], unused slots -1
 *   relations      device int32 [batch x 3], unused slots -1
 * Results are written in input order, with the same output rules as
 * kgq_execute. The plan reads only the slots a query's structure uses; in
 * checked mode a device-side check also requires every unused slot to be -1
 * and returns INVALID_ARG otherwise.
 * Errors: as kgq_execute. */
kgq_status kgq_execute_mixed(kgq_handle* h, int32_t batch, const int32_t* structure_ids,
                             const int32_t* anchors, const int32_t* relations, int32_t k,
                             float* out_scores, int32_t* out_topk_idx, float* out_topk_score,
                             void* stream);

/* Allocation-free variant of kgq_execute_mixed, for callers that cannot
 * allocate device memory while they run (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation). Same arguments,
 * outputs, batch limits and errors as kgq_execute_mixed; the difference is
 * where the call's device scratch lives. kgq_execute_mixed uses the scratch
 * the handle allocated at create; this call carves every device buffer it
 * needs (plan image, error flag, state rows, dense-layer rows, packed
 * queries, the score matrix when out_scores is NULL, top-k candidates, and,
 * as far as room is left, BetaE's chunk keys for top-k and the split
 * workspaces of small batches) out of one
 * static array of KGQ_NOALLOC_SCRATCH_BYTES per GPU, which the library holds
 * from its first use on that GPU until the process ends. The call itself
 * allocates nothing, device or pinned; it lowers the plan on the host as
 * kgq_execute_mixed does and stages it through the handle's pinned slots.
 * A batch whose buffers exceed the array is INVALID_ARG before anything is
 * enqueued (passing out_scores, or a smaller batch, reduces the need).
 * The array is shared by every call on a GPU, from every handle: calls of
 * this function that overlap on one GPU (on different streams, or from
 * different handles) race and give unspecified results; calls on one stream
 * are ordered. The array keeps the previous call's contents; the call clears
 * what must start at zero (its error flag) itself. */
#define KGQ_NOALLOC_SCRATCH_BYTES (64 << 20)
kgq_status kgq_execute_mixed_noalloc(kgq_handle* h, int32_t batch, const int32_t* structure_ids,
                                     const int32_t* anchors, const int32_t* relations, int32_t k,
                                     float* out_scores, int32_t* out_topk_idx, float* out_topk_score,
                                     void* stream);

/* Turn checked mode on (non-zero) or off for this handle. */
kgq_status kgq_set_checked(kgq_handle* h, int32_t on);

/* Which matrix cores the dense contractions run on: the dense layers (the
 * MLPs of Eq. 4 and of the intersection operators, and kgq_dense) and
 * BetaE's scoring contraction (the regrouped KL of Eq. 3's embeddings). Both
 * paths compute in FP32 precision class:
 *   KGQ_DENSE_AUTO (the default): layers with K >= 32 (K is a multiple of 4
 *     on every path) and at least 384 output tiles of 64 x 64, or 1,024 rows
 *     and 192 such tiles, run on the bf16 matrix cores, each FP32 operand
 *     split exactly into three bf16 parts and six of the nine part products
 *     kept (the dropped ones are below 2^-23 of each product; the weight
 *     parts are zero-padded to a multiple of 32 columns); smaller layers of
 *     an execute with more than 64 rows and K >= 64 split K there; the
 *     others (K < 32, layers of at most 64 rows, and kgq_dense layers below
 *     the bounds) on the FP32 matrix cores. Inputs
 *     must be finite and below 3.39e38 in magnitude on the bf16 path.
 *     BetaE scores on the bf16 path when 2d is a multiple of 32 and the call
 *     scores more than 64 rows (more than 128 when 128-row tiles would give
 *     fewer than 256 workgroups); smaller calls score on the FP32 matrix
 *     cores.
 *   KGQ_DENSE_FP32: every layer and the BetaE scorer on the FP32 matrix cores.
 *   KGQ_DENSE_BF16X3: every layer with K >= 32, and the BetaE scorer when
 *     2d is a multiple of 32, on the bf16 path, whatever the size (for
 *     tests).
 * The bf16 parts of the weights and of BetaE's entity-side scoring rows are
 * made when they are loaded, whatever the path. Takes effect for calls
 * enqueued after it. Errors: INVALID_ARG. */
typedef enum { KGQ_DENSE_AUTO = 0, KGQ_DENSE_FP32 = 1, KGQ_DENSE_BF16X3 = 2 } kgq_dense_path;
kgq_status kgq_set_dense_path(kgq_handle* h, int32_t path);

/* Describe the lowered plan of a batch (host structure ids, built-in or
 * compiled) without running it. counts receives KGQ_PLAN_NCOUNTS values, in
 * this order:
 *   0 projection chains starting at an anchor, 1 intersection groups,
 *   2 intersection inputs, 3..6 BetaE projection rows at hops 1, 2 and >= 3
 *   from the anchors and after an intersection, 7 scored rows, 8 union
 *   pairs, 9 kernel launches per execute (with top-k), 10 intersection
 *   stages, 11 unions scored as groups of four rows (3 or 4 terms),
 *   12 state rows.
 * Errors: INVALID_ARG, UNSUPPORTED. */
#define KGQ_PLAN_NCOUNTS 13
kgq_status kgq_describe_plan(const kgq_handle* h, int32_t batch, const int32_t* structure_ids,
                             int32_t* counts);

/* ---- Query structures as computation graphs -------------------------------
 * Any query structure built from the four operators can be compiled into a
 * structure id of a handle and then executed like a built-in one. This is
 * the paper's compilation pipeline (Methodology, Fig. 2):
 *   Graph Capturer (Eq. 2): the caller describes the query as a graph.
 *   Entities are value nodes (KGQ_OP_ANCHOR), each relation a projection
 *   node (KGQ_OP_PROJECT), and the connectives the functions f_and, f_or and
 *   f_not (KGQ_OP_AND, KGQ_OP_OR, KGQ_OP_NOT).
 *   Pattern Recognizer: the graph is rewritten into disjunctive normal form
 *   (Eq. 1): projection and intersection distribute over unions, the
 *   negation of a union becomes the intersection of the negations, and
 *   chains of negations reduce to their parity.
 *   Operator Fuser (Algorithm 1): each maximal run of projections on one
 *   path becomes one fused chain (horizontal fusion), each intersection one
 *   combine over all its branches (vertical fusion), and for GQE and
 *   Query2Box a run of projections that follows an intersection is folded
 *   into that combine (hybrid fusion). At execute time every fused operator
 *   of one kind and schedule position runs as a single launch for the whole
 *   batch, across structures.
 * The built-in structures 0..13 are such graphs, compiled the same way; their
 * text forms are listed with kgq_parse_structure. */
typedef enum {
    KGQ_OP_ANCHOR = 0,    /* anchor entity in anchor slot `slot` */
    KGQ_OP_PROJECT = 1,   /* projection of in[0] by the relation in relation slot `slot` */
    KGQ_OP_AND = 2,       /* intersection of in[0..] (2 to 4 inputs) */
    KGQ_OP_OR = 3,        /* union of in[0..] (2 to 4 inputs) */
    KGQ_OP_NOT = 4        /* negation of in[0] (BetaE, ConE, LogicE) */
} kgq_op;

typedef struct {
    int32_t op;      /* kgq_op */
    int32_t slot;    /* anchor or relation slot (0 .. KGQ_MAX_SLOTS-1); ignored for AND, OR, NOT */
    int32_t in[4];   /* indices of earlier nodes, from in[0]; unused entries -1 */
} kgq_node;

#define KGQ_MAX_GRAPH_NODES 64   /* nodes of one graph */
#define KGQ_MAX_SLOTS 8          /* anchor slots and relation slots of one structure */
#define KGQ_MAX_DISJUNCTS 4      /* conjunctive terms of any node in disjunctive normal form */
#define KGQ_MAX_COMPILED 64      /* compiled structures per handle */

/* Read the text form of a graph into nodes (host memory, capacity entries),
 * in post-order: every node after its inputs, the answer last.
 *   e<k>               anchor slot k            p(<x>, r<k>)  projection of x by relation slot k
 *   i(<x>, <y>[, ...]) intersection of 2-4       u(<x>, <y>[, ...]) union of 2-4
 *   n(<x>)             negation                 whitespace is ignored
 * The built-in structures, in this form:
 *   1p p(e0,r0)   2p p(p(e0,r0),r1)   3p p(p(p(e0,r0),r1),r2)   2i i(p(e0,r0),p(e1,r1))
 *   3i i(p(e0,r0),p(e1,r1),p(e2,r2))   pi i(p(p(e0,r0),r1),p(e1,r2))   ip p(i(p(e0,r0),p(e1,r1)),r2)
 *   2u u(p(e0,r0),p(e1,r1))   up p(u(p(e0,r0),p(e1,r1)),r2)   2in i(p(e0,r0),n(p(e1,r1)))
 *   3in i(p(e0,r0),p(e1,r1),n(p(e2,r2)))   inp p(i(p(e0,r0),n(p(e1,r1))),r2)
 *   pin i(p(p(e0,r0),r1),n(p(e1,r2)))   pni i(n(p(p(e0,r0),r1)),p(e1,r2))
 * *n_nodes receives the node count. The text is not checked beyond its
 * syntax (kgq_compile_structure checks the graph).
 * Errors: INVALID_ARG (NULL argument, syntax error, more than capacity or
 * KGQ_MAX_GRAPH_NODES nodes). */
kgq_status kgq_parse_structure(const char* text, kgq_node* nodes, int32_t capacity, int32_t* n_nodes);

/* Compile a graph (host nodes[n_nodes], the answer last) for this handle's
 * model and return its new structure id (>= KGQ_NUM_STRUCTURES) in
 * *structure_id, valid for this handle's kgq_execute, kgq_execute_mixed,
 * kgq_describe_plan and kgq_structure_info until kgq_destroy. A query of the
 * structure takes anchors[slot] for slots 0..A-1 and relations[slot] for
 * slots 0..R-1; both slot sets must be used without gaps (a mixed batch
 * holds at most 3 of each). Rules: inputs are earlier nodes; every node but
 * the last feeds a later one; an anchor feeds only projections; at most
 * KGQ_MAX_DISJUNCTS conjunctive terms at any node in normal form (so at most
 * 4 intersection inputs after a negated union).
 * Compiling allocates nothing on the device; the handle's scratch, sized by
 * max_batch for the built-in structures, bounds the batch of a larger
 * structure (kgq_structure_info reports the bound).
 * Errors: INVALID_ARG (NULL argument, a rule broken, KGQ_MAX_COMPILED
 * reached, a structure that does not fit even one query), UNSUPPORTED
 * (negation on GQE or Query2Box). */
kgq_status kgq_compile_structure(kgq_handle* h, const kgq_node* nodes, int32_t n_nodes, int32_t* structure_id);

/* Facts about a built-in or compiled structure on this handle. info receives
 * KGQ_INFO_NCOUNTS values: 0 anchors, 1 relations, 2 conjunctive terms of the
 * answer, 3 fused operators per query, 4 intersection stages, 5 kernel
 * launches per execute (with top-k), 6 largest batch of this structure alone
 * that the handle's scratch holds, 7 uses negation (0/1).
 * Errors: INVALID_ARG (NULL argument or unknown id), UNSUPPORTED (a
 * built-in negation structure on GQE or Query2Box). */
#define KGQ_INFO_NCOUNTS 8
kgq_status kgq_structure_info(const kgq_handle* h, int32_t structure_id, int32_t* info);

/* Filtered ranks of known answers, and ranking metrics per query (the paper
 * reports MRR; Experiments). For query q, with score row
 * scores + q * ld (N = cfg.n_entities columns, ld >= N; e.g. the out_scores
 * of an execute) and answer set A_q = ans_ids[ans_offsets[q] ..
 * ans_offsets[q + 1]) (distinct entity ids, at most KGQ_MAX_ANSWERS), the
 * filtered rank of answer a is
 *   1 + #{ e not in A_q : e ranks before a },
 * in the library's ranking order (higher score first, equal scores by lower
 * entity index: the order of the top-k). out_rank[i] receives the rank of
 * ans_ids[i]. out_metrics (or NULL) receives per query, over its hard
 * answers (ans_hard[i] != 0; ans_hard == NULL: every answer is hard), in
 * double precision: [MRR = mean 1/rank, Hits@1, Hits@3, Hits@10]; NaN for a
 * query without hard answers. All arrays are device memory; the call
 * enqueues on stream and returns.
 * Errors: INVALID_ARG (null pointers, batch < 1, ld < N), NO_DEVICE; in
 * checked mode the call synchronises and reports OUT_OF_RANGE for an answer
 * id outside [0, N) and INVALID_ARG for a list longer than KGQ_MAX_ANSWERS
 * or of negative length (such ranks are -1, such metrics NaN, in either
 * mode). */
#define KGQ_MAX_ANSWERS 1024
kgq_status kgq_rank_answers(kgq_handle* h, int32_t batch, const float* scores, int64_t ld,
                            const int32_t* ans_offsets, const int32_t* ans_ids, const int32_t* ans_hard,
                            int32_t* out_rank, double* out_metrics, void* stream);

/* Device memory the handle holds, in bytes (the paper measures peak memory
 * against batch size; Experiments, RQ2). param_bytes: every parameter and
 * derived table (entity layouts, softplus offsets, BetaE digamma / log-Beta
 * and first-layer tables). scratch_bytes: the execute scratch of all
 * concurrency lanes, sized by max_batch at create. Execute allocates
 * nothing, so their sum is the handle's peak; transient load staging is not
 * included. A validation-only handle (device = -1) holds none.
 * Either output may be NULL. Errors: INVALID_ARG (null handle). */
kgq_status kgq_memory(const kgq_handle* h, int64_t* param_bytes, int64_t* scratch_bytes);

/* Per-stage timing. kgq_profile_enable takes a bitmask of stages (bit i =
 * stage i; 0 turns profiling off). While a stage's bit is set, execute
 * records a pair of HIP events around every kernel of that stage it
 * launches, on the caller's stream.
 * kgq_profile_read synchronises on those events and returns the summed
 * milliseconds and launch count of one stage since profiling was turned
 * on (or last reset), then keeps accumulating. Stages:
 *   0 anchor gather and translation chains, 1 dense layers (MFMA),
 *   2 intersection / negation combines, 3 query packing,
 *   4 entity scoring, 5 top-k selection. */
#define KGQ_NUM_STAGES 6
kgq_status kgq_profile_enable(kgq_handle* h, int32_t on);
kgq_status kgq_profile_read(kgq_handle* h, int32_t stage, double* total_ms, int64_t* launches);
kgq_status kgq_profile_reset(kgq_handle* h);
/* Start and end (milliseconds from a time origin recorded when profiling
 * was first enabled on the handle) of every timed launch of a stage since
 * the last reset: out receives min(cap, *n) (start, end) pairs; *n is the
 * total count. Launches on different streams may overlap in time; the
 * union of the intervals is the time the stage had work on the GPU. */
kgq_status kgq_profile_intervals(kgq_handle* h, int32_t stage, double* out, int64_t cap, int64_t* n);

/* One dense layer on the device with the library's GEMM:
 * y[m][n] = act(sum_k x[m][k] * w[n][k] + b[n]) (the matmul + add (+ ReLU)
 * pattern of the paper's Eq. 4), on the matrix cores kgq_set_dense_path
 * selects; on the bf16 path, w is split into its bf16 parts on `stream` in
 * a stream-ordered allocation freed after the layer.
 *   x  device float [M x K], w device float [N x K], b device float [N] or NULL,
 *   y  device float [M x N]; K a multiple of 4, rows 16-byte aligned.
 *   act 0 = none, 1 = ReLU, 2 = BetaE regulariser clamp(v + 1, 0.05, 1e9).
 * Asynchronous on `stream`. Errors: INVALID_ARG, NO_DEVICE, OOM, DEVICE. */
kgq_status kgq_dense(kgq_handle* h, const float* x, int32_t M, int32_t K, const float* w, const float* b,
                     int32_t N, int32_t act, float* y, void* stream);

/* Free the handle and everything it owns: parameters, derived tables,
 * compiled plans and scratch (the counterpart of kgq_create). Waits for the
 * handle's work in flight first. NULL is accepted. */
kgq_status kgq_destroy(kgq_handle* h);

/* Static description of a status code. */
const char* kgq_status_string(kgq_status s);

/* Message of the last failing call on this handle ("" if none). The string
 * stays valid until the next call on the handle. */
const char* kgq_last_error(const kgq_handle* h);

/* Message of the last failing kgq_create in this thread. */
const char* kgq_create_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KGQ_H */
