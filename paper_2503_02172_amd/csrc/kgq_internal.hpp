// Internal declarations shared by the host library and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/kgq.h"

namespace kgq {

// ---- data layout constants -------------------------------------------------

// Entities are scored in blocks of 256 (the table is padded with zeros to a
// multiple of 256 entities). GQE and Query2Box points are stored block by
// block, dimension-major inside a block, element (e, k) at
//   [e / 256][k][e % 256]
// so that a VALU wavefront (64 lanes x 4 entities) reads 1 KiB contiguous per
// dimension; LogicE's bounds the same way over its 2d coordinates. ConE
// keeps two fields per dimension, [e / 256][k][sin | cos of theta/2][e % 256].
// BetaE's scoring table is row-major [e][U (d) | V (d)], the B operand of the
// matrix-core scorer.
constexpr int kEntBlock = 256;

// Largest k of a top-k request (the selection buffer lives in LDS).
constexpr int kMaxK = 1024;

// Query rows per wavefront in the VALU scorers (rows are wave-uniform and
// read through the scalar cache). Packed layout [row_block][k][field][kTq].
constexpr int kTqGqe = 24;
constexpr int kTqQ2b = 12;
constexpr int kTqCone = 8;
// BetaE query rows are packed row-major [row][alpha (d) | beta (d)] and
// padded to the matrix-core scorer's 128-row tile.
constexpr int kRowTileBetae = 128;

// LogicE scores with GQE's L1 kernel over its 2d bound coordinates.
inline int valu_form(int model) { return model == KGQ_LOGICE ? KGQ_GQE : model; }

// Scored rows are padded to a multiple of this per model.
inline int score_row_pad(int model)
{
    switch (valu_form(model)) {
    case KGQ_GQE: return kTqGqe;
    case KGQ_Q2B: return kTqQ2b;
    case KGQ_CONE: return kTqCone;
    default: return kRowTileBetae;
    }
}

// Small batches (at most kSmallScoreRows scored rows) run the GQE / Query2Box
// pack and scorer with fewer rows per wavefront: there the scorer's dimension
// loop is a latency chain on a few workgroups, whose length grows with the
// rows per wavefront. 8 and 4 divide the padding (24 and 12), so the padded
// layout holds either form; pack and scorer decide from the same row count.
constexpr int kTqGqeSmall = 8;
constexpr int kTqQ2bSmall = 4;
constexpr int kTqConeSmall = 4;
constexpr int kSmallScoreRows = 1024;
inline bool score_small(int n_rows) { return n_rows <= kSmallScoreRows; }
inline int score_tq(int model, int n_rows)
{
    const bool small = score_small(n_rows);
    switch (valu_form(model)) {
    case KGQ_GQE: return small ? kTqGqeSmall : kTqGqe;
    case KGQ_Q2B: return small ? kTqQ2bSmall : kTqQ2b;
    default: return small ? kTqConeSmall : kTqCone;
    }
}

// Models whose projection is an MLP (one dense-layer pass per hop) and that
// define negation: BetaE, ConE, LogicE.
inline bool mlp_model(int model) { return model == KGQ_BETAE || model == KGQ_CONE || model == KGQ_LOGICE; }

// Device error flag bits.
constexpr int kErrRange = 1;    // an anchor or relation id outside its table
constexpr int kErrPadding = 2;  // a mixed-batch unused slot that is not -1
constexpr int kErrAnswers = 4;  // an answer list longer than kMaxAnswers or of negative length

// Largest answer list of one query for the ranking metrics (sorted in LDS).
constexpr int kMaxAnswers = 1024;

// Dense-layer epilogues. EPI_CONE_ANGLES maps columns below epi_split to
// pi tanh(v) (ConE axes) and the others to pi/2 (tanh(2 v) + 1) (ConE
// half-apertures); EPI_SIGMOID is LogicE's sigmoid before its bound map.
enum Epilogue { EPI_NONE = 0, EPI_RELU = 1, EPI_BETA_REG = 2, EPI_CONE_ANGLES = 3, EPI_SIGMOID = 4 };

// ---- launchers (each enqueues on `s` and returns) ---------------------------

struct GemmArgs {
    const float* A; int64_t lda;       // [M x K] row-major
    const float* W; int64_t ldw;       // [N x K] row-major (y = W x + b)
    const float* bias;                 // [N] or nullptr
    float* C; int64_t ldc;             // [M x N] (row m stored at C + map(m) * ldc)
    const int32_t* c_rowmap;           // nullptr = identity
    int M, N, K;                       // K % 4 == 0, A/W 16-byte aligned rows
    int epi;
    float* ws = nullptr;               // split-K partials for small M (nullptr: never split)
    int64_t ws_elems = 0;
    int epi_split = 0;                 // EPI_CONE_ANGLES: first column of the second map
    // W split into three bf16 planes (launch_split_planes: [3][N][plane_ld(K)],
    // zero past K) or nullptr. With the planes, K >= 32 and enough output
    // tiles to fill the chip, the layer runs on the bf16 matrix cores with
    // FP32 accuracy (k_gemm_bf16x3); bf16x3_always takes that path whenever
    // K allows it.
    const uint16_t* Wp = nullptr;
    bool bf16x3_always = false;
};
void launch_gemm(const GemmArgs& g, hipStream_t s);
// Whether launch_gemm, given weight planes, runs a layer of this shape on
// the bf16 matrix cores.
bool gemm_shape_takes_bf16x3(int M, int N, int K, int64_t lda, bool always);
// Row stride of the bf16 planes of a [rows x cols] matrix: cols rounded up
// to the 32-wide stage of the bf16 tile loop.
__host__ __device__ inline int64_t plane_ld(int64_t cols) { return (cols + 31) / 32 * 32; }
// W [rows x cols] -> three bf16 planes, plane q at p + q * rows * ld with
// ld = plane_ld(cols), row r at r * ld, zeros in columns cols .. ld - 1;
// w = p0 + p1 + p2 exactly (round to nearest even at each step).
void launch_split_planes(const float* w, uint16_t* p, int64_t rows, int64_t cols, hipStream_t s);

// Epilogue value of output column n.
__device__ __forceinline__ float apply_epilogue(int epi, int split, int n, float v)
{
    if (epi == EPI_RELU) return v > 0.f ? v : 0.f;
    if (epi == EPI_BETA_REG) return fminf(fmaxf(v + 1.0f, 0.05f), 1e9f);
    if (epi == EPI_CONE_ANGLES)
        return n < split ? 3.14159265358979323846f * tanhf(v) : 1.57079632679489661923f * (tanhf(2.0f * v) + 1.0f);
    if (epi == EPI_SIGMOID) return 1.0f / (1.0f + expf(-v));
    return v;
}

// Relayout a row-major [N x d] table (fp32 or bf16 bits) into the blocked
// scorer layout (fp32), padding with zeros; also writes a row-major fp32 copy.
void launch_relayout_points(const void* src, int src_bf16, int64_t N, int d, int64_t n_blocks,
                            float* rowmajor, float* blocked, hipStream_t s);

// BetaE: decode alpha|beta [N x 2d] to fp32 row-major, and build U, V
// (blocked) and the per-entity constant E_e (double).
void launch_betae_entity_prep(const void* src, int src_bf16, int64_t N, int d, int64_t n_blocks,
                              float* ab_rowmajor, float* uv_blocked, double* e_const, hipStream_t s);

void launch_softplus(const float* src, float* dst, int64_t n, hipStream_t s);

// BetaE first-hop projections, first layer: h1[m] = ReLU(pe[anchor_m] +
// pr[rel_m]) with pe = entity alpha|beta . W1^T and pr = Rel . W1^T + b1
// (rows of width w = 4d). Ids are range-checked like the other gathers.
void launch_betae_proj1(const int32_t* anchor_ref, const int32_t* rel_ref, int M, const int32_t* anchors,
                        const int32_t* rels, const float* pe, const float* pr, int64_t n_ent, int n_rel, int w,
                        float* h1, int* flag, hipStream_t s);

void launch_clear_flag(int* flag, hipStream_t s);

// Copy n_words from pinned (device-mapped) host memory to the device with a
// kernel; both pointers 16-byte aligned, n_words rounded up to a multiple of 4.
void launch_fetch_words(const int32_t* host_src, int32_t* dst, int64_t n_words, hipStream_t s);

// Checked-mode validation of a batch's ids (and mixed padding).
void launch_validate(const int32_t* anchors, const int32_t* rels, const int32_t* sid_dev,
                     int B, int sa, int sr, int fixed_na, int fixed_nr,
                     int64_t n_ent, int n_rel, int* flag, hipStream_t s);

// GQE / Query2Box translation chains: row dst[c] = E[a] + sum_h C[r_h]
// (Q2B also offset = sum_h softplus(O[r_h])) over chain c's relations
// rel_ref[rel_off[c] .. rel_off[c+1]). Width W = d (GQE) or 2d (Q2B).
void launch_chain(int model, const int32_t* anchor_ref, const int32_t* rel_off, const int32_t* rel_ref,
                  const int32_t* dst_row, int n_chain, const int32_t* anchors, const int32_t* rels,
                  const float* ent_rm, const float* rel_c, const float* rel_o, int64_t n_ent, int n_rel, int d,
                  float* states, int* flag, hipStream_t s);

// Intersection groups of one stage. Group g reads input rows in_start[g] ..
// in_start[g] + n_in[g] - 1 of the stage's block (the `states` argument of
// the combine kernels points at the block; logits, features and BetaE's
// prepared inputs are indexed the same way) and writes row out_row[g] of
// the full state buffer. neg_mask bit j: input j is negated (BetaE). A
// folded post-chain (GQE / Query2Box) adds the relations
// post_ref[post_off[g] .. post_off[g+1]).
constexpr int kGroupInputs = 4;
struct GroupArgs {
    const int32_t* in_start; const int32_t* n_in; const int32_t* out_row;
    const int32_t* neg_mask; const int32_t* post_off; const int32_t* post_ref; int n_groups;
};
void launch_combine_center(int model, const GroupArgs& g, const float* states, int W,
                           const float* logits, const float* zfeat, float* zmean,
                           const int32_t* rels, const float* rel_c, int n_rel, int d,
                           float* out_states, int* flag, hipStream_t s);
// Query2Box offsets: min over branches times sigmoid(gate) (+ post offset).
void launch_combine_offset(const GroupArgs& g, const float* states, int W, const float* gate,
                           const int32_t* rels, const float* rel_o, int n_rel, int d,
                           float* out_states, int* flag, hipStream_t s);

// BetaE: intersection inputs (reciprocal where the branch is negated).
void launch_betae_int_prep(const GroupArgs& g, const float* states, int d, float* x_int,
                           hipStream_t s);
// BetaE: attention-weighted alpha/beta over branches.
void launch_betae_combine(const GroupArgs& g, const float* x_int, const float* logits, int d,
                          float* states, hipStream_t s);
// BetaE projection input rows x = base + Rel[r] (base = a state row, or an
// anchor entity when src_row < 0; its reciprocal where neg[m] != 0, neg may
// be NULL).
void launch_betae_proj_prep(const int32_t* src_row, const int32_t* anchor_ref, const int32_t* rel_ref,
                            const int32_t* neg, int M, const int32_t* anchors, const int32_t* rels,
                            const float* states, const float* ent_ab, const float* rel,
                            int64_t n_ent, int n_rel, int d, float* x, int* flag, hipStream_t s);

// Pack scored rows into the scorer's layout; BetaE also C_q = sum lnB(a, b)
// and the reciprocal of rows with neg[j] != 0 (neg may be NULL).
void launch_pack(int model, const int32_t* src_row, const int32_t* neg, int n_rows, int n_rows_pad,
                 const float* states, int W, int d, float* qpack, double* cq, hipStream_t s);

// ---- ConE / LogicE (k_cone_logice.hip) ----
void launch_cone_entity_prep(const float* src, int64_t N, int d, int64_t n_blocks, float* ent_rm, float* blocked,
                             hipStream_t s);
// Projection input rows: ConE x = source (complemented where neg[m]) +
// Rel[r] (width 2d); LogicE x = [source (complemented where neg[m]); Rel[r]]
// (width 3d). The source is a state row, or the anchor entity when
// src_row[m] < 0.
void launch_mlp_proj_prep(int model, const int32_t* src_row, const int32_t* anchor_ref, const int32_t* rel_ref,
                          const int32_t* neg, int M, const int32_t* anchors, const int32_t* rels,
                          const float* states, const float* ent_rm, const float* rel, int64_t n_ent, int n_rel,
                          int d, float* x, int* flag, hipStream_t s);
// LogicE: u = l + s (1 - l) in the destination rows of a projection level.
void launch_logic_bounds(const int32_t* rowmap, int M, int d, float* states, hipStream_t s);
void launch_cone_int_prep(const GroupArgs& g, const float* states, int d, float* x_int, hipStream_t s);
void launch_cone_combine_axis(const GroupArgs& g, const float* states, const float* logits, const float* hid, int d,
                              float* zmean, float* out_states, hipStream_t s);
void launch_cone_combine_arg(const GroupArgs& g, const float* states, const float* gate, int d, float* out_states,
                             hipStream_t s);
void launch_logic_combine(int tnorm, const GroupArgs& g, const float* states, int d, float* out_states,
                          hipStream_t s);
void launch_pack_cone(const int32_t* src_row, const int32_t* neg, int n_rows, int n_rows_pad, const float* states,
                      int d, float* qpack, hipStream_t s);

// Order-preserving key of a score: unsigned comparison of keys orders the
// scores as floats, -0 and +0 equal (NaNs sort by their bits, above +inf or
// below -inf by sign). Top-k selection and the chunk keys share it.
__device__ __forceinline__ uint32_t score_key(float f)
{
    if (f == 0.0f) f = 0.0f;   // -0 and +0 rank equal
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

constexpr int kKeyChunk = 64;   // entities per chunk key

// s_waitcnt vmcnt(0), other counters not waited for (expcnt 7, lgkmcnt 15).
// A vector load issued after a store waits (vmcnt) for that store too, since
// the counter counts stores as well, in issue order; kernels that store in a
// loop load what the loop needs first and wait for it once with this.
constexpr int kWaitVmcnt0 = 0x0F70;

// Threads per workgroup for a row of `width` floats: one element per thread
// (up to 1,024), so that no thread loads after it has stored.
inline int row_threads(int width) { return std::min(1024, std::max(64, (width + 63) / 64 * 64)); }

// Largest x over each DPP row of 16 lanes (all of them active): swaps of
// neighbours and of pairs inside quads, then the half-row and the row
// mirrored. The scorers' 16 lanes that hold a chunk's 64 scores form one
// DPP row.
__device__ __forceinline__ uint32_t chunk16_max(uint32_t x)
{
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0xB1, 0xF, 0xF, false));    // quad_perm 1,0,3,2
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x4E, 0xF, 0xF, false));    // quad_perm 2,3,0,1
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x141, 0xF, 0xF, false));   // row_half_mirror
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x140, 0xF, 0xF, false));   // row_mirror
    return x;
}

struct ScoreArgs {
    int model;
    const float* qpack; const float* ent; const double* cq; const double* ee;
    // Scored rows: [0, n_quad) groups of four (one output each: the max),
    // then n_pair rows in pairs, then single rows; out_dest lists the output
    // row of each group, pair and single row in that order.
    const int32_t* out_dest;
    int n_rows, n_quad, n_pair, d;
    int64_t N, n_blocks;
    float gamma, center_reg;
    float* scores; int64_t ld;
    // distance scale: score = gamma - dist_scale * distance (GQE 1, LogicE
    // 1 / (2d), ConE its modulus; Query2Box ignores it)
    float dist_scale = 1.0f;
    float* part = nullptr;             // GQE / Query2Box split-d partials for small batches
    int64_t part_elems = 0;            //   (nullptr: never split)
    // BetaE: the [U | V] rows of `ent` split into three bf16 planes (plane
    // stride n_blocks * 256 * 2d) for the bf16 matrix-core contraction, or
    // nullptr for the FP32 one
    const uint16_t* ent_planes = nullptr;
    bool split_always = false;         // the bf16 contraction at any row count (tests)
    // Per output row and chunk of kKeyChunk entities, the largest score_key
    // of the row's scores in the chunk (at least 1), [rows x key_ld] with
    // key_ld >= ceil(N / kKeyChunk), written by the BetaE bf16 contraction
    // and the VALU scorers' unsplit form; nullptr: not written
    uint32_t* chunk_key = nullptr;
    int64_t key_ld = 0;
};
// Filtered answer ranks and per-query [MRR, Hits@1, @3, @10] (k_rank.hip).
void launch_rank_answers(const float* scores, int64_t ld, int64_t N, int batch, const int32_t* off,
                         const int32_t* ids, const int32_t* hard, int32_t* rank, double* metrics, int* flag,
                         hipStream_t s);

// Output of the group, pair or single row that starts at scored row r.
__host__ __device__ inline int score_out_index(int r, int n_quad, int n_pair)
{
    if (r < n_quad) return r >> 2;
    if (r < n_quad + n_pair) return (n_quad >> 2) + ((r - n_quad) >> 1);
    return (n_quad >> 2) + (n_pair >> 1) + (r - n_quad - n_pair);
}

// Both return whether the chunk keys were written (only the bf16 BetaE
// contraction writes them, and only when a.chunk_key is set).
bool launch_score(const ScoreArgs& a, hipStream_t s);      // GQE, Query2Box: VALU
bool launch_score_kl(const ScoreArgs& a, hipStream_t s);   // BetaE: matrix cores

// Top-k works on segments of at most kTopkSegment scores per workgroup;
// longer rows take extra rounds over per-segment candidates.
constexpr int kTopkSegment = 16384;

struct TopkArgs {
    const float* scores; int64_t ld; int64_t N;
    int n_rows;                        // rows 0 .. n_rows-1 of the score buffer
    int k;
    int32_t* out_idx; float* out_score;        // [n_rows x k]
    int32_t* cand_idx[2]; float* cand_score[2]; // scratch for long rows (topk_scratch_elems each)
    // set by launch_topk for each round
    const int32_t* in_idx;             // index of each element (nullptr: its position)
    int64_t seg_len;
    int64_t out_ld;
    int out_rows_per_row;
    // the scorer's chunk keys for rows 0 .. n_rows-1 (ScoreArgs::chunk_key),
    // or nullptr; the first round skips chunks whose key is below its
    // running threshold
    const uint32_t* chunk_key = nullptr;
    int64_t key_ld = 0;
};
// Launches every round; false (nothing launched) when a round needs the
// scratch buffers and they are missing.
bool launch_topk(const TopkArgs& a, hipStream_t s);
int64_t topk_scratch_elems(int64_t n_rows, int64_t N, int k);

}  // namespace kgq
