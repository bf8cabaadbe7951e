// Operator kernels of the two cone / fuzzy-logic models the paper benchmarks
// beside BetaE (Experiments, Baselines; Table 1: ConE and LogicE). Their
// projections share BetaE's plan (per-hop MLP passes on the MFMA GEMM, with
// the first hop's first layer from precomputed tables); what differs, and
// lives here, is each model's state, negation, intersection and packing for
// the scorer.
//
// ConE   state [theta; psi]: per dimension a sector cone with axis theta in
//        [-pi, pi) and half-aperture psi in [0, pi]; an entity is a cone of
//        aperture 0.
//          projection  x = [theta + theta_r; psi + psi_r] -> 3 dense layers ->
//                      theta = pi tanh(y), psi = pi/2 (tanh(2 y') + 1)
//                      (the output maps run in the last layer's epilogue)
//          negation    the complementary cone: theta - pi (theta >= 0) or
//                      theta + pi, and pi - psi
//          intersection u_j = [theta_j - psi_j; theta_j + psi_j]; attention
//                      logits W2 ReLU(W1 u_j + b1) + b2 (2d -> d -> d),
//                      softmax across branches per dimension, axis = angle
//                      of sum_j w_j (cos theta_j, sin theta_j); psi =
//                      min_j psi_j * sigmoid(W4 mean_j ReLU(W3 u_j + b3) + b4).
//                      Both first layers read u_j: they run as one GEMM with
//                      the two weight matrices stacked ([W1; W3], 2d -> 2d).
// LogicE state [l; u]: lower and upper truth bounds in [0, 1], l <= u.
//          projection  x = [l; u; Rel[r]] (width 3d) -> 3 dense layers ->
//                      l = sigmoid(y_l), u = l + sigmoid(y_u) (1 - l)
//                      (sigmoid in the GEMM epilogue, the bound map after it)
//          negation    [l; u] -> [1 - u; 1 - l]
//          intersection a t-norm over the branches, coordinate-wise on the
//                      lower and on the upper bounds (product, minimum or
//                      Lukasiewicz max(0, a + b - 1)), folded from the first
//                      branch on.
// Negation is never a kernel of its own: the plan marks the edges that read
// a negated value (an intersection input, a projection source, a scored
// row), and the reading kernel applies it.
#include <algorithm>

#include "kgq_internal.hpp"

namespace kgq {

constexpr float kPi = 3.14159265358979323846f;

// ConE complement of one dimension's cone.
__device__ __forceinline__ void cone_negate(float& theta, float& psi)
{
    theta = theta >= 0.f ? theta - kPi : theta + kPi;
    psi = kPi - psi;
}

__device__ __forceinline__ int32_t checked_id_cl(int32_t id, int64_t n, int* flag)
{
    if (id < 0 || (int64_t)id >= n) {
        atomicOr(flag, kErrRange);
        return 0;
    }
    return id;
}

// ---------------------------------------------------------------------------
// Load time
// ---------------------------------------------------------------------------

// ConE entity tables: the anchor state [theta; 0] row-major [N x 2d], and the
// scorer's blocked table [block][k][sin(theta/2) (256) | cos(theta/2) (256)]
// (zero past N). The half-angle sines and cosines are computed once here in
// double precision.
__global__ __launch_bounds__(256) void k_cone_entity_prep(const float* src, int64_t N, int d, int64_t n_pad,
                                                          float* ent_rm, float* blocked)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n_pad) return;
    const int64_t blk = e / kEntBlock;
    const int lo = (int)(e % kEntBlock);
    float* dst = blocked + blk * (int64_t)d * 2 * kEntBlock + lo;
    for (int k = 0; k < d; ++k) {
        float s = 0.f, c = 0.f;
        if (e < N) {
            const float th = src[e * d + k];
            ent_rm[e * 2 * d + k] = th;
            ent_rm[e * 2 * d + d + k] = 0.f;
            s = (float)sin(0.5 * (double)th);
            c = (float)cos(0.5 * (double)th);
        }
        dst[(int64_t)k * 2 * kEntBlock] = s;
        dst[(int64_t)k * 2 * kEntBlock + kEntBlock] = c;
    }
}

void launch_cone_entity_prep(const float* src, int64_t N, int d, int64_t n_blocks, float* ent_rm, float* blocked,
                             hipStream_t s)
{
    const int64_t n_pad = n_blocks * kEntBlock;
    hipLaunchKernelGGL(k_cone_entity_prep, dim3((unsigned)((n_pad + 255) / 256)), dim3(256), 0, s, src, N, d, n_pad,
                       ent_rm, blocked);
}

// ---------------------------------------------------------------------------
// Projection inputs (hops whose source is not an anchor, or is negated)
// ---------------------------------------------------------------------------

// x row m: ConE (width 2d) the source state (complemented where neg[m]) plus
// Rel[r]; LogicE (width 3d) [source (complemented where neg[m]); Rel[r]].
template <int MODEL>
__global__ __launch_bounds__(1024) void k_mlp_proj_prep(const int32_t* src_row, const int32_t* anchor_ref,
                                                       const int32_t* rel_ref, const int32_t* neg,
                                                       const int32_t* anchors, const int32_t* rels,
                                                       const float* states, const float* ent_rm, const float* rel,
                                                       int64_t n_ent, int n_rel, int d, float* x, int* flag)
{
    const int m = blockIdx.x;
    const int W = 2 * d;
    const int32_t sr = src_row[m];
    const float* base;
    if (sr >= 0) {
        base = states + (int64_t)sr * W;
    } else {
        const int64_t a = checked_id_cl(anchors[anchor_ref[m]], n_ent, flag);
        base = ent_rm + a * W;
    }
    const bool inv = neg && neg[m];
    const int64_t r = checked_id_cl(rels[rel_ref[m]], n_rel, flag);
    if (MODEL == KGQ_CONE) {
        const float* rr = rel + r * W;
        float* dst = x + (int64_t)m * W;
        for (int k = threadIdx.x; k < d; k += blockDim.x) {
            float th = base[k], ps = base[d + k];
            if (inv) cone_negate(th, ps);
            dst[k] = th + rr[k];
            dst[d + k] = ps + rr[d + k];
        }
    } else {
        const float* rr = rel + r * d;
        float* dst = x + (int64_t)m * 3 * d;
        for (int k = threadIdx.x; k < d; k += blockDim.x) {
            const float l = base[k], u = base[d + k];
            dst[k] = inv ? 1.0f - u : l;
            dst[d + k] = inv ? 1.0f - l : u;
            dst[2 * d + k] = rr[k];
        }
    }
}

void launch_mlp_proj_prep(int model, const int32_t* src_row, const int32_t* anchor_ref, const int32_t* rel_ref,
                          const int32_t* neg, int M, const int32_t* anchors, const int32_t* rels,
                          const float* states, const float* ent_rm, const float* rel, int64_t n_ent, int n_rel,
                          int d, float* x, int* flag, hipStream_t s)
{
    if (M <= 0) return;
    if (model == KGQ_CONE)
        hipLaunchKernelGGL(k_mlp_proj_prep<KGQ_CONE>, dim3(M), dim3(row_threads(d)), 0, s, src_row, anchor_ref, rel_ref, neg,
                           anchors, rels, states, ent_rm, rel, n_ent, n_rel, d, x, flag);
    else
        hipLaunchKernelGGL(k_mlp_proj_prep<KGQ_LOGICE>, dim3(M), dim3(row_threads(d)), 0, s, src_row, anchor_ref, rel_ref, neg,
                           anchors, rels, states, ent_rm, rel, n_ent, n_rel, d, x, flag);
}

// LogicE projection output: the last layer wrote sigmoid(y) into both halves
// of each destination row; turn the upper half into u = l + s (1 - l).
__global__ __launch_bounds__(256) void k_logic_bounds(const int32_t* rowmap, int d, float* states)
{
    float* row = states + (int64_t)rowmap[blockIdx.x] * 2 * d;
    for (int k = threadIdx.x; k < d; k += blockDim.x) {
        const float l = row[k];
        row[d + k] = l + row[d + k] * (1.0f - l);
    }
}

void launch_logic_bounds(const int32_t* rowmap, int M, int d, float* states, hipStream_t s)
{
    if (M <= 0) return;
    hipLaunchKernelGGL(k_logic_bounds, dim3(M), dim3(256), 0, s, rowmap, d, states);
}

// ---------------------------------------------------------------------------
// Intersections (vertical fusion: all branches of a group in one pass)
// ---------------------------------------------------------------------------

// ConE: u_j = [theta_j - psi_j; theta_j + psi_j] of every input row of the
// stage (complemented first where the branch is negated), the input of the
// stacked first layers.
__global__ __launch_bounds__(256) void k_cone_int_prep(GroupArgs g, const float* states, int d, float* x_int)
{
    const int gi = blockIdx.x;
    const int i0 = g.in_start[gi];
    const int n = g.n_in[gi];
    const int neg = g.neg_mask[gi];
    for (int j = 0; j < n; ++j) {
        const bool inv = (neg >> j) & 1;
        const float* src = states + (int64_t)(i0 + j) * 2 * d;
        float* dst = x_int + (int64_t)(i0 + j) * 2 * d;
        for (int k = threadIdx.x; k < d; k += blockDim.x) {
            float th = src[k], ps = src[d + k];
            if (inv) cone_negate(th, ps);
            dst[k] = th - ps;
            dst[d + k] = th + ps;
        }
    }
}

void launch_cone_int_prep(const GroupArgs& g, const float* states, int d, float* x_int, hipStream_t s)
{
    if (g.n_groups <= 0) return;
    hipLaunchKernelGGL(k_cone_int_prep, dim3(g.n_groups), dim3(256), 0, s, g, states, d, x_int);
}

// ConE axis: attention-weighted mean of the branch axes' unit vectors; and
// the mean over branches of the aperture set function's hidden features
// (columns d .. 2d-1 of the stacked first layer's output).
__global__ __launch_bounds__(1024) void k_cone_combine_axis(GroupArgs g, const float* states, const float* logits,
                                                           const float* hid, int d, float* zmean, float* out_states)
{
    const int gi = blockIdx.x;
    const int i0 = g.in_start[gi];
    const int n = g.n_in[gi];
    const int neg = g.neg_mask[gi];
    const int64_t orow = g.out_row[gi];
    for (int k = threadIdx.x; k < d; k += blockDim.x) {
        float mx = logits[(int64_t)i0 * d + k];
        for (int j = 1; j < n; ++j) mx = fmaxf(mx, logits[(int64_t)(i0 + j) * d + k]);
        float z = 0.f, cx = 0.f, sy = 0.f, zm = 0.f;
        for (int j = 0; j < n; ++j) {
            const float w = expf(logits[(int64_t)(i0 + j) * d + k] - mx);
            float th = states[(int64_t)(i0 + j) * 2 * d + k], ps = states[(int64_t)(i0 + j) * 2 * d + d + k];
            if ((neg >> j) & 1) cone_negate(th, ps);
            float sn, cs;
            sincosf(th, &sn, &cs);
            z += w;
            cx += w * cs;
            sy += w * sn;
            zm += hid[(int64_t)(i0 + j) * 2 * d + d + k];
        }
        // the weights' common factor 1/z does not change the angle
        out_states[orow * 2 * d + k] = atan2f(sy / z, cx / z);
        zmean[(int64_t)gi * d + k] = zm / (float)n;
    }
}

void launch_cone_combine_axis(const GroupArgs& g, const float* states, const float* logits, const float* hid, int d,
                              float* zmean, float* out_states, hipStream_t s)
{
    if (g.n_groups <= 0) return;
    hipLaunchKernelGGL(k_cone_combine_axis, dim3(g.n_groups), dim3(row_threads(d)), 0, s, g, states, logits, hid, d, zmean,
                       out_states);
}

// ConE half-aperture: min over branches (complemented where negated) times
// the sigmoid gate.
__global__ __launch_bounds__(1024) void k_cone_combine_arg(GroupArgs g, const float* states, const float* gate, int d,
                                                          float* out_states)
{
    const int gi = blockIdx.x;
    const int i0 = g.in_start[gi];
    const int n = g.n_in[gi];
    const int neg = g.neg_mask[gi];
    const int64_t orow = g.out_row[gi];
    for (int k = threadIdx.x; k < d; k += blockDim.x) {
        float m = 0.f;
        for (int j = 0; j < n; ++j) {
            float ps = states[(int64_t)(i0 + j) * 2 * d + d + k];
            if ((neg >> j) & 1) ps = kPi - ps;
            m = j == 0 ? ps : fminf(m, ps);
        }
        out_states[orow * 2 * d + d + k] = m * (1.0f / (1.0f + expf(-gate[(int64_t)gi * d + k])));
    }
}

void launch_cone_combine_arg(const GroupArgs& g, const float* states, const float* gate, int d, float* out_states,
                             hipStream_t s)
{
    if (g.n_groups <= 0) return;
    hipLaunchKernelGGL(k_cone_combine_arg, dim3(g.n_groups), dim3(row_threads(d)), 0, s, g, states, gate, d, out_states);
}

// LogicE: the t-norm over the branches of each group, coordinate-wise.
template <int TNORM>
__global__ __launch_bounds__(1024) void k_logic_combine(GroupArgs g, const float* states, int d, float* out_states)
{
    const int gi = blockIdx.x;
    const int i0 = g.in_start[gi];
    const int n = g.n_in[gi];
    const int neg = g.neg_mask[gi];
    const int64_t orow = g.out_row[gi];
    for (int k = threadIdx.x; k < d; k += blockDim.x) {
        float lo = 0.f, hi = 0.f;
        for (int j = 0; j < n; ++j) {
            const float* src = states + (int64_t)(i0 + j) * 2 * d;
            float l = src[k], u = src[d + k];
            if ((neg >> j) & 1) {
                const float t = 1.0f - u;
                u = 1.0f - l;
                l = t;
            }
            if (j == 0) {
                lo = l;
                hi = u;
            } else if (TNORM == KGQ_TNORM_MIN) {
                lo = fminf(lo, l);
                hi = fminf(hi, u);
            } else if (TNORM == KGQ_TNORM_LUKASIEWICZ) {
                lo = fmaxf(lo + l - 1.0f, 0.f);
                hi = fmaxf(hi + u - 1.0f, 0.f);
            } else {
                lo *= l;
                hi *= u;
            }
        }
        out_states[orow * 2 * d + k] = lo;
        out_states[orow * 2 * d + d + k] = hi;
    }
}

void launch_logic_combine(int tnorm, const GroupArgs& g, const float* states, int d, float* out_states,
                          hipStream_t s)
{
    if (g.n_groups <= 0) return;
    if (tnorm == KGQ_TNORM_MIN)
        hipLaunchKernelGGL(k_logic_combine<KGQ_TNORM_MIN>, dim3(g.n_groups), dim3(row_threads(d)), 0, s, g, states, d,
                           out_states);
    else if (tnorm == KGQ_TNORM_LUKASIEWICZ)
        hipLaunchKernelGGL(k_logic_combine<KGQ_TNORM_LUKASIEWICZ>, dim3(g.n_groups), dim3(row_threads(d)), 0, s, g, states, d,
                           out_states);
    else
        hipLaunchKernelGGL(k_logic_combine<KGQ_TNORM_PRODUCT>, dim3(g.n_groups), dim3(row_threads(d)), 0, s, g, states, d,
                           out_states);
}

// ---------------------------------------------------------------------------
// ConE query packing for the VALU scorer: [row_block][k][field][TQ] with the
// four fields cos(theta/2), sin(theta/2), cos(psi/2), sin(psi/2) of each
// (complemented where the scored row is negated) query cone. One workgroup
// per block of TQ rows; padding rows are zero.
// ---------------------------------------------------------------------------

template <int TQ>
__global__ __launch_bounds__(256) void k_pack_cone(const int32_t* src_row, const int32_t* neg, int n_rows,
                                                   const float* states, int d, float* qpack)
{
    const int qb = blockIdx.x;
    float* out = qpack + (int64_t)qb * d * 4 * TQ;
    for (int o = threadIdx.x; o < d * TQ; o += blockDim.x) {
        const int i = o % TQ, k = o / TQ;
        const int j = qb * TQ + i;
        float ca = 0.f, sa = 0.f, cb = 0.f, sb = 0.f;
        if (j < n_rows) {
            const float* st = states + (int64_t)src_row[j] * 2 * d;
            float th = st[k], ps = st[d + k];
            if (neg && neg[j]) cone_negate(th, ps);
            sincosf(0.5f * th, &sa, &ca);
            sincosf(0.5f * ps, &sb, &cb);
        }
        float* dst = out + (int64_t)k * 4 * TQ + i;
        dst[0] = ca;
        dst[TQ] = sa;
        dst[2 * TQ] = cb;
        dst[3 * TQ] = sb;
    }
}

void launch_pack_cone(const int32_t* src_row, const int32_t* neg, int n_rows, int n_rows_pad, const float* states,
                      int d, float* qpack, hipStream_t s)
{
    if (n_rows_pad <= 0) return;
    const int tq = score_tq(KGQ_CONE, n_rows);
    const dim3 grid(n_rows_pad / tq);
    if (score_small(n_rows))
        hipLaunchKernelGGL(k_pack_cone<kTqConeSmall>, grid, dim3(256), 0, s, src_row, neg, n_rows, states, d, qpack);
    else
        hipLaunchKernelGGL(k_pack_cone<kTqCone>, grid, dim3(256), 0, s, src_row, neg, n_rows, states, d, qpack);
}

}  // namespace kgq
