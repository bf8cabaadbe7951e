// Query-plan operator kernels other than the dense layers and the scorer:
// parameter re-layout at load time, anchor gathers, translation chains,
// intersection / negation combines, query packing and id validation.
//
// Operators (the paper's Eq. 2 maps a query's relations, conjunctions and
// negations to projection, intersection and negation functions):
//   GQE   projection q + Rel[r]; intersection sum_j softmax_j(s_j) q_j with
//         s_j = W2 ReLU(W1 q_j + b1) + b2 (softmax across branches, per dim).
//   Q2B   projection (c + C[r], o + softplus(O[r])); intersection: attention
//         as above on the centers; offset min_j(o_j) * sigmoid(W4 mean_j
//         ReLU(W3 o_j + b3) + b4).
//   BetaE negation (alpha, beta) -> (1/alpha, 1/beta); intersection:
//         attention weights from [alpha; beta] (W1: 2d -> 2d, W2: 2d -> d),
//         applied to alpha and beta; projection MLP (Eq. 4) runs on the MFMA
//         GEMM, with x = [alpha; beta] + Rel[r] built here.
// Ids read from device memory are range-checked in every kernel that reads
// them: an out-of-range id raises a flag bit and is replaced by 0, so no
// access ever leaves a table.
#include <algorithm>

#include "kgq_internal.hpp"

namespace kgq {

__device__ __forceinline__ float bf16_to_f32(uint16_t h)
{
    return __uint_as_float(((uint32_t)h) << 16);
}

__device__ __forceinline__ float load_param(const void* src, int bf16, int64_t i)
{
    return bf16 ? bf16_to_f32(reinterpret_cast<const uint16_t*>(src)[i])
                : reinterpret_cast<const float*>(src)[i];
}

// ---------------------------------------------------------------------------
// Load-time kernels
// ---------------------------------------------------------------------------

// One thread per entity slot of the padded table; writes the blocked
// dimension-major layout (coalesced across threads) and a row-major copy.
__global__ void k_relayout_points(const void* src, int bf16, int64_t N, int d, int64_t n_pad,
                                  float* rowmajor, float* blocked)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n_pad) return;
    const int64_t blk = e / kEntBlock;
    const int lo = (int)(e % kEntBlock);
    float* dst = blocked + blk * (int64_t)d * kEntBlock + lo;
    for (int k = 0; k < d; ++k) {
        float v = 0.f;
        if (e < N) {
            v = load_param(src, bf16, e * d + k);
            rowmajor[e * d + k] = v;
        }
        dst[(int64_t)k * kEntBlock] = v;
    }
}

void launch_relayout_points(const void* src, int src_bf16, int64_t N, int d, int64_t n_blocks,
                            float* rowmajor, float* blocked, hipStream_t s)
{
    const int64_t n_pad = n_blocks * kEntBlock;
    hipLaunchKernelGGL(k_relayout_points, dim3((unsigned)((n_pad + 255) / 256)), dim3(256), 0, s,
                       src, src_bf16, N, d, n_pad, rowmajor, blocked);
}

// Digamma for x > 0 in double precision: shift the argument up with
// psi(x) = psi(x + 1) - 1/x until x >= 8, then the asymptotic series
// psi(x) = ln x - 1/(2x) - sum_{n>=1} B_2n / (2n x^2n), kept through B_12
// (Abramowitz & Stegun 6.3.18); the first dropped term is below 2e-14 at x = 8.
__device__ double digamma_d(double x)
{
    double shift = 0.0;
    while (x < 8.0) {
        shift -= 1.0 / x;
        x += 1.0;
    }
    const double f = 1.0 / (x * x);
    const double tail = f * (-1.0 / 12.0 + f * (1.0 / 120.0 + f * (-1.0 / 252.0 + f * (1.0 / 240.0
                      + f * (-1.0 / 132.0 + f * (691.0 / 32760.0))))));
    return shift + log(x) - 0.5 / x + tail;
}

// ln Gamma(x) for x >= 8 by Stirling's series (Abramowitz & Stegun 6.1.41),
// kept through the z^-11 term; the first dropped term is below 2e-14 at x = 8.
__device__ __forceinline__ double lngamma_stirling(double x)
{
    const double r = 1.0 / x, f = r * r;
    const double tail = r * (1.0 / 12.0 + f * (-1.0 / 360.0 + f * (1.0 / 1260.0 + f * (-1.0 / 1680.0
                      + f * (1.0 / 1188.0 + f * (-691.0 / 360360.0))))));
    return (x - 0.5) * log(x) - x + 0.91893853320467274178 + tail;   // + ln sqrt(2 pi)
}

// ln B(a, b) = ln Gamma(a) + ln Gamma(b) - ln Gamma(a + b) in double
// precision for a, b > 0. Each argument below 8 is shifted up with
// ln Gamma(x) = ln Gamma(x + 1) - ln x, and the three products of the shifted
// factors share one logarithm (at most 8 factors each, all in (0, 8), so the
// products of fp32-sourced arguments stay within double range). Other
// arguments give NaN: the Beta distribution needs positive shape parameters.
__device__ __forceinline__ double lnbeta_pos(double a, double b)
{
    if (!(a > 0.0 && b > 0.0)) return __builtin_nan("");
    double c = a + b, pa = 1.0, pb = 1.0, pc = 1.0;
    while (a < 8.0) { pa *= a; a += 1.0; }
    while (b < 8.0) { pb *= b; b += 1.0; }
    while (c < 8.0) { pc *= c; c += 1.0; }
    return lngamma_stirling(a) + lngamma_stirling(b) - lngamma_stirling(c) - log((pa / pc) * pb);
}

// The same for any arguments: those that are not positive take the library
// lgamma (for the entity table as loaded; the scored query states are
// regulariser outputs or their reciprocals, always positive).
__device__ __forceinline__ double lnbeta_d(double a, double b)
{
    if (!(a > 0.0 && b > 0.0)) return lgamma(a) + lgamma(b) - lgamma(a + b);
    return lnbeta_pos(a, b);
}

// BetaE entity tables: alpha|beta decoded to fp32 (row-major, for anchor
// gathers), U|V row-major for the matrix-core scorer (zero rows past N), and
// E_e, all from the stored values.
__global__ __launch_bounds__(128) void k_betae_entity_prep(const void* src, int bf16, int64_t N, int d, int64_t n_pad,
                                    float* ab_rowmajor, float* uv_rowmajor, double* e_const)
{
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= n_pad) return;
    float* dst = uv_rowmajor + e * 2 * d;
    double acc = 0.0;
    for (int k = 0; k < d; ++k) {
        float u = 0.f, v = 0.f;
        if (e < N) {
            const float af = load_param(src, bf16, e * 2 * d + k);
            const float bf = load_param(src, bf16, e * 2 * d + d + k);
            ab_rowmajor[e * 2 * d + k] = af;
            ab_rowmajor[e * 2 * d + d + k] = bf;
            const double a = af, b = bf;
            const double pa = digamma_d(a), pb = digamma_d(b), pab = digamma_d(a + b);
            u = (float)(pab - pa);
            v = (float)(pab - pb);
            const double lnb = lnbeta_d(a, b);
            acc += -lnb + a * pa + b * pb - (a + b) * pab;
        }
        dst[k] = u;
        dst[d + k] = v;
    }
    e_const[e] = acc;
}

void launch_betae_entity_prep(const void* src, int src_bf16, int64_t N, int d, int64_t n_blocks,
                              float* ab_rowmajor, float* uv_rowmajor, double* e_const, hipStream_t s)
{
    const int64_t n_pad = n_blocks * kEntBlock;
    hipLaunchKernelGGL(k_betae_entity_prep, dim3((unsigned)((n_pad + 127) / 128)), dim3(128), 0, s,
                       src, src_bf16, N, d, n_pad, ab_rowmajor, uv_rowmajor, e_const);
}

__global__ void k_softplus(const float* src, float* dst, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const double x = src[i];
    dst[i] = (float)((x > 0.0 ? x : 0.0) + log1p(exp(-fabs(x))));
}

void launch_softplus(const float* src, float* dst, int64_t n, hipStream_t s)
{
    hipLaunchKernelGGL(k_softplus, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, dst, n);
}

// ---------------------------------------------------------------------------
// Validation
// ---------------------------------------------------------------------------

__global__ void k_clear_flag(int* flag) { *flag = 0; }

void launch_clear_flag(int* flag, hipStream_t s)
{
    hipLaunchKernelGGL(k_clear_flag, dim3(1), dim3(1), 0, s, flag);
}

// Plan upload: 16-byte words read from pinned host memory (over the bus)
// and written to the device slot, by a kernel in the caller's stream order.
__global__ __launch_bounds__(256) void k_fetch_words(const int4* __restrict__ src, int4* __restrict__ dst,
                                                     int64_t n4)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256)
        dst[i] = src[i];
}

void launch_fetch_words(const int32_t* host_src, int32_t* dst, int64_t n_words, hipStream_t s)
{
    const int64_t n4 = (n_words + 3) / 4;
    if (n4 <= 0) return;
    const int grid = (int)std::min<int64_t>(64, (n4 + 255) / 256);
    hipLaunchKernelGGL(k_fetch_words, dim3(grid), dim3(256), 0, s, reinterpret_cast<const int4*>(host_src),
                       reinterpret_cast<int4*>(dst), n4);
}

__device__ __forceinline__ int32_t checked_id(int32_t id, int64_t n, int* flag)
{
    if (id < 0 || (int64_t)id >= n) {
        atomicOr(flag, kErrRange);
        return 0;
    }
    return id;
}

// arity: one thread per query. For a mixed batch na_q / nr_q hold the
// per-query arity (from the plan) and unused slots must be -1.
__global__ void k_validate(const int32_t* anchors, const int32_t* rels, const int32_t* arity_q,
                           int B, int sa, int sr, int fixed_na, int fixed_nr,
                           int64_t n_ent, int n_rel, int* flag)
{
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= B) return;
    const int na = arity_q ? arity_q[2 * q] : fixed_na;
    const int nr = arity_q ? arity_q[2 * q + 1] : fixed_nr;
    int bits = 0;
    for (int s = 0; s < sa; ++s) {
        const int32_t v = anchors[(int64_t)q * sa + s];
        if (s < na) { if (v < 0 || (int64_t)v >= n_ent) bits |= kErrRange; }
        else if (v != -1) bits |= kErrPadding;
    }
    for (int s = 0; s < sr; ++s) {
        const int32_t v = rels[(int64_t)q * sr + s];
        if (s < nr) { if (v < 0 || v >= n_rel) bits |= kErrRange; }
        else if (v != -1) bits |= kErrPadding;
    }
    if (bits) atomicOr(flag, bits);
}

void launch_validate(const int32_t* anchors, const int32_t* rels, const int32_t* arity_q,
                     int B, int sa, int sr, int fixed_na, int fixed_nr,
                     int64_t n_ent, int n_rel, int* flag, hipStream_t s)
{
    hipLaunchKernelGGL(k_validate, dim3((B + 255) / 256), dim3(256), 0, s, anchors, rels, arity_q,
                       B, sa, sr, fixed_na, fixed_nr, n_ent, n_rel, flag);
}

// ---------------------------------------------------------------------------
// GQE / Query2Box translation chains (horizontal fusion of consecutive
// projections: the whole chain is one pass over the row)
// ---------------------------------------------------------------------------

__global__ void k_chain(int model, const int32_t* anchor_ref, const int32_t* rel_off, const int32_t* rel_ref,
                        const int32_t* dst_row, const int32_t* anchors, const int32_t* rels, const float* ent_rm,
                        const float* rel_c, const float* rel_o, int64_t n_ent, int n_rel, int d, float* states,
                        int* flag)
{
    const int c = blockIdx.x;
    const int64_t a = checked_id(anchors[anchor_ref[c]], n_ent, flag);
    const int h0 = rel_off[c], h1 = rel_off[c + 1];
    const int W = model == 0 ? d : 2 * d;
    float* out = states + (int64_t)dst_row[c] * W;
    // d is a multiple of 4: 128-bit accesses, one float4 per thread per step
    for (int k = threadIdx.x * 4; k < d; k += blockDim.x * 4) {
        float4 x = *reinterpret_cast<const float4*>(ent_rm + a * d + k);
        float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int h = h0; h < h1; ++h) {
            const int64_t r = checked_id(rels[rel_ref[h]], n_rel, flag);
            const float4 v = *reinterpret_cast<const float4*>(rel_c + r * d + k);
            x.x += v.x; x.y += v.y; x.z += v.z; x.w += v.w;
            if (model == 1) {
                const float4 u = *reinterpret_cast<const float4*>(rel_o + r * d + k);
                o.x += u.x; o.y += u.y; o.z += u.z; o.w += u.w;
            }
        }
        *reinterpret_cast<float4*>(out + k) = x;
        if (model == 1) *reinterpret_cast<float4*>(out + d + k) = o;
    }
}

void launch_chain(int model, const int32_t* anchor_ref, const int32_t* rel_off, const int32_t* rel_ref,
                  const int32_t* dst_row, int n_chain, const int32_t* anchors, const int32_t* rels,
                  const float* ent_rm, const float* rel_c, const float* rel_o, int64_t n_ent, int n_rel, int d,
                  float* states, int* flag, hipStream_t s)
{
    if (n_chain <= 0) return;
    hipLaunchKernelGGL(k_chain, dim3(n_chain), dim3(128), 0, s, model, anchor_ref, rel_off, rel_ref, dst_row,
                       anchors, rels, ent_rm, rel_c, rel_o, n_ent, n_rel, d, states, flag);
}

// ---------------------------------------------------------------------------
// Intersections (vertical fusion: all branches of a group in one pass)
// ---------------------------------------------------------------------------

// Attention weights across the n (2 .. kGroupInputs) branches of one
// dimension. Unrolled over the maximum with a guard, so that w stays in
// registers.
__device__ __forceinline__ void softmax_branches(const float* logits, int64_t ld, int n, int k,
                                                 float (&w)[kGroupInputs])
{
    float mx = logits[k];
#pragma unroll
    for (int j = 1; j < kGroupInputs; ++j)
        if (j < n) mx = fmaxf(mx, logits[j * ld + k]);
    float z = 0.f;
#pragma unroll
    for (int j = 0; j < kGroupInputs; ++j) {
        w[j] = j < n ? expf(logits[j * ld + k] - mx) : 0.f;
        z += w[j];
    }
    const float inv = 1.0f / z;
#pragma unroll
    for (int j = 0; j < kGroupInputs; ++j) w[j] *= inv;
}

__global__ void k_combine_center(int model, GroupArgs g, const float* states, int W,
                                 const float* logits, const float* zfeat, float* zmean,
                                 const int32_t* rels, const float* rel_c, int n_rel, int d,
                                 float* out_states, int* flag)
{
    const int gi = blockIdx.x;
    const int i0 = g.in_start[gi];
    const int n = g.n_in[gi];
    const int64_t orow = g.out_row[gi];
    const int p0 = g.post_off[gi], p1 = g.post_off[gi + 1];
    for (int k = threadIdx.x; k < d; k += blockDim.x) {
        float w[kGroupInputs];
        softmax_branches(logits + (int64_t)i0 * d, d, n, k, w);
        float c = 0.f;
        for (int j = 0; j < n; ++j) c += w[j] * states[(int64_t)(i0 + j) * W + k];
        // folded post-chain: the translations of the projections that follow
        for (int h = p0; h < p1; ++h) c += rel_c[(int64_t)checked_id(rels[g.post_ref[h]], n_rel, flag) * d + k];
        out_states[orow * W + k] = c;
        if (model == 1) {
            float z = 0.f;
            for (int j = 0; j < n; ++j) z += zfeat[(int64_t)(i0 + j) * d + k];
            zmean[(int64_t)gi * d + k] = z / (float)n;
        }
    }
}

void launch_combine_center(int model, const GroupArgs& g, const float* states, int W,
                           const float* logits, const float* zfeat, float* zmean,
                           const int32_t* rels, const float* rel_c, int n_rel, int d,
                           float* out_states, int* flag, hipStream_t s)
{
    if (g.n_groups <= 0) return;
    hipLaunchKernelGGL(k_combine_center, dim3(g.n_groups), dim3(row_threads(d)), 0, s, model, g, states, W, logits,
                       zfeat, zmean, rels, rel_c, n_rel, d, out_states, flag);
}

__global__ void k_combine_offset(GroupArgs g, const float* states, int W, const float* gate,
                                 const int32_t* rels, const float* rel_o, int n_rel, int d,
                                 float* out_states, int* flag)
{
    const int gi = blockIdx.x;
    const int i0 = g.in_start[gi];
    const int n = g.n_in[gi];
    const int64_t orow = g.out_row[gi];
    const int p0 = g.post_off[gi], p1 = g.post_off[gi + 1];
    for (int k = threadIdx.x; k < d; k += blockDim.x) {
        float m = states[(int64_t)i0 * W + d + k];
        for (int j = 1; j < n; ++j) m = fminf(m, states[(int64_t)(i0 + j) * W + d + k]);
        const float gv = gate[(int64_t)gi * d + k];
        float o = m * (1.0f / (1.0f + expf(-gv)));
        for (int h = p0; h < p1; ++h) o += rel_o[(int64_t)checked_id(rels[g.post_ref[h]], n_rel, flag) * d + k];
        out_states[orow * W + d + k] = o;
    }
}

void launch_combine_offset(const GroupArgs& g, const float* states, int W, const float* gate,
                           const int32_t* rels, const float* rel_o, int n_rel, int d,
                           float* out_states, int* flag, hipStream_t s)
{
    if (g.n_groups <= 0) return;
    hipLaunchKernelGGL(k_combine_offset, dim3(g.n_groups), dim3(row_threads(d)), 0, s, g, states, W, gate, rels,
                       rel_o, n_rel, d, out_states, flag);
}

// BetaE: copy each intersection input row, inverting both shape parameters
// of negated branches (negation), into the attention MLP input buffer.
__global__ void k_betae_int_prep(GroupArgs g, const float* states, int d, float* x_int)
{
    const int gi = blockIdx.x;
    const int i0 = g.in_start[gi];
    const int n = g.n_in[gi];
    const int neg = g.neg_mask[gi];
    const int W = 2 * d;
    // every input's value read before any is stored: a load issued after a
    // store waits (vmcnt) for that store too
    for (int k = threadIdx.x; k < W; k += blockDim.x) {
        float v[kGroupInputs];
#pragma unroll
        for (int j = 0; j < kGroupInputs; ++j)
            if (j < n) {
                const float x = states[(int64_t)(i0 + j) * W + k];
                v[j] = ((neg >> j) & 1) ? 1.0f / x : x;
            }
#pragma unroll
        for (int j = 0; j < kGroupInputs; ++j)
            if (j < n) x_int[(int64_t)(i0 + j) * W + k] = v[j];
    }
}


void launch_betae_int_prep(const GroupArgs& g, const float* states, int d, float* x_int, hipStream_t s)
{
    if (g.n_groups <= 0) return;
    hipLaunchKernelGGL(k_betae_int_prep, dim3(g.n_groups), dim3(row_threads(2 * d)), 0, s, g, states, d, x_int);
}

__global__ void k_betae_combine(GroupArgs g, const float* x_int, const float* logits, int d, float* states)
{
    const int gi = blockIdx.x;
    const int i0 = g.in_start[gi];
    const int n = g.n_in[gi];
    const int64_t orow = g.out_row[gi];
    const int W = 2 * d;
    for (int k = threadIdx.x; k < d; k += blockDim.x) {
        float w[kGroupInputs];
        softmax_branches(logits + (int64_t)i0 * d, d, n, k, w);
        float al = 0.f, be = 0.f;
        for (int j = 0; j < n; ++j) {
            al += w[j] * x_int[(int64_t)(i0 + j) * W + k];
            be += w[j] * x_int[(int64_t)(i0 + j) * W + d + k];
        }
        states[orow * W + k] = al;
        states[orow * W + d + k] = be;
    }
}

void launch_betae_combine(const GroupArgs& g, const float* x_int, const float* logits, int d,
                          float* states, hipStream_t s)
{
    if (g.n_groups <= 0) return;
    hipLaunchKernelGGL(k_betae_combine, dim3(g.n_groups), dim3(row_threads(d)), 0, s, g, x_int, logits, d, states);
}

__global__ void k_betae_proj_prep(const int32_t* src_row, const int32_t* anchor_ref, const int32_t* rel_ref,
                                  const int32_t* neg, const int32_t* anchors, const int32_t* rels,
                                  const float* states, const float* ent_ab, const float* rel, int64_t n_ent,
                                  int n_rel, int d, float* x, int* flag)
{
    const int m = blockIdx.x;
    const int W = 2 * d;
    const int32_t sr = src_row[m];
    const float* base;
    if (sr >= 0) {
        base = states + (int64_t)sr * W;
    } else {
        const int64_t a = checked_id(anchors[anchor_ref[m]], n_ent, flag);
        base = ent_ab + a * W;
    }
    const bool inv = neg && neg[m];   // negated source: reciprocal of both shape parameters
    const int64_t r = checked_id(rels[rel_ref[m]], n_rel, flag);
    const float* rr = rel + r * W;
    float* dst = x + (int64_t)m * W;
    for (int k = threadIdx.x; k < W; k += blockDim.x) {
        const float v = base[k];
        dst[k] = (inv ? 1.0f / v : v) + rr[k];
    }
}

void launch_betae_proj_prep(const int32_t* src_row, const int32_t* anchor_ref, const int32_t* rel_ref,
                            const int32_t* neg, int M, const int32_t* anchors, const int32_t* rels,
                            const float* states, const float* ent_ab, const float* rel,
                            int64_t n_ent, int n_rel, int d, float* x, int* flag, hipStream_t s)
{
    if (M <= 0) return;
    hipLaunchKernelGGL(k_betae_proj_prep, dim3(M), dim3(row_threads(2 * d)), 0, s, src_row, anchor_ref, rel_ref, neg, anchors,
                       rels, states, ent_ab, rel, n_ent, n_rel, d, x, flag);
}

// BetaE first-hop projection, first layer, from the precomputed tables: the
// layer is linear in its input [alpha; beta] + Rel[r], so
// W1 (E[a] + Rel[r]) + b1 = (E W1^T)[a] + (Rel W1^T + b1)[r].
__global__ __launch_bounds__(256) void k_betae_proj1(const int32_t* anchor_ref, const int32_t* rel_ref,
                                                     const int32_t* anchors, const int32_t* rels, const float* pe,
                                                     const float* pr, int64_t n_ent, int n_rel, int w, float* h1,
                                                     int* flag)
{
    const int m = blockIdx.x;
    const int64_t a = checked_id(anchors[anchor_ref[m]], n_ent, flag);
    const int64_t r = checked_id(rels[rel_ref[m]], n_rel, flag);
    const float* x = pe + a * w;
    const float* y = pr + r * w;
    float* dst = h1 + (int64_t)m * w;
    for (int k = 4 * threadIdx.x; k < w; k += 4 * 256) {      // w = 4d is a multiple of 16
        const float4 u = *reinterpret_cast<const float4*>(x + k);
        const float4 v = *reinterpret_cast<const float4*>(y + k);
        float4 o;
        o.x = fmaxf(u.x + v.x, 0.f);
        o.y = fmaxf(u.y + v.y, 0.f);
        o.z = fmaxf(u.z + v.z, 0.f);
        o.w = fmaxf(u.w + v.w, 0.f);
        *reinterpret_cast<float4*>(dst + k) = o;
    }
}

void launch_betae_proj1(const int32_t* anchor_ref, const int32_t* rel_ref, int M, const int32_t* anchors,
                        const int32_t* rels, const float* pe, const float* pr, int64_t n_ent, int n_rel, int w,
                        float* h1, int* flag, hipStream_t s)
{
    if (M <= 0) return;
    hipLaunchKernelGGL(k_betae_proj1, dim3(M), dim3(256), 0, s, anchor_ref, rel_ref, anchors, rels, pe, pr, n_ent,
                       n_rel, w, h1, flag);
}

// ---------------------------------------------------------------------------
// Query packing for the VALU scorers (GQE, Query2Box, LogicE): [row_block][k][field][TQ].
// One workgroup per block of TQ rows transposes through LDS, KC dimensions at
// a time (as many as a 32 KiB tile holds, so that all loads of a chunk are in
// flight together): the state rows are read along k and the packed block is
// written in its own order, both contiguous.
// ---------------------------------------------------------------------------

// NEGL (LogicE): a row with neg[j] != 0 is packed complemented, [1 - u; 1 - l]
// of its state [l; u] (d = 2 * half coordinates): coordinate c reads the
// state's coordinate (c + half) mod d and packs 1 minus it.
template <int TQ, int F, bool NEGL>
__global__ __launch_bounds__(256) void k_pack(const int32_t* src_row, const int32_t* neg, int half, int n_rows,
                                              const float* states, int W, int d, float* qpack)
{
    // dimensions per chunk: up to a 32 KiB tile (d = 400: one or two
    // chunks), a multiple of 4 so that no float4 straddles two fields
    constexpr int KC = 8192 / (TQ * F) / 4 * 4;
    constexpr int RS = F * KC + 1;            // padded LDS row: the transposed reads hit distinct banks
    __shared__ float tile[TQ * RS];
    __shared__ int srcs[TQ];
    __shared__ int negs[TQ];
    const int qb = blockIdx.x;
    const int t = threadIdx.x;
    if (t < TQ) {
        const int j = qb * TQ + t;
        srcs[t] = j < n_rows ? src_row[j] : -1;
        negs[t] = (NEGL && j < n_rows && neg) ? neg[j] : 0;
    }
    __syncthreads();
    float* out = qpack + (int64_t)qb * d * F * TQ;
    for (int k0 = 0; k0 < d; k0 += KC) {
        const int kc = min(KC, d - k0);           // a multiple of 4
        const int n4 = TQ * F * kc / 4;            // float4 elements of this chunk
        constexpr int PER4 = (TQ * F * KC / 4 + 255) / 256;   // float4 loads per thread (the last may be idle)
        // All loads of the chunk are issued before any is used: each reads a
        // valid address (row 0 for padding rows or past the chunk's end) and
        // the empty asm keeps the compiler from moving a load into the
        // validity branch, where the loads would wait for each other.
        float4 v[PER4];
#pragma unroll
        for (int u = 0; u < PER4; ++u) {
            const int e = 4 * (t + 256 * u);
            const int i = min(e / (F * kc), TQ - 1), rem = e - i * (F * kc);
            const int f = rem / kc, kk = rem - f * kc;
            const int src = srcs[i];
            const bool ok = t + 256 * u < n4 && src >= 0;
            int col = f * d + k0 + kk;
            if (NEGL && negs[i]) col = col >= half ? col - half : col + half;
            const int64_t off = ok ? (int64_t)src * W + col : 0;
            v[u] = *reinterpret_cast<const float4*>(states + off);
        }
#pragma unroll
        for (int u = 0; u < PER4; ++u) asm volatile("" : "+v"(v[u].x), "+v"(v[u].y), "+v"(v[u].z), "+v"(v[u].w));
#pragma unroll
        for (int u = 0; u < PER4; ++u) {
            if (t + 256 * u >= n4) break;
            const int e = 4 * (t + 256 * u);
            const int i = e / (F * kc), rem = e - i * (F * kc);
            const int f = rem / kc, kk = rem - f * kc;
            const bool ok = srcs[i] >= 0;
            float* dst = tile + i * RS + f * KC + kk;
            float4 x = v[u];
            if (NEGL && negs[i]) x = make_float4(1.0f - x.x, 1.0f - x.y, 1.0f - x.z, 1.0f - x.w);
            dst[0] = ok ? x.x : 0.f;
            dst[1] = ok ? x.y : 0.f;
            dst[2] = ok ? x.z : 0.f;
            dst[3] = ok ? x.w : 0.f;
        }
        __syncthreads();
        for (int o = t; o < kc * F * TQ; o += 256) {
            const int i = o % TQ, f = (o / TQ) % F, kk = o / (TQ * F);
            out[(int64_t)k0 * F * TQ + o] = tile[i * RS + f * KC + kk];
        }
        __syncthreads();
    }
}

// BetaE: the query rows row-major, [row][alpha (d) | beta (d)], the A operand
// of the matrix-core scorer, and C_q = sum_i lnB(alpha_i, beta_i) per row in
// double precision (rows are regulariser outputs or their reciprocals, so
// positive; lnbeta_pos keeps the kernel at 45 VGPRs where the library lgamma
// fallback took 176). A negated answer row (neg[j] != 0) is packed as the
// reciprocals of its shape parameters. One workgroup per row; padding rows
// are zero with C_q = 0.
__global__ __launch_bounds__(256) void k_pack_rows(const int32_t* src_row, const int32_t* neg, int n_rows,
                                                   const float* states, int d, float* qrows, double* cq)
{
    __shared__ double part[4];
    const int j = blockIdx.x;
    const int t = threadIdx.x;
    const int src = j < n_rows ? src_row[j] : -1;
    const bool inv = src >= 0 && neg && neg[j];
    const float* st = states + (int64_t)(src >= 0 ? src : 0) * 2 * d;
    float* dst = qrows + (int64_t)j * 2 * d;
    for (int k = 4 * t; k < 2 * d; k += 4 * 256) {
        float4 v = *reinterpret_cast<const float4*>(st + k);
        if (inv) v = make_float4(1.0f / v.x, 1.0f / v.y, 1.0f / v.z, 1.0f / v.w);
        *reinterpret_cast<float4*>(dst + k) = src >= 0 ? v : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    double lnb = 0.0;
    if (src >= 0) {
        for (int k = t; k < d; k += 256) {
            float af = st[k], bf = st[d + k];
            if (inv) {
                af = 1.0f / af;
                bf = 1.0f / bf;
            }
            const double a = af, b = bf;
            lnb += lnbeta_pos(a, b);
        }
    }
    for (int off = 32; off > 0; off >>= 1) lnb += __shfl_xor(lnb, off, 64);
    if ((t & 63) == 0) part[t >> 6] = lnb;
    __syncthreads();
    if (t == 0) cq[j] = (part[0] + part[1]) + (part[2] + part[3]);
}

void launch_pack(int model, const int32_t* src_row, const int32_t* neg, int n_rows, int n_rows_pad,
                 const float* states, int W, int d, float* qpack, double* cq, hipStream_t s)
{
    if (n_rows_pad <= 0) return;
    if (model == KGQ_BETAE) {
        hipLaunchKernelGGL(k_pack_rows, dim3(n_rows_pad), dim3(256), 0, s, src_row, neg, n_rows, states, d, qpack,
                           cq);
        return;
    }
    if (model == KGQ_CONE) {
        launch_pack_cone(src_row, neg, n_rows, n_rows_pad, states, d, qpack, s);
        return;
    }
    const int tq = score_tq(model, n_rows);
    const bool small = score_small(n_rows);
    const dim3 grid(n_rows_pad / tq);          // n_rows_pad is a multiple of score_row_pad, hence of tq
    if (model == KGQ_GQE) {
        if (small) hipLaunchKernelGGL((k_pack<kTqGqeSmall, 1, false>), grid, dim3(256), 0, s, src_row, nullptr, 0, n_rows, states, W, d, qpack);
        else hipLaunchKernelGGL((k_pack<kTqGqe, 1, false>), grid, dim3(256), 0, s, src_row, nullptr, 0, n_rows, states, W, d, qpack);
    } else if (model == KGQ_LOGICE) {
        // the 2d bound coordinates as one field (d here is the width 2d)
        if (small) hipLaunchKernelGGL((k_pack<kTqGqeSmall, 1, true>), grid, dim3(256), 0, s, src_row, neg, d / 2, n_rows, states, W, d, qpack);
        else hipLaunchKernelGGL((k_pack<kTqGqe, 1, true>), grid, dim3(256), 0, s, src_row, neg, d / 2, n_rows, states, W, d, qpack);
    } else {
        if (small) hipLaunchKernelGGL((k_pack<kTqQ2bSmall, 2, false>), grid, dim3(256), 0, s, src_row, nullptr, 0, n_rows, states, W, d, qpack);
        else hipLaunchKernelGGL((k_pack<kTqQ2b, 2, false>), grid, dim3(256), 0, s, src_row, nullptr, 0, n_rows, states, W, d, qpack);
    }
}

}  // namespace kgq
