// Entity scoring for GQE, Query2Box, ConE and LogicE: the entity-similarity
// step that the paper times together with operator execution (Experiments,
// Metrics): every query embedding is scored against every entity. (BetaE's
// regrouped KL score is a dense contraction and runs on the matrix cores,
// k_score_kl.hip.) LogicE's score is GQE's L1 distance over its 2d bound
// coordinates, scaled by 1 / (2d).
//
// This is VALU work, not a dense contraction: per (query, entity, dim)
// triple GQE needs |q - e| accumulated, Query2Box a box distance. The kernel
// is organised like a register-blocked GEMM without the multiply-add:
//   - a lane owns 4 consecutive entities (one 128-bit load per dimension
//     from the blocked, dimension-major entity table);
//   - a wavefront owns kTq query rows that are uniform across its lanes, so
//     the query values come through the scalar cache into SGPRs and feed the
//     VALU as scalar operands: no LDS traffic and no cross-lane reduction;
//   - the 4 wavefronts of a workgroup share one entity block (L1 reuse), and
//     workgroups are ordered in chunks of query groups (~2 MiB of packed
//     queries), each swept against every entity block: the chunk's queries
//     stay in L2 for the whole sweep and the entity table is fetched once
//     per chunk (entity-block-major order would instead re-fetch every query
//     once per entity block).
//
// Per-triple work (one non-packed VALU op each):
//   GQE     d = e - q;  acc += |d|                                       (2)
//   Q2B     t = |e - c|: acc1 += t; acc2 += min(t, o)                    (4)
//           score = gamma - acc1 + (1 - center_reg) * acc2, the exact
//           regrouping of dist_out + center_reg * dist_in
//           (t <= o: center_reg * t; t > o: (t - o) + center_reg * o)
//   ConE    with the entity's half-angle sine / cosine (Se, Ce) from the
//           table and the query's (Ca, Sa) of theta/2 and (Cb, Sb) of psi/2:
//           s = Se Ca - Ce Sa = sin((theta_e - theta)/2),
//           c = Ce Ca + Se Sa = cos((theta_e - theta)/2),
//           t = |s| Cb - |c| Sb;  acc1 += max(t, 0);  acc2 += min(|s|, Sb) (10,
//           plus Cb and Sb moved to vector registers once per row and step)
//           score = gamma - modulus (acc1 + center_reg acc2). This is the
//           sector distance exactly: min(|sin(a + b)|, |sin(a - b)|) =
//           ||sin a| cos b - |cos a| sin b| for b = psi/2 in [0, pi/2], and
//           the bracket is negative exactly when |sin a| < sin b, i.e. inside
//           the sector, where the outside distance is 0.
// Union (disjunctive normal form, Eq. 1 of the paper): a query whose answer
// has 2 conjunctive terms has two adjacent rows (a pair), one with 3 or 4
// terms a group of four rows; its score is the max over the rows' scores.
// Groups come first, then pairs, then single rows, so that every group and
// pair lies inside one lane's TQ rows.
#include <algorithm>
#include <type_traits>

#include "kgq_internal.hpp"

namespace kgq {

// A lane's four consecutive scores of one output row: one 16-byte
// non-temporal store (rows start only 4-byte aligned; gfx950 takes
// dword-aligned multi-dword global stores), element stores at the ragged end
// of the row. Non-temporal: the score matrix streams past L2 instead of
// evicting the packed queries that the other entity blocks still read, and
// a wavefront writes whole lines.
typedef float f4u_t __attribute__((ext_vector_type(4), aligned(4)));

__device__ __forceinline__ void store_scores4(float* dst, int64_t e0, int64_t N, const float (&v)[4])
{
    if (e0 + 3 < N) {
        __builtin_nontemporal_store((f4u_t){v[0], v[1], v[2], v[3]}, reinterpret_cast<f4u_t*>(dst + e0));
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            if (e0 + j < N) __builtin_nontemporal_store(v[j], dst + e0 + j);
    }
}

// score_key in integer operations only (this file is built without NaN
// semantics, so no float compare decides it): -0 becomes +0, then the sign
// flips the other bits or sets the top one.
__device__ __forceinline__ uint32_t score_key_bits(float f)
{
    uint32_t u = __float_as_uint(f);
    u = u == 0x80000000u ? 0u : u;
    return u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
}

// One output row's four scores of the lane (entities e0 .. e0 + 3): stored,
// and, when keys are wanted, folded into the row's chunk key (the 16 lanes of
// a 64-entity chunk are one DPP row; entities past N count as key 0). Called
// by the whole wavefront.
__device__ __forceinline__ void store_row(const ScoreArgs& a, int64_t orow, int64_t e0, int lane, const float (&v)[4])
{
    if (a.chunk_key) {
        uint32_t kx = 0u;
#pragma unroll
        for (int j = 0; j < 4; ++j) kx = max(kx, e0 + j < a.N ? score_key_bits(v[j]) : 0u);
        kx = chunk16_max(kx);
        if ((lane & 15) == 0 && e0 < a.N) a.chunk_key[orow * a.key_ld + e0 / kKeyChunk] = max(kx, 1u);
    }
    store_scores4(a.scores + orow * a.ld, e0, a.N, v);
}

template <int MODEL, int TQ>
__global__ __launch_bounds__(256) void k_score(ScoreArgs a, int nqg, int qchunk, int total_wg, int wg_per_xcd,
                                               int kslice)
{
    // XCD-aware mapping: workgroup b runs on XCD b % 8 (round-robin dispatch),
    // so XCD x executes positions [x * wg_per_xcd, (x + 1) * wg_per_xcd) of
    // the global order, in order. The global order is: query chunks of qchunk
    // query groups (the last one may be short); within a chunk, entity blocks;
    // within an entity block, the chunk's query groups.
    const int b = blockIdx.x;
    const int L = (b & 7) * wg_per_xcd + (b >> 3);
    if (L >= total_wg) return;
    const int chunk_wg = qchunk * (int)a.n_blocks;
    const int c = L / chunk_wg;
    const int r = L - c * chunk_wg;
    const int qcc = min(qchunk, nqg - c * qchunk);     // query groups in this chunk
    const int eb = r / qcc;
    const int qg = c * qchunk + (r - eb * qcc);
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    const int qb = qg * 4 + wave;
    if (qb * TQ >= a.n_rows) return;

    constexpr int F = (MODEL == 0) ? 1 : (MODEL == 1 ? 2 : 4);   // query fields per row
    constexpr int EF = (MODEL == 3) ? 2 : 1;                       // entity fields per dimension
    constexpr bool TWO = MODEL != 0;                               // two accumulators per triple
    constexpr int AF = TWO ? 2 : 1;                                // accumulator fields (split-d partials)
    // Small batches split the dimensions over blockIdx.y: slice z covers
    // [z * kslice, z * kslice + d) (kslice and d multiples of 4) and writes
    // its raw accumulators to a.part instead of scores.
    const int k_begin = blockIdx.y * kslice;
    const int d = min(kslice, a.d - k_begin);
    const float* __restrict__ qp = a.qpack + ((int64_t)qb * a.d + k_begin) * F * TQ;
    const float* __restrict__ ep = a.ent + ((int64_t)eb * a.d + k_begin) * EF * kEntBlock + lane * 4;

    float acc[TQ][4];
    float acc2[TWO ? TQ : 1][4];
#pragma unroll
    for (int i = 0; i < TQ; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
#pragma unroll
    for (int i = 0; i < (TWO ? TQ : 1); ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc2[i][j] = 0.f;

    // Software pipeline, two steps per trip with named buffers A and B: a
    // step's entity vector(s) are requested a step ahead, and its query
    // scalars half a step ahead, after the previous wait (scalar loads may
    // return out of order, so each wait on them covers every one
    // outstanding). d is even (a multiple of 4).
    constexpr int QN = F * TQ;
    // The packed queries are read-only for the whole kernel; reading them
    // through the constant address space keeps them on scalar loads.
    const __attribute__((address_space(4))) float* qc = (const __attribute__((address_space(4))) float*)qp;
    // a step's entity vectors: EF float4 (ConE: sines, then cosines)
    struct EVec {
        float4 v[EF];
    };
    auto load_e = [&](int k, EVec& u) {
#pragma unroll
        for (int f = 0; f < EF; ++f)
            u.v[f] = *reinterpret_cast<const float4*>(ep + ((int64_t)k * EF + f) * kEntBlock);
    };
    // rows [R0, R1) of one step
    auto compute = [&](const EVec& eu, const float* qv, auto R0c, auto R1c) {
        constexpr int R0 = decltype(R0c)::value, R1 = decltype(R1c)::value;
        const float e4[4] = {eu.v[0].x, eu.v[0].y, eu.v[0].z, eu.v[0].w};
#pragma unroll
        for (int i = R0; i < R1; ++i) {
            const float c = qv[i];
            if (MODEL == 0) {
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] += fabsf(e4[j] - c);
            } else if (MODEL == 3) {
                const float ce4[4] = {eu.v[EF - 1].x, eu.v[EF - 1].y, eu.v[EF - 1].z, eu.v[EF - 1].w};
                const float sa = qv[TQ + i];
                // the aperture's cosine and sine as vector operands: the VALU
                // takes a scalar operand on at most every other issue cycle,
                // and with them in SGPRs 7 of the triple's 10 instructions
                // would read one (2 moves per row and step, per 4 triples:
                // the scorer at the 14,505-entity ConE workload went from
                // 4.75 to 4.00 ms)
                float cb, sb;
                asm("v_mov_b32 %0, %1" : "=v"(cb) : "s"(qv[2 * TQ + i]));
                asm("v_mov_b32 %0, %1" : "=v"(sb) : "s"(qv[3 * TQ + i]));
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float sn = fmaf(-ce4[j], sa, e4[j] * c);    // sin((theta_e - theta) / 2)
                    const float cs = fmaf(e4[j], sa, ce4[j] * c);     // cos((theta_e - theta) / 2)
                    const float as = fabsf(sn);
                    const float t = fmaf(-fabsf(cs), sb, as * cb);
                    acc[i][j] += __builtin_fmaxf(t, 0.f);
                    acc2[i][j] += __builtin_fminf(as, sb);
                }
            } else {
                const float o = qv[TQ + i];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float t = fabsf(e4[j] - c);
                    acc[i][j] += t;
                    acc2[i][j] += __builtin_fminf(t, o);
                }
            }
        }
    };
    using H0 = std::integral_constant<int, 0>;
    using H1 = std::integral_constant<int, TQ / 2>;
    using H2 = std::integral_constant<int, TQ>;
    EVec ua, ub;
    float qa[QN], qb2[QN];
    load_e(0, ua);
#pragma unroll
    for (int t = 0; t < QN; ++t) qa[t] = qc[t];
    for (int k = 0; k < d; k += 2) {
        load_e(k + 1, ub);                                  // B <- step k + 1
        __builtin_amdgcn_sched_barrier(0);
        compute(ua, qa, H0{}, H1{});
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < QN; ++t) qb2[t] = qc[(k + 1) * QN + t];
        __builtin_amdgcn_sched_barrier(0);
        compute(ua, qa, H1{}, H2{});
        const int k2 = (k + 2 < d) ? k + 2 : k + 1;         // A <- step k + 2 (last trip: in bounds, unused)
        load_e(k2, ua);
        __builtin_amdgcn_sched_barrier(0);
        compute(ub, qb2, H0{}, H1{});
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int t = 0; t < QN; ++t) qa[t] = qc[k2 * QN + t];
        __builtin_amdgcn_sched_barrier(0);
        compute(ub, qb2, H1{}, H2{});
    }

    // Epilogue: finish the scores, merge union pairs, store.
    const int64_t e0 = (int64_t)eb * kEntBlock + lane * 4;
    if (a.part) {
        // split-d: raw accumulators of this slice, [slice][field][row][entity]
        // over the padded rows (nqg * 4 * TQ) and entities (n_blocks * 256)
        const int64_t n_pad = a.n_blocks * kEntBlock, rows_pad = (int64_t)nqg * 4 * TQ;
        float* pz = a.part + (int64_t)blockIdx.y * AF * rows_pad * n_pad;
#pragma unroll
        for (int i = 0; i < TQ; ++i) {
            const int64_t row = (int64_t)qb * TQ + i;
            *reinterpret_cast<float4*>(pz + row * n_pad + e0) = make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
            if (TWO)
                *reinterpret_cast<float4*>(pz + (rows_pad + row) * n_pad + e0) =
                    make_float4(acc2[i][0], acc2[i][1], acc2[i][2], acc2[i][3]);
        }
        return;
    }
    const int n_grouped = a.n_quad + a.n_pair;
    // Output row of each of the wavefront's rows (a group's or pair's rows
    // share theirs), loaded before the first store and waited for once: a
    // load issued between the stores would wait (vmcnt) for the stores before
    // it as well. Lane i loads row i's (rows past the last clamped to it),
    // and each is then read from its lane.
    static_assert(TQ <= 64, "one row per lane");
    const int32_t od_lane =
        a.out_dest[score_out_index(min(qb * TQ + min(lane, TQ - 1), a.n_rows - 1), a.n_quad, a.n_pair)];
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    int32_t od[TQ];
#pragma unroll
    for (int i = 0; i < TQ; ++i) od[i] = __builtin_amdgcn_readlane(od_lane, i);
#pragma unroll
    for (int i = 0; i < TQ; i += 4) {
        const int row = qb * TQ + i;
        if (row >= a.n_rows) break;
        float sc[4][4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (MODEL == 0) sc[u][j] = a.gamma - a.dist_scale * acc[i + u][j];
                else if (MODEL == 3) sc[u][j] = a.gamma - a.dist_scale * fmaf(a.center_reg, acc2[i + u][j], acc[i + u][j]);
                else sc[u][j] = a.gamma - acc[i + u][j] + (1.0f - a.center_reg) * acc2[i + u][j];
            }
        if (row < a.n_quad) {
            float v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = fmaxf(fmaxf(sc[0][j], sc[1][j]), fmaxf(sc[2][j], sc[3][j]));
            store_row(a, od[i], e0, lane, v);
            continue;
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int r = row + 2 * h;
            if (r >= a.n_rows) break;
            if (r < n_grouped) {
                float v[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) v[j] = fmaxf(sc[2 * h][j], sc[2 * h + 1][j]);
                store_row(a, od[i + 2 * h], e0, lane, v);
            } else {
                store_row(a, od[i + 2 * h], e0, lane, sc[2 * h]);
                if (r + 1 < a.n_rows) store_row(a, od[i + 2 * h + 1], e0, lane, sc[2 * h + 1]);
            }
        }
    }
}

// Split-d finish: output o (groups of four, then pairs, then single rows,
// the order of out_dest) and entity e: sum the slices in order, score, max
// over the output's rows, store.
template <int MODEL>
__global__ __launch_bounds__(256) void k_score_sum(ScoreArgs a, int splits, int64_t rows_pad, int n_out)
{
    constexpr int F = (MODEL == 0) ? 1 : 2;     // accumulator fields of the partials (as AF in k_score)
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= (int64_t)n_out * a.N) return;
    const int o = (int)(t / a.N);
    const int64_t e = t - (int64_t)o * a.N;
    const int64_t n_pad = a.n_blocks * kEntBlock;
    const int nq = a.n_quad >> 2, np = a.n_pair >> 1;
    int r0, nr;
    if (o < nq) {
        r0 = 4 * o;
        nr = 4;
    } else if (o < nq + np) {
        r0 = a.n_quad + 2 * (o - nq);
        nr = 2;
    } else {
        r0 = a.n_quad + a.n_pair + (o - nq - np);
        nr = 1;
    }
    float best = 0.f;
    for (int u = 0; u < nr; ++u) {
        float s1 = 0.f, s2 = 0.f;
        for (int z = 0; z < splits; ++z) {
            const float* pz = a.part + (int64_t)z * F * rows_pad * n_pad;
            s1 += pz[(int64_t)(r0 + u) * n_pad + e];
            if (MODEL != 0) s2 += pz[(rows_pad + r0 + u) * n_pad + e];
        }
        const float v = MODEL == 0   ? a.gamma - a.dist_scale * s1
                        : MODEL == 3 ? a.gamma - a.dist_scale * fmaf(a.center_reg, s2, s1)
                                     : a.gamma - s1 + (1.0f - a.center_reg) * s2;
        best = u == 0 ? v : fmaxf(best, v);
    }
    a.scores[(int64_t)a.out_dest[o] * a.ld + e] = best;
}

bool launch_score(const ScoreArgs& a, hipStream_t s)
{
    if (a.n_rows <= 0) return false;
    if (a.model == KGQ_BETAE) return launch_score_kl(a, s);
    const int form = valu_form(a.model);           // LogicE runs GQE's kernel
    const int tq = score_tq(a.model, a.n_rows);    // the pack's layout for this row count
    const bool small = score_small(a.n_rows);
    const int nqb = (a.n_rows + tq - 1) / tq;
    const int nqg = (nqb + 3) / 4;
    const int total = (int)(a.n_blocks * nqg);
    const int per_xcd = (total + 7) / 8;
    const int QF = form == KGQ_GQE ? 1 : (form == KGQ_Q2B ? 2 : 4);   // query fields
    // query chunk: as many query groups as ~2 MiB of packed queries (about
    // half an XCD's L2); the entity table is streamed once per chunk, and the
    // XCDs split the global order evenly whatever the chunk size
    const int64_t qg_bytes = (int64_t)4 * tq * a.d * QF * 4;   // packed queries of one group
    const int qc = (int)std::min<int64_t>(nqg, std::max<int64_t>(1, (int64_t)(2 << 20) / qg_bytes));
    // Small batches: with fewer than 128 workgroups the dimension loop is a
    // latency chain on a few compute units, so the dimensions are split over
    // up to 16 slices (each at least 16 dimensions) whose partials fit the
    // lane's workspace; a second kernel sums them.
    const int F = form == KGQ_GQE ? 1 : 2;         // accumulator fields
    const int64_t rows_pad = (int64_t)nqg * 4 * tq, n_pad = a.n_blocks * kEntBlock;
    int splits = 1;
    if (a.part && total < 128 && a.d >= 32) {
        splits = std::min({16, (512 + total - 1) / total, a.d / 16});
        while (splits > 1 && (int64_t)splits * F * rows_pad * n_pad > a.part_elems) --splits;
    }
    ScoreArgs b = a;
    int kslice = a.d, z = 1;
    if (splits > 1) {
        kslice = (((a.d + splits - 1) / splits) + 3) / 4 * 4;
        z = (a.d + kslice - 1) / kslice;
    } else {
        b.part = nullptr;
    }
    if (splits > 1) b.chunk_key = nullptr;   // the split-d sum writes no keys
    dim3 grid(per_xcd * 8, z);
    if (form == KGQ_GQE) {
        if (small) hipLaunchKernelGGL((k_score<0, kTqGqeSmall>), grid, dim3(256), 0, s, b, nqg, qc, total, per_xcd, kslice);
        else hipLaunchKernelGGL((k_score<0, kTqGqe>), grid, dim3(256), 0, s, b, nqg, qc, total, per_xcd, kslice);
    } else if (form == KGQ_Q2B) {
        if (small) hipLaunchKernelGGL((k_score<1, kTqQ2bSmall>), grid, dim3(256), 0, s, b, nqg, qc, total, per_xcd, kslice);
        else hipLaunchKernelGGL((k_score<1, kTqQ2b>), grid, dim3(256), 0, s, b, nqg, qc, total, per_xcd, kslice);
    } else {
        if (small) hipLaunchKernelGGL((k_score<3, kTqConeSmall>), grid, dim3(256), 0, s, b, nqg, qc, total, per_xcd, kslice);
        else hipLaunchKernelGGL((k_score<3, kTqCone>), grid, dim3(256), 0, s, b, nqg, qc, total, per_xcd, kslice);
    }
    if (z > 1) {
        const int n_out = (a.n_quad >> 2) + (a.n_pair >> 1) + (a.n_rows - a.n_quad - a.n_pair);
        const int64_t tot = (int64_t)n_out * a.N;
        const dim3 g2((unsigned)((tot + 255) / 256));
        if (form == KGQ_GQE)
            hipLaunchKernelGGL((k_score_sum<0>), g2, dim3(256), 0, s, b, z, rows_pad, n_out);
        else if (form == KGQ_Q2B)
            hipLaunchKernelGGL((k_score_sum<1>), g2, dim3(256), 0, s, b, z, rows_pad, n_out);
        else
            hipLaunchKernelGGL((k_score_sum<3>), g2, dim3(256), 0, s, b, z, rows_pad, n_out);
    }
    return b.chunk_key != nullptr;
}

}  // namespace kgq
