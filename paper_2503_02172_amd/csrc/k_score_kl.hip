// BetaE entity scoring on the FP32 matrix cores of gfx950.
//
// The score of query row q against entity e is gamma minus the KL divergence
// of the entity's Beta embedding from the query's, summed over dimensions
// (Eq. 3 of the paper defines the Beta embedding). Regrouped exactly,
//   sum_i KL(Beta(a_i, b_i) || Beta(alpha_i, beta_i))
//     = C_q + E_e + sum_i (alpha_i * U_i + beta_i * V_i),
// with U = psi(a + b) - psi(a), V = psi(a + b) - psi(b) and the per-entity
// constant E_e built at load time, the per-query constant C_q built by the
// pack kernel. The sum is a dense [rows x 2d] . [2d x N] contraction of the
// packed query rows [alpha | beta] with the entity rows [U | V], so it runs
// on v_mfma_f32_16x16x4_f32 (full FP32 inputs and accumulation); the VALU
// form is bound by the half-rate FMA issue of the vector units.
//
// Tiling: a workgroup of 4 wavefronts (2 x 2) owns a 64-row x 128-entity tile
// of scores; each wavefront computes 2 x 4 MFMA tiles of 16 x 16. K advances
// 32 at a time through double-buffered LDS (one barrier per step), the next
// step's global loads in registers while the current step computes. Within
// a 16-wide K slice, lane group g = lane / 16 feeds k = 4g .. 4g + 3 to four
// consecutive MFMAs from one 128-bit LDS read (a permutation of the
// reduction order). The epilogue adds C_q + E_e in double precision, takes
// the max over union pairs (two adjacent rows, held by the same lane), and
// scatters rows to their output positions. Workgroups are ordered so that
// each XCD takes a chunk of row tiles and sweeps every entity tile.
#include <algorithm>

#include "kgq_internal.hpp"

namespace kgq {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int KL_BM = 64;           // query rows per workgroup tile
constexpr int KL_BN = 128;          // entities per workgroup tile
constexpr int KL_BK = 32;           // K per LDS stage
constexpr int KL_LD = KL_BK + 4;    // padded LDS row (floats)

__global__ __launch_bounds__(256, 2) void k_score_kl(ScoreArgs a, int n_mt, int n_nt, int qchunk, int total,
                                                     int per_xcd)
{
    __shared__ float As[2][KL_BM * KL_LD];
    __shared__ float Bs[2][KL_BN * KL_LD];

    // XCD-aware order (workgroup b runs on XCD b % 8): chunks of qchunk row
    // tiles, then entity tiles, then the chunk's row tiles.
    const int b = blockIdx.x;
    const int L = (b & 7) * per_xcd + (b >> 3);
    if (L >= total) return;
    const int chunk_wg = qchunk * n_nt;
    const int c = L / chunk_wg;
    const int r = L - c * chunk_wg;
    const int qcc = min(qchunk, n_mt - c * qchunk);
    const int nt = r / qcc;
    const int mt = c * qchunk + (r - nt * qcc);
    const int m0 = mt * KL_BM, n0 = nt * KL_BN;

    const int K = 2 * a.d;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;   // wavefront tile: rows [wm*32, +32), entities [wn*64, +64)
    const int grp = lane >> 4, li = lane & 15;

    // global -> register staging: thread t loads k = (t % 8) * 4 .. +3 of
    // rows t / 8 + 32 h (A: h < 2, B: h < 4). The query rows are padded to a
    // multiple of 64 and the entity rows to a multiple of 256, so every row
    // index is inside its buffer; only the K tail needs a check.
    const int lrow = tid >> 3, lk = (tid & 7) * 4;
    const float* __restrict__ A = a.qpack + (int64_t)(m0 + lrow) * K + lk;
    const float* __restrict__ B = a.ent + (int64_t)(n0 + lrow) * K + lk;
    float4 ra[2], rb[4];
    auto load = [&](int k0) {
        const bool ok = k0 + lk < K;
#pragma unroll
        for (int h = 0; h < 2; ++h)
            ra[h] = ok ? *reinterpret_cast<const float4*>(A + (int64_t)h * 32 * K + k0) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int h = 0; h < 4; ++h)
            rb[h] = ok ? *reinterpret_cast<const float4*>(B + (int64_t)h * 32 * K + k0) : make_float4(0.f, 0.f, 0.f, 0.f);
    };
    auto stash = [&](int buf) {
#pragma unroll
        for (int h = 0; h < 2; ++h) *reinterpret_cast<float4*>(&As[buf][(lrow + 32 * h) * KL_LD + lk]) = ra[h];
#pragma unroll
        for (int h = 0; h < 4; ++h) *reinterpret_cast<float4*>(&Bs[buf][(lrow + 32 * h) * KL_LD + lk]) = rb[h];
    };

    v4f acc[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    const int nk = (K + KL_BK - 1) / KL_BK;
    load(0);
    stash(0);
    __syncthreads();
    int buf = 0;
    for (int kt = 0; kt < nk; ++kt) {
        if (kt + 1 < nk) load((kt + 1) * KL_BK);
#pragma unroll
        for (int s = 0; s < KL_BK / 16; ++s) {
            float4 av[2], bv[4];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                av[i] = *reinterpret_cast<const float4*>(&As[buf][(wm * 32 + i * 16 + li) * KL_LD + s * 16 + grp * 4]);
#pragma unroll
            for (int j = 0; j < 4; ++j)
                bv[j] = *reinterpret_cast<const float4*>(&Bs[buf][(wn * 64 + j * 16 + li) * KL_LD + s * 16 + grp * 4]);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].x, bv[j].x, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].y, bv[j].y, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].z, bv[j].z, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].w, bv[j].w, acc[i][j], 0, 0, 0);
                }
        }
        if (kt + 1 < nk) {
            buf ^= 1;
            stash(buf);
            __syncthreads();
        }
    }

    // Epilogue. MFMA output layout: lane holds entity column li of its tile
    // and rows 4 * grp + r, r = 0..3. Union pairs are rows (2p, 2p + 1),
    // i.e. r = 0, 1 and r = 2, 3 of one lane.
    const int nu_pairs = a.n_union_rows >> 1;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int64_t n = n0 + wn * 64 + j * 16 + li;
        if (n >= a.N) continue;
        const double ee = a.ee[n];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int mb = m0 + wm * 32 + i * 16 + grp * 4;
            float s[4];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                s[q] = (float)((double)a.gamma - (a.cq[mb + q] + ee + (double)acc[i][j][q]));
#pragma unroll
            for (int pr = 0; pr < 2; ++pr) {
                const int m = mb + 2 * pr;
                if (m >= a.n_rows) break;
                if (m < a.n_union_rows) {
                    a.scores[(int64_t)a.out_dest[m >> 1] * a.ld + n] = fmaxf(s[2 * pr], s[2 * pr + 1]);
                } else {
                    const int o = nu_pairs + (m - a.n_union_rows);
                    a.scores[(int64_t)a.out_dest[o] * a.ld + n] = s[2 * pr];
                    if (m + 1 < a.n_rows) a.scores[(int64_t)a.out_dest[o + 1] * a.ld + n] = s[2 * pr + 1];
                }
            }
        }
    }
}

void launch_score_kl(const ScoreArgs& a, hipStream_t s)
{
    if (a.n_rows <= 0) return;
    const int n_mt = (a.n_rows + KL_BM - 1) / KL_BM;
    const int n_nt = (int)((a.N + KL_BN - 1) / KL_BN);
    const int total = n_mt * n_nt;
    const int per_xcd = (total + 7) / 8;
    // row-tile chunk per XCD: an eighth of the row tiles, at most ~2 MiB of queries
    const int64_t tile_bytes = (int64_t)KL_BM * 2 * a.d * 4;
    int qchunk = (n_mt + 7) / 8;
    qchunk = (int)std::min<int64_t>(qchunk, std::max<int64_t>(1, (int64_t)(2 << 20) / tile_bytes));
    hipLaunchKernelGGL(k_score_kl, dim3(per_xcd * 8), dim3(256), 0, s, a, n_mt, n_nt, qchunk, total, per_xcd);
}

}  // namespace kgq
