// BetaE entity scoring on the matrix cores of gfx950.
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
// on the matrix cores; the VALU form is bound by the half-rate FMA issue of
// the vector units.
//
// Tiling (mfma_tile.hpp). When 2d is a multiple of 32 and the [U | V] rows
// have been split into three bf16 planes at load, the contraction runs on
// v_mfma_f32_16x16x32_bf16 with the query rows split in registers and six
// part products kept: FP32 accuracy at 0.375 of the FP32 matrix-core time per
// k range (MfmaTileBf16x3 with 128-row x 128-entity tiles, 4 x 1
// wavefronts and raised issue priority while fragments are read and split,
// an 80 KiB LDS ring; 1.7x faster than the FP32 loop at the 63,361-entity
// workload, and 6% faster than 128 x 64 tiles).
// Otherwise 64-row x 64-entity tiles, 2 x 2 MFMA tiles of 16 x 16 per
// wavefront, on v_mfma_f32_16x16x4_f32 with full FP32 inputs: through the
// direct-to-LDS ring of three stages when 2d is a multiple of 16 (measured
// faster, epilogue included, than 128 x 64, 64 x 128 or 128 x 128 tiles and
// than two or four stages), else the register-staged loop with 128 x 128
// tiles. The epilogue adds
// C_q + E_e in double precision, stages the output tile in LDS, takes the
// max over union groups of four and pairs of rows and writes each output
// row with 16-byte non-temporal stores. On the 128-entity bf16 tiles it also
// writes, per output row and chunk of 64 entities, the largest key of the
// chunk's scores, from which top-k skips the chunks that cannot hold an
// answer.
// Workgroups are ordered in chunks of row tiles (about 2 MiB of query rows),
// each swept against every entity tile: the chunk's rows stay in L2 while
// the entity table streams past.
#include <algorithm>

#include "kgq_internal.hpp"
#include "mfma_tile.hpp"

namespace kgq {

// Workgroup tiles: 64 x 64 on the direct-to-LDS loop; on the register-staged
// loop 128 x 128, or 64 x 64 for small batches, where the larger tile leaves
// the chip underfilled and each workgroup's K loop is a latency chain. Query
// rows are padded to 128 (kRowTileBetae), a multiple of every tile's rows.
template <class KlTile>
__global__ __launch_bounds__(256, 2) void k_score_kl(ScoreArgs a, int n_mt, int n_nt, int qchunk, int total,
                                                     int per_xcd)
{
    constexpr int KL_BM = KlTile::kBM, KL_BN = KlTile::kBN;
    extern __shared__ __align__(16) float sm[];   // KlTile::SMEM floats, set at launch

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

    // Query rows are padded (with zeros) to a multiple of 128 and entity
    // rows to a multiple of 256, so the whole tile is inside both buffers.
    const int K = 2 * a.d;
    const int n_ent_pad = (int)(a.n_blocks * kEntBlock);
    v4f acc[KlTile::TM][KlTile::TN];
    if constexpr (KlTile::kBf16x3)
        KlTile::run(a.qpack, K, n_mt * KL_BM, a.n_rows, a.ent_planes, (int64_t)n_ent_pad * K, K, n_ent_pad, K, m0,
                    n0, sm, acc);
    else
        KlTile::run(a.qpack, K, n_mt * KL_BM, a.ent, K, n_ent_pad, K, m0, n0, sm, acc);

    // Epilogue, staged through LDS (the ring is free after the K loop):
    //   1. each lane subtracts E_e and its accumulators from gamma - C_q (one
    //      per row, hoisted) in double precision
    //      and writes the scores of its 4 rows x 1 column per MFMA tile into
    //      a BM x BN tile (rows padded by 4 floats: the 16 lanes of a column
    //      group and the 4 row groups hit distinct banks, and rows stay
    //      16-byte aligned);
    //   2. BN / 4 threads per row read whole rows back, take the max over a
    //      union group of four rows or a pair (groups start at multiples of
    //      4, pairs at even rows, neither crosses a tile) and write each
    //      output row with 16-byte non-temporal stores, so the score matrix
    //      streams past L2 in whole lines instead of 64-byte pieces that
    //      evict the entity rows still to be read.
    // Query rows are padded to a multiple of 128 (C_q = 0 there) and E_e to
    // the entity blocks, so the constant reads are in bounds for every row
    // and column of the tile; padding never reaches the output.
    constexpr int TLD = KL_BN + 4;
    static_assert(KL_BM * TLD <= KlTile::SMEM, "output tile fits the LDS ring");
    static_assert(KL_BN % 4 == 0 && 256 % (KL_BN / 4) == 0, "output row pieces");
    // The output rows of the thread's rows in step 2, loaded now and waited
    // for once before it: a load inside its loop would wait (vmcnt) for the
    // stores issued before it as well. (Rows past the last are clamped to
    // it: no branch, so the loads issue back to back.)
    constexpr int C4 = KL_BN / 4, RPP = 256 / C4;     // 16-byte pieces per row, rows per pass
    constexpr int NIT = KL_BM / RPP;
    const int r0 = threadIdx.x / C4;
    int32_t od[NIT];
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int m = min(m0 + r0 + it * RPP, a.n_rows - 1);
        od[it] = a.out_dest[score_out_index(m, a.n_quad, a.n_pair)];
    }
    __syncthreads();                                  // every wavefront is done with the ring
    float* T = sm;
    double gq[KlTile::TM][4];                         // gamma - C_q of the lane's rows, once per tile
#pragma unroll
    for (int i = 0; i < KlTile::TM; ++i)
#pragma unroll
        for (int q = 0; q < 4; ++q) gq[i][q] = (double)a.gamma - a.cq[m0 + KlTile::row_of(i) + q];
#pragma unroll
    for (int j = 0; j < KlTile::TN; ++j) {
        const int cj = KlTile::col_of(j);
        const double ee = a.ee[n0 + cj];
#pragma unroll
        for (int i = 0; i < KlTile::TM; ++i) {
            const int rb = KlTile::row_of(i);
#pragma unroll
            for (int q = 0; q < 4; ++q) T[(rb + q) * TLD + cj] = (float)((gq[i][q] - ee) - (double)acc[i][j][q]);
        }
    }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);          // the output rows
    __syncthreads();
    const int c4 = threadIdx.x % C4;
    const int64_t n = n0 + 4 * c4;
    // Chunk keys (128-entity tiles only): the 16 lanes of a chunk are one DPP
    // row, and every lane of a row stays in the loop below (the row-uniform
    // branches keep its DPP rows whole); lanes past N add key 0.
    constexpr bool KEYS = KlTile::kBf16x3 && KL_BN == 2 * kKeyChunk;
    const bool keys = KEYS && a.chunk_key != nullptr;
    const bool tail = n0 + KL_BN > a.N;               // the last entity tile
    if (!keys && n >= a.N) return;
    const int n_grouped = a.n_quad + a.n_pair;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
        const int r = r0 + it * RPP;
        const int m = m0 + r;
        if (m >= a.n_rows) break;                     // rows only grow along the loop
        int cnt = 1;
        if (m < a.n_quad) {
            if (m & 3) continue;                      // inside a group of four
            cnt = 4;
        } else if (m < n_grouped) {
            if ((m - a.n_quad) & 1) continue;         // second row of a pair
            cnt = 2;
        }
        const float* t = T + r * TLD + 4 * c4;
        float4 v = *reinterpret_cast<const float4*>(t);
        for (int u = 1; u < cnt; ++u) {
            const float4 w = *reinterpret_cast<const float4*>(t + u * TLD);
            v = make_float4(fmaxf(v.x, w.x), fmaxf(v.y, w.y), fmaxf(v.z, w.z), fmaxf(v.w, w.w));
        }
        const int64_t orow = od[it];
        if constexpr (KEYS) {
            if (keys) {
                // An upper bound of the keys of the lane's scores: the key of
                // their float maximum (the scores order as their keys, NaN
                // aside), or the largest key when one is NaN; columns past N
                // count as -inf (in the last entity tile only).
                float4 kv = v;
                if (tail) {
                    const float ninf = -__builtin_inff();
                    kv = make_float4(n < a.N ? kv.x : ninf, n + 1 < a.N ? kv.y : ninf, n + 2 < a.N ? kv.z : ninf,
                                     n + 3 < a.N ? kv.w : ninf);
                }
                const float mx = fmaxf(fmaxf(kv.x, kv.y), fmaxf(kv.z, kv.w));
                const bool nan = __builtin_isunordered(kv.x, kv.y) || __builtin_isunordered(kv.z, kv.w);
                const uint32_t u = __float_as_uint(mx == 0.0f ? 0.0f : mx);
                const uint32_t kx = chunk16_max(nan ? 0xFFFFFFFFu : u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u));
                if ((c4 & 15) == 0 && n < a.N) a.chunk_key[orow * a.key_ld + n / kKeyChunk] = max(kx, 1u);
            }
        }
        float* dst = a.scores + orow * a.ld + n;
        if (n + 3 < a.N) {
            // rows start only 4-byte aligned; gfx950 takes dword-aligned
            // multi-dword global stores
            typedef float f4u_t __attribute__((ext_vector_type(4), aligned(4)));
            __builtin_nontemporal_store((f4u_t){v.x, v.y, v.z, v.w}, reinterpret_cast<f4u_t*>(dst));
        } else {
            const float e4[4] = {v.x, v.y, v.z, v.w};
            for (int jj = 0; jj < 4; ++jj)
                if (n + jj < a.N) __builtin_nontemporal_store(e4[jj], dst + jj);
        }
    }
}

template <class Tile>
static void launch_tiles(const ScoreArgs& a, hipStream_t s)
{
    constexpr int BM = Tile::kBM, BN = Tile::kBN;
    const int n_mt = (a.n_rows + BM - 1) / BM;
    const int n_nt = (int)((a.N + BN - 1) / BN);
    const int total = n_mt * n_nt;
    const int per_xcd = (total + 7) / 8;
    // Row-tile chunk: as many row tiles as ~2 MiB of query rows (about half an
    // XCD's L2). The entity table is streamed once per chunk, and the XCDs
    // split the global order evenly whatever the chunk size, so larger
    // chunks cost no balance.
    const int64_t tile_bytes = (int64_t)BM * 2 * a.d * 4;
    const int qchunk = (int)std::min<int64_t>(n_mt, std::max<int64_t>(1, (int64_t)(2 << 20) / tile_bytes));
    // LDS is dynamic so that rings above the 64 KiB static limit fit; the
    // limit is raised once per device and tile
    constexpr int lds = Tile::SMEM * 4;
    if (lds > 65536) {
        static bool raised[64] = {};
        int dev = 0;
        if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64 && !raised[dev]) {
            if (hipFuncSetAttribute((const void*)k_score_kl<Tile>, hipFuncAttributeMaxDynamicSharedMemorySize, lds) ==
                hipSuccess)
                raised[dev] = true;
        }
    }
    hipLaunchKernelGGL((k_score_kl<Tile>), dim3(per_xcd * 8), dim3(256), lds, s, a, n_mt, n_nt, qchunk, total,
                       per_xcd);
}

constexpr int kScoreKlFp32Rows = 64;   // scored rows up to which the FP32 tile runs

bool launch_score_kl(const ScoreArgs& a, hipStream_t s)
{
    if (a.n_rows <= 0) return false;
    using LdsTile = MfmaTileLds<64, 64, 3>;
    using LdsTileHalf = MfmaTileLds<64, 64, 3, true>;
    using SplitTile = MfmaTileBf16x3<128, 128, 4, true>;
    // The bf16 split tile pays from 65 scored rows on: at fewer, its
    // 128-row tile is mostly padding and its entity-tile grid too small to
    // fill the chip (B = 1: 142 us per 1p query at 63,361 entities, 92 us at
    // 14,505, against 131 and 77 us on the FP32 64 x 64 tile). Up to 128
    // rows it also needs a workgroup per compute unit (96 rows at 14,505
    // entities, 114 tiles: 1.12 against 1.04 us per query); from 129 rows
    // it wins with fewer (160 and 240 rows at 14,505: 0.71 and 0.50 against
    // 0.74 and 0.57 us per query).
    const int64_t split_tiles = (int64_t)((a.n_rows + 127) / 128) * ((a.N + 127) / 128);
    const bool split_pays =
        a.split_always || (a.n_rows > kScoreKlFp32Rows && (a.n_rows > 128 || split_tiles >= 256));
    if (a.ent_planes && (2 * a.d) % 32 == 0 && split_pays) {   // planes: row stride 2d
        launch_tiles<SplitTile>(a, s);
        return a.chunk_key != nullptr;
    }
    if (LdsTile::supports(2 * a.d)) {
        launch_tiles<LdsTile>(a, s);
    } else if (LdsTileHalf::supports(2 * a.d)) {
        launch_tiles<LdsTileHalf>(a, s);
    } else {
        const int64_t big_tiles = (int64_t)((a.n_rows + 127) / 128) * ((a.N + 127) / 128);
        if (big_tiles < 512) launch_tiles<MfmaTileReg<64, 64>>(a, s);
        else launch_tiles<MfmaTileReg<kRowTileBetae, 128>>(a, s);
    }
    return false;
}

}  // namespace kgq
