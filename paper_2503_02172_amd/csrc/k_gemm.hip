// Dense layers on the FP32 matrix cores of gfx950:  C = epi(A W^T + b).
//
// These are the dense contractions of the operators: the projection MLPs of
// BetaE, ConE and LogicE (Eq. 4 of the paper: three matmul + bias layers with
// ReLU between them) and the attention / set-function MLPs of the
// intersection operators. Both
// operands are K-contiguous (A rows, W rows). The tile loop (mfma_tile.hpp)
// runs 64 x 64 workgroup tiles: at the path's shapes (M of a few hundred to a
// few thousand rows, N and K of 400 to 1,600) they give enough workgroups to
// fill the chip, and measured faster than 64 x 128, 128 x 64 or 128 x 128
// tiles there. K a multiple of 16 takes the direct-to-LDS ring of three
// stages, any other K the register-staged loop. Tiles are dispatched in
// row-major order split into one contiguous range per XCD, so each XCD's L2
// sees few distinct rows of A at a time.
// The epilogue adds the bias, applies the activation and stores each row m at
// C + map(m) * ldc.
//
// Layers with enough output tiles run instead on the bf16 matrix cores at
// FP32 accuracy (k_gemm_bf16x3, below): v_mfma_f32_16x16x32_bf16 does 16
// times the work of v_mfma_f32_16x16x4_f32 per cycle, and six of its products
// per k range reproduce one FP32 product.
#include <algorithm>
#include <type_traits>

#include "kgq_internal.hpp"
#include "mfma_tile.hpp"

namespace kgq {

using GemmTileLds = MfmaTileLds<64, 64, 3>;
using GemmTileLdsHalf = MfmaTileLds<64, 64, 3, true>;
using GemmTileReg = MfmaTileReg<64, 64>;

// Epilogue of a tile: bias, activation, row map, stores. The bias of the
// lane's columns and the row map of its rows are loaded first (indices
// clamped, so the loads issue back to back) and waited for once: a load
// issued between the stores would wait (vmcnt) for the stores before it as
// well, and the stores would go out one acknowledgement at a time.
template <class Tile>
__device__ __forceinline__ void store_tile(const GemmArgs& g, int m0, int n0, const v4f (&acc)[Tile::TM][Tile::TN])
{
    float bias[Tile::TN];
    int64_t row[Tile::TM][4];
#pragma unroll
    for (int j = 0; j < Tile::TN; ++j) bias[j] = g.bias ? g.bias[min(n0 + Tile::col_of(j), g.N - 1)] : 0.f;
#pragma unroll
    for (int i = 0; i < Tile::TM; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = m0 + Tile::row_of(i) + r;
            row[i][r] = g.c_rowmap ? (int64_t)g.c_rowmap[min(m, g.M - 1)] : (int64_t)m;
        }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
#pragma unroll
    for (int j = 0; j < Tile::TN; ++j) {
        const int n = n0 + Tile::col_of(j);
        if (n >= g.N) continue;
#pragma unroll
        for (int i = 0; i < Tile::TM; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + Tile::row_of(i) + r;
                if (m >= g.M) continue;
                g.C[row[i][r] * g.ldc + n] = apply_epilogue(g.epi, g.epi_split, n, acc[i][j][r] + bias[j]);
            }
    }
}

template <class GemmTile>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g, int tm, int tn, int per_xcd)
{
    __shared__ float sm[GemmTile::SMEM];
    // workgroup b runs on XCD b % 8, which takes positions
    // [x * per_xcd, (x + 1) * per_xcd) of the row-major tile order
    const int b = blockIdx.x;
    const int L = (b & 7) * per_xcd + (b >> 3);
    if (L >= tm * tn) return;
    const int mt = L / tn, nt = L - mt * tn;
    const int m0 = mt * 64, n0 = nt * 64;
    v4f acc[GemmTile::TM][GemmTile::TN];
    GemmTile::run(g.A, g.lda, g.M, g.W, g.ldw, g.N, g.K, m0, n0, sm, acc);

    store_tile<GemmTile>(g, m0, n0, acc);
}

// Split-K for small M: with few 64 x 64 output tiles the K loop is a latency
// chain (one stage of 32 per LDS round trip) on a handful of compute units.
// Each of S workgroups per tile runs a K slice and writes its partial tile;
// a second kernel adds the S partials in slice order (deterministic), then
// the bias and activation, and stores through the row map.
// Slices before the last have kc of K (a multiple of 32) and run on
// SliceTile; the last has the rest and runs on LastTile.
template <class SliceTile, class LastTile>
__global__ __launch_bounds__(256) void k_gemm_part(GemmArgs g, int kc)
{
    using GemmTile = SliceTile;
    static_assert(SliceTile::SMEM == LastTile::SMEM && SliceTile::TM == LastTile::TM &&
                  SliceTile::TN == LastTile::TN, "tile loops of one shape");
    __shared__ float sm[GemmTile::SMEM];
    const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
    const int k0 = blockIdx.z * kc;
    const int kn = min(kc, g.K - k0);
    v4f acc[GemmTile::TM][GemmTile::TN];
    if (blockIdx.z + 1 < gridDim.z)
        SliceTile::run(g.A + k0, g.lda, g.M, g.W + k0, g.ldw, g.N, kn, m0, n0, sm, acc);
    else
        LastTile::run(g.A + k0, g.lda, g.M, g.W + k0, g.ldw, g.N, kn, m0, n0, sm, acc);
    float* part = g.ws + (int64_t)blockIdx.z * g.M * g.N;
#pragma unroll
    for (int j = 0; j < GemmTile::TN; ++j) {
        const int n = n0 + GemmTile::col_of(j);
        if (n >= g.N) continue;
#pragma unroll
        for (int i = 0; i < GemmTile::TM; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + GemmTile::row_of(i) + r;
                if (m < g.M) part[(int64_t)m * g.N + n] = acc[i][j][r];
            }
    }
}

__global__ __launch_bounds__(256) void k_gemm_reduce(GemmArgs g, int splits)
{
    const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (t >= (int64_t)g.M * g.N) return;
    const int m = (int)(t / g.N), n = (int)(t - (int64_t)m * g.N);
    float v = 0.f;
    for (int z = 0; z < splits; ++z) v += g.ws[(int64_t)z * g.M * g.N + t];
    v += g.bias ? g.bias[n] : 0.f;
    v = apply_epilogue(g.epi, g.epi_split, n, v);
    const int64_t row = g.c_rowmap ? (int64_t)g.c_rowmap[m] : (int64_t)m;
    g.C[row * g.ldc + n] = v;
}


// ---- FP32-accurate layers on the bf16 matrix cores ---------------------------
//
// The tile loop (MfmaTileBf16x3, mfma_tile.hpp) splits each FP32 value
// exactly into three bf16 parts and keeps six of the nine part products:
// the result has the error class of an FP32 GEMM at 0.375 of the FP32
// matrix-core time per k range. The weights are split once, when they are
// loaded (launch_split_planes); the inputs A are split in registers as their
// fragments are read from LDS, so A keeps its FP32 layout and the producers
// of the layer inputs are unchanged. Epilogue and tile order as in k_gemm.
__global__ __launch_bounds__(256) void k_split_planes(const float* __restrict__ w, uint16_t* __restrict__ p,
                                                      int64_t cols, int64_t ld, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int64_t row = i / ld, c = i - row * ld;
    const float x = c < cols ? w[row * cols + c] : 0.f;
    const uint32_t H = pack_bf16_rne(x, 0.f);
    const float r = x - __uint_as_float(H << 16);
    const uint32_t Mm = pack_bf16_rne(r, 0.f);
    const float t = r - __uint_as_float(Mm << 16);
    p[i] = (uint16_t)H;
    p[n + i] = (uint16_t)Mm;
    p[2 * n + i] = (uint16_t)pack_bf16_rne(t, 0.f);
}

void launch_split_planes(const float* w, uint16_t* p, int64_t rows, int64_t cols, hipStream_t s)
{
    const int64_t ld = plane_ld(cols), n = rows * ld;
    if (n <= 0) return;
    hipLaunchKernelGGL(k_split_planes, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, w, p, cols, ld, n);
}

template <int BM, int BN, bool PRIO>
__device__ __forceinline__ void gemm_bf16x3_tile(const GemmArgs& g, int tm, int tn, int per_xcd, float* sm)
{
    using Tile = MfmaTileBf16x3<BM, BN, 4, PRIO>;
    const int b = blockIdx.x;
    const int L = (b & 7) * per_xcd + (b >> 3);
    if (L >= tm * tn) return;
    const int mt = L / tn, nt = L - mt * tn;
    const int m0 = mt * BM, n0 = nt * BN;
    v4f acc[Tile::TM][Tile::TN];
    const int64_t ldp = plane_ld(g.K);
    Tile::run(g.A, g.lda, g.M, g.M, g.Wp, (int64_t)g.N * ldp, ldp, g.N, g.K, m0, n0, sm, acc);

    store_tile<Tile>(g, m0, n0, acc);
}

template <int BM, int BN>
__global__ __launch_bounds__(256) void k_gemm_bf16x3(GemmArgs g, int tm, int tn, int per_xcd)
{
    __shared__ float sm[MfmaTileBf16x3<BM, BN, 4, BM == 64>::SMEM];
    gemm_bf16x3_tile<BM, BN, BM == 64>(g, tm, tn, per_xcd, sm);   // raised read priority: see the tile
}

// 128 x 128 tiles (the BetaE scorer's): an 80 KiB ring, above the static LDS
// limit, two workgroups per compute unit, raised read priority
__global__ __launch_bounds__(256, 2) void k_gemm_bf16x3_128(GemmArgs g, int tm, int tn, int per_xcd)
{
    extern __shared__ __align__(16) float sm_dyn[];
    gemm_bf16x3_tile<128, 128, true>(g, tm, tn, per_xcd, sm_dyn);
}

// Split K on the bf16 matrix cores: each of S workgroups per 64 x 64 tile
// multiplies a K slice (a multiple of 32) and writes its partial tile;
// k_gemm_reduce then adds the S partials in slice order (deterministic), the
// bias and the activation, and stores through the row map.
__global__ __launch_bounds__(256) void k_gemm_bf16x3_part(GemmArgs g, int kc)
{
    using Tile = MfmaTileBf16x3<64, 64, 4, true>;
    __shared__ float sm[Tile::SMEM];
    const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
    const int k0 = blockIdx.z * kc;
    const int kn = min(kc, g.K - k0);
    v4f acc[Tile::TM][Tile::TN];
    const int64_t ldp = plane_ld(g.K);
    Tile::run(g.A + k0, g.lda, g.M, g.M, g.Wp + k0, (int64_t)g.N * ldp, ldp, g.N, kn, m0, n0, sm, acc);
    float* part = g.ws + (int64_t)blockIdx.z * g.M * g.N;
#pragma unroll
    for (int j = 0; j < Tile::TN; ++j) {
        const int n = n0 + Tile::col_of(j);
        if (n >= g.N) continue;
#pragma unroll
        for (int i = 0; i < Tile::TM; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + Tile::row_of(i) + r;
                if (m < g.M) part[(int64_t)m * g.N + n] = acc[i][j][r];
            }
    }
}

// Whether a layer of this shape runs on the bf16 matrix cores (given the
// weight planes): K is a multiple of 4 and at least one 32-wide stage (the
// planes are zero-padded to a whole stage), A's rows are 16-byte aligned,
// and (unless forced) the layer has at least 384 output tiles of
// 64 x 64 (1.5 per compute unit), or 1,024 rows and 192 tiles. Fewer rows on
// fewer tiles lost to the FP32 loop as a whole-K tile loop (512 x 1,600
// layers, 200 tiles: 21.5 and 36.3 us against 22.4 and 40.2 us; 1,024 x
// 800 x 1,600, 208 tiles: bf16 34.2 us against 37.5 us); launch_gemm splits
// their K on the bf16 path when it has a workspace.
bool gemm_shape_takes_bf16x3(int M, int N, int K, int64_t lda, bool always)
{
    if (M <= 0 || N <= 0 || K < 32 || K % 4 != 0 || lda % 4 != 0) return false;
    const int64_t tiles = (int64_t)((M + 63) / 64) * ((N + 63) / 64);
    return always || tiles >= 384 || (M >= 1024 && tiles >= 192);
}

static bool use_bf16x3(const GemmArgs& g)
{
    return g.Wp && gemm_shape_takes_bf16x3(g.M, g.N, g.K, g.lda, g.bf16x3_always);
}

static void launch_gemm_bf16x3(const GemmArgs& g, hipStream_t s)
{
    // 128 x 64 tiles for the largest layers (half the B fragment reads per
    // product), 64 x 64 otherwise (more workgroups per compute unit).
    // Measured on the 14,505-entity BetaE step: dense stage 0.576 ms, against
    // 0.597 ms with 64 x 128 tiles for the largest layers, 0.594 ms with
    // 128 x 64 tiles for every layer of 4,096 rows or more, 0.628 ms with
    // 64 x 64 tiles throughout; on the 63,361-entity step, 128 x 64 tiles from
    // 2,048 rows (its 3,947-row layers) took the stage from 0.534 to 0.516 ms.
    // A layer whose 128 x 64 tiles need a second round of the 512 resident
    // workgroups while 128 x 128 tiles fit one takes those (3,947 x 1,600 x
    // 1,600: 775 tiles of 128 x 64 in 142 us, 403 of 128 x 128 in 125 us).
    // 128 x 128 for every layer of 2,048 rows or more with 192-512 such
    // tiles (the N = 800 layers too) made both BetaE dense stages slower.
    const int64_t t128 = (int64_t)((g.M + 127) / 128) * ((g.N + 127) / 128);
    const int64_t t64 = (int64_t)((g.M + 127) / 128) * ((g.N + 63) / 64);
    if (g.M >= 2048 && g.N >= 1024 && t128 <= 512 && t64 > 512) {
        constexpr int lds = MfmaTileBf16x3<128, 128, 4, true>::SMEM * 4;
        static bool raised[64] = {};
        int dev = 0;
        if (hipGetDevice(&dev) == hipSuccess && dev >= 0 && dev < 64 && !raised[dev]) {
            if (hipFuncSetAttribute((const void*)k_gemm_bf16x3_128, hipFuncAttributeMaxDynamicSharedMemorySize, lds) ==
                hipSuccess)
                raised[dev] = true;
        }
        const int tm = (g.M + 127) / 128, tn = (g.N + 127) / 128, per_xcd = (tm * tn + 7) / 8;
        hipLaunchKernelGGL(k_gemm_bf16x3_128, dim3(per_xcd * 8), dim3(256), lds, s, g, tm, tn, per_xcd);
    } else if (g.M >= 2048 && g.N >= 1024) {
        const int tm = (g.M + 127) / 128, tn = (g.N + 63) / 64, per_xcd = (tm * tn + 7) / 8;
        hipLaunchKernelGGL((k_gemm_bf16x3<128, 64>), dim3(per_xcd * 8), dim3(256), 0, s, g, tm, tn, per_xcd);
    } else {
        const int tm = (g.M + 63) / 64, tn = (g.N + 63) / 64, per_xcd = (tm * tn + 7) / 8;
        hipLaunchKernelGGL((k_gemm_bf16x3<64, 64>), dim3(per_xcd * 8), dim3(256), 0, s, g, tm, tn, per_xcd);
    }
}

void launch_gemm(const GemmArgs& g, hipStream_t s)
{
    if (g.M <= 0 || g.N <= 0) return;
    if (use_bf16x3(g)) {
        launch_gemm_bf16x3(g, s);
        return;
    }
    const int tn = (g.N + 63) / 64, tm = (g.M + 63) / 64;
    const int tiles = tn * tm;
    // smaller layers with the weight planes: split K on the bf16 matrix
    // cores, about 1.5 workgroups per compute unit, slices of whole 32-wide
    // stages, at least two (the last slice ends at K, which may cut it short).
    // Layers of at most 64 rows stay on the FP32 loop's split K, whose tile
    // has no split work for its one partly used row tile (3p queries at
    // B = 64: 2.45 against 2.54 us per query at 14,505 BetaE entities).
    if (g.Wp && g.ws && g.M > 64 && g.K >= 64 && g.K % 4 == 0 && g.lda % 4 == 0) {
        int sb = std::min({16, (384 + tiles - 1) / tiles, g.K / 64});
        while (sb > 1 && (int64_t)sb * g.M * g.N > g.ws_elems) --sb;
        if (sb > 1) {
            const int kc = (((g.K + sb - 1) / sb) + 31) / 32 * 32;
            const int z = (g.K + kc - 1) / kc;
            hipLaunchKernelGGL(k_gemm_bf16x3_part, dim3(tn, tm, z), dim3(256), 0, s, g, kc);
            const int64_t total = (int64_t)g.M * g.N;
            hipLaunchKernelGGL(k_gemm_reduce, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, g, z);
            return;
        }
    }
    // split K when the tiles alone leave most of the chip idle, keeping at
    // least two stages (64 of K) per slice
    int splits = 1;
    if (g.ws && tiles < 128 && g.K >= 128) {
        splits = std::min({16, (256 + tiles - 1) / tiles, g.K / 64});
        while (splits > 1 && (int64_t)splits * g.M * g.N > g.ws_elems) --splits;
    }
    if (splits > 1) {
        const int kc = (((g.K + splits - 1) / splits) + 31) / 32 * 32;   // slice: a multiple of the 32-wide stage
        const int z = (g.K + kc - 1) / kc;
        // every slice but the last has kc (a multiple of 32) of K; the last
        // has K - (z - 1) * kc, congruent to K modulo 32
        if (GemmTileLds::supports(g.K))
            hipLaunchKernelGGL((k_gemm_part<GemmTileLds, GemmTileLds>), dim3(tn, tm, z), dim3(256), 0, s, g, kc);
        else if (GemmTileLdsHalf::supports(g.K))
            hipLaunchKernelGGL((k_gemm_part<GemmTileLds, GemmTileLdsHalf>), dim3(tn, tm, z), dim3(256), 0, s, g, kc);
        else
            hipLaunchKernelGGL((k_gemm_part<GemmTileReg, GemmTileReg>), dim3(tn, tm, z), dim3(256), 0, s, g, kc);
        const int64_t total = (int64_t)g.M * g.N;
        hipLaunchKernelGGL(k_gemm_reduce, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, g, z);
        return;
    }
    const int per_xcd = (tiles + 7) / 8;
    const dim3 grid(per_xcd * 8);
    if (GemmTileLds::supports(g.K))
        hipLaunchKernelGGL(k_gemm<GemmTileLds>, grid, dim3(256), 0, s, g, tm, tn, per_xcd);
    else if (GemmTileLdsHalf::supports(g.K))
        hipLaunchKernelGGL(k_gemm<GemmTileLdsHalf>, grid, dim3(256), 0, s, g, tm, tn, per_xcd);
    else
        hipLaunchKernelGGL(k_gemm<GemmTileReg>, grid, dim3(256), 0, s, g, tm, tn, per_xcd);
}

}  // namespace kgq
