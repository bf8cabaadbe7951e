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

#pragma unroll
    for (int j = 0; j < GemmTile::TN; ++j) {
        const int n = n0 + GemmTile::col_of(j);
        if (n >= g.N) continue;
        const float b = g.bias ? g.bias[n] : 0.f;
#pragma unroll
        for (int i = 0; i < GemmTile::TM; ++i) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + GemmTile::row_of(i) + r;
                if (m >= g.M) continue;
                const float v = apply_epilogue(g.epi, g.epi_split, n, acc[i][j][r] + b);
                const int64_t row = g.c_rowmap ? (int64_t)g.c_rowmap[m] : (int64_t)m;
                g.C[row * g.ldc + n] = v;
            }
        }
    }
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
// Split. Every FP32 value x is written exactly as x = h + m + l with h, m, l
// bf16: h = bf16(x), m = bf16(x - h), l = x - h - m (round to nearest even at
// each step). Both subtractions are exact in FP32, and l has at most 8
// significant bits, so it is a bf16 value and the sum is exact. |m| <= 2^-8 |x|
// and |l| <= 2^-16 |x|, up to rounding.
// Products. x w = hh' + hm' + mh' + mm' + hl' + lh' + (ml' + lm' + ll'); the
// first six are kept, the dropped three are below 2^-23 |x w| together. Each
// bf16 x bf16 product is exact in FP32 and the matrix core accumulates in
// FP32, so a layer has the error class of an FP32 GEMM. Per 32 of K, the six
// 16x16x32 bf16 MFMAs (16 cycles each) replace eight 16x16x4 FP32 MFMAs (32
// cycles each).
// Operands. The weights are split once, when they are loaded
// (launch_split_planes); the inputs A are split in registers as their
// fragments are read from LDS, so A keeps its FP32 layout and producers are
// unchanged. Values must be finite and below the largest bf16 (3.39e38):
// h would round to infinity above it.
// Tiles. A workgroup of 4 wavefronts (2 x 2) owns a BM x BN output tile, each
// wavefront (BM/32) x (BN/32) 16x16 blocks. Stages of 32 of K go through a
// two-slot LDS ring by direct-to-LDS loads: A as FP32 rows (128 bytes, 16-byte
// chunks XOR-swizzled by row), W as three planes of bf16 rows (64 bytes,
// chunks swizzled by row / 2), so that the fragment reads of 16 rows at one
// chunk fall in distinct banks. Lane l supplies row l % 16 of a block at
// k = 8 (l / 16) .. + 7 (the builtin's operand layout) and holds the output
// rows 4 (l / 16) .. + 3 of column l % 16, as in the FP32 loop. Stage kt + 1's
// fragments are read while stage kt's products run; stage kt + 2 is loaded
// into the slot stage kt leaves.
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

struct Bf16x3 {
    v4u h, m, l;   // 8 bf16 each, element e in half e % 2 of word e / 2
};

__device__ __forceinline__ uint32_t pack_bf16_rne(float a, float b)
{
    typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
    typedef float v2f __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((v2f){a, b}, v2bf));
}

// 8 FP32 values (lo: elements 0..3, hi: 4..7) -> their three bf16 planes
__device__ __forceinline__ Bf16x3 split_bf16x3(const v4u& lo, const v4u& hi)
{
    const float x[8] = {__uint_as_float(lo.x), __uint_as_float(lo.y), __uint_as_float(lo.z), __uint_as_float(lo.w),
                        __uint_as_float(hi.x), __uint_as_float(hi.y), __uint_as_float(hi.z), __uint_as_float(hi.w)};
    Bf16x3 f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const float a = x[2 * p], b = x[2 * p + 1];
        const uint32_t H = pack_bf16_rne(a, b);
        const float ra = a - __uint_as_float(H << 16), rb = b - __uint_as_float(H & 0xffff0000u);
        const uint32_t Mm = pack_bf16_rne(ra, rb);
        const float sa = ra - __uint_as_float(Mm << 16), sb = rb - __uint_as_float(Mm & 0xffff0000u);
        f.h[p] = H;
        f.m[p] = Mm;
        f.l[p] = pack_bf16_rne(sa, sb);
    }
    return f;
}

__global__ __launch_bounds__(256) void k_split_planes(const float* __restrict__ w, uint16_t* __restrict__ p, int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const float x = w[i];
    const uint32_t H = pack_bf16_rne(x, 0.f);
    const float r = x - __uint_as_float(H << 16);
    const uint32_t Mm = pack_bf16_rne(r, 0.f);
    const float t = r - __uint_as_float(Mm << 16);
    p[i] = (uint16_t)H;
    p[n + i] = (uint16_t)Mm;
    p[2 * n + i] = (uint16_t)pack_bf16_rne(t, 0.f);
}

void launch_split_planes(const float* w, uint16_t* p, int64_t n, hipStream_t s)
{
    if (n <= 0) return;
    hipLaunchKernelGGL(k_split_planes, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, w, p, n);
}

__device__ __forceinline__ v4f mfma_bf16(const v4u& a, const v4u& b, v4f c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0, 0,
                                                   0);
}

template <int BM, int BN>
struct TileBf16x3 {
    static constexpr int BK = 32;
    static constexpr int AROW = BK * 4;                // bytes of one A row per stage (FP32)
    static constexpr int WROW = BK * 2;                // bytes of one W row per stage and plane (bf16)
    static constexpr int ABYTES = BM * AROW;
    static constexpr int STAGE = ABYTES + 3 * BN * WROW;
    static constexpr int TM = BM / 32, TN = BN / 32;   // 16x16 blocks per wavefront
    static constexpr int AI = BM / 32;                 // A load instructions per wavefront and stage (8 rows each)
    static constexpr int WI = 3 * BN / 64;             // W load instructions per wavefront and stage (16 rows each)
    static constexpr int LPS = AI + WI;
    static_assert(BM % 32 == 0 && BN % 64 == 0 && LPS < 64, "tile shape");
    static_assert(2 * STAGE <= 65536, "LDS");
    __device__ static int aswz(int row) { return (row & 7) ^ ((row >> 3) & 1); }
    __device__ static int wswz(int row) { return (row >> 1) & 3; }
};

template <int BM, int BN>
__global__ __launch_bounds__(256) void k_gemm_bf16x3(GemmArgs g, int tm, int tn, int per_xcd)
{
    using T = TileBf16x3<BM, BN>;
    __shared__ __align__(16) char sm[2 * T::STAGE];
    const int b = blockIdx.x;
    const int L = (b & 7) * per_xcd + (b >> 3);
    if (L >= tm * tn) return;
    const int mt = L / tn, nt = L - mt * tn;
    const int m0 = mt * BM, n0 = nt * BN;
    const int M = g.M, N = g.N, nk = g.K / T::BK;
    const int64_t plane = (int64_t)N * g.K;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave >> 1, wn = wave & 1;
    const int grp = lane >> 4, li = lane & 15;

    // A: load instruction t = h * 4 + wave writes rows 8t .. 8t + 7 (1 KiB);
    // lane l lands at row 8t + l / 8, chunk position l % 8
    const float* ag[T::AI];
#pragma unroll
    for (int h = 0; h < T::AI; ++h) {
        const int row = (h * 4 + wave) * 8 + (lane >> 3);
        ag[h] = g.A + (int64_t)min(m0 + row, M - 1) * g.lda + ((lane & 7) ^ T::aswz(row)) * 4;
    }
    // W: load instruction u = h * 4 + wave writes plane u / (BN / 16), rows
    // 16 (u % (BN / 16)) .. + 15; lane l lands at row + l / 4, position l % 4
    const uint16_t* wg[T::WI];
    int wdst[T::WI];
#pragma unroll
    for (int h = 0; h < T::WI; ++h) {
        const int u = h * 4 + wave;
        const int p = u / (BN / 16), rb = u % (BN / 16);
        const int row = rb * 16 + (lane >> 2);
        wg[h] = g.Wp + p * plane + (int64_t)min(n0 + row, N - 1) * g.K + ((lane & 3) ^ T::wswz(row)) * 8;
        wdst[h] = T::ABYTES + (p * BN + rb * 16) * T::WROW;
    }
    auto issue = [&](int kt, int slot) {
        char* st = sm + slot * T::STAGE;
#pragma unroll
        for (int h = 0; h < T::AI; ++h)
            __builtin_amdgcn_global_load_lds((const void*)(ag[h] + kt * T::BK),
                                             (lds_void*)(st + (h * 4 + wave) * 8 * T::AROW), 16, 0, 0);
#pragma unroll
        for (int h = 0; h < T::WI; ++h)
            __builtin_amdgcn_global_load_lds((const void*)(wg[h] + kt * T::BK), (lds_void*)(st + wdst[h]), 16, 0, 0);
    };

    // fragment offsets in a stage: A block i, k = 8 grp .. + 7 (chunks 2 grp, 2 grp + 1); W block j, chunk grp
    int aoff[T::TM][2], woff[T::TN];
#pragma unroll
    for (int i = 0; i < T::TM; ++i) {
        const int row = wm * (BM / 2) + i * 16 + li;
#pragma unroll
        for (int q = 0; q < 2; ++q) aoff[i][q] = row * T::AROW + ((2 * grp + q) ^ T::aswz(row)) * 16;
    }
#pragma unroll
    for (int j = 0; j < T::TN; ++j) {
        const int row = wn * (BN / 2) + j * 16 + li;
        woff[j] = T::ABYTES + row * T::WROW + (grp ^ T::wswz(row)) * 16;
    }

    v4f acc[T::TM][T::TN];
#pragma unroll
    for (int i = 0; i < T::TM; ++i)
#pragma unroll
        for (int j = 0; j < T::TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    Bf16x3 fa[T::TM];          // stage kt, split
    v4u fw[3][T::TN];
    v4u ra[T::TM][2];          // stage kt + 1, as read
    v4u rw[3][T::TN];
    auto read = [&](int slot) {
        const char* st = sm + slot * T::STAGE;
#pragma unroll
        for (int i = 0; i < T::TM; ++i) {
            ra[i][0] = *reinterpret_cast<const v4u*>(st + aoff[i][0]);
            ra[i][1] = *reinterpret_cast<const v4u*>(st + aoff[i][1]);
        }
#pragma unroll
        for (int p = 0; p < 3; ++p)
#pragma unroll
            for (int j = 0; j < T::TN; ++j) rw[p][j] = *reinterpret_cast<const v4u*>(st + woff[j] + p * BN * T::WROW);
    };
    auto take = [&]() {
#pragma unroll
        for (int i = 0; i < T::TM; ++i) fa[i] = split_bf16x3(ra[i][0], ra[i][1]);
#pragma unroll
        for (int p = 0; p < 3; ++p)
#pragma unroll
            for (int j = 0; j < T::TN; ++j) fw[p][j] = rw[p][j];
    };
    // the six kept products, largest first; consecutive MFMAs update
    // different accumulators
    auto products = [&]() {
#pragma unroll
        for (int q = 0; q < 6; ++q)
#pragma unroll
            for (int i = 0; i < T::TM; ++i)
#pragma unroll
                for (int j = 0; j < T::TN; ++j) {
                    const v4u& a = (q == 0 || q == 1 || q == 4) ? fa[i].h : (q == 5 ? fa[i].l : fa[i].m);
                    const v4u& w = (q == 0 || q == 2 || q == 5) ? fw[0][j] : (q == 4 ? fw[2][j] : fw[1][j]);
                    acc[i][j] = mfma_bf16(a, w, acc[i][j]);
                }
    };

    // The vmcnt counts below are this loop's loads only: nothing else is
    // outstanding on entry.
    issue(0, 0);
    if (nk > 1) issue(1, 1);
    if (nk > 1) wait_vm_barrier<T::LPS>();   // stage 0 landed
    else wait_vm_barrier<0>();
    read(0);
    take();
    for (int kt = 0; kt < nk; ++kt) {
        if (kt + 1 < nk) {
            // stage kt + 1 landed (stage kt + 2 is not issued yet), and every
            // wavefront holds stage kt's fragments, so its slot is free
            wait_vm_barrier<0>();
            if (kt + 2 < nk) issue(kt + 2, kt & 1);
            read((kt + 1) & 1);
        }
        products();
        if (kt + 1 < nk) take();
    }

#pragma unroll
    for (int j = 0; j < T::TN; ++j) {
        const int n = n0 + wn * (BN / 2) + j * 16 + li;
        if (n >= N) continue;
        const float bb = g.bias ? g.bias[n] : 0.f;
#pragma unroll
        for (int i = 0; i < T::TM; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm * (BM / 2) + i * 16 + grp * 4 + r;
                if (m >= M) continue;
                const float v = apply_epilogue(g.epi, g.epi_split, n, acc[i][j][r] + bb);
                const int64_t row = g.c_rowmap ? (int64_t)g.c_rowmap[m] : (int64_t)m;
                g.C[row * g.ldc + n] = v;
            }
    }
}

// Whether a layer of this shape runs on the bf16 matrix cores (given the
// weight planes): K is a multiple of the 32-wide stage, A's rows are 16-byte
// aligned, and (unless forced) the layer has at least 192 output tiles of
// 64 x 64, below which the FP32 path with its split-K mode measured as fast
// or faster.
bool gemm_shape_takes_bf16x3(int M, int N, int K, int64_t lda, bool always)
{
    if (M <= 0 || N <= 0 || K < 32 || K % 32 != 0 || lda % 4 != 0) return false;
    return always || (int64_t)((M + 63) / 64) * ((N + 63) / 64) >= 192;
}

static bool use_bf16x3(const GemmArgs& g)
{
    return g.Wp && gemm_shape_takes_bf16x3(g.M, g.N, g.K, g.lda, g.bf16x3_always);
}

static void launch_gemm_bf16x3(const GemmArgs& g, hipStream_t s)
{
    // 64 x 128 tiles for the largest layers (fewer A fragment splits per
    // product), 64 x 64 otherwise (more workgroups per compute unit)
    if (g.M >= 4096 && g.N >= 1024) {
        const int tm = (g.M + 63) / 64, tn = (g.N + 127) / 128, per_xcd = (tm * tn + 7) / 8;
        hipLaunchKernelGGL((k_gemm_bf16x3<64, 128>), dim3(per_xcd * 8), dim3(256), 0, s, g, tm, tn, per_xcd);
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
