// Dense layers on the FP32 matrix cores of gfx950:  C = epi(A W^T + b).
//
// These are the only dense contractions on the path: BetaE's projection
// MLP (Eq. 4 of the paper: three matmul + bias layers with ReLU between
// them) and the attention / set-function MLPs of the intersection
// operators. Both operands are K-contiguous (A rows, W rows).
//
// Tiling: a workgroup of 4 wavefronts owns a 64x64 tile of C (BM = 64) or a
// 32x64 tile (BM = 32, for small M so that the grid still fills 256 CUs).
// Each wavefront computes 2x2 (or 1x2) v_mfma_f32_16x16x4_f32 tiles.
// K advances in steps of 16 staged through LDS with register double
// buffering. Inside a 16-wide K step, lane group g = lane / 16 reads the
// four consecutive k = 4g .. 4g+3 with one 128-bit LDS read and feeds them to
// four MFMAs; the reduction order over k is a permutation of 0..15, which
// the sum does not depend on.
#include "kgq_internal.hpp"

namespace kgq {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int GBK = 16;
constexpr int GPAD = 4;           // LDS row padding (floats)
constexpr int GLD = GBK + GPAD;   // LDS row stride

template <int BM>
__global__ __launch_bounds__(256) void k_gemm(GemmArgs g)
{
    constexpr int BN = 64;
    constexpr int TM = BM / 32;   // 16x16 MFMA tiles per wave along M (1 or 2)
    __shared__ float As[2][BM * GLD];
    __shared__ float Bs[2][BN * GLD];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave >> 1;   // wave row (0..1): rows [wm * BM/2, +BM/2)
    const int wn = wave & 1;    // wave col (0..1): cols [wn * 32, +32)
    const int m0 = blockIdx.y * BM;
    const int n0 = blockIdx.x * BN;

    // global -> register staging: one float4 per thread per operand
    // (A: BM rows x 16 k; for BM = 32 only the first 128 threads load A).
    const int lrow = tid >> 2;
    const int lk = (tid & 3) * 4;
    const bool a_loader = lrow < BM;

    auto load_a = [&](int k0) -> float4 {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        int m = m0 + lrow;
        if (a_loader && m < g.M && k0 + lk < g.K)
            v = *reinterpret_cast<const float4*>(g.A + (int64_t)m * g.lda + k0 + lk);
        return v;
    };
    auto load_b = [&](int k0) -> float4 {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        int n = n0 + lrow;
        if (n < g.N && k0 + lk < g.K)
            v = *reinterpret_cast<const float4*>(g.W + (int64_t)n * g.ldw + k0 + lk);
        return v;
    };

    v4f acc[TM][2];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    const int nk = (g.K + GBK - 1) / GBK;
    float4 ra = load_a(0), rb = load_b(0);
    int buf = 0;
    if (a_loader) *reinterpret_cast<float4*>(&As[0][lrow * GLD + lk]) = ra;
    *reinterpret_cast<float4*>(&Bs[0][lrow * GLD + lk]) = rb;
    __syncthreads();

    const int grp = lane >> 4;   // k sub-block 4*grp .. 4*grp+3
    const int li = lane & 15;

    for (int kt = 0; kt < nk; ++kt) {
        if (kt + 1 < nk) {
            ra = load_a((kt + 1) * GBK);
            rb = load_b((kt + 1) * GBK);
        }
        float4 av[TM], bv[2];
#pragma unroll
        for (int i = 0; i < TM; ++i)
            av[i] = *reinterpret_cast<const float4*>(&As[buf][(wm * (BM / 2) + i * 16 + li) * GLD + grp * 4]);
#pragma unroll
        for (int j = 0; j < 2; ++j)
            bv[j] = *reinterpret_cast<const float4*>(&Bs[buf][(wn * 32 + j * 16 + li) * GLD + grp * 4]);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].x, bv[j].x, acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].y, bv[j].y, acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].z, bv[j].z, acc[i][j], 0, 0, 0);
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i].w, bv[j].w, acc[i][j], 0, 0, 0);
            }
        if (kt + 1 < nk) {
            buf ^= 1;
            if (a_loader) *reinterpret_cast<float4*>(&As[buf][lrow * GLD + lk]) = ra;
            *reinterpret_cast<float4*>(&Bs[buf][lrow * GLD + lk]) = rb;
            __syncthreads();
        }
    }

    // Output layout of a 16x16 MFMA tile: lane holds column (lane % 16) and
    // rows 4 * (lane / 16) + r, r = 0..3.
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int n = n0 + wn * 32 + j * 16 + li;
            if (n >= g.N) continue;
            const float b = g.bias ? g.bias[n] : 0.f;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm * (BM / 2) + i * 16 + grp * 4 + r;
                if (m >= g.M) continue;
                float v = acc[i][j][r] + b;
                if (g.epi == EPI_RELU) v = v > 0.f ? v : 0.f;
                else if (g.epi == EPI_BETA_REG) v = fminf(fmaxf(v + 1.0f, 0.05f), 1e9f);
                const int64_t row = g.c_rowmap ? (int64_t)g.c_rowmap[m] : (int64_t)m;
                g.C[row * g.ldc + n] = v;
            }
        }
}

void launch_gemm(const GemmArgs& g, hipStream_t s)
{
    if (g.M <= 0 || g.N <= 0) return;
    const int nb = (g.N + 63) / 64;
    // Prefer the 64-row tile when it already gives two workgroups per CU.
    const int64_t wg64 = (int64_t)nb * ((g.M + 63) / 64);
    if (wg64 >= 512) {
        dim3 grid(nb, (g.M + 63) / 64);
        hipLaunchKernelGGL(k_gemm<64>, grid, dim3(256), 0, s, g);
    } else {
        dim3 grid(nb, (g.M + 31) / 32);
        hipLaunchKernelGGL(k_gemm<32>, grid, dim3(256), 0, s, g);
    }
}

}  // namespace kgq
