// Dense layers on the FP32 matrix cores of gfx950:  C = epi(A W^T + b).
//
// These are the dense contractions of the operators: BetaE's projection MLP
// (Eq. 4 of the paper: three matmul + bias layers with ReLU between them)
// and the attention / set-function MLPs of the intersection operators. Both
// operands are K-contiguous (A rows, W rows). The tile loop is MfmaTile
// (mfma_tile.hpp) with 64 x 64 workgroup tiles: at the path's shapes (M of a
// few thousand rows, N and K of 400 to 1,600) it gives enough workgroups to
// fill the chip, and measured faster than 64 x 128 or 128 x 128 tiles there.
// The epilogue adds the bias, applies the activation and stores each row m at
// C + map(m) * ldc.
#include "kgq_internal.hpp"
#include "mfma_tile.hpp"

namespace kgq {

using GemmTile = MfmaTile<64, 64>;

__global__ __launch_bounds__(256) void k_gemm(GemmArgs g)
{
    __shared__ float sm[GemmTile::SMEM];
    const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
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
                float v = acc[i][j][r] + b;
                if (g.epi == EPI_RELU) v = v > 0.f ? v : 0.f;
                else if (g.epi == EPI_BETA_REG) v = fminf(fmaxf(v + 1.0f, 0.05f), 1e9f);
                const int64_t row = g.c_rowmap ? (int64_t)g.c_rowmap[m] : (int64_t)m;
                g.C[row * g.ldc + n] = v;
            }
        }
    }
}

void launch_gemm(const GemmArgs& g, hipStream_t s)
{
    if (g.M <= 0 || g.N <= 0) return;
    dim3 grid((g.N + 63) / 64, (g.M + 63) / 64);
    hipLaunchKernelGGL(k_gemm, grid, dim3(256), 0, s, g);
}

}  // namespace kgq
