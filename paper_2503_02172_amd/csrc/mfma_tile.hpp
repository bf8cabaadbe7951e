// Device-side FP32 matrix-core tile loop shared by the dense layers and the
// BetaE scorer: acc = A[m0 : m0 + BM, :K] . B[n0 : n0 + BN, :K]^T, both
// operands row-major with K contiguous (A rows: inputs or query rows; B rows:
// weight rows or entity rows).
//
// A workgroup of 4 wavefronts (2 x 2) owns a BM x BN tile; each wavefront
// computes (BM / 32) x (BN / 32) tiles of v_mfma_f32_16x16x4_f32. K advances
// BK = 32 at a time through double-buffered LDS with one barrier per stage;
// the next stage's global loads sit in registers while the current stage
// computes. Within a 16-wide K slice, lane group g = lane / 16 feeds
// k = 4g .. 4g + 3 to four consecutive MFMAs from one 128-bit LDS read (a
// permutation of the reduction order over k).
//
// Edges: rows of A at or past M and rows of B at or past N are read from the
// last valid row (their products only reach outputs the caller discards);
// K positions at or past K read as zero. K must be a multiple of 4 and rows
// 16-byte aligned.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kgq {

typedef float v4f __attribute__((ext_vector_type(4)));

template <int BM, int BN>
struct MfmaTile {
    static constexpr int BK = 32;
    static constexpr int LD = BK + 4;                  // padded LDS row (floats)
    static constexpr int TM = BM / 32, TN = BN / 32;   // MFMA tiles per wavefront
    static constexpr int AL = BM / 32, BL = BN / 32;   // 128-bit loads per thread per stage
    static constexpr int SMEM = 2 * (BM + BN) * LD;    // floats

    __device__ static void run(const float* __restrict__ A, int64_t lda, int M, const float* __restrict__ B,
                               int64_t ldb, int N, int K, int m0, int n0, float* sm, v4f (&acc)[TM][TN])
    {
        float* As = sm;                    // [2][BM * LD]
        float* Bs = sm + 2 * BM * LD;      // [2][BN * LD]
        const int tid = threadIdx.x;
        const int lane = tid & 63;
        const int wave = tid >> 6;
        const int wm = wave >> 1, wn = wave & 1;
        const int grp = lane >> 4, li = lane & 15;

        // thread t stages k = (t % 8) * 4 .. +3 of tile rows t / 8 + 32 h
        const int lrow = tid >> 3, lk = (tid & 7) * 4;
        const float* ap[AL];
        const float* bp[BL];
#pragma unroll
        for (int h = 0; h < AL; ++h) ap[h] = A + (int64_t)min(m0 + lrow + 32 * h, M - 1) * lda + lk;
#pragma unroll
        for (int h = 0; h < BL; ++h) bp[h] = B + (int64_t)min(n0 + lrow + 32 * h, N - 1) * ldb + lk;
        float4 ra[AL], rb[BL];
        auto load = [&](int k0) {
            const bool ok = k0 + lk < K;
            const int kk = ok ? k0 : 0;
#pragma unroll
            for (int h = 0; h < AL; ++h) {
                const float4 v = *reinterpret_cast<const float4*>(ap[h] + kk);
                ra[h] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int h = 0; h < BL; ++h) {
                const float4 v = *reinterpret_cast<const float4*>(bp[h] + kk);
                rb[h] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        };
        auto stash = [&](int buf) {
#pragma unroll
            for (int h = 0; h < AL; ++h)
                *reinterpret_cast<float4*>(&As[buf * BM * LD + (lrow + 32 * h) * LD + lk]) = ra[h];
#pragma unroll
            for (int h = 0; h < BL; ++h)
                *reinterpret_cast<float4*>(&Bs[buf * BN * LD + (lrow + 32 * h) * LD + lk]) = rb[h];
        };

#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

        const int nk = (K + BK - 1) / BK;
        load(0);
        stash(0);
        __syncthreads();
        int buf = 0;
        for (int kt = 0; kt < nk; ++kt) {
            if (kt + 1 < nk) load((kt + 1) * BK);
            const float* as = As + buf * BM * LD + (wm * (BM / 2) + li) * LD + grp * 4;
            const float* bs = Bs + buf * BN * LD + (wn * (BN / 2) + li) * LD + grp * 4;
#pragma unroll
            for (int s = 0; s < BK / 16; ++s) {
                float4 av[TM], bv[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) av[i] = *reinterpret_cast<const float4*>(as + i * 16 * LD + s * 16);
#pragma unroll
                for (int j = 0; j < TN; ++j) bv[j] = *reinterpret_cast<const float4*>(bs + j * 16 * LD + s * 16);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) {
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
    }

    // Output position of acc[i][j][r] within the workgroup tile: row
    // wm * BM/2 + i * 16 + 4 * grp + r, column wn * BN/2 + j * 16 + li.
    __device__ static int row_of(int i) { return ((threadIdx.x >> 6) >> 1) * (BM / 2) + i * 16 + ((threadIdx.x & 63) >> 4) * 4; }
    __device__ static int col_of(int j) { return ((threadIdx.x >> 6) & 1) * (BN / 2) + j * 16 + (threadIdx.x & 15); }
};

}  // namespace kgq
