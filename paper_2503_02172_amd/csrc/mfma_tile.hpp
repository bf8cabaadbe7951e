// Device-side FP32 matrix-core tile loops shared by the dense layers and the
// BetaE scorer: acc = A[m0 : m0 + BM, :K] . B[n0 : n0 + BN, :K]^T, both
// operands row-major with K contiguous (A rows: inputs or query rows; B rows:
// weight rows or entity rows).
//
// Common to both loops: a workgroup of 4 wavefronts (2 x 2) owns a BM x BN
// tile; each wavefront computes (BM / 32) x (BN / 32) tiles of
// v_mfma_f32_16x16x4_f32. Within a 16-wide K slice, lane group g = lane / 16
// feeds k = 4g .. 4g + 3 to four consecutive MFMAs from one 128-bit LDS read
// (a permutation of the reduction order over k, the same in both loops, so
// they give identical results). Rows of A at or past M and rows of B at or
// past N are read from the last valid row (their products only reach outputs
// the caller discards). Rows must be 16-byte aligned.
//
// MfmaTileLds (K a multiple of 16): a ring of S LDS stages of BK = 32 filled
//   by direct-to-LDS loads (global_load_lds_dwordx4: each wave instruction
//   writes 1 KiB of LDS, no staging registers, no LDS store instructions).
//   Stage kt + S - 1 is requested while stage kt computes; one barrier per
//   stage. Rows are stored unpadded with their 16-byte chunks XOR-swizzled by
//   row (chunk c of row r at position c ^ (r & 7)), so the fragment reads of
//   16 rows at one chunk hit distinct banks. The fragment registers are
//   double-buffered: the second half-stage's fragments, and the next stage's
//   first, are read before the current MFMAs issue. The HALF instantiation
//   serves K an odd multiple of 16: one more stage holds the last 16 of K,
//   its lanes whose chunk lies past K load a chunk 16 floats lower in the
//   same row instead (in bounds, never read), and it runs its first half
//   only. (Kept out of the other instantiation, whose loop it slowed by 3%.)
// MfmaTileReg (any K multiple of 4): double-buffered LDS, the next stage's
//   global loads held in registers while the current stage computes, padded
//   LDS rows; the K tail reads as zero.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace kgq {

typedef float v4f __attribute__((ext_vector_type(4)));

template <int BM, int BN>
struct MfmaTileReg {
    static constexpr int kBM = BM, kBN = BN;
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

// s_waitcnt vmcnt(N) lgkmcnt(0); s_barrier. Written as one asm statement with
// a memory clobber: the compiler neither moves LDS accesses across it nor
// adds its own vmcnt(0) (which a __syncthreads() would, draining every
// outstanding direct-to-LDS load of later stages).
template <int N>
__device__ __forceinline__ void wait_vm_barrier()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

typedef __attribute__((address_space(3))) void lds_void;

template <int BM, int BN, int S, bool HALF = false>
struct MfmaTileLds {
    static constexpr int kBM = BM, kBN = BN;
    static constexpr int BK = 32;
    static constexpr int CH = BK / 4;                  // 16-byte chunks per row per stage
    static constexpr int RPI = 64 / CH;                // rows written by one wave instruction
    static constexpr int AI = BM / (RPI * 4), BI = BN / (RPI * 4);   // instructions per wave per stage
    static constexpr int LPS = AI + BI;
    static constexpr int TM = BM / 32, TN = BN / 32;
    static constexpr int STAGE = (BM + BN) * BK;       // floats
    static constexpr int SMEM = S * STAGE;             // floats
    static_assert(S >= 2 && AI >= 1 && BI >= 1, "tile shape");
    static_assert((S - 2) * LPS < 64, "vmcnt range");

    __device__ static int swz(int row) { return row & 7; }
    static bool supports(int K) { return K > 0 && K % BK == (HALF ? 16 : 0); }

    __device__ static void run(const float* __restrict__ A, int64_t lda, int M, const float* __restrict__ B,
                               int64_t ldb, int N, int K, int m0, int n0, float* sm, v4f (&acc)[TM][TN])
    {
        const int tid = threadIdx.x, lane = tid & 63;
        const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int wm = wave >> 1, wn = wave & 1;
        const int grp = lane >> 4, li = lane & 15;

        // Loads: wave instruction t = h * 4 + wave writes rows t * RPI ..
        // t * RPI + RPI - 1 of the stage's A (or B) block; its lane l lands at
        // row t * RPI + l / CH, chunk position l % CH, so it reads the global
        // chunk (l % CH) ^ swz(row).
        const int lr = lane / CH, lp = lane % CH;
        const int nfull = K / BK;                       // full stages
        const int nk = nfull + (HALF ? 1 : 0);          // HALF: one more stage holding 16 of K
        const float* ag[AI];
        const float* bg[BI];
        bool aup[AI], bup[BI];                           // loads a chunk of the upper half-stage
#pragma unroll
        for (int h = 0; h < AI; ++h) {
            const int row = (h * 4 + wave) * RPI + lr, c = lp ^ swz(row);
            ag[h] = A + (int64_t)min(m0 + row, M - 1) * lda + c * 4;
            aup[h] = c >= 4;
        }
#pragma unroll
        for (int h = 0; h < BI; ++h) {
            const int row = (h * 4 + wave) * RPI + lr, c = lp ^ swz(row);
            bg[h] = B + (int64_t)min(n0 + row, N - 1) * ldb + c * 4;
            bup[h] = c >= 4;
        }
        auto issue = [&](int kt, int slot) {
            float* st = sm + slot * STAGE;
#pragma unroll
            for (int h = 0; h < AI; ++h)
                __builtin_amdgcn_global_load_lds((const void*)(ag[h] + kt * BK),
                                                 (lds_void*)(st + (h * 4 + wave) * RPI * BK), 16, 0, 0);
#pragma unroll
            for (int h = 0; h < BI; ++h)
                __builtin_amdgcn_global_load_lds((const void*)(bg[h] + kt * BK),
                                                 (lds_void*)(st + BM * BK + (h * 4 + wave) * RPI * BK), 16, 0, 0);
        };
        // the half stage: chunks past K come from 16 floats lower in the row
        auto issue_half = [&](int kt, int slot) {
            float* st = sm + slot * STAGE;
#pragma unroll
            for (int h = 0; h < AI; ++h)
                __builtin_amdgcn_global_load_lds((const void*)(ag[h] + kt * BK - (aup[h] ? 16 : 0)),
                                                 (lds_void*)(st + (h * 4 + wave) * RPI * BK), 16, 0, 0);
#pragma unroll
            for (int h = 0; h < BI; ++h)
                __builtin_amdgcn_global_load_lds((const void*)(bg[h] + kt * BK - (bup[h] ? 16 : 0)),
                                                 (lds_void*)(st + BM * BK + (h * 4 + wave) * RPI * BK), 16, 0, 0);
        };
        auto issue_any = [&](int kt, int slot) {
            if constexpr (HALF) {
                if (kt == nfull) {
                    issue_half(kt, slot);
                    return;
                }
            }
            issue(kt, slot);
        };

        // Fragment offsets within a stage (floats): half-stage s covers
        // chunks 4s .. 4s + 3, lane group grp reads chunk 4s + grp.
        int aoff[TM][2], boff[TN][2];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int row = wm * (BM / 2) + i * 16 + li;
#pragma unroll
            for (int s = 0; s < 2; ++s) aoff[i][s] = row * BK + ((s * 4 + grp) ^ swz(row)) * 4;
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int row = wn * (BN / 2) + j * 16 + li;
#pragma unroll
            for (int s = 0; s < 2; ++s) boff[j][s] = BM * BK + row * BK + ((s * 4 + grp) ^ swz(row)) * 4;
        }
        v4f fa[2][TM], fb[2][TN];
        auto read = [&](int slot, int s, int f) {
            const float* st = sm + slot * STAGE;
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[f][i] = *reinterpret_cast<const v4f*>(st + aoff[i][s]);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[f][j] = *reinterpret_cast<const v4f*>(st + boff[j][s]);
        };
        auto mma = [&](int f) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[f][i][q], fb[f][j][q], acc[i][j], 0, 0, 0);
        };

#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

        // The vmcnt accounting below counts only this loop's loads: the
        // caller has no vector-memory load outstanding on entry.
#pragma unroll
        for (int s = 0; s < S - 1; ++s)
            if (s < nk) issue_any(s, s);
        if (nk >= S - 1) wait_vm_barrier<(S - 2) * LPS>();   // stage 0 landed
        else wait_vm_barrier<0>();
        read(0, 0, 0);
        for (int kt = 0; kt < nfull; ++kt) {
            // Slot (kt + S - 1) % S was last read in stage kt - 1; every wave
            // passed the barrier after finishing those reads.
            const bool more = kt + S - 1 < nk;
            if (more) issue_any(kt + S - 1, (kt + S - 1) % S);
            read(kt % S, 1, 1);
            mma(0);
            if (kt + 1 < nk) {
                // stage kt + 1 landed for this wave (later stages may still be
                // in flight); the barrier makes it so for every wave
                if (more) wait_vm_barrier<(S - 2) * LPS>();
                else wait_vm_barrier<0>();
                read((kt + 1) % S, 0, 0);
            }
            mma(1);
        }
        // the half stage: its first half-stage fragments are in buffer 0
        if constexpr (HALF) mma(0);
    }

    __device__ static int row_of(int i) { return ((threadIdx.x >> 6) >> 1) * (BM / 2) + i * 16 + ((threadIdx.x & 63) >> 4) * 4; }
    __device__ static int col_of(int j) { return ((threadIdx.x >> 6) & 1) * (BN / 2) + j * 16 + (threadIdx.x & 15); }
};

}  // namespace kgq
