// Device-side matrix-core tile loops shared by the dense layers and the
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
// MfmaTileBf16x3 (K a multiple of 32): FP32 accuracy on the bf16 matrix
//   cores. B comes as three bf16 planes (split beforehand), A as FP32 and is
//   split in registers; six of the nine part products per k range, on
//   v_mfma_f32_16x16x32_bf16 with FP32 accumulation (details at the struct).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace kgq {

typedef float v4f __attribute__((ext_vector_type(4)));

template <int BM, int BN>
struct MfmaTileReg {
    static constexpr int kBM = BM, kBN = BN;
    static constexpr bool kBf16x3 = false;
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
    static constexpr bool kBf16x3 = false;
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

// ---- FP32 accuracy on the bf16 matrix cores ---------------------------------
//
// Split. Every FP32 value x is written exactly as x = h + m + l with h, m, l
// bf16: h = bf16(x), m = bf16(x - h), l = x - h - m (round to nearest even at
// each step). Both subtractions are exact in FP32, and l has at most 8
// significant bits, so it is a bf16 value and the sum is exact; |m| <= 2^-8 |x|
// and |l| <= 2^-16 |x|, up to rounding. Values must be finite and below the
// largest bf16 (3.39e38), above which h would round to infinity.
// Products. x y = hh' + hm' + mh' + mm' + hl' + lh' + (ml' + lm' + ll'): the
// first six are kept, the dropped three are below 2^-23 |x y| together. A
// bf16 x bf16 product is exact in FP32 and the matrix core accumulates in
// FP32, so a contraction has the error class of an FP32 one. Per 32 of K, six
// 16x16x32 bf16 MFMAs (16 cycles each) replace eight 16x16x4 FP32 MFMAs (32
// cycles each).
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

// 8 FP32 values (lo: elements 0..3, hi: 4..7) -> their three bf16 parts
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

__device__ __forceinline__ v4f mfma_bf16(const v4u& a, const v4u& b, v4f c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0, 0,
                                                   0);
}

// Tiles. A workgroup of 4 wavefronts owns a BM x BN tile; the wavefronts
// are stacked WM x (4 / WM) (4 x 1 by default: each splits a different part
// of A, so no A fragment is split twice in a workgroup), each with
// (BM / WM / 16) x (BN / (4 / WM) / 16) 16x16 blocks. Stages of 32 of K go
// through a two-slot LDS ring by direct-to-LDS loads: A as FP32 rows (128
// bytes, 16-byte chunks XOR-swizzled by row), B as three planes of bf16 rows
// (64 bytes, chunks swizzled by row / 2), so that the fragment reads of 16
// rows at one chunk fall in distinct banks. Lane l supplies row l % 16 of a
// block at k = 8 (l / 16) .. + 7 (the builtin's operand layout) and holds the
// output rows 4 (l / 16) .. + 3 of column l % 16, as in the FP32 loops. Rows
// of A at or past M and of B at or past N are read from the last valid row.
// Measured on the BetaE scorer (63,361 entities): 128 x 128 tiles with 4 x 1
// wavefronts and fragments read when their stage is multiplied ran 1.21 ms,
// 128 x 64 tiles 1.28-1.31 ms, against 1.37 ms with the next stage's
// fragments read ahead (which needs a second register set), 1.42-1.50 ms
// with 2 x 2 wavefronts, and 1.48 ms for 64 x 64 tiles with 2 x 2 wavefronts.
template <int BM, int BN, int WM = 4, bool PRIO = false>
struct MfmaTileBf16x3 {
    static constexpr int kBM = BM, kBN = BN;
    static constexpr bool kBf16x3 = true;
    static constexpr int BK = 32;
    static constexpr int WN = 4 / WM;                  // wavefronts along N
    static constexpr int AROW = BK * 4;                // bytes of one A row per stage (FP32)
    static constexpr int BROW = BK * 2;                // bytes of one B row per stage and plane (bf16)
    static constexpr int ABYTES = BM * AROW;
    static constexpr int STAGE = ABYTES + 3 * BN * BROW;
    static constexpr int SMEM = 2 * STAGE / 4;         // floats
    static constexpr int TM = BM / WM / 16, TN = BN / WN / 16;   // 16x16 blocks per wavefront
    static constexpr int AI = BM / 32;                 // A load instructions per wavefront and stage (8 rows each)
    static constexpr int BI = 3 * BN / 64;             // B load instructions per wavefront and stage (16 rows each)
    static constexpr int LPS = AI + BI;
    static_assert((WM == 2 || WM == 4) && TM >= 1 && TN >= 1 && BM % 32 == 0 && BN % 64 == 0 && LPS < 64,
                  "tile shape");
    static_assert(2 * STAGE <= 160 * 1024, "LDS");   // above 64 KiB only as dynamic LDS

    // K a multiple of 4 of at least one stage; when K is not a multiple of 32
    // the B planes must hold zeros from K to the next multiple of 32 (their
    // rows padded to it), and the last stage's A chunks past K re-read the
    // previous stage's (finite values, multiplied by those zeros)
    static bool supports(int K) { return K >= BK && K % 4 == 0; }
    __device__ static int aswz(int row) { return (row & 7) ^ ((row >> 3) & 1); }
    __device__ static int bswz(int row) { return (row >> 1) & 3; }

    // acc = A[m0 : m0 + BM, :K] . B[n0 : n0 + BN, :K]^T; B's planes are
    // Bp, Bp + plane, Bp + 2 plane (row stride ldb elements, zero-padded
    // past K as above). A's rows are read up to M - 1; a wavefront whose rows
    // all lie at or past live_rows (output rows the caller drops) takes its
    // share of the loads and the barriers but no products, and its acc stays
    // zero.
    __device__ static void run(const float* __restrict__ A, int64_t lda, int M, int live_rows,
                               const uint16_t* __restrict__ Bp, int64_t plane, int64_t ldb, int N, int K, int m0,
                               int n0, float* sm_f, v4f (&acc)[TM][TN])
    {
        char* sm = reinterpret_cast<char*>(sm_f);
        const int nk = (K + BK - 1) / BK;
        const int tid = threadIdx.x, lane = tid & 63;
        const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
        const int wm = wave / WN, wn = wave % WN;
        const int grp = lane >> 4, li = lane & 15;

        // A: load instruction t = h * 4 + wave writes rows 8t .. 8t + 7
        // (1 KiB); lane l lands at row 8t + l / 8, chunk position l % 8.
        // With K not a multiple of 32, a lane whose chunk of the last stage
        // starts at or past K reads the chunk one stage back: inside the row,
        // since K >= 32, or the caller's A starts at least a stage into it.
        const float* ag[AI];
        bool past[AI];
        const int k_last = (nk - 1) * BK;
#pragma unroll
        for (int h = 0; h < AI; ++h) {
            const int row = (h * 4 + wave) * 8 + (lane >> 3);
            const int chunk = (lane & 7) ^ aswz(row);
            ag[h] = A + (int64_t)min(m0 + row, M - 1) * lda + chunk * 4;
            past[h] = k_last + chunk * 4 >= K;
        }
        // B: load instruction u = h * 4 + wave writes plane u / (BN / 16),
        // rows 16 (u % (BN / 16)) .. + 15; lane l lands at row + l / 4,
        // chunk position l % 4
        const uint16_t* bg[BI];
        int bdst[BI];
#pragma unroll
        for (int h = 0; h < BI; ++h) {
            const int u = h * 4 + wave;
            const int p = u / (BN / 16), rb = u % (BN / 16);
            const int row = rb * 16 + (lane >> 2);
            bg[h] = Bp + p * plane + (int64_t)min(n0 + row, N - 1) * ldb + ((lane & 3) ^ bswz(row)) * 8;
            bdst[h] = ABYTES + (p * BN + rb * 16) * BROW;
        }
        auto issue = [&](int kt, int slot) {
            char* st = sm + slot * STAGE;
            const bool tail = kt == nk - 1 && (K % BK) != 0;
#pragma unroll
            for (int h = 0; h < AI; ++h)
                __builtin_amdgcn_global_load_lds((const void*)(ag[h] + (kt - (tail && past[h] ? 1 : 0)) * BK),
                                                 (lds_void*)(st + (h * 4 + wave) * 8 * AROW), 16, 0, 0);
#pragma unroll
            for (int h = 0; h < BI; ++h)
                __builtin_amdgcn_global_load_lds((const void*)(bg[h] + kt * BK), (lds_void*)(st + bdst[h]), 16, 0,
                                                 0);
        };

        // fragment offsets in a stage: A block i at k = 8 grp .. + 7
        // (chunks 2 grp, 2 grp + 1), B block j at chunk grp
        int aoff[TM][2], boff[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int row = wm * (BM / WM) + i * 16 + li;
#pragma unroll
            for (int q = 0; q < 2; ++q) aoff[i][q] = row * AROW + ((2 * grp + q) ^ aswz(row)) * 16;
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int row = wn * (BN / WN) + j * 16 + li;
            boff[j] = ABYTES + row * BROW + (grp ^ bswz(row)) * 16;
        }

#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

        Bf16x3 fa[TM];          // the stage being multiplied: A split, B as read
        v4u fb[3][TN];
        auto read_split = [&](int slot) {
            const char* st = sm + slot * STAGE;
            v4u ra[TM][2];
#pragma unroll
            for (int i = 0; i < TM; ++i) {
                ra[i][0] = *reinterpret_cast<const v4u*>(st + aoff[i][0]);
                ra[i][1] = *reinterpret_cast<const v4u*>(st + aoff[i][1]);
            }
#pragma unroll
            for (int p = 0; p < 3; ++p)
#pragma unroll
                for (int j = 0; j < TN; ++j) fb[p][j] = *reinterpret_cast<const v4u*>(st + boff[j] + p * BN * BROW);
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[i] = split_bf16x3(ra[i][0], ra[i][1]);
        };
        // the six kept products, largest first; consecutive MFMAs update
        // different accumulators
        auto products = [&]() {
#pragma unroll
            for (int q = 0; q < 6; ++q)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) {
                        const v4u& a = (q == 0 || q == 1 || q == 4) ? fa[i].h : (q == 5 ? fa[i].l : fa[i].m);
                        const v4u& b = (q == 0 || q == 2 || q == 5) ? fb[0][j] : (q == 4 ? fb[2][j] : fb[1][j]);
                        acc[i][j] = mfma_bf16(a, b, acc[i][j]);
                    }
        };

        // A stage's fragments are read when it is multiplied (the other
        // workgroups on the compute unit cover the LDS latency). With PRIO
        // the wavefront raises its issue priority while it reads and splits
        // them, so that a wavefront about to feed the matrix core is served
        // before one whose products are already queued: measured on the
        // 63,361-entity BetaE scorer 1.209 -> 1.166 ms per launch, and on
        // the 64 x 64 tiles; the 128 x 64 dense tiles gained nothing. One barrier
        // per stage: past it, stage kt has landed for every wavefront and
        // every wavefront has read stage kt - 1, whose slot then takes stage
        // kt + 1 while stage kt is multiplied. The wait counts this loop's
        // loads only: the caller has no vector-memory load outstanding on
        // entry, and at the wait stage kt's are the only ones in flight.
        issue(0, 0);
        if (m0 + wm * (BM / WM) < live_rows) {
            for (int kt = 0; kt < nk; ++kt) {
                wait_vm_barrier<0>();
                if (kt + 1 < nk) issue(kt + 1, (kt + 1) & 1);
                if constexpr (PRIO) __builtin_amdgcn_s_setprio(1);
                read_split(kt & 1);
                if constexpr (PRIO) __builtin_amdgcn_s_setprio(0);
                products();
            }
        } else {
            for (int kt = 0; kt < nk; ++kt) {
                wait_vm_barrier<0>();
                if (kt + 1 < nk) issue(kt + 1, (kt + 1) & 1);
            }
        }
    }

    // Output position of acc[i][j][r] within the workgroup tile.
    __device__ static int row_of(int i) { return ((threadIdx.x >> 6) / WN) * (BM / WM) + i * 16 + ((threadIdx.x & 63) >> 4) * 4; }
    __device__ static int col_of(int j) { return ((threadIdx.x >> 6) % WN) * (BN / WN) + j * 16 + (threadIdx.x & 15); }
};

}  // namespace kgq
