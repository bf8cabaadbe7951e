// Top-k selection over each query's N entity scores (the ranking the paper
// evaluates with MRR, Experiments/Metrics). Order: score descending, equal
// scores by entity index ascending.
//
// One workgroup of 1024 threads selects the top k of one segment of at most
// 16 Ki scores, held in registers (KPT keys per thread, element i =
// j * 1024 + tid). Scores map to order-preserving 32-bit keys. Bits that
// every key of the segment shares (typically the sign and most of the
// exponent) are found with a block-wide OR / AND and skipped. One histogram
// pass over the next 11 bits then locates the bin that holds the k-th key;
// every key in that bin or above (k plus the bin's other members) is
// compacted into LDS as (key, index) composites and sorted, and the first k
// are the answer, ties included (the composite orders equal keys by index).
// If that candidate set would exceed the LDS buffer (very many equal or
// nearly equal scores), exact radix passes of 8 bits narrow the threshold key
// T down instead, and the keys above T plus the lowest-index keys equal to T
// are taken. Compaction uses a prefix over per-(step, wavefront) ballot
// counts, so it needs no atomics. Sorting runs in registers inside one
// wavefront for up to 256 candidates, in LDS across the workgroup otherwise.
//
// Rows longer than one segment take two (or more) launches: each segment of
// a row yields its top k, then the same kernel selects the top k of those
// candidates through an index map. Segments are contiguous index ranges and
// each segment's list is ordered by (score desc, index asc), so among equal
// scores candidate position order is global index order, and the tie rule
// carries through. A segment shorter than k pads its list with -inf
// entries, which never outrank a real score.
#include "kgq_internal.hpp"

namespace kgq {

constexpr int TK_THREADS = 1024;
constexpr int TK_WAVES = TK_THREADS / 64;

__device__ __forceinline__ uint32_t score_key(float f)
{
    if (f == 0.0f) f = 0.0f;   // -0 and +0 rank equal
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_score(uint32_t key)
{
    return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// composite c = key << 32 | (2^32 - 1 - index): descending c = score
// descending, then index ascending
__device__ __forceinline__ uint64_t composite(uint32_t key, int32_t idx)
{
    return ((uint64_t)key << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)idx);
}

__device__ __forceinline__ void store_one(const TopkArgs& a, int64_t orow, int p, uint64_t c)
{
    a.out_idx[orow * a.out_ld + p] = (int32_t)(0xFFFFFFFFu - (uint32_t)c);
    a.out_score[orow * a.out_ld + p] = key_score((uint32_t)(c >> 32));
}

// Sort the n selected entries inside one wavefront (P = 64 * E >= n
// positions, lane l holds positions e * 64 + l; padding sorts last) and
// write out the first k.
template <int E>
__device__ __forceinline__ void bitonic_wave(const uint64_t* sel, int n, int k, int64_t orow, int lane,
                                             const TopkArgs& a)
{
    constexpr int P = 64 * E;
    uint64_t v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int p = e * 64 + lane;
        v[e] = p < n ? sel[p] : 0ull;
    }
#pragma unroll
    for (int size = 2; size <= P; size <<= 1) {
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            if (stride >= 64) {
                const int es = stride >> 6;
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const int f = e ^ es;
                    if (f > e) {
                        const bool desc = ((e * 64 + lane) & size) == 0;
                        const uint64_t a0 = v[e], a1 = v[f];
                        const bool sw = desc ? (a0 < a1) : (a0 > a1);
                        v[e] = sw ? a1 : a0;
                        v[f] = sw ? a0 : a1;
                    }
                }
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const uint32_t lo = __shfl_xor((uint32_t)v[e], stride, 64);
                    const uint32_t hi = __shfl_xor((uint32_t)(v[e] >> 32), stride, 64);
                    const uint64_t w = ((uint64_t)hi << 32) | lo;
                    const bool desc = ((e * 64 + lane) & size) == 0;
                    const bool lower = (lane & stride) == 0;   // this position is the lower of the pair
                    const uint64_t mx = v[e] > w ? v[e] : w, mn = v[e] > w ? w : v[e];
                    v[e] = (desc == lower) ? mx : mn;
                }
            }
        }
    }
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int p = e * 64 + lane;
        if (p < k) store_one(a, orow, p, v[e]);
    }
}

// Exclusive prefix, in place, over the KPT * 16 per-(step, wavefront) counts
// in (step, wavefront) order, which is element index order. Run by the whole
// workgroup; only wavefront 0 works.
template <int KPT>
__device__ __forceinline__ void block_exclusive_prefix(int* cnt, int tid)
{
    if (tid >= 64) return;
    constexpr int NC = KPT * TK_WAVES;
    constexpr int PER = (NC + 63) / 64;
    int s = 0;
#pragma unroll
    for (int t = 0; t < PER; ++t) {
        const int c = tid * PER + t;
        if (c < NC) s += cnt[c];
    }
    int incl = s;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off, 64);
        if (tid >= off) incl += v;
    }
    int b = incl - s;
#pragma unroll
    for (int t = 0; t < PER; ++t) {
        const int c = tid * PER + t;
        if (c < NC) {
            const int v = cnt[c];
            cnt[c] = b;
            b += v;
        }
    }
}

template <int KPT>
__global__ __launch_bounds__(TK_THREADS) void k_topk(TopkArgs a)
{
    __shared__ uint32_t hist[2048];
    __shared__ uint64_t sel[kMaxK];
    __shared__ int sh_bin, sh_rem;
    __shared__ uint32_t sh_or[TK_WAVES], sh_and[TK_WAVES];
    __shared__ int cnt_gt[KPT * TK_WAVES], cnt_eq[KPT * TK_WAVES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t row = blockIdx.y;
    const int64_t seg0 = (int64_t)blockIdx.x * a.seg_len;     // first element of this segment
    int64_t n = a.N - seg0;
    if (n > a.seg_len) n = a.seg_len;
    const float* __restrict__ sr = a.scores + row * a.ld + seg0;
    const int32_t* __restrict__ ir = a.in_idx ? a.in_idx + row * a.ld + seg0 : nullptr;
    const int k = a.k < n ? a.k : (int)n;   // a segment shorter than k yields all of it

    uint32_t keys[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j) {
        const int64_t i = (int64_t)j * TK_THREADS + tid;
        keys[j] = i < n ? score_key(sr[i]) : 0u;
    }

    // bits shared by every key: OR and AND over the segment
    {
        uint32_t o = 0u, an = 0xFFFFFFFFu;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            if ((int64_t)j * TK_THREADS + tid < n) { o |= keys[j]; an &= keys[j]; }
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            o |= __shfl_xor(o, off, 64);
            an &= __shfl_xor(an, off, 64);
        }
        if (lane == 0) { sh_or[wave] = o; sh_and[wave] = an; }
    }
    __syncthreads();
    uint32_t all_or = 0u, all_and = 0xFFFFFFFFu;
#pragma unroll
    for (int w = 0; w < TK_WAVES; ++w) { all_or |= sh_or[w]; all_and &= sh_and[w]; }
    const uint32_t diff = all_or ^ all_and;            // bits that differ somewhere
    int top = diff ? 31 - __clz(diff) : -1;            // highest differing bit

    // bits above `top` are common to all keys: they start the prefix
    uint32_t pmask = diff ? ~(0xFFFFFFFFu >> (31 - top)) : 0xFFFFFFFFu;
    uint32_t prefix = all_and & pmask;

    // --- one wide histogram pass: the bin of the k-th key -------------------
    // digit = bits [wlo, top], at most 11 bits
    const int wlo = top >= 10 ? top - 10 : 0;
    const uint32_t wmask = top >= 0 ? ((2u << (top - wlo)) - 1u) : 0u;
    int n_cand = (int)n;       // candidates: keys whose digit is >= the k-th key's digit
    uint32_t dmin = 0;         // smallest candidate digit
    if (top >= 0) {
        for (int b = tid; b < 2048; b += TK_THREADS) hist[b] = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const int64_t i = (int64_t)j * TK_THREADS + tid;
            const bool act = i < n;
            const uint32_t bin = (keys[j] >> wlo) & wmask;
            const uint64_t am = __ballot(act);
            if (act) {
                const int first = __ffsll((unsigned long long)am) - 1;
                const uint32_t b0 = __shfl(bin, first, 64);
                const uint64_t same = __ballot(bin == b0);
                if ((same & am) == am) {
                    if (lane == first) atomicAdd(&hist[b0], (uint32_t)__popcll(am));
                } else {
                    atomicAdd(&hist[bin], 1u);
                }
            }
        }
        __syncthreads();
        if (tid < 64) {
            // lane l owns bins 32l .. 32l+31; inclusive suffix sum over lanes
            uint32_t s = 0;
#pragma unroll
            for (int t = 0; t < 32; ++t) s += hist[32 * tid + t];
            uint32_t incl = s;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const uint32_t v = __shfl_down(incl, off, 64);
                if (tid + off < 64) incl += v;
            }
            const uint32_t above = incl - s;
            if (above < (uint32_t)k && (uint32_t)k <= incl) {
                uint32_t cum = above;
                for (int t = 31; t >= 0; --t) {
                    const uint32_t c = hist[32 * tid + t];
                    if ((uint32_t)k <= cum + c) {
                        sh_bin = 32 * tid + t;
                        sh_rem = (int)(cum + c);      // candidates: bins >= this one
                        break;
                    }
                    cum += c;
                }
            }
        }
        __syncthreads();
        dmin = (uint32_t)sh_bin;
        n_cand = sh_rem;
    }

    int n_sel;                 // entries placed in sel[]
    if (n_cand <= kMaxK) {
        // --- candidates fit: take every key whose digit is >= dmin ----------
        n_sel = n_cand;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const int64_t i = (int64_t)j * TK_THREADS + tid;
            const uint64_t bc = __ballot(i < n && ((keys[j] >> wlo) & wmask) >= dmin);
            if (lane == 0) cnt_gt[j * TK_WAVES + wave] = __popcll(bc);
        }
        __syncthreads();
        block_exclusive_prefix<KPT>(cnt_gt, tid);
        __syncthreads();
        const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const int64_t i = (int64_t)j * TK_THREADS + tid;
            const bool f = i < n && ((keys[j] >> wlo) & wmask) >= dmin;
            const uint64_t bc = __ballot(f);
            if (f) {
                const int slot = cnt_gt[j * TK_WAVES + wave] + __popcll(bc & lt);
                if (slot < kMaxK) sel[slot] = composite(keys[j], ir ? ir[i] : (int32_t)(seg0 + i));
            }
        }
    } else {
        // --- too many candidates: exact radix passes find T ------------------
        int rem = k;
        for (int lo = top - 7; top >= 0; lo -= 8) {
            // digit = bits [max(lo, 0), top] of the key
            const int shift = lo > 0 ? lo : 0;
            const int width = top - shift + 1;
            const uint32_t dmask = (1u << width) - 1u;      // width <= 8
            if (tid < 256) hist[tid] = 0;
            __syncthreads();
#pragma unroll
            for (int j = 0; j < KPT; ++j) {
                const int64_t i = (int64_t)j * TK_THREADS + tid;
                const uint32_t key = keys[j];
                const bool act = i < n && (key & pmask) == prefix;
                const uint32_t bin = (key >> shift) & dmask;
                const uint64_t am = __ballot(act);
                if (act) {
                    const int first = __ffsll((unsigned long long)am) - 1;
                    const uint32_t b0 = __shfl(bin, first, 64);
                    const uint64_t same = __ballot(bin == b0);
                    if ((same & am) == am) {
                        if (lane == first) atomicAdd(&hist[b0], (uint32_t)__popcll(am));
                    } else {
                        atomicAdd(&hist[bin], 1u);
                    }
                }
            }
            __syncthreads();
            if (tid < 64) {
                // lane l owns bins 4l..4l+3; inclusive suffix sum over lanes
                uint32_t c[4], s = 0;
#pragma unroll
                for (int t = 0; t < 4; ++t) { c[t] = hist[4 * tid + t]; s += c[t]; }
                uint32_t incl = s;
#pragma unroll
                for (int off = 1; off < 64; off <<= 1) {
                    const uint32_t v = __shfl_down(incl, off, 64);
                    if (tid + off < 64) incl += v;
                }
                const uint32_t above = incl - s;
                if (above < (uint32_t)rem && (uint32_t)rem <= incl) {
                    uint32_t cum = above;
                    for (int t = 3; t >= 0; --t) {
                        if ((uint32_t)rem <= cum + c[t]) {
                            sh_bin = 4 * tid + t;
                            sh_rem = rem - (int)cum;
                            break;
                        }
                        cum += c[t];
                    }
                }
            }
            __syncthreads();
            prefix |= (uint32_t)sh_bin << shift;
            pmask |= dmask << shift;
            rem = sh_rem;
            __syncthreads();
            top = shift - 1;
        }
        // prefix is now the exact key T of the k-th element; the k - rem keys
        // above T and the first rem keys equal to T (index order) are selected.
        const uint32_t T = prefix;
        const int n_gt = k - rem;
        n_sel = k;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const int64_t i = (int64_t)j * TK_THREADS + tid;
            const uint64_t bg = __ballot(i < n && keys[j] > T);
            const uint64_t be = __ballot(i < n && keys[j] == T);
            if (lane == 0) {
                cnt_gt[j * TK_WAVES + wave] = __popcll(bg);
                cnt_eq[j * TK_WAVES + wave] = __popcll(be);
            }
        }
        __syncthreads();
        block_exclusive_prefix<KPT>(cnt_gt, tid);
        __syncthreads();
        block_exclusive_prefix<KPT>(cnt_eq, tid);
        __syncthreads();
        const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const int64_t i = (int64_t)j * TK_THREADS + tid;
            const bool fg = i < n && keys[j] > T, fe = i < n && keys[j] == T;
            const uint64_t bg = __ballot(fg);
            const uint64_t be = __ballot(fe);
            int slot = -1;
            if (fg) slot = cnt_gt[j * TK_WAVES + wave] + __popcll(bg & lt);
            else if (fe) {
                const int r = cnt_eq[j * TK_WAVES + wave] + __popcll(be & lt);
                if (r < rem) slot = n_gt + r;
            }
            // slots stay below k by construction; the check keeps LDS accesses
            // inside the buffer regardless
            if (slot >= 0 && slot < k)
                sel[slot] = composite(keys[j], ir ? ir[i] : (int32_t)(seg0 + i));
        }
    }
    __syncthreads();

    // order the n_sel selected entries and write the first k; a short
    // segment pads its list to a.k entries with -inf
    const int64_t orow = row * a.out_rows_per_row + blockIdx.x;
    for (int p = k + tid; p < a.k; p += TK_THREADS) {
        a.out_idx[orow * a.out_ld + p] = 0x7FFFFFFF;
        a.out_score[orow * a.out_ld + p] = -__builtin_inff();
    }
    if (n_sel <= 256) {
        if (tid < 64) {
            if (n_sel <= 64) bitonic_wave<1>(sel, n_sel, k, orow, lane, a);
            else if (n_sel <= 128) bitonic_wave<2>(sel, n_sel, k, orow, lane, a);
            else bitonic_wave<4>(sel, n_sel, k, orow, lane, a);
        }
    } else {
        int P = 512;
        while (P < n_sel) P <<= 1;             // 512 or 1024
        for (int p = n_sel + tid; p < P; p += TK_THREADS) sel[p] = 0ull;
        for (int size = 2; size <= P; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                __syncthreads();
                if (tid < P) {
                    const int q = tid ^ stride;
                    if (q > tid) {
                        const bool desc = (tid & size) == 0;
                        const uint64_t a0 = sel[tid], a1 = sel[q];
                        if (desc ? (a0 < a1) : (a0 > a1)) { sel[tid] = a1; sel[q] = a0; }
                    }
                }
            }
        }
        __syncthreads();
        if (tid < k) store_one(a, orow, tid, sel[tid]);
    }
}

static void launch_segments(const TopkArgs& a, hipStream_t s)
{
    const int64_t per = (a.seg_len + TK_THREADS - 1) / TK_THREADS;
    dim3 grid((unsigned)((a.N + a.seg_len - 1) / a.seg_len), (unsigned)a.n_rows), block(TK_THREADS);
    if (per <= 1) hipLaunchKernelGGL(k_topk<1>, grid, block, 0, s, a);
    else if (per <= 2) hipLaunchKernelGGL(k_topk<2>, grid, block, 0, s, a);
    else if (per <= 4) hipLaunchKernelGGL(k_topk<4>, grid, block, 0, s, a);
    else if (per <= 8) hipLaunchKernelGGL(k_topk<8>, grid, block, 0, s, a);
    else hipLaunchKernelGGL(k_topk<16>, grid, block, 0, s, a);
}

int64_t topk_scratch_elems(int64_t n_rows, int64_t N, int k)
{
    const int64_t segs = (N + kTopkSegment - 1) / kTopkSegment;
    return segs > 1 ? n_rows * segs * k : 0;
}

void launch_topk(const TopkArgs& in, hipStream_t s)
{
    if (in.n_rows <= 0) return;
    TopkArgs a = in;
    a.in_idx = nullptr;
    a.out_ld = a.k;
    a.out_rows_per_row = 1;
    // Rounds: segments of kTopkSegment -> per-segment top-k candidates laid
    // out [row][segment][k] in a scratch buffer, until one segment holds a
    // row's whole candidate list. Each round's output is smaller than the
    // first's, so two buffers of topk_scratch_elems() entries suffice.
    int ping = 0;
    while (a.N > kTopkSegment) {
        const int64_t segs = (a.N + kTopkSegment - 1) / kTopkSegment;
        TopkArgs r = a;
        r.seg_len = kTopkSegment;
        r.out_idx = in.cand_idx[ping];
        r.out_score = in.cand_score[ping];
        r.out_ld = a.k;
        r.out_rows_per_row = (int)segs;
        launch_segments(r, s);
        a.scores = in.cand_score[ping];
        a.in_idx = in.cand_idx[ping];
        a.ld = segs * a.k;
        a.N = segs * a.k;
        ping ^= 1;
    }
    a.seg_len = a.N;
    launch_segments(a, s);
}

}  // namespace kgq
