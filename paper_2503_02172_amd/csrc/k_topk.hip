// Top-k selection over each query's N entity scores (the ranking the paper
// evaluates with MRR, Experiments/Metrics). Order: score descending, equal
// scores by entity index ascending. Scores map to order-preserving 32-bit
// keys; equal keys are ordered by index through a (key, ~index) composite.
//
// Two kernels, chosen per round by launch_topk:
//
// Streaming (k <= 256 with enough rows to occupy the chip, the path of large
// batches): one wavefront per row (or per segment of a row when rows are
// few), no workgroup barriers. The wavefront streams its scores once and
// keeps only those at or above a running threshold in an LDS candidate
// buffer; the threshold starts from the k-th largest of the column maxima
// of the first 1,536 scores and rises whenever the buffer is pruned. The end is a last prune
// and a sort of at most 256 candidates inside the wavefront. Its cost per
// score is a compare and a ballot, so it runs near the rate the scores
// stream in.
//
// Register-resident (k > 256, or small batches, where latency matters more
// than throughput): one workgroup of 256 threads selects the top k of one
// segment of at most 16 Ki scores, held in registers (KPT keys per thread,
// element i = j * 256 + tid), all loads issued at once.
//   Common case (k <= 256): each thread's largest key is taken, and the k-th
//   largest of those 256 maxima, L, is a lower bound of the segment's k-th
//   key (k distinct keys, one per thread, are at least L). Only slightly
//   more than k keys usually reach L (about 120 for k = 100 among 14,505
//   scores); they are compacted into LDS, with ranges per wavefront from
//   ballot counts and no atomics, and one wavefront sorts them in registers.
//   Histogram case (k > 256, or more than 256 keys at or above L: masses of
//   equal or nearly equal scores): bits shared by every key are skipped, one
//   histogram pass over the next 11 bits locates the bin of the k-th key,
//   and every key in it or above is compacted and sorted; a second 11-bit
//   histogram narrows a crowded bin, and exact radix passes of 8 bits handle
//   what would still overflow LDS (the keys above the threshold T plus the
//   lowest-index keys equal to T are taken). Sorting runs in registers inside
//   one wavefront for up to 256 candidates, in LDS across the workgroup
//   otherwise.
//
// Rows cut into several segments take two (or more) launches: each segment
// yields its top k, then the next round selects the top k of those
// candidates through an index map. Segments are contiguous index ranges and
// the composite carries the global index, so the tie rule holds across
// segments. A segment shorter than k pads its list with -inf entries (index
// 0x7FFFFFFF), which never outrank a real score.
#include <algorithm>

#include "kgq_internal.hpp"

namespace kgq {


__device__ __forceinline__ float key_score(uint32_t key)
{
    return __uint_as_float((key & 0x80000000u) ? (key & 0x7FFFFFFFu) : ~key);
}

// Key of segment position j * NT + tid through the segment's buffer resource;
// positions past the end give the padding key 0.
template <int NT>
__device__ __forceinline__ uint32_t fetch_key(__amdgpu_buffer_rsrc_t rsrc, int tid, int j, int n)
{
    const uint32_t u = __builtin_amdgcn_raw_buffer_load_b32(rsrc, tid * 4, j * NT * 4, 0);
    return (tid < n - j * NT) ? max(score_key(__uint_as_float(u)), 1u) : 0u;
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
// write out the first k. Entry p is the composite of sel_key[p] and sel_idx[p].
template <int E>
__device__ __forceinline__ void bitonic_wave(const uint32_t* sel_key, const uint32_t* sel_idx, int n, int k,
                                             int64_t orow, int lane, const TopkArgs& a)
{
    constexpr int P = 64 * E;
    uint64_t v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int p = e * 64 + lane;
        v[e] = p < n ? (((uint64_t)sel_key[p] << 32) | sel_idx[p]) : 0ull;
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

// Sort 256 keys descending inside one wavefront: lane l holds positions
// e * 64 + l in v[e] (the network of bitonic_wave, on 32-bit keys).
__device__ __forceinline__ void sort256_desc(uint32_t (&v)[4], int lane)
{
#pragma unroll
    for (int size = 2; size <= 256; size <<= 1) {
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            if (stride >= 64) {
                const int es = stride >> 6;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int f = e ^ es;
                    if (f > e) {
                        const bool desc = ((e * 64 + lane) & size) == 0;
                        const uint32_t a0 = v[e], a1 = v[f];
                        const bool sw = desc ? (a0 < a1) : (a0 > a1);
                        v[e] = sw ? a1 : a0;
                        v[f] = sw ? a0 : a1;
                    }
                }
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t w = __shfl_xor(v[e], stride, 64);
                    const bool desc = ((e * 64 + lane) & size) == 0;
                    const bool lower = (lane & stride) == 0;
                    v[e] = (desc == lower) ? max(v[e], w) : min(v[e], w);
                }
            }
        }
    }
}

// Exclusive prefix, in place, over the KPT * NT / 64 per-(step, wavefront)
// counts in (step, wavefront) order, which is element index order. Run by the
// whole workgroup; only wavefront 0 works.
template <int NT, int KPT>
__device__ __forceinline__ void block_exclusive_prefix(int* cnt, int tid)
{
    if (tid >= 64) return;
    constexpr int NC = KPT * (NT / 64);
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

// At 64 keys per thread the kernel needs 99 VGPRs, three above the budget
// of five wavefronts per SIMD; asking for five (a few values spill to
// scratch) keeps five rows in flight per compute unit instead of four:
// measured 110 -> 100 us over 4,608 rows of 14,505 scores.
template <int NT, int KPT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(5))) void k_topk(TopkArgs a)
{
    constexpr int TK_THREADS = NT;
    constexpr int TK_WAVES = NT / 64;
    // The selected entries are kept as separate 32-bit key and inverted-index
    // arrays (a key never has to sit in the high half of a 64-bit register
    // pair, which would cost a second register per key). The LDS sort for
    // long candidate lists builds 64-bit composites in the histogram's
    // storage, which is free by then.
    __shared__ uint64_t srt[kMaxK];
    __shared__ uint32_t sel_key[kMaxK], sel_idx[kMaxK];
    uint32_t* hist = reinterpret_cast<uint32_t*>(srt);    // 2048 bins
    __shared__ int sh_bin, sh_rem, sh_binc;
    __shared__ uint32_t sh_or[TK_WAVES], sh_and[TK_WAVES];   // per-wavefront max / min key
    __shared__ int cnt_gt[KPT * TK_WAVES], cnt_eq[KPT * TK_WAVES];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    // one-dimensional grid, row-major over (row, segment): gridDim.y is too
    // small for large batches
    const int64_t nseg = (a.N + a.seg_len - 1) / a.seg_len;
    const int64_t row = (int64_t)blockIdx.x / nseg;
    const int64_t seg = (int64_t)blockIdx.x - row * nseg;
    const int64_t seg0 = seg * a.seg_len;                      // first element of this segment
    int64_t n = a.N - seg0;
    if (n > a.seg_len) n = a.seg_len;
    const float* __restrict__ sr = a.scores + row * a.ld + seg0;
    const int32_t* __restrict__ ir = a.in_idx ? a.in_idx + row * a.ld + seg0 : nullptr;
    const int k = a.k < n ? a.k : (int)n;   // a segment shorter than k yields all of it

    // Positions past the segment's end hold key 0; real keys are at least 1
    // (only the one NaN pattern whose key would be 0 moves up to 1), so no
    // per-element validity mask has to stay live through the passes below.
    // Buffer loads against a resource sized to the segment: every position
    // loads (past the end the hardware returns 0), so the loads carry no
    // branch, share one address register and are all in flight together.
    const int nn = (int)n;
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(sr), (short)0, nn * 4, 0x00020000);
    uint32_t keys[KPT];
#pragma unroll
    for (int j = 0; j < KPT; ++j)
        keys[j] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, tid * 4, j * TK_THREADS * 4, 0);
    // The empty asm uses every loaded value unconditionally, so the compiler
    // cannot move a load into the validity branch below (which would make
    // the loads wait for each other one by one).
#pragma unroll
    for (int j = 0; j < KPT; ++j) asm volatile("" : "+v"(keys[j]));
#pragma unroll
    for (int j = 0; j < KPT; ++j)
        keys[j] = (tid < nn - j * TK_THREADS) ? max(score_key(__uint_as_float(keys[j])), 1u) : 0u;

    // Bits shared by every key: the keys' common leading bits are those of the
    // smallest and the largest key. Padding (0) drops out of the maximum, and
    // of the minimum taken over key - 1 (where it wraps to the top).
    {
        uint32_t mx = 0u, mn1 = 0xFFFFFFFFu;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            mx = max(mx, keys[j]);
            mn1 = min(mn1, keys[j] - 1u);
        }
        hist[tid] = mx;    // this thread's largest key (0: no key), for the threshold below
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            mx = max(mx, (uint32_t)__shfl_xor(mx, off, 64));
            mn1 = min(mn1, (uint32_t)__shfl_xor(mn1, off, 64));
        }
        if (lane == 0) { sh_or[wave] = mx; sh_and[wave] = mn1 + 1u; }
    }
    __syncthreads();
    uint32_t kmax = 0u, kmin = 0xFFFFFFFFu;
#pragma unroll
    for (int w = 0; w < TK_WAVES; ++w) { kmax = max(kmax, sh_or[w]); kmin = min(kmin, sh_and[w]); }
    const uint32_t diff = kmax ^ kmin;                 // zero iff all keys are equal
    int top = diff ? 31 - __clz(diff) : -1;            // highest differing bit

    // bits above `top` are common to all keys: they start the prefix
    uint32_t pmask = diff ? ~(0xFFFFFFFFu >> (31 - top)) : 0xFFFFFFFFu;
    uint32_t prefix = kmax & pmask;

    // Bin of the need-th key from the top in hist[0 .. 2047] (run by wavefront
    // 0; need is at least 1 and at most the histogram's total): sh_bin = that
    // bin, sh_rem = keys in it and above, sh_binc = keys in it.
    auto find_bin = [&](uint32_t need) {
        if (tid >= 64) return;
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
        if (above < need && need <= incl) {
            uint32_t cum = above;
            for (int t = 31; t >= 0; --t) {
                const uint32_t c = hist[32 * tid + t];
                if (need <= cum + c) {
                    sh_bin = 32 * tid + t;
                    sh_rem = (int)(cum + c);
                    sh_binc = (int)c;
                    break;
                }
                cum += c;
            }
        }
    };

    // --- threshold from the thread maxima --------------------------------
    // At least k threads hold a key (positions 0 .. n-1 are spread over the
    // threads and k <= n), and the k-th largest of their maxima, L, has k
    // distinct keys at or above it: L is at most the k-th largest key, so
    // every key of the top k is >= L. Typically only a few more than k keys
    // are (about 120 for k = 100 among 14,505 normal scores), so they are
    // compacted directly: no histogram, no atomics. More than 256 (masses of
    // equal scores at L) take the histogram passes below instead.
    int n_sel = -1;            // entries placed in sel_key[] / sel_idx[]
    if (k <= TK_THREADS && top >= 0) {
        if (tid < 64) {
            uint32_t v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = e * 64 + lane < TK_THREADS ? hist[e * 64 + lane] : 0u;
            sort256_desc(v, lane);
            const int p = k - 1, ep = p >> 6;
            const uint32_t sel = ep == 0 ? v[0] : ep == 1 ? v[1] : ep == 2 ? v[2] : v[3];
            const uint32_t L = __shfl(sel, p & 63, 64);
            if (lane == 0) sh_bin = (int)L;
        }
        __syncthreads();
        const uint32_t L = max((uint32_t)sh_bin, 1u);
        int wc = 0;
#pragma unroll
        for (int j = 0; j < KPT; ++j) wc += __popcll(__ballot(keys[j] >= L));
        if (lane == 0) cnt_gt[wave] = wc;
        __syncthreads();
        int base = 0, total = 0;
#pragma unroll
        for (int w = 0; w < TK_WAVES; ++w) {
            base += w < wave ? cnt_gt[w] : 0;
            total += cnt_gt[w];
        }
        if (total <= 256) {
            n_sel = total;
            const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
            for (int j = 0; j < KPT; ++j) {
                const bool f = keys[j] >= L;
                const uint64_t bc = __ballot(f);
                if (f) {
                    const int i = j * TK_THREADS + tid;
                    const int slot = base + __popcll(bc & lt);
                    sel_key[slot] = keys[j];
                    sel_idx[slot] = 0xFFFFFFFFu - (uint32_t)(ir ? ir[i] : (int32_t)seg0 + i);
                }
                base += __popcll(bc);
            }
        }
        __syncthreads();       // hist, sh_bin and cnt_gt are reused below
    }
    if (n_sel < 0) {
    // --- one wide histogram pass: the bin of the k-th key -------------------
    // digit = bits [wlo, top], at most 11 bits
    const int wlo = top >= 10 ? top - 10 : 0;
    const uint32_t wmask = top >= 0 ? ((2u << (top - wlo)) - 1u) : 0u;
    int n_cand = (int)n;       // candidates: keys whose digit is >= the k-th key's digit
    uint32_t dmin = 0;         // smallest candidate digit
    // every key >= thr is a candidate (thr >= 1 keeps the padding out)
    uint32_t thr = max(prefix, 1u);
    if (top >= 0) {
        for (int b = tid; b < 2048; b += TK_THREADS) hist[b] = 0;
        __syncthreads();
#pragma unroll
        for (int j = 0; j < KPT; ++j) atomicAdd(&hist[(keys[j] >> wlo) & wmask], 1u);
        __syncthreads();
        // the padding landed in bin 0 (thread 0 is in the wavefront that reads
        // the histogram next, and one wavefront's LDS accesses stay in order)
        if (tid == 0) hist[0] -= (uint32_t)(KPT * TK_THREADS - nn);
        find_bin((uint32_t)k);
        __syncthreads();
        dmin = (uint32_t)sh_bin;
        n_cand = sh_rem;
        // All keys share the bits above `top`, so digit >= dmin is the same
        // as key >= (common bits, dmin, zeros).
        thr = max(prefix | (dmin << wlo), 1u);
        if (n_cand > 256 && wlo > 0) {
            // The k-th key's bin is crowded (scores spanning the sign or many
            // exponents make the top 11 bits coarse), so the candidates would
            // need the LDS sort (more than 256) or the radix passes (more than
            // kMaxK): a second histogram over the next lower bits of that
            // bin's keys, still in registers, finds the sub-bin of the key the
            // bin must contribute.
            const int above = n_cand - sh_binc;                   // keys in higher bins
            const int wlo2 = wlo >= 11 ? wlo - 11 : 0;
            const uint32_t wmask2 = (1u << (wlo - wlo2)) - 1u;
            for (int b = tid; b < 2048; b += TK_THREADS) hist[b] = 0;
            __syncthreads();
#pragma unroll
            for (int j = 0; j < KPT; ++j) {
                // (the empty asm keeps the compiler from hoisting this pass's
                // per-key tests above the first pass, where they would stay
                // live in registers beside the keys)
                uint32_t kj = keys[j];
                asm volatile("" : "+v"(kj));
                if (kj != 0u && ((kj >> wlo) & wmask) == dmin) atomicAdd(&hist[(kj >> wlo2) & wmask2], 1u);
            }
            __syncthreads();
            find_bin((uint32_t)(k - above));
            __syncthreads();
            n_cand = above + sh_rem;
            thr = max(prefix | (dmin << wlo) | ((uint32_t)sh_bin << wlo2), 1u);
        }
    }

    if (n_cand <= kMaxK) {
        // --- candidates fit: take every key >= thr ---------------------------
        n_sel = n_cand;
        // The sort below orders candidates completely by (key, index), so
        // their slots only need to be distinct: each wavefront takes a range
        // sized by its candidate count and fills it in step order.
        int wc = 0;
#pragma unroll
        for (int j = 0; j < KPT; ++j) wc += __popcll(__ballot(keys[j] >= thr));
        if (lane == 0) cnt_gt[wave] = wc;
        __syncthreads();
        int base = 0;
        for (int w = 0; w < wave; ++w) base += cnt_gt[w];
        const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const bool f = keys[j] >= thr;
            const uint64_t bc = __ballot(f);
            if (f) {
                const int i = j * TK_THREADS + tid;
                const int slot = base + __popcll(bc & lt);
                if (slot < kMaxK) {
                    sel_key[slot] = keys[j];
                    sel_idx[slot] = 0xFFFFFFFFu - (uint32_t)(ir ? ir[i] : (int32_t)seg0 + i);
                }
            }
            base += __popcll(bc);
        }
    } else {
        // --- too many candidates: exact radix passes find T ------------------
        // (rare: very many equal or nearly equal scores). Keys are fetched
        // again from memory in loops that are not unrolled, so this path adds
        // no register pressure to the common one above.
        int rem = k;
        for (int lo = top - 7; top >= 0; lo -= 8) {
            // digit = bits [max(lo, 0), top] of the key
            const int shift = lo > 0 ? lo : 0;
            const int width = top - shift + 1;
            const uint32_t dmask = (1u << width) - 1u;      // width <= 8
            for (int b = tid; b < 256; b += TK_THREADS) hist[b] = 0;
            __syncthreads();
#pragma unroll 1
            for (int j = 0; j < KPT; ++j) {
                const uint32_t key = fetch_key<NT>(rsrc, tid, j, nn);
                const bool act = key != 0u && (key & pmask) == prefix;
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
#pragma unroll 1
        for (int j = 0; j < KPT; ++j) {
            const uint32_t key = fetch_key<NT>(rsrc, tid, j, nn);
            const uint64_t bg = __ballot(key > T);
            const uint64_t be = __ballot(key == T);
            if (lane == 0) {
                cnt_gt[j * TK_WAVES + wave] = __popcll(bg);
                cnt_eq[j * TK_WAVES + wave] = __popcll(be);
            }
        }
        __syncthreads();
        block_exclusive_prefix<NT, KPT>(cnt_gt, tid);
        __syncthreads();
        block_exclusive_prefix<NT, KPT>(cnt_eq, tid);
        __syncthreads();
        const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll 1
        for (int j = 0; j < KPT; ++j) {
            const int i = j * TK_THREADS + tid;
            const uint32_t key = fetch_key<NT>(rsrc, tid, j, nn);
            const bool fg = key > T, fe = key == T;
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
            if (slot >= 0 && slot < k) {
                sel_key[slot] = key;
                sel_idx[slot] = 0xFFFFFFFFu - (uint32_t)(ir ? ir[i] : (int32_t)seg0 + i);
            }
        }
    }
    }   // histogram passes
    __syncthreads();

    // order the n_sel selected entries and write the first k; a short
    // segment pads its list to a.k entries with -inf
    const int64_t orow = row * a.out_rows_per_row + seg;
    for (int p = k + tid; p < a.k; p += TK_THREADS) {
        a.out_idx[orow * a.out_ld + p] = 0x7FFFFFFF;
        a.out_score[orow * a.out_ld + p] = -__builtin_inff();
    }
    if (n_sel <= 256) {
        if (tid < 64) {
            if (n_sel <= 64) bitonic_wave<1>(sel_key, sel_idx, n_sel, k, orow, lane, a);
            else if (n_sel <= 128) bitonic_wave<2>(sel_key, sel_idx, n_sel, k, orow, lane, a);
            else bitonic_wave<4>(sel_key, sel_idx, n_sel, k, orow, lane, a);
        }
    } else {
        int P = 512;
        while (P < n_sel) P <<= 1;             // 512 or 1024
        for (int p = tid; p < P; p += TK_THREADS)
            srt[p] = p < n_sel ? (((uint64_t)sel_key[p] << 32) | sel_idx[p]) : 0ull;
        for (int size = 2; size <= P; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                __syncthreads();
                // P / 2 compare-exchange pairs per stage; pair t is (p, p + stride)
                for (int t = tid; t < P / 2; t += TK_THREADS) {
                    const int p = ((t & ~(stride - 1)) << 1) | (t & (stride - 1));
                    const int q = p + stride;
                    const bool desc = (p & size) == 0;
                    const uint64_t a0 = srt[p], a1 = srt[q];
                    if (desc ? (a0 < a1) : (a0 > a1)) { srt[p] = a1; srt[q] = a0; }
                }
            }
        }
        __syncthreads();
        for (int p = tid; p < k; p += TK_THREADS) store_one(a, orow, p, srt[p]);
    }
}

// ---------------------------------------------------------------------------
// Streaming selection (k <= kStreamK): one wavefront per segment, no
// workgroup barriers. The wavefront reads its segment once, four coalesced
// 256-byte loads per step, with several steps in flight, and compares each
// score with a running threshold score tf. Scores not below it are appended,
// as (raw bits, element index) pairs, to the wavefront's candidate buffer in
// LDS: ballot ranges, no atomics, no branches, a few instructions per 64
// scores. When fewer free slots remain than one group of steps could fill,
// the buffer is pruned: its entries become order-preserving keys, and a radix
// select over them (one bit at a time from their highest differing bit,
// counting with ballots) raises the threshold T = (key, inverted index) to a
// bound that at least k of them still reach and at most max(k, kStreamKeep)
// do; masses of equal keys are narrowed by index, which makes T exact. T
// never exceeds the k-th largest (key, index) seen so far, so no element of
// the top k is dropped; the score compare only admits a superset (ties with
// T, NaN), which the prunes sort out. At the end the buffer is pruned to at
// most 64, 128 or 256 entries (by k) and sorted inside the wavefront.
// Over a score matrix whose scorer also wrote chunk keys (the largest key of
// every kKeyChunk scores of a row), the first round reads only the chunks
// whose key reaches the k-th largest chunk key (k_topk_listed).
// ---------------------------------------------------------------------------
constexpr int kStreamK = 256;        // largest k on the streaming path
constexpr int kPruneChunks = 1024;   // chunk keys per segment on the listed stream (65,536 scores)
constexpr int kStreamKeep = 128;     // a prune leaves at most max(k, this) entries
constexpr int kStreamWaves = 2;      // wavefronts (segments) per workgroup
constexpr int kStreamGroup = 1;      // load steps per group
constexpr int kStreamDepth = 6;      // groups held in registers (depth - 1 in flight)
constexpr int kStreamCap = 768;      // candidate buffer entries per wavefront

// Smallest buffer (entries per wavefront) for H-step groups: one group of
// appends on top of what a prune leaves (at most kStreamK, plus fewer than k
// copies of the padding pair in later rounds, whose lists hold the padding
// of short segments).
template <int H, bool IDX>
constexpr int stream_min_cap() { return kStreamK + (IDX ? kStreamK : 0) + 256 * H; }

__device__ __forceinline__ uint64_t ballot64(bool f) { return __builtin_amdgcn_ballot_w64(f); }

__device__ __forceinline__ int lanes_below(uint64_t m)
{
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Number of keys at or above x >= 1 (empty slots hold key 0).
template <int E>
__device__ __forceinline__ int stream_count_ge(const uint32_t (&key)[E], uint32_t x)
{
    int c = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) c += __popcll(ballot64(key[e] >= x));
    return c;
}

// Raise the threshold (tk, ti) so that at least k and at most `keep` of the
// cnt buffered entries reach it (cnt > keep >= k). key[e] holds the key of
// entry e * 64 + lane (0 past cnt); inv_of(e) gives its inverted index.
template <int E, bool TIES = true, typename Inv>
__device__ __forceinline__ void stream_threshold(const uint32_t (&key)[E], Inv inv_of, int cnt, int k, int keep,
                                                 uint32_t& tk, uint32_t& ti)
{
    // common leading bits of the buffered keys (valid keys are >= 1; empty
    // slots drop out of the maximum, and out of the minimum over key - 1)
    uint32_t mx = 0u, mn1 = 0xFFFFFFFFu;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        mx = max(mx, key[e]);
        mn1 = min(mn1, key[e] - 1u);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        mx = max(mx, (uint32_t)__shfl_xor(mx, off, 64));
        mn1 = min(mn1, (uint32_t)__shfl_xor(mn1, off, 64));
    }
    // (the reduced values are uniform: keep them, and all that follows from
    // them, in scalar registers)
    mx = __builtin_amdgcn_readfirstlane(mx);
    mn1 = __builtin_amdgcn_readfirstlane(mn1);
    const uint32_t diff = mx ^ (mn1 + 1u);
    const int top = diff ? 31 - __clz(diff) : -1;
    // p: the k-th largest key with the bits below the current one cleared
    // (every key >= p until the loop moves it); np = keys >= p
    uint32_t p = diff ? mx & ~((2u << top) - 1u) : mx;
    int np = cnt;
    for (int b = top; b >= 0 && np > keep; --b) {
        const uint32_t c = p | (1u << b);
        const int n = stream_count_ge(key, c);
        if (n >= k) { p = c; np = n; }
    }
    uint32_t q = 0u;
    if (TIES && np > keep) {
        // p is the k-th largest key and too many keys equal it: select among
        // those by inverted index, down to k entries (distinct indices)
        const int above = p == 0xFFFFFFFFu ? 0 : stream_count_ge(key, p + 1u);
        const int need = k - above;
        int nq = np - above;
        for (int b = 31; b >= 0 && above + nq > keep; --b) {
            const uint32_t c = q | (1u << b);
            int n = 0;
#pragma unroll
            for (int e = 0; e < E; ++e) n += __popcll(ballot64(key[e] == p && inv_of(e) >= c));
            if (n >= need) { q = c; nq = n; }
        }
    }
    // the threshold only rises
    if (p > tk || (p == tk && q > ti)) { tk = p; ti = q; }
}

// Prune while the stream runs (its loads in flight hold registers): keys in
// registers, indices read from LDS. Entries reaching the new threshold are
// compacted to the front, in place, as (score bits, index). Copies of one
// (key, index) pair come only from the padding of short segments' lists
// (fewer than k per row), so at most keep + k - 1 entries remain.
template <int E>
__device__ __forceinline__ void stream_prune(uint2* buf, int& cnt, uint32_t& tk, uint32_t& ti, int k, int keep,
                                             int lane)
{
    uint32_t key[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int p = e * 64 + lane;
        key[e] = p < cnt ? max(score_key(__uint_as_float(buf[p].x)), 1u) : 0u;
    }
    stream_threshold<E>(key, [&](int e) { return ~buf[e * 64 + lane].y; }, cnt, k, keep, tk, ti);
    // In place: chunk e's entries move to slots below (e + 1) * 64, which
    // hold entries of chunks up to e, already read (a wavefront's LDS
    // accesses complete in order).
    int base = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int p = e * 64 + lane;
        const uint32_t idx = buf[p].y;
        const bool f = p < cnt && (key[e] > tk || (key[e] == tk && ~idx >= ti));
        const uint64_t bc = ballot64(f);
        if (f) buf[base + lanes_below(bc)] = make_uint2(__float_as_uint(key_score(key[e])), idx);
        base += __popcll(bc);
    }
    cnt = base;
}

// Final prune (nothing in flight; cnt <= 64 E): keys and indices in
// registers. Keeps at most `keep` entries, those above the threshold and
// then copies of the threshold pair (identical, so any copies do), and
// writes them as (key, inverted index) for the sort.
template <int E>
__device__ __forceinline__ void stream_prune_final(uint2* buf, int& cnt, uint32_t& tk, uint32_t& ti, int k, int keep,
                                                   int lane)
{
    uint32_t key[E], inv[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int p = e * 64 + lane;
        const uint2 b = p < cnt ? buf[p] : make_uint2(0u, 0xFFFFFFFFu);
        key[e] = p < cnt ? max(score_key(__uint_as_float(b.x)), 1u) : 0u;
        inv[e] = ~b.y;
    }
    if (cnt > keep) stream_threshold<E>(key, [&](int e) { return inv[e]; }, cnt, k, keep, tk, ti);
    int base = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const bool f = (e * 64 + lane < cnt) && (key[e] > tk || (key[e] == tk && inv[e] > ti));
        const uint64_t bc = ballot64(f);
        if (f) buf[base + lanes_below(bc)] = make_uint2(key[e], inv[e]);
        base += __popcll(bc);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const bool f = (e * 64 + lane < cnt) && key[e] == tk && inv[e] == ti;
        const uint64_t bc = ballot64(f);
        const int slot = base + lanes_below(bc);
        if (f && slot < keep) buf[slot] = make_uint2(key[e], inv[e]);
        base = min(base + __popcll(bc), keep);
    }
    cnt = base;
}

// Sort the n (key, inverted index) entries of buf inside one wavefront and
// write the first k (the network of bitonic_wave).
template <int E>
__device__ __forceinline__ void stream_sort(const uint2* buf, int n, int k, int64_t orow, int lane, const TopkArgs& a)
{
    constexpr int P = 64 * E;
    uint64_t v[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int p = e * 64 + lane;
        v[e] = p < n ? (((uint64_t)buf[p].x << 32) | buf[p].y) : 0ull;
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
                    const bool lower = (lane & stride) == 0;
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

// State of one wavefront's stream.
struct StreamState {
    uint2* buf;                        // (score bits, element index) pairs
    int cnt;                           // buffered entries (wave-uniform)
    uint32_t tk, ti;                   // threshold; (0, 0): everything passes
    float tf;                          // score of tk (NaN: every score passes)
};

// Append the scores of step s not below tf (NaN scores included; all of
// them while tf is NaN). y: the elements' indices when IDX, else position
// + seg0. CHECK: the step reaches past the segment's end (positions past it
// read as 0 and are masked). No memory is read here: a load would wait for
// every load in flight before it (the vector memory counter is in order).
template <bool IDX, bool CHECK>
__device__ __forceinline__ void stream_step(StreamState& st, const float (&x)[4], const int32_t (&y)[4], int s, int nn,
                                            int32_t seg0, int dummy, int lane)
{
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int i = s * 256 + c * 64 + lane;
        const bool f = (!CHECK || i < nn) && !(x[c] < st.tf);
        const uint64_t bc = ballot64(f);
        if (bc != 0ull) {
            // every lane writes: those not appending to a slot of their own
            // past the buffer (no exec-mask changes on this path)
            const int slot = f ? st.cnt + lanes_below(bc) : dummy + lane;
            st.buf[slot] = make_uint2(__float_as_uint(x[c]), IDX ? (uint32_t)y[c] : (uint32_t)(seg0 + i));
            st.cnt += __popcll(bc);
        }
    }
}

// Loads of the H steps from s0 (positions past the segment read as 0), and
// of the elements' indices when IDX.
template <int H, bool IDX>
__device__ __forceinline__ void stream_load(float (&v)[H][4], int32_t (&w)[H][4], __amdgpu_buffer_rsrc_t rsrc,
                                            __amdgpu_buffer_rsrc_t irsrc, int s0, int lane)
{
#pragma unroll
    for (int h = 0; h < H; ++h)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int off = lane * 4 + ((s0 + h) * 256 + c * 64) * 4;
            v[h][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsrc, off, 0, 0));
            if (IDX) w[h][c] = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(irsrc, off, 0, 0);
        }
}

// One group of H steps (first step s0) held in v / w: room for all of them
// first, then each step's appends (checked only where the segment ends).
template <int H, bool IDX, int CAP, int KEEP>
__device__ __forceinline__ void stream_group(StreamState& st, const float (&v)[H][4], const int32_t (&w)[H][4], int s0,
                                             int nsteps, int nn, int32_t seg0, int k, int lane)
{
    static_assert(CAP % 64 == 0, "the dummy slots follow the buffer");
    if (st.cnt > CAP - 256 * H) {
        stream_prune<CAP / 64>(st.buf, st.cnt, st.tk, st.ti, k, k > KEEP ? k : KEEP, lane);
        st.tf = key_score(st.tk);
    }
#pragma unroll
    for (int h = 0; h < H; ++h) {
        const int s = s0 + h;
        if ((s + 1) * 256 <= nn) stream_step<IDX, false>(st, v[h], w[h], s, nn, seg0, CAP, lane);
        else if (s < nsteps) stream_step<IDX, true>(st, v[h], w[h], s, nn, seg0, CAP, lane);
    }
}

// Final prune of the buffer to at most 64, 128 or 256 entries (by k), which
// also turns them into keys, then the sort, written to output row orow (and
// padding past k).
template <int CAP>
__device__ __forceinline__ void stream_finish(StreamState& st, int k, int64_t orow, int lane, const TopkArgs& a)
{
    const int fin = k <= 64 ? 64 : k <= 128 ? 128 : 256;     // sort size
    if (st.cnt <= 256) stream_prune_final<4>(st.buf, st.cnt, st.tk, st.ti, k, fin, lane);
    else if (st.cnt <= 512) stream_prune_final<8>(st.buf, st.cnt, st.tk, st.ti, k, fin, lane);
    else stream_prune_final<CAP / 64>(st.buf, st.cnt, st.tk, st.ti, k, fin, lane);
    for (int p = k + lane; p < a.k; p += 64) {
        a.out_idx[orow * a.out_ld + p] = 0x7FFFFFFF;
        a.out_score[orow * a.out_ld + p] = -__builtin_inff();
    }
    if (st.cnt <= 64) stream_sort<1>(st.buf, st.cnt, k, orow, lane, a);
    else if (st.cnt <= 128) stream_sort<2>(st.buf, st.cnt, k, orow, lane, a);
    else stream_sort<4>(st.buf, st.cnt, k, orow, lane, a);
}

// H: steps per group; D groups held in registers, D - 1 of them in flight
// while one is compared. IDX: element indices come from in_idx (later
// rounds).
template <int H, int D, bool IDX, int CAP, int KEEP, int W>
__global__ __launch_bounds__(64 * W) void k_topk_stream(TopkArgs a)
{
    static_assert(CAP >= stream_min_cap<H, IDX>() && CAP % 64 == 0 && KEEP <= kStreamK, "stream buffer too small");
    __shared__ uint2 s_buf[W][CAP + 64];     // + 64 slots for the lanes that append nothing
    const int lane = threadIdx.x & 63;
    // (readfirstlane: the wavefront index is uniform, so the segment's
    // addresses and its buffer resource stay in scalar registers)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nseg = (a.N + a.seg_len - 1) / a.seg_len;
    const int64_t unit = (int64_t)blockIdx.x * W + wave;   // (row, segment), row-major
    if (unit >= nseg * a.n_rows) return;
    const int64_t row = unit / nseg;
    const int64_t seg = unit - row * nseg;
    const int64_t seg0 = seg * a.seg_len;
    int64_t n64 = a.N - seg0;
    if (n64 > a.seg_len) n64 = a.seg_len;
    const int nn = (int)n64;
    const int k = a.k < nn ? a.k : nn;
    StreamState st{s_buf[wave], 0, 0u, 0u, key_score(0u)};

    // Step s covers positions s * 256 + c * 64 + lane, c = 0 .. 3. All offsets
    // go in the per-lane offset, which the buffer range check covers: loads
    // past the segment's end return 0 (and are masked in the append).
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.scores + row * a.ld + seg0), (short)0, nn * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t irsrc = __builtin_amdgcn_make_buffer_rsrc(
        IDX ? const_cast<int32_t*>(a.in_idx + row * a.ld + seg0) : nullptr, (short)0, IDX ? nn * 4 : 0, 0x00020000);
    const int nsteps = (nn + 255) >> 8;
    float v[D][H][4];
    int32_t w[D][H][4];
    // (the scheduling barriers keep the groups' loads in order, so that
    // waiting for the oldest group leaves the others in flight)
#pragma unroll
    for (int g = 0; g < D; ++g) {
        stream_load<H, IDX>(v[g], w[g], rsrc, irsrc, g * H, lane);
        __builtin_amdgcn_sched_barrier(0);
    }
    // Initial threshold: each (lane, column) takes the largest of its scores
    // in the first D * H steps, which are all inside the segment and still in
    // registers, and the threshold is the k-th largest of those 256 maxima
    // (radix select). Each maximum is a distinct element, so k elements reach
    // it: it bounds the k-th largest of the segment from below. From there on
    // few scores reach the threshold and the stream rarely prunes.
    if (nn >= D * H * 256) {
        uint32_t key[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float m = v[0][0][c];
#pragma unroll
            for (int t = 1; t < D * H; ++t) m = fmaxf(m, v[t / H][t % H][c]);
            key[c] = max(score_key(m), 1u);
        }
        stream_threshold<4, false>(key, [](int) { return 0u; }, 256, k, k, st.tk, st.ti);
        st.tf = key_score(st.tk);
    }
    // Oldest-first issue would let the first wavefronts of a compute unit
    // run ahead and leave the last ones to finish alone, with too few loads
    // in flight to keep memory busy. Instead each wavefront lowers its
    // priority as it advances (3 .. 0 by quarters of its segment), so the
    // ones behind issue first and all finish together.
    const int q1 = nsteps >> 2, q2 = nsteps >> 1, q3 = (3 * nsteps) >> 2;
    __builtin_amdgcn_s_setprio(3);
    for (int s0 = 0; s0 < nsteps; s0 += D * H) {
        if (s0 >= q3) __builtin_amdgcn_s_setprio(0);
        else if (s0 >= q2) __builtin_amdgcn_s_setprio(1);
        else if (s0 >= q1) __builtin_amdgcn_s_setprio(2);
#pragma unroll
        for (int g = 0; g < D; ++g) {
            stream_group<H, IDX, CAP, KEEP>(st, v[g], w[g], s0 + g * H, nsteps, nn, (int32_t)seg0, k, lane);
            __builtin_amdgcn_sched_barrier(0);
            stream_load<H, IDX>(v[g], w[g], rsrc, irsrc, s0 + (g + D) * H, lane);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    __builtin_amdgcn_s_setprio(0);
    // Every score of the segment reached the threshold or is below the k-th
    // largest, so the buffer holds the top k (all nn when nn <= k).
    stream_finish<CAP>(st, k, row * a.out_rows_per_row + seg, lane, a);
}

// Pruned first round over a score matrix with chunk keys (at most
// kPruneChunks per segment). The threshold starts at the k-th largest chunk
// key of the segment (the chunks are disjoint, so at least k elements reach
// it), the chunks whose key reaches it are listed in LDS, and the wavefront
// streams that list alone, G chunks (one load each) per group, D groups in
// flight, appending and pruning as the full stream does. A chunk left out
// holds only elements below the threshold, none of them among the k largest,
// so the result is the full stream's. At most about k chunks of a row hold
// an element of its top k: the rest of the row is never read.
template <int E>
__device__ __forceinline__ int list_chunks(const uint32_t* src, uint32_t* list, int nchunk, int k, StreamState& st,
                                           int lane)
{
    uint32_t key[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = e * 64 + lane;
        key[e] = j < nchunk ? src[j] : 0u;
    }
    if (nchunk > k) {
        stream_threshold<E, false>(key, [](int) { return 0u; }, nchunk, k, k, st.tk, st.ti);
        st.tf = key_score(st.tk);
    }
    int n = 0;
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int j = e * 64 + lane;
        const bool f = j < nchunk && key[e] >= st.tk;
        const uint64_t bc = ballot64(f);
        if (f) list[n + lanes_below(bc)] = (uint32_t)j;
        n += __popcll(bc);
    }
    return n;
}

template <int G, int D, int CAP, int KEEP, int W>
__global__ __launch_bounds__(64 * W) void k_topk_listed(TopkArgs a)
{
    static_assert(CAP >= kStreamK + 64 * G && CAP % 64 == 0 && KEEP <= kStreamK && G == 4, "listed stream shape");
    __shared__ uint2 s_buf[W][CAP + 64];     // + 64 slots for the lanes that append nothing
    __shared__ __align__(16) uint32_t s_list[W][kPruneChunks];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nseg = (a.N + a.seg_len - 1) / a.seg_len;
    const int64_t unit = (int64_t)blockIdx.x * W + wave;   // (row, segment), row-major
    if (unit >= nseg * a.n_rows) return;
    const int64_t row = unit / nseg;
    const int64_t seg = unit - row * nseg;
    const int64_t seg0 = seg * a.seg_len;                    // a multiple of 256
    int64_t n64 = a.N - seg0;
    if (n64 > a.seg_len) n64 = a.seg_len;
    const int nn = (int)n64;
    const int k = a.k < nn ? a.k : nn;
    StreamState st{s_buf[wave], 0, 0u, 0u, key_score(0u)};
    uint32_t* list = s_list[wave];
    const uint32_t* src = a.chunk_key + row * a.key_ld + seg0 / kKeyChunk;
    const int nchunk = (nn + kKeyChunk - 1) / kKeyChunk;
    int nlist;
    if (nchunk <= 256) nlist = list_chunks<4>(src, list, nchunk, k, st, lane);
    else if (nchunk <= 512) nlist = list_chunks<8>(src, list, nchunk, k, st, lane);
    else nlist = list_chunks<kPruneChunks / 64>(src, list, nchunk, k, st, lane);
    nlist = __builtin_amdgcn_readfirstlane(nlist);

    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(a.scores + row * a.ld + seg0), (short)0, nn * 4, 0x00020000);
    // Group q holds list entries q * G .. q * G + G - 1; an entry past the
    // list (chunk -1) loads at offset nn * 4, past the segment: the buffer
    // range check returns 0 without a memory access, and nothing is appended.
    const int ngroups = (nlist + G - 1) / G;
    float v[D][G];
    int ch[D][G];
    auto issue = [&](int g, int q) {
        int c4[G] = {-1, -1, -1, -1};
        if (q * G < nlist) {
            const uint4 l = *reinterpret_cast<const uint4*>(list + q * G);
            const int idx[G] = {(int)l.x, (int)l.y, (int)l.z, (int)l.w};
#pragma unroll
            for (int c = 0; c < G; ++c)
                c4[c] = q * G + c < nlist ? __builtin_amdgcn_readfirstlane(idx[c]) : -1;
        }
#pragma unroll
        for (int c = 0; c < G; ++c) {
            ch[g][c] = c4[c];
            const int off = c4[c] >= 0 ? (c4[c] * kKeyChunk + lane) * 4 : nn * 4;
            v[g][c] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsrc, off, 0, 0));
        }
    };
#pragma unroll
    for (int g = 0; g < D; ++g) {
        issue(g, g);
        __builtin_amdgcn_sched_barrier(0);
    }
    for (int q0 = 0; q0 < ngroups; q0 += D) {
#pragma unroll
        for (int g = 0; g < D; ++g) {
            if (st.cnt > CAP - 64 * G) {
                stream_prune<CAP / 64>(st.buf, st.cnt, st.tk, st.ti, k, k > KEEP ? k : KEEP, lane);
                st.tf = key_score(st.tk);
            }
#pragma unroll
            for (int c = 0; c < G; ++c) {
                if (ch[g][c] < 0) continue;
                const int pos = ch[g][c] * kKeyChunk + lane;
                const bool f = pos < nn && !(v[g][c] < st.tf);
                const uint64_t bc = ballot64(f);
                if (bc != 0ull) {
                    // every lane writes: those not appending to a slot of
                    // their own past the buffer
                    const int slot = f ? st.cnt + lanes_below(bc) : CAP + lane;
                    st.buf[slot] = make_uint2(__float_as_uint(v[g][c]), (uint32_t)(seg0 + pos));
                    st.cnt += __popcll(bc);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
            issue(g, q0 + g + D);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    stream_finish<CAP>(st, k, row * a.out_rows_per_row + seg, lane, a);
}

static void launch_segments(const TopkArgs& a, hipStream_t s)
{
    // (rows x segments fits 32 bits: the score buffer holds rows x N floats)
    dim3 grid((unsigned)(((a.N + a.seg_len - 1) / a.seg_len) * a.n_rows));
    // 256 threads with up to 64 keys each for long segments; short ones
    // (k-candidate lists of later rounds) use as many keys per thread as fit
    const int64_t per = (a.seg_len + 255) / 256;
    if (per <= 4) hipLaunchKernelGGL((k_topk<256, 4>), grid, dim3(256), 0, s, a);
    else if (per <= 8) hipLaunchKernelGGL((k_topk<256, 8>), grid, dim3(256), 0, s, a);
    else if (per <= 16) hipLaunchKernelGGL((k_topk<256, 16>), grid, dim3(256), 0, s, a);
    else if (per <= 32) hipLaunchKernelGGL((k_topk<256, 32>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_topk<256, 64>), grid, dim3(256), 0, s, a);
}

int64_t topk_scratch_elems(int64_t n_rows, int64_t N, int k)
{
    const int64_t segs = (N + kTopkSegment - 1) / kTopkSegment;
    return segs > 1 ? n_rows * segs * k : 0;
}

// Streaming rounds want at least kStreamMinUnits (row, segment) wavefronts
// (8 per compute unit): one per row when the rows alone give that many,
// however long the rows; otherwise long rows are split until they do, which
// costs one more (short) round over the per-segment lists. Below that the
// chip is mostly idle and the register-resident kernel, which issues a whole
// segment's loads at once, has the lower latency.
constexpr int64_t kStreamMinUnits = 2048;

static void launch_stream(const TopkArgs& a, hipStream_t s)
{
    const int64_t units = ((a.N + a.seg_len - 1) / a.seg_len) * a.n_rows;
    const dim3 grid((unsigned)((units + kStreamWaves - 1) / kStreamWaves));
    if (!a.in_idx && a.chunk_key && (a.seg_len + kKeyChunk - 1) / kKeyChunk <= kPruneChunks)
        hipLaunchKernelGGL((k_topk_listed<4, kStreamDepth, kStreamCap, kStreamKeep, kStreamWaves>), grid,
                           dim3(64 * kStreamWaves), 0, s, a);
    else if (a.in_idx)
        hipLaunchKernelGGL((k_topk_stream<kStreamGroup, kStreamDepth, true, kStreamCap, kStreamKeep, kStreamWaves>),
                           grid, dim3(64 * kStreamWaves), 0, s, a);
    else
        hipLaunchKernelGGL((k_topk_stream<kStreamGroup, kStreamDepth, false, kStreamCap, kStreamKeep, kStreamWaves>),
                           grid, dim3(64 * kStreamWaves), 0, s, a);
}

bool launch_topk(const TopkArgs& in, hipStream_t s)
{
    if (in.n_rows <= 0) return true;
    TopkArgs a = in;
    a.in_idx = nullptr;
    a.out_ld = a.k;
    a.out_rows_per_row = 1;
    // Rounds: each row is cut into segments, each segment yields its top k
    // laid out [row][segment][k] in a scratch buffer, and the next round
    // selects over those lists, until one segment holds a row. A streaming
    // round cuts rows only as far as kStreamMinUnits asks, a register-
    // resident round into segments of kTopkSegment; neither makes more
    // segments than the kTopkSegment cut, so each round's output fits the two
    // buffers of topk_scratch_elems() entries, used in turn.
    int ping = 0;
    for (;;) {
        const int64_t max_segs = (a.N + kTopkSegment - 1) / kTopkSegment;
        const int64_t fit = a.n_rows >= kStreamMinUnits
                                ? 1
                                : std::min<int64_t>(max_segs, (kStreamMinUnits + a.n_rows - 1) / a.n_rows);
        const bool stream = a.k <= kStreamK && a.n_rows * fit >= kStreamMinUnits;
        int64_t segs = stream ? fit : max_segs;
        int64_t seg_len = a.N;
        if (segs > 1) {
            seg_len = stream ? ((a.N + segs - 1) / segs + 255) / 256 * 256 : kTopkSegment;
            segs = (a.N + seg_len - 1) / seg_len;
        }
        if (segs == 1) {
            a.seg_len = a.N;
            if (stream) launch_stream(a, s);
            else launch_segments(a, s);
            return true;
        }
        // a round of several segments writes its lists to the scratch buffers
        if (!in.cand_idx[ping] || !in.cand_score[ping]) return false;
        TopkArgs r = a;
        r.seg_len = seg_len;
        r.out_idx = in.cand_idx[ping];
        r.out_score = in.cand_score[ping];
        r.out_ld = a.k;
        r.out_rows_per_row = (int)segs;
        if (stream) launch_stream(r, s);
        else launch_segments(r, s);
        a.scores = in.cand_score[ping];
        a.in_idx = in.cand_idx[ping];
        a.ld = segs * a.k;
        a.N = segs * a.k;
        ping ^= 1;
    }
}

}  // namespace kgq
