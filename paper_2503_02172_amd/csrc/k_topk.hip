// Top-k selection over each query's N entity scores (the ranking the paper
// evaluates with MRR, Experiments/Metrics). Order: score descending, equal
// scores by entity index ascending.
//
// One workgroup of NT threads (256, or 1024 for the short candidate lists of
// later rounds) selects the top k of one segment of at most 16 Ki scores, held
// in registers (KPT keys per thread, element i = j * NT + tid). Small
// workgroups keep several rows in flight per compute unit, which hides the
// latency of the selection's barrier-separated phases. Scores map to
// order-preserving 32-bit keys; equal keys are ordered by index through a
// (key, ~index) composite.
//
// Common path (k <= 256): each thread's largest key is taken, and the k-th
// largest of those 256 maxima, L, is a lower bound of the segment's k-th key
// (k distinct keys, one per thread, are at least L). Only slightly more than
// k keys usually reach L (about 120 for k = 100 among 14,505 scores), so they
// are compacted straight into LDS, with ranges per wavefront from ballot
// counts and no atomics, and one wavefront sorts them in registers; the
// first k are the answer.
//
// Histogram path (k > 256, or more than 256 keys at or above L: masses of
// equal or nearly equal scores). Bits that every key of the segment shares
// are found with a block-wide OR / AND and skipped. One histogram pass over
// the next 11 bits locates the bin that holds the k-th key; every key in that
// bin or above is compacted and sorted. If that bin is crowded, a second
// 11-bit histogram over the bin's keys, still in registers, narrows it. If
// the candidate set would still exceed the LDS buffer, exact radix passes of
// 8 bits narrow the threshold key T down instead, and the keys above T plus
// the lowest-index keys equal to T are taken. Sorting runs in registers
// inside one wavefront for up to 256 candidates, in LDS across the workgroup
// otherwise.
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
