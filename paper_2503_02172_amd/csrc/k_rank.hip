// Filtered ranks of known answers and ranking metrics (the paper reports
// MRR; Experiments). For query q with answer set A (distinct entity ids) and
// score row s, the filtered rank of answer a is
//   1 + #{ e not in A : e ranks before a },
// in the library's ranking order: higher score first, equal scores by lower
// entity index (the order of the top-k). Per query, over its hard answers:
// MRR = mean of 1 / rank, Hits@{1, 3, 10} = share of ranks <= 1, 3, 10.
//
// One workgroup of 256 threads per query:
//   1. the answers' (key, index) composites (the top-k's order-preserving
//      score key in the high half, the inverted index in the low half, so
//      that "ranks before" is "composite greater") are sorted ascending in
//      LDS, at most kMaxAnswers of them;
//   2. one pass over the score row: each entity finds, by a branch-free
//      binary search, how many answer composites lie below its own (the
//      answers it outranks) and counts itself in that bin of an LDS histogram;
//   3. a suffix sum over the bins gives each answer the number of entities
//      ranked before it; the answers among those are exactly the answers
//      sorted above it, which are subtracted;
//   4. the metrics are summed in double precision in answer-list order.
// The pass over the scores reads each row once; placing each entity among
// the answers, not the read, bounds it.
//
// Lists of at most kRankShort answers (the common case) take a streaming
// kernel instead: one wavefront per query, no workgroup barriers. The
// wavefront sorts its answers in registers (one per lane), streams the row
// with several 256-entity steps in flight, counts for each answer the
// entities that outrank it (per-lane counters against answer keys in scalar
// registers for up to 8 answers; otherwise each entity's place among the
// answers, from scalar-register pivots and a short search in its own LDS,
// into per-lane histograms), and computes ranks and metrics in registers. The workgroup kernel
// then runs only for the other lists (longer, empty or invalid), which it
// leaves to the streaming kernel otherwise.
#include <algorithm>

#include "kgq_internal.hpp"

namespace kgq {

constexpr int RK_THREADS = 256;

__device__ __forceinline__ uint64_t rank_composite(float f, int64_t e)
{
    if (f == 0.0f) f = 0.0f;   // -0 and +0 rank equal
    const uint32_t u = __float_as_uint(f);
    const uint32_t key = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
    return ((uint64_t)key << 32) | (uint32_t)(0xFFFFFFFFu - (uint32_t)e);
}

constexpr int kRankShort = 32;       // longest answer list of the streaming kernel

// One query by the whole workgroup.
__device__ __forceinline__ void rank_query_wg(int64_t q, const float* scores, int64_t ld, int64_t N,
                                              const int32_t* off, const int32_t* ids, const int32_t* hard,
                                              int32_t* rank, double* metrics, int* flag)
{
    __shared__ uint64_t key[kMaxAnswers];
    __shared__ int32_t pos[kMaxAnswers];
    __shared__ uint32_t hist[kMaxAnswers + 1];
    __shared__ int32_t rk[kMaxAnswers];      // rank by original list position
    __shared__ int sh_bad;

    const int tid = threadIdx.x;
    const int32_t lo = off[q];
    const int n = off[q + 1] - lo;
    double* met = metrics ? metrics + 4 * q : nullptr;
    const double qnan = __builtin_nan("");
    if (n <= 0 || n > kMaxAnswers) {
        if (n != 0 && tid == 0) atomicOr(flag, kErrAnswers);
        for (int i = tid; i < n; i += RK_THREADS) rank[lo + i] = -1;
        if (met && tid < 4) met[tid] = qnan;
        return;
    }
    const float* row = scores + q * ld;
    if (tid == 0) sh_bad = 0;
    int P = 1;
    while (P < n) P <<= 1;
    __syncthreads();
    for (int i = tid; i < P; i += RK_THREADS) {
        if (i < n) {
            const int32_t id = ids[lo + i];
            if (id < 0 || (int64_t)id >= N) {
                key[i] = 0ull;                    // sorts first; its rank is reported as -1
                atomicOr(&sh_bad, 1);
            } else {
                key[i] = rank_composite(row[id], id);
            }
            pos[i] = i;
        } else {
            key[i] = ~0ull;                       // padding sorts last
            pos[i] = -1;
        }
    }
    // bitonic sort, ascending
    for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            __syncthreads();
            for (int t = tid; t < P / 2; t += RK_THREADS) {
                const int p = ((t & ~(stride - 1)) << 1) | (t & (stride - 1));
                const int r = p + stride;
                const bool up = (p & size) == 0;
                const uint64_t a = key[p], b = key[r];
                if (up ? (a > b) : (a < b)) {
                    key[p] = b; key[r] = a;
                    const int32_t x = pos[p]; pos[p] = pos[r]; pos[r] = x;
                }
            }
        }
    }
    for (int i = tid; i <= n; i += RK_THREADS) hist[i] = 0;
    __syncthreads();
    if (tid == 0 && sh_bad) atomicOr(flag, kErrRange);

    // pass over the row: entity e outranks the answers whose composite is
    // below its own; a = their count, and e adds to bin a (suffix sums
    // below; bin 0 is never summed). a is a branch-free lower bound over the
    // P sorted keys (padding ~0 sorts last): one step per halving, the same
    // for every lane, and the U entities of a thread step together so that
    // their LDS reads overlap. Loads are unconditional at clamped positions;
    // entity indices fit 32 bits (n_entities < 2^31).
    constexpr int U = 8;
    const uint32_t Nu = (uint32_t)N;
    for (uint32_t e0 = tid; e0 < Nu; e0 += RK_THREADS * U) {
        float v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = row[min(e0 + (uint32_t)(u * RK_THREADS), Nu - 1)];
        uint64_t c[U];
        int a[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            c[u] = rank_composite(v[u], (int64_t)(e0 + (uint32_t)(u * RK_THREADS)));
            a[u] = 0;
        }
        for (int step = P >> 1; step > 0; step >>= 1) {
#pragma unroll
            for (int u = 0; u < U; ++u) a[u] += key[a[u] + step - 1] < c[u] ? step : 0;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) a[u] += key[a[u]] < c[u] ? 1 : 0;   // a was at most P - 1
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (e0 + (uint32_t)(u * RK_THREADS) < Nu && a[u] > 0) atomicAdd(&hist[a[u]], 1u);
    }
    __syncthreads();

    // suffix sums by one wavefront: before(i) = sum of hist[j], j > i
    if (tid < 64) {
        constexpr int PER = (kMaxAnswers + 1 + 63) / 64;
        uint32_t v[PER], s = 0;
#pragma unroll
        for (int t = 0; t < PER; ++t) {
            const int j = tid * PER + t;
            v[t] = j <= n ? hist[j] : 0u;
            s += v[t];
        }
        uint32_t incl = s;                        // inclusive suffix over lanes
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t x = __shfl_down(incl, o, 64);
            if (tid + o < 64) incl += x;
        }
        uint32_t above = incl - s;                // bins of higher lanes
#pragma unroll
        for (int t = PER - 1; t >= 0; --t) {
            const int i = tid * PER + t;          // answer i receives bins j > i
            if (i < n) {
                const int p = pos[i];
                const int32_t r = key[i] == 0ull ? -1 : (int32_t)(1 + above - (uint32_t)(n - 1 - i));
                rank[lo + p] = r;
                rk[p] = r;
            }
            above += v[t];
        }
    }
    __syncthreads();

    if (met && tid == 0) {
        double mrr = 0.0, h1 = 0.0, h3 = 0.0, h10 = 0.0;
        int nh = 0;
        for (int i = 0; i < n; ++i) {
            if (hard && !hard[lo + i]) continue;
            ++nh;
            const int r = rk[i];
            mrr += 1.0 / (double)r;
            h1 += r <= 1 ? 1.0 : 0.0;
            h3 += r <= 3 ? 1.0 : 0.0;
            h10 += r <= 10 ? 1.0 : 0.0;
        }
        if (nh == 0 || sh_bad) {
            met[0] = met[1] = met[2] = met[3] = qnan;
        } else {
            met[0] = mrr / nh;
            met[1] = h1 / nh;
            met[2] = h3 / nh;
            met[3] = h10 / nh;
        }
    }
}

// One workgroup per query; skip_short: lists of 1 .. kRankShort answers are
// left to the streaming kernel.
__global__ __launch_bounds__(RK_THREADS) void k_rank_answers(const float* scores, int64_t ld, int64_t N,
                                                             const int32_t* off, const int32_t* ids,
                                                             const int32_t* hard, int32_t* rank, double* metrics,
                                                             int* flag, int skip_short)
{
    const int64_t q = blockIdx.x;
    const int n = off[q + 1] - off[q];       // the same for the whole workgroup
    if (skip_short && n >= 1 && n <= kRankShort) return;
    rank_query_wg(q, scores, ld, N, off, ids, hard, rank, metrics, flag);
}

// ---------------------------------------------------------------------------
// Streaming kernel: queries with 1 .. kRankShort answers, one wavefront each.
//
// Answer i (of the n sorted ascending, padded to P with ~0) is outranked by
// count_i = #{ e : composite(e) > t_i } entities, the answers sorted above it
// among them.
//   P <= 8: each lane keeps P counters and adds one 64-bit compare of each
//   entity against each answer composite, held in scalar registers; one
//   wave sum per answer at the end.
//   P = 16, 32: an entity's place among the answers, a = #{ i : t_i < c },
//   comes from seven pivots in scalar registers (the last answer of each of
//   the first seven blocks of P / 8) and a binary search inside the block in
//   LDS; it adds one to bin a of the lane's own histogram (16-bit counters,
//   two bins a word, bin-major so that each lane keeps to one LDS bank: no
//   conflicts, no atomics shared between lanes). count_i is the sum of bins
//   above i over all lanes.
// ---------------------------------------------------------------------------
constexpr int kRankWaves = 2;        // wavefronts (queries) per workgroup
constexpr int kRankDepth = 6;        // 256-entity steps held in registers (5 in flight)
constexpr int kRankHistWords = kRankShort / 2 + 1;   // bins 0 .. kRankShort, two a word

struct RankLds {
    uint64_t key[kRankShort];        // answer composites, ascending (padding ~0)
    uint32_t hist[kRankHistWords][64];   // [bin pair][lane], 16-bit counters
    int32_t rk[kRankShort];          // rank by list position
};

// The pass over row (positions past N read as 0 through the buffer range
// check; body decides what they count for). Per step of 4 x 64 entities,
// body(x, base) gets the four scores of positions base + cc * 64
// (cc = 0 .. 3), base = step * 256 + lane.
template <typename Body>
__device__ __forceinline__ void rank_stream_row(const float* row, int64_t N, int lane, Body body)
{
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(row), (short)0, (int)(N * 4), 0x00020000);
    const int nsteps = (int)((N + 255) >> 8);
    // (the caller passes the wavefront's part of a row: row and N relative to
    // it; body adds the part's first index)
    float v[kRankDepth][4];
#pragma unroll
    for (int g = 0; g < kRankDepth; ++g) {
#pragma unroll
        for (int cc = 0; cc < 4; ++cc)
            v[g][cc] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rsrc, lane * 4 + (g * 256 + cc * 64) * 4, 0, 0));
        __builtin_amdgcn_sched_barrier(0);
    }
    // wave priority falls with progress (as in the streaming top-k)
    const int q1 = nsteps >> 2, q2 = nsteps >> 1, q3 = (3 * nsteps) >> 2;
    __builtin_amdgcn_s_setprio(3);
    for (int s0 = 0; s0 < nsteps; s0 += kRankDepth) {
        if (s0 >= q3) __builtin_amdgcn_s_setprio(0);
        else if (s0 >= q2) __builtin_amdgcn_s_setprio(1);
        else if (s0 >= q1) __builtin_amdgcn_s_setprio(2);
#pragma unroll
        for (int g = 0; g < kRankDepth; ++g) {
            const int s = s0 + g;
            if (s < nsteps) body(v[g], (uint32_t)(s * 256 + lane));
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int cc = 0; cc < 4; ++cc)
                v[g][cc] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(
                    rsrc, lane * 4 + ((s + kRankDepth) * 256 + cc * 64) * 4, 0, 0));
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    __builtin_amdgcn_s_setprio(0);
}

__device__ __forceinline__ uint64_t rank_lane_key(uint64_t t_lane, int i)
{
    // (readlane returns int: through uint32_t, or the low half would
    // sign-extend over the high one)
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(t_lane >> 32), i) << 32) |
           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)t_lane, i);
}

// Wave sum of x, the same in every lane.
__device__ __forceinline__ uint32_t rank_wave_sum(uint32_t x)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

// count_i by counters (P <= 8; lane i holds t_i): returns lane i's count.
template <int P>
__device__ __forceinline__ uint32_t rank_counts(const float* row, int64_t N, uint32_t p0, int lane, uint64_t t_lane)
{
    uint64_t t[P];
#pragma unroll
    for (int i = 0; i < P; ++i) t[i] = rank_lane_key(t_lane, i);
    uint32_t cnt[P];
#pragma unroll
    for (int i = 0; i < P; ++i) cnt[i] = 0u;
    const uint32_t Nu = (uint32_t)N;
    rank_stream_row(row, N, lane, [&](const float (&x)[4], uint32_t base) {
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            const uint32_t e = base + cc * 64;
            const uint64_t c = e < Nu ? rank_composite(x[cc], (int64_t)(p0 + e)) : 0ull;   // past the part: outranks nothing
#pragma unroll
            for (int i = 0; i < P; ++i) cnt[i] += c > t[i] ? 1u : 0u;
        }
    });
    uint32_t mine = 0u;
#pragma unroll
    for (int i = 0; i < P; ++i) {
        const uint32_t x = rank_wave_sum(cnt[i]);
        mine = lane == i ? x : mine;
    }
    return mine;
}

// count_i by place and per-lane histogram (P = 16, 32; the sorted keys in
// L.key, lane i holds t_i): returns lane i's count.
template <int P>
__device__ __forceinline__ uint32_t rank_counts_place(RankLds& L, const float* row, int64_t N, uint32_t p0, int lane,
                                                      uint64_t t_lane)
{
    constexpr int BK = P / 8;                    // block size
    constexpr int W = P / 2 + 1;                 // histogram words (bins 0 .. P)
    uint64_t piv[7];
#pragma unroll
    for (int j = 0; j < 7; ++j) piv[j] = rank_lane_key(t_lane, (j + 1) * BK - 1);
#pragma unroll
    for (int w = 0; w < W; ++w) L.hist[w][lane] = 0u;
    const uint32_t Nu = (uint32_t)N;
    rank_stream_row(row, N, lane, [&](const float (&x)[4], uint32_t base) {
        uint64_t c[4];
        int a[4];
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            c[cc] = rank_composite(x[cc], (int64_t)(p0 + base + cc * 64));
            int below = 0;
#pragma unroll
            for (int j = 0; j < 7; ++j) below += piv[j] < c[cc] ? 1 : 0;
            a[cc] = below * BK;
        }
#pragma unroll
        for (int step = BK / 2; step > 0; step >>= 1) {
#pragma unroll
            for (int cc = 0; cc < 4; ++cc) a[cc] += L.key[a[cc] + step - 1] < c[cc] ? step : 0;
        }
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) a[cc] += L.key[a[cc]] < c[cc] ? 1 : 0;   // a was at most P - 1
#pragma unroll
        for (int cc = 0; cc < 4; ++cc) {
            // bin a of this lane's own counters (one LDS bank per lane: no
            // conflicts); bin 0 is never summed, past the part counts nothing
            if (base + cc * 64 < Nu && a[cc] > 0) atomicAdd(&L.hist[a[cc] >> 1][lane], 1u << ((a[cc] & 1) * 16));
        }
    });
    // count_i = sum over lanes of the bins j > i
    uint32_t mine = 0u, above = 0u;
#pragma unroll
    for (int w = W - 1; w >= 0; --w) {
        const uint32_t x = L.hist[w][lane];
        const uint32_t hi = rank_wave_sum(x >> 16);      // bin 2w + 1
        const uint32_t lo = rank_wave_sum(x & 0xFFFFu);  // bin 2w
        // answer 2w + 1 gets the bins above 2w + 1; answer 2w also bin 2w + 1
        if (lane == 2 * w + 1) mine = above;
        above += hi;
        if (lane == 2 * w) mine = above;
        above += lo;
    }
    return mine;
}

// QW wavefronts per query, each over its own part of the row (QW = 1: two
// queries per workgroup, one wavefront each).
template <int QW>
__global__ __launch_bounds__(64 * (QW == 1 ? kRankWaves : QW)) void k_rank_stream(
    const float* scores, int64_t ld, int64_t N, const int32_t* off, const int32_t* ids, const int32_t* hard,
    int32_t* rank, double* metrics, int* flag, int batch)
{
    constexpr int WG = QW == 1 ? kRankWaves : QW;
    __shared__ RankLds lds[WG];
    __shared__ uint32_t part_cnt[QW][kRankShort];
    const int lane = threadIdx.x & 63;
    // (readfirstlane: the wavefront index is uniform, so the query's
    // addresses stay in scalar registers)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t q = QW == 1 ? (int64_t)blockIdx.x * kRankWaves + wave : (int64_t)blockIdx.x;
    const int part = QW == 1 ? 0 : wave;
    if (q >= batch) return;                  // (QW > 1: the whole workgroup)
    const int32_t lo = off[q];
    const int n = off[q + 1] - lo;
    if (n < 1 || n > kRankShort) return;     // the workgroup kernel's (the whole workgroup for QW > 1)
    RankLds& L = lds[wave];
    const float* row = scores + q * ld;

    // the answers, one per lane, sorted ascending with their list positions
    uint64_t c = ~0ull;                      // padding sorts last
    int32_t pos = lane;
    bool bad = false;
    if (lane < n) {
        const int32_t id = ids[lo + lane];
        bad = id < 0 || (int64_t)id >= N;
        c = bad ? 0ull : rank_composite(row[id], id);   // an invalid id sorts first; its rank is -1
    }
    if (__builtin_amdgcn_ballot_w64(bad) != 0ull && lane == 0 && part == 0) atomicOr(flag, kErrRange);
#pragma unroll
    for (int size = 2; size <= 64; size <<= 1) {
#pragma unroll
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            const uint32_t olo = __shfl_xor((uint32_t)c, stride, 64);
            const uint32_t ohi = __shfl_xor((uint32_t)(c >> 32), stride, 64);
            const int32_t opos = __shfl_xor(pos, stride, 64);
            const uint64_t o = ((uint64_t)ohi << 32) | olo;
            const bool up = (lane & size) == 0;            // ascending run
            const bool lower = (lane & stride) == 0;
            const bool take = (up == lower) ? (o < c) : (o > c);   // keep the min in the lower slot of an up run
            c = take ? o : c;
            pos = take ? opos : pos;
        }
    }
    int P = 1;
    while (P < n) P <<= 1;

    // this wavefront's part of the row: positions [p0, p0 + len)
    const int64_t plen = QW == 1 ? N : (((N + QW - 1) / QW + 255) / 256) * 256;
    const int64_t p0 = part * plen;
    const int64_t len = p0 >= N ? 0 : (N - p0 < plen ? N - p0 : plen);
    const float* prow = row + p0;
    uint32_t cnt = 0u;                       // lane i: count_i over the part
    if (len > 0) {
        switch (P) {
        case 1: cnt = rank_counts<1>(prow, len, (uint32_t)p0, lane, c); break;
        case 2: cnt = rank_counts<2>(prow, len, (uint32_t)p0, lane, c); break;
        case 4: cnt = rank_counts<4>(prow, len, (uint32_t)p0, lane, c); break;
        case 8: cnt = rank_counts<8>(prow, len, (uint32_t)p0, lane, c); break;
        case 16:
            if (lane < kRankShort) L.key[lane] = c;      // (lanes >= n hold the padding ~0)
            cnt = rank_counts_place<16>(L, prow, len, (uint32_t)p0, lane, c);
            break;
        default:
            if (lane < kRankShort) L.key[lane] = c;
            cnt = rank_counts_place<32>(L, prow, len, (uint32_t)p0, lane, c);
            break;
        }
    }
    if (QW > 1) {
        // the parts' counts add up (one barrier; every wavefront of the
        // workgroup serves the same query and gets here)
        if (lane < kRankShort) part_cnt[part][lane] = cnt;
        __syncthreads();
        if (part != 0) return;
        cnt = 0u;
#pragma unroll
        for (int w = 0; w < QW; ++w) cnt += lane < kRankShort ? part_cnt[w][lane] : 0u;
    }
    // the n - 1 - i answers sorted above answer i are among its count
    if (lane < n) {
        const int32_t r = c == 0ull ? -1 : (int32_t)(1 + cnt - (uint32_t)(n - 1 - lane));
        rank[lo + pos] = r;
        L.rk[pos] = r;
    }
    if (!metrics) return;
    // metrics over the hard answers, summed in double in list order (each
    // lane holds list position `lane`; a non-hard answer adds 0)
    const bool any_bad = __builtin_amdgcn_ballot_w64(lane < n && L.rk[lane] < 0) != 0ull;
    const bool hd = lane < n && (!hard || hard[lo + lane] != 0);
    const int r = lane < n ? L.rk[lane] : 1;
    const double t_mrr = hd ? 1.0 / (double)r : 0.0;
    const double t_h1 = hd && r <= 1 ? 1.0 : 0.0;
    const double t_h3 = hd && r <= 3 ? 1.0 : 0.0;
    const double t_h10 = hd && r <= 10 ? 1.0 : 0.0;
    const int nh = __popcll(__builtin_amdgcn_ballot_w64(hd));
    double mrr = 0.0, h1 = 0.0, h3 = 0.0, h10 = 0.0;
    for (int p = 0; p < n; ++p) {
        mrr += __shfl(t_mrr, p, 64);
        h1 += __shfl(t_h1, p, 64);
        h3 += __shfl(t_h3, p, 64);
        h10 += __shfl(t_h10, p, 64);
    }
    if (lane == 0) {
        double* met = metrics + 4 * q;
        if (nh == 0 || any_bad) {
            const double qnan = __builtin_nan("");
            met[0] = met[1] = met[2] = met[3] = qnan;
        } else {
            met[0] = mrr / nh;
            met[1] = h1 / nh;
            met[2] = h3 / nh;
            met[3] = h10 / nh;
        }
    }
}

void launch_rank_answers(const float* scores, int64_t ld, int64_t N, int batch, const int32_t* off,
                         const int32_t* ids, const int32_t* hard, int32_t* rank, double* metrics, int* flag,
                         hipStream_t s)
{
    if (batch <= 0) return;
    // rows of more than 64 x 65,535 entities go to the workgroup kernel alone
    // (the streaming kernel's lanes count up to 65,535 entities a bin, and its
    // buffer resource spans a row in bytes as a 32-bit count)
    const int stream = N <= (int64_t)64 * 65535;
    if (stream) {
        // wavefronts per query: one per 16 Ki entities of the row, more when
        // the batch is too small to give 2,048 wavefronts; parts of at least
        // 4,096 entities, at most 4 (measured: 4,608 rows of 14,505 run best
        // with one, 2,048 rows of 63,361 with four)
        const int64_t by_row = (N + 16383) / 16384;
        const int64_t by_batch = batch < 2048 ? (2048 + batch - 1) / batch : 1;
        const int qw = (int)std::max<int64_t>(
            1, std::min<int64_t>({std::max(by_row, by_batch), (N + 4095) / 4096, 4}));
        if (qw == 1)
            hipLaunchKernelGGL(k_rank_stream<1>, dim3((batch + kRankWaves - 1) / kRankWaves), dim3(64 * kRankWaves), 0,
                               s, scores, ld, N, off, ids, hard, rank, metrics, flag, batch);
        else if (qw == 2)
            hipLaunchKernelGGL(k_rank_stream<2>, dim3(batch), dim3(128), 0, s, scores, ld, N, off, ids, hard, rank,
                               metrics, flag, batch);
        else if (qw == 3)
            hipLaunchKernelGGL(k_rank_stream<3>, dim3(batch), dim3(192), 0, s, scores, ld, N, off, ids, hard, rank,
                               metrics, flag, batch);
        else
            hipLaunchKernelGGL(k_rank_stream<4>, dim3(batch), dim3(256), 0, s, scores, ld, N, off, ids, hard, rank,
                               metrics, flag, batch);
    }
    hipLaunchKernelGGL(k_rank_answers, dim3(batch), dim3(RK_THREADS), 0, s, scores, ld, N, off, ids, hard, rank,
                       metrics, flag, stream);
}

}  // namespace kgq
