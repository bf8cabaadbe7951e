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

__global__ __launch_bounds__(RK_THREADS) void k_rank_answers(const float* scores, int64_t ld, int64_t N,
                                                             const int32_t* off, const int32_t* ids,
                                                             const int32_t* hard, int32_t* rank, double* metrics,
                                                             int* flag)
{
    __shared__ uint64_t key[kMaxAnswers];
    __shared__ int32_t pos[kMaxAnswers];
    __shared__ uint32_t hist[kMaxAnswers + 1];
    __shared__ int32_t rk[kMaxAnswers];      // rank by original list position
    __shared__ int sh_bad;

    const int tid = threadIdx.x;
    const int64_t q = blockIdx.x;
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

void launch_rank_answers(const float* scores, int64_t ld, int64_t N, int batch, const int32_t* off,
                         const int32_t* ids, const int32_t* hard, int32_t* rank, double* metrics, int* flag,
                         hipStream_t s)
{
    if (batch <= 0) return;
    hipLaunchKernelGGL(k_rank_answers, dim3(batch), dim3(RK_THREADS), 0, s, scores, ld, N, off, ids, hard, rank,
                       metrics, flag);
}

}  // namespace kgq
