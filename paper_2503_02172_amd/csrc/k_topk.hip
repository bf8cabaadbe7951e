// Top-k selection over each query's N entity scores (the ranking the paper
// evaluates with MRR, Experiments/Metrics). Order: score descending, equal
// scores by entity index ascending.
//
// One workgroup of 1024 threads per query row. Scores map to order-
// preserving 32-bit keys; an exact radix select over 4 passes of 8 bits
// (MSB first) finds the key T of the k-th element and how many elements
// equal to T are taken. With N <= 64 Ki the row is read from memory once and
// kept in registers (KPT keys per thread, element i = j * 1024 + tid);
// longer rows are re-read per pass. Elements above T are gathered through an
// LDS counter; elements equal to T are taken all at once when every one of
// them fits, otherwise in index order through a block-wide scan. The k
// selected elements are ordered by counting, for each, the elements that
// rank before it.
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

template <int KPT>   // KPT == 0: re-read the row from memory in every pass
__global__ __launch_bounds__(TK_THREADS) void k_topk(TopkArgs a)
{
    __shared__ uint32_t hist[256];
    __shared__ uint32_t sel_key[kMaxK];
    __shared__ int32_t sel_idx[kMaxK];
    __shared__ int sh_bin, sh_rem, sh_eq, sh_gt, sh_eqslot;
    __shared__ int wave_cnt[TK_WAVES];

    const int tid = threadIdx.x;
    const int row = blockIdx.x;
    const float* __restrict__ sr = a.scores + (int64_t)row * a.ld;
    const int64_t N = a.N;
    const int k = a.k;

    uint32_t keys[KPT > 0 ? KPT : 1];
    if (KPT > 0) {
#pragma unroll
        for (int j = 0; j < KPT; ++j) {
            const int64_t i = (int64_t)j * TK_THREADS + tid;
            keys[j] = i < N ? score_key(sr[i]) : 0u;
        }
    }
    // visit every valid element: f(index, key)
    auto for_each = [&](auto&& f) {
        if (KPT > 0) {
#pragma unroll
            for (int j = 0; j < (KPT > 0 ? KPT : 1); ++j) {
                const int64_t i = (int64_t)j * TK_THREADS + tid;
                if (i < N) f(i, keys[j]);
            }
        } else {
            for (int64_t i = tid; i < N; i += TK_THREADS) f(i, score_key(sr[i]));
        }
    };

    uint32_t prefix = 0, pmask = 0;
    int rem = k;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        if (tid < 256) hist[tid] = 0;
        __syncthreads();
        for_each([&](int64_t, uint32_t key) {
            if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
        });
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
            const uint32_t above = incl - s;   // elements in bins above this lane's
            if (above < (uint32_t)rem && (uint32_t)rem <= incl) {
                uint32_t cum = above;
                for (int t = 3; t >= 0; --t) {
                    if ((uint32_t)rem <= cum + c[t]) {
                        sh_bin = 4 * tid + t;
                        sh_rem = rem - (int)cum;
                        sh_eq = (int)c[t];
                        break;
                    }
                    cum += c[t];
                }
            }
        }
        __syncthreads();
        prefix |= (uint32_t)sh_bin << shift;
        pmask |= 0xFFu << shift;
        rem = sh_rem;
        __syncthreads();
    }
    // prefix is now the exact key T of the k-th element; rem elements equal
    // to T are taken; sh_eq holds the number of elements equal to T.
    const uint32_t T = prefix;
    const int n_gt = k - rem;
    const bool take_all_eq = (sh_eq == rem);
    if (tid == 0) { sh_gt = 0; sh_eqslot = n_gt; }
    __syncthreads();
    for_each([&](int64_t i, uint32_t key) {
        if (key > T) {
            const int slot = atomicAdd(&sh_gt, 1);
            sel_key[slot] = key;
            sel_idx[slot] = (int32_t)i;
        } else if (key == T && take_all_eq) {
            const int slot = atomicAdd(&sh_eqslot, 1);
            sel_key[slot] = key;
            sel_idx[slot] = (int32_t)i;
        }
    });
    if (!take_all_eq) {
        // lowest indices first: elements are visited in index order
        // i = j * 1024 + tid, j outer, with a block-wide scan per step.
        const int lane = tid & 63, wave = tid >> 6;
        int base = 0;
        for (int64_t j0 = 0; j0 < N && base < rem; j0 += TK_THREADS) {
            const int64_t i = j0 + tid;
            uint32_t key = 0;
            if (i < N) key = (KPT > 0) ? 0u : score_key(sr[i]);
            if (KPT > 0) {
                const int jj = (int)(j0 / TK_THREADS);
#pragma unroll
                for (int j = 0; j < (KPT > 0 ? KPT : 1); ++j)
                    if (j == jj) key = keys[j];
            }
            const bool flag = (i < N) && key == T;
            const uint64_t ballot = __ballot(flag);
            const int before = __popcll(ballot & ((1ull << lane) - 1ull));
            if (lane == 0) wave_cnt[wave] = __popcll(ballot);
            __syncthreads();
            int off = 0, tot = 0;
            for (int w = 0; w < TK_WAVES; ++w) {
                if (w < wave) off += wave_cnt[w];
                tot += wave_cnt[w];
            }
            const int rank = base + off + before;
            if (flag && rank < rem) {
                sel_key[n_gt + rank] = key;
                sel_idx[n_gt + rank] = (int32_t)i;
            }
            base += tot;
            __syncthreads();
        }
    }
    __syncthreads();
    if (tid < k) {
        const uint32_t mk = sel_key[tid];
        const int32_t mi = sel_idx[tid];
        int r = 0;
        for (int u = 0; u < k; ++u) {
            const uint32_t ok = sel_key[u];
            r += (ok > mk) || (ok == mk && sel_idx[u] < mi);
        }
        a.out_idx[(int64_t)row * k + r] = mi;
        a.out_score[(int64_t)row * k + r] = sr[mi];
    }
}

void launch_topk(const TopkArgs& a, hipStream_t s)
{
    if (a.n_rows <= 0) return;
    const int64_t per = (a.N + TK_THREADS - 1) / TK_THREADS;
    dim3 grid(a.n_rows), block(TK_THREADS);
    if (per <= 4) hipLaunchKernelGGL(k_topk<4>, grid, block, 0, s, a);
    else if (per <= 16) hipLaunchKernelGGL(k_topk<16>, grid, block, 0, s, a);
    else if (per <= 32) hipLaunchKernelGGL(k_topk<32>, grid, block, 0, s, a);
    else if (per <= 64) hipLaunchKernelGGL(k_topk<64>, grid, block, 0, s, a);
    else hipLaunchKernelGGL(k_topk<0>, grid, block, 0, s, a);
}

}  // namespace kgq
