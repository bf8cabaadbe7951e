// FP32 VALU issue-rate microbenchmark for gfx950.
//
// Register-only loops with the instruction mixes of the entity scorers (no
// memory traffic inside the loop; query values come from a 1 KiB buffer that
// stays in the scalar cache), run with enough workgroups to fill every SIMD.
// It prints lane-operations per second for each mix; the scorers' roofline
// fractions are quoted against the chip's 78.64 T peak and these measured
// ceilings. Built with the same flags as the library (packed FP32 disabled).
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cmath>
#define CHECK(x) do { hipError_t e = (x); if (e != hipSuccess) { printf("err %s line %d\n", hipGetErrorString(e), __LINE__); return 1; } } while (0)

// mix 0: acc += |e - q| (2 ops), 1: Q2B mix (4 ops), 2: two FMAs with scalar operands (2 ops), 3: plain adds (1 op)
template <int MIX>
__global__ __launch_bounds__(256) void k(const float* __restrict__ q, float* out, int iters)
{
    float e[4], acc[8][4], acc2[8][4];
    for (int j = 0; j < 4; ++j) e[j] = threadIdx.x * 0.001f + j;
    for (int i = 0; i < 8; ++i) for (int j = 0; j < 4; ++j) { acc[i][j] = 0.f; acc2[i][j] = 0.f; }
    for (int it = 0; it < iters; ++it) {
        const float* qq = q + (it & 15) * 16;   // uniform, scalar-cache resident
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float c = qq[i], o = qq[8 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                if (MIX == 0) acc[i][j] += fabsf(e[j] - c);
                if (MIX == 1) { const float t = fabsf(e[j] - c); acc[i][j] += t; acc2[i][j] += __builtin_fminf(t, o); }
                if (MIX == 2) acc[i][j] = fmaf(o, e[j], fmaf(c, e[j], acc[i][j]));
                if (MIX == 3) acc[i][j] += c;
            }
        }
    }
    float s = 0.f;
    for (int i = 0; i < 8; ++i) for (int j = 0; j < 4; ++j) s += acc[i][j] + acc2[i][j];
    out[blockIdx.x * blockDim.x + threadIdx.x] = s;
}

template <int MIX>
int run(const char* name, int ops_per_pair, const float* dq, float* dout, int grid)
{
    const int iters = 2000;
    hipEvent_t a, b; CHECK(hipEventCreate(&a)); CHECK(hipEventCreate(&b));
    hipLaunchKernelGGL(k<MIX>, dim3(grid), dim3(256), 0, 0, dq, dout, 10);
    CHECK(hipDeviceSynchronize());
    CHECK(hipEventRecord(a, 0));
    hipLaunchKernelGGL(k<MIX>, dim3(grid), dim3(256), 0, 0, dq, dout, iters);
    CHECK(hipEventRecord(b, 0));
    CHECK(hipEventSynchronize(b));
    float ms; CHECK(hipEventElapsedTime(&ms, a, b));
    double lane_ops = (double)grid * 256 * iters * 8 * 4 * ops_per_pair;
    printf("%-28s grid %6d: %.3f ms  %.2f T lane-ops/s  (%.1f%% of 39.32, %.1f%% of 78.64)\n", name, grid, ms,
           lane_ops / ms / 1e9, lane_ops / ms / 1e9 / 39.32 * 100, lane_ops / ms / 1e9 / 78.64 * 100);
    return 0;
}

int main()
{
    float hq[256]; for (int i = 0; i < 256; ++i) hq[i] = 0.01f * i;
    float* dq; float* dout; const int maxgrid = 256 * 16;
    CHECK(hipMalloc(&dq, sizeof(hq))); CHECK(hipMemcpy(dq, hq, sizeof(hq), hipMemcpyHostToDevice));
    CHECK(hipMalloc(&dout, sizeof(float) * maxgrid * 256));
    for (int g : {1024, 4096}) {
        run<3>("add (1 op)", 1, dq, dout, g);
        run<0>("gqe |e-q| (2 ops)", 2, dq, dout, g);
        run<1>("q2b mix (4 ops)", 4, dq, dout, g);
        run<2>("betae 2 fma (2 ops)", 2, dq, dout, g);
    }
    return 0;
}
