// Plain device-to-device copy of a known size, for two purposes:
//  - calibrating HBM byte counters: under `rocprofv3 --pmc FETCH_SIZE` (or
//    WRITE_SIZE) each dispatch of k_copy moves exactly `bytes` in each
//    direction, so counter / bytes is the counter's scale;
//  - the achievable copy bandwidth (printed), next to the 8 TB/s HBM3E peak.
// Usage: hbm_copy [MiB per buffer, default 512] [repetitions, default 20]
#include <hip/hip_runtime.h>
#include <cstdio>
#include <cstdlib>
#define CHECK(x) do { hipError_t e = (x); if (e != hipSuccess) { printf("error %s at line %d\n", hipGetErrorString(e), __LINE__); return 1; } } while (0)

// one float4 per thread; the grid covers the buffer exactly
__global__ __launch_bounds__(256) void k_copy(const float4* __restrict__ src, float4* __restrict__ dst, long n4)
{
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n4) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void k_fill(float4* dst, long n4)
{
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n4) dst[i] = make_float4((float)i, 1.f, 2.f, 3.f);
}

int main(int argc, char** argv)
{
    const long mib = argc > 1 ? atol(argv[1]) : 512;
    const int reps = argc > 2 ? atoi(argv[2]) : 20;
    if (mib <= 0 || mib > 16384 || reps <= 0) { printf("bad arguments\n"); return 1; }
    const long bytes = mib << 20;
    const long n4 = bytes / 16;
    float4 *src = nullptr, *dst = nullptr;
    CHECK(hipMalloc(&src, bytes));
    CHECK(hipMalloc(&dst, bytes));
    const unsigned blocks = (unsigned)((n4 + 255) / 256);
    hipLaunchKernelGGL(k_fill, dim3(blocks), dim3(256), 0, 0, src, n4);
    hipLaunchKernelGGL(k_copy, dim3(blocks), dim3(256), 0, 0, src, dst, n4);   // warm-up
    CHECK(hipDeviceSynchronize());
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    CHECK(hipEventRecord(e0, 0));
    for (int r = 0; r < reps; ++r) hipLaunchKernelGGL(k_copy, dim3(blocks), dim3(256), 0, 0, src, dst, n4);
    CHECK(hipEventRecord(e1, 0));
    CHECK(hipEventSynchronize(e1));
    float ms = 0.f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    const double s = ms * 1e-3 / reps;
    printf("k_copy: %ld bytes read + %ld bytes written per dispatch, %.1f us, %.0f GB/s (read + write)\n",
           bytes, bytes, s * 1e6, 2.0 * bytes / s / 1e9);
    CHECK(hipFree(src));
    CHECK(hipFree(dst));
    return 0;
}
