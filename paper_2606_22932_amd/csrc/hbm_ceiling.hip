// hbm_ceiling -- measured HBM bandwidth of this device for the access mixes of the fused
// step, used as context for its roofline (the published peak stays the reference):
//   read     one stream read
//   write    one stream written
//   copy     one stream read, another written
//   rmw3     three streams each read and written in place (the state traffic of a fused
//            step: W, m and v read and written back)
// Buffers are sized well past the memory-side cache; 16 bytes per lane, grid-stride,
// non-temporal; each figure is the best over grids of 4-32 workgroups per CU and three
// repetitions.  Prints one JSON object on stdout.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

namespace {

__global__ void __launch_bounds__(256) k_read(const u32x4_t *a, size_t n, u32x4_t *sink)
{
    u32x4_t acc = {0u, 0u, 0u, 0u};
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        acc ^= __builtin_nontemporal_load(a + i);
    if ((acc[0] ^ acc[1] ^ acc[2] ^ acc[3]) == 0x9e3779b9u) sink[0] = acc;   // keeps the loads
}

__global__ void __launch_bounds__(256) k_write(u32x4_t *a, size_t n)
{
    const u32x4_t v = {1u, 2u, 3u, 4u};
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        __builtin_nontemporal_store(v, a + i);
}

__global__ void __launch_bounds__(256) k_copy(const u32x4_t *a, u32x4_t *b, size_t n)
{
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        __builtin_nontemporal_store(__builtin_nontemporal_load(a + i), b + i);
}

__global__ void __launch_bounds__(256) k_rmw3(u32x4_t *w, u32x4_t *m, u32x4_t *v, size_t n)
{
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
        const u32x4_t x = __builtin_nontemporal_load(w + i);
        const u32x4_t y = __builtin_nontemporal_load(m + i);
        const u32x4_t z = __builtin_nontemporal_load(v + i);
        __builtin_nontemporal_store(x + 1u, w + i);
        __builtin_nontemporal_store(y ^ x, m + i);
        __builtin_nontemporal_store(z + y, v + i);
    }
}

bool ok(hipError_t e, const char *what)
{
    if (e == hipSuccess) return true;
    fprintf(stderr, "hbm_ceiling: %s: %s\n", what, hipGetErrorString(e));
    return false;
}

}  // namespace

int main(int argc, char **argv)
{
    // bytes per stream (default 12 GiB: 36 GiB for rmw3, far past the 256 MiB MALL)
    const size_t bytes = (argc > 1 ? strtoull(argv[1], nullptr, 10) : 12ull) << 30;
    const size_t n = bytes / 16;
    u32x4_t *A = nullptr, *B = nullptr, *C = nullptr, *sink = nullptr;
    if (!ok(hipMalloc(&A, bytes), "hipMalloc") || !ok(hipMalloc(&B, bytes), "hipMalloc") ||
        !ok(hipMalloc(&C, bytes), "hipMalloc") || !ok(hipMalloc(&sink, 64), "hipMalloc"))
        return 1;
    if (!ok(hipMemset(A, 0, bytes), "hipMemset") || !ok(hipMemset(B, 0, bytes), "hipMemset") ||
        !ok(hipMemset(C, 0, bytes), "hipMemset"))
        return 1;
    int ncu = 0;
    if (!ok(hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, 0), "attribute")) return 1;
    hipEvent_t e0, e1;
    if (!ok(hipEventCreate(&e0), "event") || !ok(hipEventCreate(&e1), "event")) return 1;
    const char *names[4] = {"read", "write", "copy", "rmw3"};
    double gbs[4];
    // the ceiling of a mix: the best of several grid sizes (workgroups per CU) and repetitions
    const int mults[4] = {4, 8, 16, 32};
    for (int kind = 0; kind < 4; ++kind) {
        float best = 1e30f;
        for (int rep = 0; rep < 4 * 4; ++rep) {
            const int grid = ncu * mults[rep % 4];
            if (!ok(hipEventRecord(e0), "record")) return 1;
            if (kind == 0) k_read<<<grid, 256>>>(A, n, sink);
            if (kind == 1) k_write<<<grid, 256>>>(A, n);
            if (kind == 2) k_copy<<<grid, 256>>>(A, B, n);
            if (kind == 3) k_rmw3<<<grid, 256>>>(A, B, C, n);
            if (!ok(hipGetLastError(), "launch") || !ok(hipEventRecord(e1), "record") ||
                !ok(hipEventSynchronize(e1), "sync"))
                return 1;
            float ms = 0.0f;
            if (!ok(hipEventElapsedTime(&ms, e0, e1), "elapsed")) return 1;
            if (rep >= 4 && ms < best) best = ms;    // the first pass over the grids warms up
        }
        const double moved = (kind < 2 ? 1.0 : kind == 2 ? 2.0 : 6.0) * (double)bytes;
        gbs[kind] = moved / (best * 1e-3) / 1e9;
    }
    printf("{\"unit\": \"GB/s\", \"bytes_per_stream\": %zu", bytes);
    for (int kind = 0; kind < 4; ++kind) printf(", \"%s\": %.1f", names[kind], gbs[kind]);
    printf("}\n");
    (void)hipFree(A); (void)hipFree(B); (void)hipFree(C); (void)hipFree(sink);
    return 0;
}
