// Measurement probe, not part of the library: the device's plain streaming
// read rate, as the reference for the fused kernel's key stream.  A 16 GiB
// buffer is read once per pass with 16-byte nontemporal loads (a wave
// instruction reads 1 KiB contiguous), grid-stride, ILP loads in flight per
// lane; every configuration is timed over 5 passes after one warm-up pass.
//
//   hipcc --offload-arch=gfx950 -O3 -Xclang -target-feature -Xclang -packed-fp32-ops probe_stream.hip -o probe_stream
#include <hip/hip_runtime.h>

#include <cstdio>

#define CHECK(x)                                                                  \
    do {                                                                          \
        hipError_t e_ = (x);                                                      \
        if (e_ != hipSuccess) {                                                   \
            printf("HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            return 1;                                                             \
        }                                                                         \
    } while (0)

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

template <int ILP>
__global__ void __launch_bounds__(256) read_pass(const u32x4* __restrict__ p, size_t n, unsigned* out) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    unsigned acc = 0;
    for (; i + (ILP - 1) * stride < n; i += ILP * stride) {
        u32x4 v[ILP];
#pragma unroll
        for (int k = 0; k < ILP; ++k) v[k] = __builtin_nontemporal_load(p + i + k * stride);
#pragma unroll
        for (int k = 0; k < ILP; ++k) acc ^= v[k].x ^ v[k].w;
    }
    for (; i < n; i += stride) acc ^= p[i].x;
    if (acc == 0x9e3779b9u) out[0] = acc;   // keeps the loads; never true for the fill below
}

template <int ILP>
int run(const u32x4* p, size_t n, unsigned* out, int grid, hipEvent_t a, hipEvent_t b) {
    read_pass<ILP><<<grid, 256>>>(p, n, out);
    CHECK(hipDeviceSynchronize());
    CHECK(hipEventRecord(a));
    for (int r = 0; r < 5; ++r) read_pass<ILP><<<grid, 256>>>(p, n, out);
    CHECK(hipEventRecord(b));
    CHECK(hipEventSynchronize(b));
    float ms = 0.0f;
    CHECK(hipEventElapsedTime(&ms, a, b));
    printf("| %d | %d | %.3f | %.2f |\n", grid, ILP, ms / 5, n * 16.0 / (ms / 5 * 1e-3) / 1e12);
    return 0;
}

int main() {
    const size_t bytes = (size_t)16 << 30;
    const size_t n = bytes / 16;
    u32x4* p = nullptr;
    unsigned* out = nullptr;
    CHECK(hipMalloc(&p, bytes));
    CHECK(hipMalloc(&out, 4));
    CHECK(hipMemset(p, 1, bytes));
    hipEvent_t a, b;
    CHECK(hipEventCreate(&a));
    CHECK(hipEventCreate(&b));
    printf("| workgroups (256 threads) | loads in flight per lane | ms per 16 GiB pass | TB/s |\n|---:|---:|---:|---:|\n");
    for (int grid : {256, 512, 768, 1024, 2048, 8192}) {
        if (run<4>(p, n, out, grid, a, b) || run<8>(p, n, out, grid, a, b)) return 1;
    }
    CHECK(hipFree(p));
    CHECK(hipFree(out));
    return 0;
}
