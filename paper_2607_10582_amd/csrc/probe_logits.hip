// Measurement, not part of the library: the logits of the fused observation
// kernel's key stream computed two ways, to decide between matrix cores and
// the vector ALU for the GQA group (the G query heads of one KV head):
//   MODE 1: MFMA 16x16x32 bf16, the G heads as the B operand's columns and
//           the float32 query split exactly into three bf16 terms (what the
//           fused kernel does);
//   MODE 2: a GEMV on the vector ALU in float32 (bf16 keys widened, one FMA
//           per product), each lane holding 32 dims of one token and the
//           four lanes of a token adding their partial sums by shuffles.
// Same grid (512 workgroups of four waves), the same units of 4 tiles per
// wave, block-interleaved pool and two-row load ring as the fused kernel;
// every logit goes into a running maximum that is written out, so nothing
// is dead code.  Build and run:
//   hipcc --offload-arch=gfx950 -O3 -std=c++17 \
//     -Xclang -target-feature -Xclang -packed-fp32-ops probe_logits.hip -o probe_logits
//   ./probe_logits
#include <hip/hip_runtime.h>
#include <stdio.h>
#include <stdlib.h>
#include <stdint.h>
#include <vector>
#include <algorithm>
#include <random>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

#define CHECK(x) do { hipError_t e_ = (x); if (e_ != hipSuccess) { printf("HIP error %s at %d\n", hipGetErrorString(e_), __LINE__); exit(1); } } while (0)

__device__ __forceinline__ uint32_t bf16_trunc(float f) { return __float_as_uint(f) >> 16; }

template <int MODE, int G>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2)))
probe(const uint16_t* __restrict__ pool, const int* __restrict__ perm, const float* __restrict__ q,
      float* __restrict__ out, int n_units, int LHkv) {
    __shared__ uint32_t qs[2][3][G][64];
    __shared__ float qf[2][G][128];
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int h = lane & 15, g = lane >> 4, hh = h < G ? h : G - 1;
    const uint32_t voff = 16u * lane;
    float best = -INFINITY;
    for (int unit = blockIdx.x; unit < n_units; unit += gridDim.x) {
        int page[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) page[u] = perm[unit * 16 + wv * 4 + u];
        auto load_tile = [&](u32x4 (&rg)[4], int r, int u) {
            const int rr = r < LHkv ? r : 0;
            const unsigned char* base = reinterpret_cast<const unsigned char*>(pool) +
                                        (((size_t)page[u] * LHkv + rr) * 16) * 128 * 2;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                rg[j] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(base + voff + 1024 * j));
        };
        auto stage_q = [&](int r) {   // row r's G heads into LDS buffer r & 1
            const int rr = r < LHkv ? r : 0;
            for (int i = threadIdx.x; i < G * 128; i += 256) {
                const float v = q[(size_t)rr * G * 128 + i];
                const int hd = i >> 7, d = i & 127;
                qf[r & 1][hd][d] = v;
                const uint32_t hi = bf16_trunc(v);
                const float r1 = v - __uint_as_float(hi << 16);
                const uint32_t mid = bf16_trunc(r1);
                const float r2 = r1 - __uint_as_float(mid << 16);
                const uint32_t lo = bf16_trunc(r2);
                uint16_t* p0 = reinterpret_cast<uint16_t*>(&qs[r & 1][0][hd][0]);
                uint16_t* p1 = reinterpret_cast<uint16_t*>(&qs[r & 1][1][hd][0]);
                uint16_t* p2 = reinterpret_cast<uint16_t*>(&qs[r & 1][2][hd][0]);
                p0[d] = (uint16_t)hi;
                p1[d] = (uint16_t)mid;
                p2[d] = (uint16_t)lo;
            }
        };
        u32x4 ringA[4][4], ringB[4][4];
        __syncthreads();
        stage_q(0);
#pragma unroll
        for (int u = 0; u < 4; ++u) load_tile(ringA[u], 0, u);
#pragma unroll
        for (int u = 0; u < 4; ++u) load_tile(ringB[u], 1, u);
        __syncthreads();
        auto do_row = [&](u32x4 (&ring)[4][4], int row) {
            if constexpr (MODE == 1) {
                const uint32_t* qb = &qs[row & 1][0][hh][4 * g];
                f32x4 c[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) c[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    u32x4 bq[3];
#pragma unroll
                    for (int p = 0; p < 3; ++p) bq[p] = *reinterpret_cast<const u32x4*>(qb + p * G * 64 + 16 * j);
#pragma unroll
                    for (int u = 0; u < 4; ++u)
#pragma unroll
                        for (int p = 0; p < 3; ++p)
                            c[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, ring[u][j]),
                                                                           __builtin_bit_cast(bf16x8, bq[p]), c[u], 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < 4; ++u)
                    best = fmaxf(best, fmaxf(fmaxf(c[u][0], c[u][1]), fmaxf(c[u][2], c[u][3])));
            } else {
                // lane (token h, dims block g): dims 32 j + 8 g .. +7 of token h
                for (int hd = 0; hd < G; ++hd) {
                    float qv[4][8];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const f32x4 a = *reinterpret_cast<const f32x4*>(&qf[row & 1][hd][32 * j + 8 * g]);
                        const f32x4 b = *reinterpret_cast<const f32x4*>(&qf[row & 1][hd][32 * j + 8 * g + 4]);
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            qv[j][e] = a[e];
                            qv[j][4 + e] = b[e];
                        }
                    }
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        float acc = 0.0f;
#pragma unroll
                        for (int j = 0; j < 4; ++j)
#pragma unroll
                            for (int w = 0; w < 4; ++w) {
                                const uint32_t x = ring[u][j][w];
                                acc = fmaf(__uint_as_float(x << 16), qv[j][2 * w], acc);
                                acc = fmaf(__uint_as_float(x & 0xffff0000u), qv[j][2 * w + 1], acc);
                            }
                        acc += __shfl_xor(acc, 16);
                        acc += __shfl_xor(acc, 32);
                        best = fmaxf(best, acc);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) load_tile(ring[u], row + 2, u);
            if (row + 1 < LHkv) stage_q(row + 1);
            __syncthreads();
        };
        int row = 0;
        for (; row + 1 < LHkv; row += 2) {
            do_row(ringA, row);
            do_row(ringB, row + 1);
        }
        if (row < LHkv) do_row(ringA, row);
    }
    out[blockIdx.x * 256 + threadIdx.x] = best;
}

__global__ void fill(uint16_t* p, size_t n, uint32_t seed) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
        uint32_t x = (uint32_t)i * 2654435761u ^ seed;
        x ^= x >> 13; x *= 0x5bd1e995u; x ^= x >> 15;
        const float f = ((float)(x & 0xffff) / 65536.0f - 0.5f) * 3.0f;
        p[i] = (uint16_t)(__float_as_uint(f) >> 16);
    }
}

template <int MODE, int G>
float run(const uint16_t* pool, const int* perm, const float* q, float* out, int n_units, int LHkv, int reps) {
    hipEvent_t a, b;
    CHECK(hipEventCreate(&a));
    CHECK(hipEventCreate(&b));
    probe<MODE, G><<<512, 256>>>(pool, perm, q, out, n_units, LHkv);
    CHECK(hipGetLastError());
    CHECK(hipDeviceSynchronize());
    CHECK(hipEventRecord(a));
    for (int i = 0; i < reps; ++i) probe<MODE, G><<<512, 256>>>(pool, perm, q, out, n_units, LHkv);
    CHECK(hipEventRecord(b));
    CHECK(hipEventSynchronize(b));
    float ms = 0;
    CHECK(hipEventElapsedTime(&ms, a, b));
    return ms / reps;
}

template <int G>
void shape(int L, int n_pages) {
    const int LHkv = L * 2;
    const size_t elems = (size_t)n_pages * LHkv * 16 * 128;
    uint16_t* pool;
    CHECK(hipMalloc(&pool, elems * 2));
    fill<<<4096, 256>>>(pool, elems, 12345u);
    std::vector<int> hp(n_pages);
    for (int i = 0; i < n_pages; ++i) hp[i] = i;
    std::mt19937 rng(7);
    std::shuffle(hp.begin(), hp.end(), rng);
    int* perm;
    CHECK(hipMalloc(&perm, n_pages * sizeof(int)));
    CHECK(hipMemcpy(perm, hp.data(), n_pages * sizeof(int), hipMemcpyHostToDevice));
    std::vector<float> hq((size_t)LHkv * G * 128);
    for (auto& v : hq) v = std::normal_distribution<float>(0.f, 1.f)(rng);
    float* q;
    CHECK(hipMalloc(&q, hq.size() * 4));
    CHECK(hipMemcpy(q, hq.data(), hq.size() * 4, hipMemcpyHostToDevice));
    float* out;
    CHECK(hipMalloc(&out, 512 * 256 * 4));
    const int n_units = n_pages / 16;   // n_pages is a multiple of 16
    const double bytes = (double)elems * 2;
    const float t1 = run<1, G>(pool, perm, q, out, n_units, LHkv, 10);
    const float t2 = run<2, G>(pool, perm, q, out, n_units, LHkv, 10);
    printf("G=%d L=%d pages=%d (%.2f GB of keys, %d units): MFMA %.1f us (%.2f TB/s)  GEMV %.1f us (%.2f TB/s)\n",
           G, L, n_pages, bytes / 1e9, n_units, t1 * 1e3, bytes / t1 / 1e9, t2 * 1e3, bytes / t2 / 1e9);
    CHECK(hipFree(pool));
    CHECK(hipFree(perm));
    CHECK(hipFree(q));
    CHECK(hipFree(out));
}

int main() {
    shape<6>(28, 8192);     // 1.5B shape, one unit per workgroup (the 32k batch's steady step)
    shape<6>(28, 32768);    // four units per workgroup
    shape<8>(36, 8192);     // 3B shape
    shape<8>(36, 32768);
    return 0;
}
