// Device helpers shared by the gfx950 kernels of the retention step.
#pragma once

#include <math.h>

#include "md_internal.h"

namespace md {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// log2(e) / sqrt(128): logits are kept in base 2 so that 2^(x - m) is the
// softmax numerator exp(q.k/sqrt(d) - m').
constexpr float kLogitScale = (float)(1.4426950408889634074 / 11.313708498984760390);

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// 2^x on the transcendental unit (v_exp_f32, about 1 ulp).  Results below
// 2^-126 come out as zero or denormal; softmax weights that small are
// negligible next to the row maximum's weight of 1.
__device__ __forceinline__ float hw_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
    return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__device__ __forceinline__ int load_agent(const int32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive prefix of one int per thread across the whole block (any multiple
// of 64 threads up to 1024).  lds needs 17 ints.  Contains __syncthreads.
// N exclusive block-wide scans side by side, with one pair of barriers
// (lds: 17 N ints).
template <int N>
__device__ inline void block_exclusive_scan_n(const int (&v)[N], int* lds, int (&ex)[N], int (&total)[N]) {
    const int lane = lane_id(), wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int incl[N];
#pragma unroll
    for (int k = 0; k < N; ++k) incl[k] = v[k];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1)
#pragma unroll
        for (int k = 0; k < N; ++k) {
            const int t = __shfl_up(incl[k], o);
            if (lane >= o) incl[k] += t;
        }
    if (lane == 63)
#pragma unroll
        for (int k = 0; k < N; ++k) lds[17 * k + wid] = incl[k];
    __syncthreads();
    if ((int)threadIdx.x < N) {
        int* l = lds + 17 * threadIdx.x;
        int acc = 0;
        for (int w = 0; w < nw; ++w) {
            const int t = l[w];
            l[w] = acc;
            acc += t;
        }
        l[16] = acc;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < N; ++k) {
        ex[k] = lds[17 * k + wid] + incl[k] - v[k];
        total[k] = lds[17 * k + 16];
    }
    __syncthreads();
}

__device__ inline int block_exclusive_scan(int v, int* lds, int* total) {
    const int lane = lane_id(), wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int t = __shfl_up(incl, o);
        if (lane >= o) incl += t;
    }
    if (lane == 63) lds[wid] = incl;
    __syncthreads();
    if (threadIdx.x == 0) {
        int acc = 0;
        for (int w = 0; w < nw; ++w) {
            const int t = lds[w];
            lds[w] = acc;
            acc += t;
        }
        lds[16] = acc;
    }
    __syncthreads();
    const int res = lds[wid] + incl - v;
    *total = lds[16];
    __syncthreads();
    return res;
}

// Largest s in [0, S) with pref[s] <= x, given pref[0] <= x < pref[S].
__device__ __forceinline__ int find_session(const int* pref, int S, int x) {
    int lo = 0, hi = S;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (pref[mid] <= x) lo = mid; else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ bool counters_ok(int np, int nt, const Dims& dm) {
    if (np < 0 || np > dm.MP) return false;
    if (np == 0) return nt == 0;
    return nt > (np - 1) * dm.P && nt <= np * dm.P;
}

// Split a float32 into three bfloat16 terms with x == hi + mid + lo exactly:
// hi and mid truncate (the differences are exact by Sterbenz's lemma), and
// what is left has at most 8 significant bits, so lo holds it exactly.
__device__ __forceinline__ void split3(float x, uint32_t& hi, uint32_t& mid, uint32_t& lo) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t h = u & 0xFFFF0000u;
    const float r1 = x - __uint_as_float(h);
    const uint32_t m = __float_as_uint(r1) & 0xFFFF0000u;
    const float r2 = r1 - __uint_as_float(m);
    hi = h >> 16;
    mid = m >> 16;
    lo = __float_as_uint(r2) >> 16;
}


// Retention score of an unpinned token (Eq. 4): base priority b and decay
// rate lam of its region, age t - t_ref, importance a.
__device__ __forceinline__ float retention_score(float b, float lam, int t, int t_ref, float alpha, float a) {
    return b * expf(-lam * (float)(t - t_ref)) + alpha * a;
}

// Page score (Eq. 5) over the P consecutive lanes that hold one page's
// tokens: the mean of the unpinned members' scores, +inf when any member is
// pinned.  Returns false when the page has no live member.  Every lane of
// the page gets the same bits.
__device__ __forceinline__ bool page_score_of(float score, bool live, bool pinned, int P, float* out) {
    float sum = (live && !pinned) ? score : 0.0f;
    int cnt = live ? 1 : 0;
    int anyp = pinned ? 1 : 0;
    for (int o = 1; o < P; o <<= 1) {
        sum += __shfl_xor(sum, o);
        cnt += __shfl_xor(cnt, o);
        anyp |= __shfl_xor(anyp, o);
    }
    *out = anyp ? INFINITY : sum / (float)cnt;
    return cnt > 0;
}

// Eight FP8 E4M3 key codes (bytes 8 half .. 8 half + 7 of v) as eight bf16
// values in the MFMA operand order.  The hardware widens two codes at a time
// to float32 (exactly); E4M3 values have four significant bits, so their
// bf16 halves are exact too, and the product with the query stays exact.
template <bool HIGH>
__device__ __forceinline__ uint32_t codes_pair_to_bf16(uint32_t x) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    const f32x2 f = __builtin_amdgcn_cvt_pk_f32_fp8((int)x, HIGH);
    return (__float_as_uint(f[0]) >> 16) | (__float_as_uint(f[1]) & 0xffff0000u);
}
template <int HALF>
__device__ __forceinline__ u32x4 codes_to_bf16(u32x4 v) {
    const uint32_t w0 = HALF ? v[2] : v[0], w1 = HALF ? v[3] : v[1];
    return u32x4{codes_pair_to_bf16<false>(w0), codes_pair_to_bf16<true>(w0), codes_pair_to_bf16<false>(w1),
                 codes_pair_to_bf16<true>(w1)};
}

// The FP8 E4M3 code (OCP: bias 7, no infinities) nearest to v, ties to even,
// magnitudes above 448 saturating to 448; the sign bit is set for v < 0.
// Exact steps only: a power-of-two scaling, Sterbenz subtraction, rint.
__device__ __forceinline__ uint32_t e4m3_encode(float v) {
    const uint32_t sign = v < 0.0f ? 0x80u : 0u;
    const float a = fabsf(v);
    uint32_t bits;
    if (a < 0.015625f) {                 // below 2^-6: steps of 2^-9; 8 is the smallest normal
        bits = (uint32_t)rintf(a * 512.0f);
    } else {
        int ex;
        const float m = frexpf(a, &ex);  // a = m 2^ex, m in [0.5, 1)
        int q = (int)rintf((2.0f * m - 1.0f) * 8.0f);
        int e = ex - 1;
        if (q == 8) {
            q = 0;
            e += 1;
        }
        bits = min((uint32_t)(((e + 7) << 3) | q), 0x7Eu);
    }
    return sign | bits;
}

// Weight of the attention term of Eq. 4: alpha, or alpha * |K_t| when the
// term is measured against the uniform attention level 1/|K_t|.
__device__ __forceinline__ float attention_weight(float alpha, int norm, int n_tokens) {
    return norm ? alpha * (float)n_tokens : alpha;
}

// Wave-uniform value kept in a scalar register.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

typedef const __attribute__((address_space(1))) uint8_t* gbytes;
typedef const __attribute__((address_space(1))) u32x4* gvec;

// A wave-uniform global pointer held in scalar registers.
__device__ __forceinline__ gbytes uni_ptr(const void* p) {
    const uint64_t u = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
    return (gbytes)(((uint64_t)hi << 32) | lo);
}

}  // namespace md
