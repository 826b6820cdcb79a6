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

// Inclusive prefix sum over the 64 lanes of a wave with DPP moves: shifts
// by 1, 2, 4 and 8 lanes inside each row of 16, then the last lane of each
// row added to the rows after it (row broadcasts of lanes 15 and 31).  A
// lane whose source lies outside its row, or whose row the mask leaves out,
// adds the identity.
__device__ __forceinline__ int wave_incl_sum(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);   // row_bcast:15 into rows 1, 3
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);   // row_bcast:31 into rows 2, 3
    return v;
}

// Minimum over the 64 lanes of a wave (the same DPP steps; the last lane
// ends with the minimum of all, read back to every lane).
template <int Ctrl, int RowMask>
__device__ __forceinline__ uint32_t dpp_min_step(uint32_t v) {
    // -1 = 0xFFFFFFFF, the identity of the unsigned minimum
    const uint32_t o = (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, Ctrl, RowMask, 0xf, false);
    return v < o ? v : o;
}

__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
    v = dpp_min_step<0x111, 0xf>(v);
    v = dpp_min_step<0x112, 0xf>(v);
    v = dpp_min_step<0x114, 0xf>(v);
    v = dpp_min_step<0x118, 0xf>(v);
    v = dpp_min_step<0x142, 0xa>(v);
    v = dpp_min_step<0x143, 0xc>(v);
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// N exclusive block-wide scans side by side (any multiple of 64 threads up
// to 1024; lds: 17 N ints).  Each wave scans its lanes (DPP) and publishes
// its total; after one barrier every wave scans the (at most 16) wave totals
// itself, so no thread walks them serially.  Ends with a barrier, after
// which lds may be reused.
template <int N>
__device__ inline void block_exclusive_scan_n(const int (&v)[N], int* lds, int (&ex)[N], int (&total)[N]) {
    const int lane = lane_id(), wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
    int incl[N];
#pragma unroll
    for (int k = 0; k < N; ++k) incl[k] = wave_incl_sum(v[k]);
    if (lane == 63)
#pragma unroll
        for (int k = 0; k < N; ++k) lds[17 * k + wid] = incl[k];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < N; ++k) {
        const int t = wave_incl_sum(lane < nw ? lds[17 * k + lane] : 0);
        const int before = __builtin_amdgcn_readlane(t, wid > 0 ? wid - 1 : 0);
        ex[k] = (wid > 0 ? before : 0) + incl[k] - v[k];
        total[k] = __builtin_amdgcn_readlane(t, nw - 1);
    }
    __syncthreads();
}

// Exclusive prefix of one int per thread across the whole block; *total is
// the block's sum.  lds needs 17 ints.  Ends with a barrier.
__device__ inline int block_exclusive_scan(int v, int* lds, int* total) {
    const int m[1] = {v};
    int ex[1], tot[1];
    block_exclusive_scan_n<1>(m, lds, ex, tot);
    *total = tot[0];
    return ex[0];
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
// values in the MFMA operand order.  One instruction widens two codes to a
// pair of bf16 values (scale 1): E4M3 values have four significant bits and
// exponents inside bf16's range, so the conversion is exact, and the
// product with the query stays exact.
template <bool HIGH>
__device__ __forceinline__ uint32_t codes_pair_to_bf16(uint32_t x) {
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(x, 1.0f, HIGH));
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
