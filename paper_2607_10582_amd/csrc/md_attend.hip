// gfx950 fused observation kernel: attention mass (Sec. III-C), EWMA (Eq. 2)
// and refresh (Eq. 3) of every cached token in one pass over the key cache,
// with the logits of the step held in LDS instead of HBM.
//
// The attention mass of token i averages, over every (layer, query head) row,
// the token's softmax weight in that row.  A row's softmax needs the row's
// maximum and sum over all of the session's tokens, so the logits of a block
// of tokens cannot be normalised where they are produced.  Here a session's
// tokens are split into units of T tokens, one workgroup per unit, all units
// of a session resident at once.  Each workgroup walks the (layer, KV head)
// rows in order: it computes the logits of its tokens for the G query heads of
// the row on MFMA, keeps them in an LDS ring of kRowBufs rows, publishes the
// row's (max, sum) to the other units of the session, and kConsumeLag rows
// later, when every unit's statistics of that row are in, turns the held
// logits into softmax weights and adds them to its tokens' mass.  The key
// cache is read once and nothing per (token, row) is written back.
//
// Workgroup = kProducers producer waves + one manager wave.
//   producers  own 16-token tiles of the unit; stream K tiles through a
//              four-deep register ring across row boundaries, MFMA, write
//              base-2 logits into the LDS ring, keep per-lane (max, sum),
//              and at each row end hand the row statistics to the manager and
//              normalise the row kConsumeLag rows back.
//   manager    stages the query terms of upcoming rows in LDS, merges the
//              producers' row statistics and publishes them with a tag.  The
//              manager of the session's first unit (the leader) gathers all
//              units' statistics of the previous row into the row normaliser
//              (max M, 1 / sum) and publishes it; the other managers read it
//              a row later.  Traffic per row is linear in the unit count.
// Producer <-> manager hand-offs are LDS counters; unit <-> unit hand-offs are
// 64-bit words (tag << 32 | float bits, the tag being the step's epoch)
// written and polled with agent-scope atomics, so a word is either absent or
// complete.  Every wait is bounded; a
// wait that runs out sets MD_DEV_TIMEOUT and stops all further waits of the
// workgroup, so the grid always drains.

#include "md_device.h"

namespace md {

namespace {

struct AttendDims {
    int L, Hq, Hkv, G, P, Pshift, MP, NP, R, LHkv, Tstride, U_cap;
    float rho, tau_scale;
};

struct AttendArgs {
    const uint16_t* k_pool;
    const int32_t* page_table;
    const int32_t* n_tokens;
    const int32_t* clock;
    float* imp;
    int32_t* t_ref;
    const float* q;
    float* abar_out;
    const int32_t* ustart;
    const int32_t* plan;
    const int32_t* epoch;
    unsigned long long* ustat;
    unsigned long long* nstat;
    int32_t* status;
    int32_t* probe;    // check mode only: [arrivals, least seen]
};

// LDS flags: rows finished by each producer (one counter per producer: the
// producers drift apart by up to a few rows, so a shared count could reach
// a target while one of them is still short), query rows staged, rows
// normalised, stop.
enum { kFlagProd = 0, kFlagQ = kProducers, kFlagNorm = kProducers + 1, kFlagStop = kProducers + 2,
       kFlagCount = kProducers + 3 };

struct Lds {
    float* rowbuf;    // [kRowBufs][G][Tstride] base-2 logits of the held rows
    uint32_t* qs;     // [2][3][G][64] hi, mid, lo bf16 query terms (pairs) of two rows
    float* qraw;      // [2][qraw_floats(G)] float32 query rows as loaded
    float2* wstat;    // [kStatBufs][kProducers][16] producer row statistics
    float2* norm;     // [kNormBufs][16] row normalisers (M, 1 / Lambda)
    int* flags;       // [kFlagCount]
};

__host__ __device__ inline size_t rowbuf_bytes(int G, int Tstride) {
    return (size_t)kRowBufs * G * Tstride * sizeof(float);
}
__host__ __device__ inline size_t qs_bytes(int G) { return (size_t)2 * 3 * G * 64 * sizeof(uint32_t); }
// A query row (G heads x 128 floats) rounded up to whole 64-lane x 16-byte
// direct-to-LDS loads.
__host__ __device__ inline int qraw_floats(int G) { return (G * kHeadDim + 255) / 256 * 256; }
constexpr size_t kWstatBytes = (size_t)kStatBufs * kProducers * 16 * sizeof(float2);
constexpr size_t kNormBytes = (size_t)kNormBufs * 16 * sizeof(float2);
constexpr size_t kFlagBytes = 8 * sizeof(int);
static_assert(kFlagCount <= 8, "LDS flag words");

__device__ __forceinline__ Lds carve(unsigned char* smem, int G, int Tstride) {
    Lds l;
    size_t o = 0;
    l.rowbuf = reinterpret_cast<float*>(smem + o);
    o += rowbuf_bytes(G, Tstride);
    l.qs = reinterpret_cast<uint32_t*>(smem + o);
    o += qs_bytes(G);
    l.qraw = reinterpret_cast<float*>(smem + o);
    o += (size_t)2 * qraw_floats(G) * sizeof(float);
    l.wstat = reinterpret_cast<float2*>(smem + o);
    o += kWstatBytes;
    l.norm = reinterpret_cast<float2*>(smem + o);
    o += kNormBytes;
    l.flags = reinterpret_cast<int*>(smem + o);
    return l;
}

// LDS hand-offs inside the workgroup use workgroup-scope acquire / release;
// on gfx950 these order LDS accesses only (lgkmcnt waits) and leave the
// global loads in flight untouched.
__device__ __forceinline__ int lds_get(int* p) {
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void lds_publish(int* p, int v) {
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Wait until *p >= target.  False when the wait ran out or the workgroup
// stopped waiting after an earlier time-out.
// Time limits of the waits, in ticks of the 100 MHz real-time counter.
// Waits inside a workgroup outlast waits on other workgroups, so a stalled
// session is reported by the wait that polls the other units.
constexpr uint64_t kLdsWaitTicks = 40000000ull;      // 400 ms
constexpr uint64_t kGlobalWaitTicks = 20000000ull;   // 200 ms

__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

__device__ __forceinline__ void stop_all(int* flags, int32_t* status) {
    __hip_atomic_store(flags + kFlagStop, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    atomicOr(status, MD_DEV_TIMEOUT);
}

__device__ __forceinline__ bool lds_wait(int* p, int target, int* flags, int32_t* status) {
    if (lds_get(p) >= target) return true;
    const uint64_t t0 = now_ticks();
    while (lds_get(p) < target) {
        if (lds_get(flags + kFlagStop)) return false;
        if (now_ticks() - t0 > kLdsWaitTicks) {
            stop_all(flags, status);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    return true;
}

__device__ __forceinline__ void merge_stat(float& m, float& l, float m2, float l2) {
    const float M = fmaxf(m, m2);
    l = (M == -INFINITY) ? 0.0f : l * hw_exp2(m - M) + l2 * hw_exp2(m2 - M);
    m = M;
}

struct Unit {
    int s, j, T, kt, ntok, nt_s, nu, us;
};

// First query row (layer * Hq + KV head * G) of (layer, KV head) row r.
__device__ __forceinline__ int qrow0(const AttendDims& dm, int r) {
    const int l = r / dm.Hkv;
    return l * dm.Hq + (r - l * dm.Hkv) * dm.G;
}

// ------------------------------------------------------------ producer

__device__ __forceinline__ void producer(const AttendDims& dm, const AttendArgs& a, const Lds& sm,
                                         const Unit& un, int wv) {
    const int lane = lane_id();
    const int h = lane & 15;          // MFMA column: query head of the group
    const int g = lane >> 4;          // k-group of A/B, row quad of C
    const int hh = min(h, dm.G - 1);  // in-bounds head for the unused columns
    const uint32_t voff = 256u * h + 16u * g;
    const int kt = un.kt;
    const int wtok0 = wv * kt * 16;   // first unit-local token of this producer
    int* flags = sm.flags;

    // lane i < kt: slot (physical page * P + offset) of tile i's first token
    int myslot = 0;
    bool myok = false;
    if (lane < kt) {
        const int tok = un.j * un.T + wtok0 + 16 * lane;
        if (tok < un.nt_s) {
            const int p = a.page_table[(size_t)un.s * dm.MP + (tok >> dm.Pshift)];
            if ((unsigned)p < (unsigned)dm.NP) {
                myslot = (p << dm.Pshift) + (tok & (dm.P - 1));
                myok = true;
            } else {
                atomicOr(a.status, kDevCorrupt);
            }
        }
    }
    const unsigned long long vmask = __ballot(myok);

    // K tile (row, tile) in the MFMA A layout; a tile without cached tokens,
    // or past the last row, reads the pool's first tile (its logits are
    // masked), so loads never branch.
    int lrow = 0, lti = 0;
    auto load_next = [&](u32x4 (&r)[4]) {
        const bool ok = lrow < dm.LHkv && ((vmask >> lti) & 1ull);
        const int slot = __builtin_amdgcn_readlane(myslot, lti);
        const size_t e = ok ? ((size_t)(slot >> dm.Pshift) * dm.LHkv + lrow) * dm.P + (slot & (dm.P - 1)) : 0;
        gbytes base = uni_ptr(a.k_pool + e * kHeadDim);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            r[j] = __builtin_nontemporal_load(reinterpret_cast<gvec>(base + voff + 64 * j));
        if (++lti == kt) {
            lti = 0;
            ++lrow;
        }
    };

    u32x4 bq[4][3];
    auto read_bq = [&](int r) {
        const uint32_t* qb = sm.qs + (size_t)(r & 1) * 3 * dm.G * 64;
#pragma unroll
        for (int p = 0; p < 3; ++p)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                bq[j][p] = *reinterpret_cast<const u32x4*>(qb + (p * dm.G + hh) * 64 + 16 * j + 4 * g);
    };

    float acc_tok[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    const int my_tokens = kt * 16;
    auto consume = [&](int rc) {
        lds_wait(flags + kFlagNorm, rc + 1, flags, a.status);
        const float* rb = sm.rowbuf + (size_t)(rc % kRowBufs) * dm.G * dm.Tstride;
        const float2* nm = sm.norm + (rc % kNormBufs) * 16;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int lt = lane + 64 * k;
            if (lt < my_tokens && wtok0 + lt < un.ntok) {
                float sum = 0.0f;
                for (int hd = 0; hd < dm.G; ++hd) {
                    const float2 n = nm[hd];
                    sum += hw_exp2(rb[hd * dm.Tstride + wtok0 + lt] - n.x) * n.y;
                }
                acc_tok[k] += sum;
            }
        }
    };

    lds_wait(flags + kFlagQ, 1, flags, a.status);
    read_bq(0);
    u32x4 ring[4][4];
#pragma unroll
    for (int u = 0; u < 4; ++u) load_next(ring[u]);

    int row = 0, ti = 0;
    float m = -INFINITY, lsum = 0.0f;
    const int n_loop = (kt * dm.LHkv + 3) & ~3;
    for (int n = 0; n < n_loop; n += 4) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            f32x4 c = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
#pragma unroll
                for (int p = 0; p < 3; ++p)
                    c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, ring[u][j]), __builtin_bit_cast(bf16x8, bq[j][p]), c, 0, 0,
                        0);
            }
            load_next(ring[u]);
            if (row < dm.LHkv) {
                const int lt0 = wtok0 + 16 * ti + 4 * g;   // unit-local token of c[0]
                const bool tok_ok = (vmask >> ti) & 1ull;
                float x[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) x[i] = (tok_ok && lt0 + i < un.ntok) ? c[i] * kLogitScale : -INFINITY;
                const float mn = fmaxf(m, fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
                const bool live = mn != -INFINITY;
                const float ms = live ? mn : 0.0f;
                const float part = (hw_exp2(x[0] - ms) + hw_exp2(x[1] - ms)) +
                                   (hw_exp2(x[2] - ms) + hw_exp2(x[3] - ms));
                lsum = live ? lsum * hw_exp2(m - ms) + part : lsum;
                m = live ? mn : m;
                if (h < dm.G)
                    *reinterpret_cast<f32x4*>(sm.rowbuf + ((size_t)(row % kRowBufs) * dm.G + h) * dm.Tstride + lt0) =
                        f32x4{x[0], x[1], x[2], x[3]};
                if (++ti == kt) {
                    // row end: hand the row's statistics to the manager
#pragma unroll
                    for (int o = 16; o <= 32; o <<= 1) merge_stat(m, lsum, __shfl_xor(m, o), __shfl_xor(lsum, o));
                    if (g == 0 && h < dm.G)
                        sm.wstat[((row % kStatBufs) * kProducers + wv) * 16 + h] = make_float2(m, lsum);
                    m = -INFINITY;
                    lsum = 0.0f;
                    if (lane == 0) lds_publish(flags + kFlagProd + wv, row + 1);
                    if (row + 1 < dm.LHkv) {
                        lds_wait(flags + kFlagQ, row + 2, flags, a.status);
                        read_bq(row + 1);
                    }
                    if (row >= kConsumeLag) consume(row - kConsumeLag);
                    ti = 0;
                    ++row;
                }
            }
        }
    }
    for (int rc = max(0, dm.LHkv - kConsumeLag); rc < dm.LHkv; ++rc) consume(rc);

    // Eq. 2 and Eq. 3 for this producer's tokens.
    const float one_m_rho = 1.0f - dm.rho;
    const float tau = dm.tau_scale / (float)un.nt_s;
    const int t_now = a.clock[un.s];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int lt = lane + 64 * k;
        const int tile = min(lt >> 4, 63);
        const int slot0 = __shfl(myslot, tile);
        if (lt < my_tokens && wtok0 + lt < un.ntok && ((vmask >> tile) & 1ull)) {
            const float abar = acc_tok[k] / (float)dm.R;
            const size_t si = (size_t)slot0 + (lt & 15);
            a.imp[si] = fmaf(dm.rho, a.imp[si], one_m_rho * abar);
            if (abar >= tau) a.t_ref[si] = t_now;
            if (a.abar_out != nullptr) a.abar_out[si] = abar;
        }
    }
}

// ------------------------------------------------------------ manager

__device__ __forceinline__ void manager(const AttendDims& dm, const AttendArgs& a, const Lds& sm,
                                        const Unit& un, uint32_t tag) {
    const int lane = lane_id();
    int* flags = sm.flags;
    const int G = dm.G;

    // Query row r: G heads x 128 floats, copied straight into LDS (no
    // registers held while the copy is in flight), then split into the three
    // bf16 terms the producers' B operands take.
    const int qn = G * kHeadDim;
    auto load_q = [&](int r) {
        const float* qr = a.q + ((size_t)un.s * dm.L * dm.Hq + qrow0(dm, r)) * kHeadDim;
        float* dst = sm.qraw + (size_t)(r & 1) * qraw_floats(G);
        for (int i = 0; i < qraw_floats(G); i += 256) {
            const int f = i + 4 * lane;
            const float* src = qr + (f < qn ? f : 0);
            __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                             (__attribute__((address_space(3))) void*)(dst + i), 16, 0, 0);
        }
    };
    auto store_q = [&](int r) {
        __builtin_amdgcn_s_waitcnt(0x0f70);   // vmcnt(0): the direct-to-LDS copy has landed
        const float* src = sm.qraw + (size_t)(r & 1) * qraw_floats(G);
        uint32_t* qb = sm.qs + (size_t)(r & 1) * 3 * G * 64;
        bool bad = false;
#pragma unroll 1
        for (int f = lane; f < G * 32; f += 64) {
            const f32x4 x = *reinterpret_cast<const f32x4*>(src + 4 * f);
            const int hd = f >> 5, d2 = 2 * (f & 31);
            uint32_t t[3][4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                bad |= !isfinite(x[e]);
                split3(x[e], t[0][e], t[1][e], t[2][e]);
            }
#pragma unroll
            for (int p = 0; p < 3; ++p)
                *reinterpret_cast<uint2*>(qb + (p * G + hd) * 64 + d2) =
                    make_uint2(t[p][0] | (t[p][1] << 16), t[p][2] | (t[p][3] << 16));
        }
        if (bad) atomicOr(a.status, MD_DEV_NONFINITE);
    };

    // Bounded poll of tagged words until every active lane holds words with
    // this step's tag; false after a time-out (or a stop seen).
    auto poll_words = [&](auto&& load_all) -> bool {
        if (__all(load_all())) return true;
        const uint64_t t0 = now_ticks();
        while (true) {
            __builtin_amdgcn_s_sleep(8);   // back off: many units may poll the same words
            if (__all(load_all())) return true;
            if (lds_get(flags + kFlagStop)) return false;
            if (now_ticks() - t0 > kGlobalWaitTicks) {
                stop_all(flags, a.status);
                return false;
            }
        }
    };
    auto set_norm = [&](int rc, int hd, float M, float inv) {
        sm.norm[(rc % kNormBufs) * 16 + hd] = make_float2(M, inv);
    };
    const unsigned long long hi_tag = (unsigned long long)tag << 32;

    // Leader (unit 0 of the session): every unit's statistics of row rc ->
    // the row normaliser, eight heads at a time (lane k holds units k, k + 64,
    // ...; a butterfly merges the lanes), published to the session's other
    // units as tagged words and kept for this workgroup.
    auto lead = [&](int rc) {
        const int r0 = qrow0(dm, rc);
        for (int h0 = 0; h0 < G; h0 += 8) {
            float Mh[8], Lh[8];
#pragma unroll
            for (int hd = 0; hd < 8; ++hd) {
                Mh[hd] = -INFINITY;
                Lh[hd] = 0.0f;
            }
            for (int c0 = 0; c0 < un.nu; c0 += 64) {
                const int k = c0 + lane;
                const bool act = k < un.nu;
                unsigned long long* p = a.ustat + (((size_t)(un.us + (act ? k : 0)) * dm.R + r0 + h0) << 1);
                unsigned long long w[8][2];
                poll_words([&]() {
                    bool ok = true;
#pragma unroll
                    for (int hd = 0; hd < 8; ++hd) {
                        if (h0 + hd < G && act) {
                            w[hd][0] = __hip_atomic_load(p + 2 * hd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            w[hd][1] = __hip_atomic_load(p + 2 * hd + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        }
                    }
#pragma unroll
                    for (int hd = 0; hd < 8; ++hd)
                        if (h0 + hd < G && act)
                            ok &= (uint32_t)(w[hd][0] >> 32) == tag && (uint32_t)(w[hd][1] >> 32) == tag;
                    return ok;
                });
#pragma unroll
                for (int hd = 0; hd < 8; ++hd)
                    if (h0 + hd < G && act)
                        merge_stat(Mh[hd], Lh[hd], __uint_as_float((uint32_t)w[hd][0]),
                                   __uint_as_float((uint32_t)w[hd][1]));
            }
            float mine_m = 0.0f, mine_l = 1.0f;
#pragma unroll
            for (int hd = 0; hd < 8; ++hd) {
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) merge_stat(Mh[hd], Lh[hd], __shfl_xor(Mh[hd], o), __shfl_xor(Lh[hd], o));
                if (lane == hd) {
                    mine_m = Mh[hd];
                    mine_l = Lh[hd];
                }
            }
            if (lane < 8 && h0 + lane < G) {
                const float inv = 1.0f / mine_l;
                set_norm(rc, h0 + lane, mine_m, inv);
                if (un.nu > 1) {
                    unsigned long long* q = a.nstat + (((size_t)un.s * dm.R + r0 + h0 + lane) << 1);
                    __hip_atomic_store(q, hi_tag | __float_as_uint(mine_m), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(q + 1, hi_tag | __float_as_uint(inv), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        }
        lds_publish(flags + kFlagNorm, rc + 1);
    };

    // Other units: the leader's normaliser of row rc.
    auto follow = [&](int rc) {
        const int r0 = qrow0(dm, rc);
        const bool act = lane < G;
        unsigned long long* q = a.nstat + (((size_t)un.s * dm.R + r0 + (act ? lane : 0)) << 1);
        unsigned long long w0 = 0, w1 = 0;
        poll_words([&]() {
            if (!act) return true;
            w0 = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            w1 = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return (uint32_t)(w0 >> 32) == tag && (uint32_t)(w1 >> 32) == tag;
        });
        if (act) set_norm(rc, lane, __uint_as_float((uint32_t)w0), __uint_as_float((uint32_t)w1));
        lds_publish(flags + kFlagNorm, rc + 1);
    };

    const bool leader = un.j == 0;
    load_q(0);
    store_q(0);
    if (dm.LHkv > 1) {
        load_q(1);
        store_q(1);
    }
    lds_publish(flags + kFlagQ, min(2, dm.LHkv));
    if (dm.LHkv > 2) load_q(2);
    // Iteration r: publish row r's statistics; the leader reduces row r - 1
    // (every unit has had a row's time to publish it), the others read the
    // leader's normaliser of row r - 2.
    for (int r = 0; r <= dm.LHkv + 1; ++r) {
        if (r < dm.LHkv) {
#pragma unroll
            for (int w = 0; w < kProducers; ++w) lds_wait(flags + kFlagProd + w, r + 1, flags, a.status);
            // query row r + 2 (its copy was started an iteration ago) into the
            // buffer row r used: every producer has read row r's terms by now
            if (r + 2 < dm.LHkv) {
                store_q(r + 2);
                lds_publish(flags + kFlagQ, r + 3);
            }
            if (lane < G) {
                float m = -INFINITY, l = 0.0f;
#pragma unroll
                for (int w = 0; w < kProducers; ++w) {
                    const float2 st = sm.wstat[((r % kStatBufs) * kProducers + w) * 16 + lane];
                    merge_stat(m, l, st.x, st.y);
                }
                unsigned long long* p = a.ustat + (((size_t)(un.us + un.j) * dm.R + qrow0(dm, r) + lane) << 1);
                __hip_atomic_store(p, hi_tag | __float_as_uint(m), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(p + 1, hi_tag | __float_as_uint(l), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            if (r + 3 < dm.LHkv) load_q(r + 3);
        }
        if (leader) {
            if (r >= 1 && r <= dm.LHkv) lead(r - 1);
        } else if (r >= 2) {
            follow(r - 2);
        }
    }
}

// ------------------------------------------------------------ kernel

__global__ void __launch_bounds__(kAttendThreads) __attribute__((amdgpu_waves_per_eu(3)))
k_attend(AttendDims dm, AttendArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    if (a.probe != nullptr) {
        // Check mode: every wave stays until all workgroups have arrived
        // (bounded by ~20 ms), so the fewest arrivals seen is the number of
        // workgroups that are really resident together.
        if (threadIdx.x == 0) atomicAdd(a.probe, 1);
        if (lane_id() == 0) {
            const uint64_t t0 = now_ticks();
            int seen = 0;
            while (true) {
                seen = __hip_atomic_load(a.probe, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (seen >= (int)gridDim.x || now_ticks() - t0 > 2000000ull) break;
                __builtin_amdgcn_s_sleep(10);
            }
            atomicMin(a.probe + 1, seen);
        }
        return;
    }
    const Lds sm = carve(smem, dm.G, dm.Tstride);
    const int wv = uni(threadIdx.x >> 6);
    const uint32_t tag = (uint32_t)a.epoch[0];
    const int n_pass = a.plan[0];
    const int w = blockIdx.x;
    for (int ps = 0; ps < n_pass; ++ps) {
        const int T = a.plan[1 + 3 * ps], sb = a.plan[2 + 3 * ps], se = a.plan[3 + 3 * ps];
        const int u0 = a.ustart[sb];
        if (w >= a.ustart[se] - u0) continue;
        // session of unit u0 + w: largest s in [sb, se) with ustart[s] <= u0 + w
        int lo = sb, hi = se;
        while (hi - lo > 1) {
            const int mid = (lo + hi) >> 1;
            if (a.ustart[mid] <= u0 + w) lo = mid; else hi = mid;
        }
        Unit un;
        un.s = lo;
        un.us = a.ustart[lo];
        un.nu = a.ustart[lo + 1] - un.us;
        un.j = u0 + w - un.us;
        un.T = T;
        un.kt = T / kUnitQuantum;
        un.nt_s = a.n_tokens[lo];
        un.ntok = min(T, un.nt_s - un.j * T);
        __syncthreads();   // the previous unit is done with the LDS
        if (threadIdx.x < kFlagCount) sm.flags[threadIdx.x] = 0;
        __syncthreads();
        if (wv < kProducers) producer(dm, a, sm, un, wv);
        else manager(dm, a, sm, un, tag);
    }
}

}  // namespace

size_t attend_lds_bytes(int G, int Tstride) {
    return rowbuf_bytes(G, Tstride) + qs_bytes(G) + (size_t)2 * qraw_floats(G) * sizeof(float) + kWstatBytes +
           kNormBytes + kFlagBytes;
}

const void* attend_kernel() { return reinterpret_cast<const void*>(&k_attend); }

hipError_t launch_attend(const Dims& dm, const View& v, const Scratch& sc, const float* q, float* abar_out,
                         hipStream_t st) {
    AttendDims ad{dm.L, dm.Hq, dm.Hkv, dm.G, dm.P, dm.Pshift, dm.MP, dm.NP, dm.R, dm.LHkv, dm.Tstride, dm.U_cap,
                  dm.rho, dm.tau_scale};
    AttendArgs aa{v.k_pool, v.page_table, v.n_tokens, v.clock, v.imp, v.t_ref, q, abar_out,
                  sc.ustart, sc.plan, sc.epoch, sc.ustat, sc.nstat, sc.status, nullptr};
    void* args[] = {&ad, &aa};
    return hipLaunchCooperativeKernel(attend_kernel(), dim3(dm.n_wg), dim3(kAttendThreads), args,
                                      (unsigned)attend_lds_bytes(dm.G, dm.Tstride), st);
}

hipError_t launch_attend_check(const Dims& dm, int32_t* probe, int n_wg, hipStream_t st) {
    AttendDims ad{};
    AttendArgs aa{};
    aa.probe = probe;
    hipError_t e = hipMemsetD32Async(reinterpret_cast<hipDeviceptr_t>(probe), 0, 1, st);
    if (e == hipSuccess) e = hipMemsetD32Async(reinterpret_cast<hipDeviceptr_t>(probe + 1), 1 << 30, 1, st);
    if (e != hipSuccess) return e;
    void* args[] = {&ad, &aa};
    return hipLaunchCooperativeKernel(attend_kernel(), dim3(n_wg), dim3(kAttendThreads), args,
                                      (unsigned)attend_lds_bytes(dm.G, dm.Tstride), st);
}

}  // namespace md
