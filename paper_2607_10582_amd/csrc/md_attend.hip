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
//              producers' row statistics and publishes them with a tag, and
//              gathers every unit's statistics of an earlier row into the row
//              normaliser (max M, 1 / sum).  Each unit reads the others'
//              words itself (one hop; the words are a few KB per row and stay
//              in the caches).
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
    uint32_t* qs;     // [kQBufs][3][G][64] hi, mid, lo bf16 query terms (pairs) of staged rows
    float2* wstat;    // [kStatBufs][kProducers][16] producer row statistics
    float2* norm;     // [kNormBufs][16] row normalisers (M, 1 / Lambda)
    int* flags;       // [kFlagCount]
};

__host__ __device__ inline size_t rowbuf_bytes(int G, int Tstride) {
    return (size_t)kRowBufs * G * Tstride * sizeof(float);
}
__host__ __device__ inline size_t qs_bytes(int G) { return (size_t)kQBufs * 3 * G * 64 * sizeof(uint32_t); }
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
    l.wstat = reinterpret_cast<float2*>(smem + o);
    o += kWstatBytes;
    l.norm = reinterpret_cast<float2*>(smem + o);
    o += kNormBytes;
    l.flags = reinterpret_cast<int*>(smem + o);
    return l;
}

// LDS hand-offs inside the workgroup.  A wave's LDS operations complete in
// issue order, so publishing a flag after the data only needs the data's LDS
// writes done (lgkmcnt) and the compiler kept from reordering; a C++
// release store would also wait for the wave's outstanding global loads and
// stores (vmcnt), which would drain the producers' load ring and stall the
// manager on its in-flight requests.
__device__ __forceinline__ int lds_get(int* p) {
    const int v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    asm volatile("" ::: "memory");
    return v;
}

__device__ __forceinline__ void lds_publish(int* p, int v) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Time limits of the waits, in ticks of the 100 MHz real-time counter.
// Waits inside a workgroup outlast waits on other workgroups, so a stalled
// session is reported by the wait that polls the other units.
constexpr uint64_t kLdsWaitTicks = 10000000ull;      // 100 ms
constexpr uint64_t kGlobalWaitTicks = 5000000ull;    // 50 ms
constexpr uint64_t kRecheckTicks = 300;              // 3 us: re-check an unanswered request
constexpr uint64_t kUnitTicks = 100000000ull;        // 1 s: a unit stops waiting after this

__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

__device__ __forceinline__ void stop_all(int* flags, int32_t* status) {
    __hip_atomic_store(flags + kFlagStop, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    atomicOr(status, MD_DEV_TIMEOUT);
}

// Wait until *p >= target.  False when the wait ran out (at its own limit
// or the unit's deadline) or the workgroup stopped waiting after an earlier
// time-out.
__device__ __forceinline__ bool lds_wait(int* p, int target, int* flags, int32_t* status, uint64_t deadline) {
    if (lds_get(p) >= target) return true;
    const uint64_t t0 = now_ticks();
    while (lds_get(p) < target) {
        if (lds_get(flags + kFlagStop)) return false;
        const uint64_t t = now_ticks();
        if (t - t0 > kLdsWaitTicks || t > deadline) {
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

// Wave-wide max and sum with DPP row shifts and row broadcasts (VALU only;
// no LDS round trips).  Kogge-Stone within each 16-lane row (shifts 1, 2, 4,
// 8; a lane whose source falls outside its row keeps the identity), then
// lane 15 of rows 0 and 2 is folded into rows 1 and 3, and lane 31 into
// rows 2 and 3: lane 63 ends with the reduction of all 64 lanes, read as a
// wave-uniform value.
#define MD_DPP(old, v, ctrl, rm) \
    __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(old), __float_as_int(v), ctrl, rm, 0xf, false))
__device__ __forceinline__ float wave_max_dpp(float v) {
    const float id = -INFINITY;
    v = fmaxf(v, MD_DPP(id, v, 0x111, 0xf));   // row_shr:1
    v = fmaxf(v, MD_DPP(id, v, 0x112, 0xf));   // row_shr:2
    v = fmaxf(v, MD_DPP(id, v, 0x114, 0xf));   // row_shr:4
    v = fmaxf(v, MD_DPP(id, v, 0x118, 0xf));   // row_shr:8
    v = fmaxf(v, MD_DPP(id, v, 0x142, 0xa));   // row_bcast:15 into rows 1, 3
    v = fmaxf(v, MD_DPP(id, v, 0x143, 0xc));   // row_bcast:31 into rows 2, 3
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
__device__ __forceinline__ float wave_sum_dpp(float v) {
    const float id = 0.0f;
    v += MD_DPP(id, v, 0x111, 0xf);
    v += MD_DPP(id, v, 0x112, 0xf);
    v += MD_DPP(id, v, 0x114, 0xf);
    v += MD_DPP(id, v, 0x118, 0xf);
    v += MD_DPP(id, v, 0x142, 0xa);
    v += MD_DPP(id, v, 0x143, 0xc);
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}
#undef MD_DPP

struct Unit {
    int s, j, T, kt, ntok, nt_s, nu, us;
    uint64_t deadline;   // real-time tick after which the unit stops waiting
};

// First query row (layer * Hq + KV head * G) of (layer, KV head) row r.
__device__ __forceinline__ int qrow0(const AttendDims& dm, int r) {
    const int l = r / dm.Hkv;
    return l * dm.Hq + (r - l * dm.Hkv) * dm.G;
}

// ------------------------------------------------------------ producer

__device__ __forceinline__ void producer(const AttendDims& dm, const AttendArgs& a, const Lds& sm,
                                         const Unit& un, int wv, int lane, uint32_t tag) {
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
        const uint32_t* qb = sm.qs + (size_t)(r % kQBufs) * 3 * dm.G * 64;
#pragma unroll
        for (int p = 0; p < 3; ++p)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                bq[j][p] = *reinterpret_cast<const u32x4*>(qb + (p * dm.G + hh) * 64 + 16 * j + 4 * g);
    };

    float acc_tok[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    const int my_tokens = kt * 16;
    auto consume = [&](int rc) {
        lds_wait(flags + kFlagNorm, rc + 1, flags, a.status, un.deadline);
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

    lds_wait(flags + kFlagQ, 1, flags, a.status, un.deadline);
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
                    if (wv == 0) {
                        // Producer 0 publishes the unit's statistics of the
                        // row for the other units (the manager issues no
                        // stores: its waits on its own loads must not wait
                        // for a store's round trip too).
#pragma unroll
                        for (int pw = 1; pw < kProducers; ++pw)
                            lds_wait(flags + kFlagProd + pw, row + 1, flags, a.status, un.deadline);
                        if (lane < dm.G) {
                            float um = -INFINITY, ul = 0.0f;
#pragma unroll
                            for (int pw = 0; pw < kProducers; ++pw) {
                                const float2 st = sm.wstat[((row % kStatBufs) * kProducers + pw) * 16 + lane];
                                merge_stat(um, ul, st.x, st.y);
                            }
                            unsigned long long* p =
                                a.ustat + (((size_t)(un.us + un.j) * dm.R + qrow0(dm, row) + lane) << 1);
                            const unsigned long long hi = (unsigned long long)tag << 32;
                            __hip_atomic_store(p, hi | __float_as_uint(um), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            __hip_atomic_store(p + 1, hi | __float_as_uint(ul), __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_AGENT);
                        }
                    }
                    if (row + 1 < dm.LHkv) {
                        lds_wait(flags + kFlagQ, row + 2, flags, a.status, un.deadline);
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
                                        const Unit& un, uint32_t tag, int lane) {
    int* flags = sm.flags;
    const int G = dm.G;

    // Query row r: G heads x 128 floats, loaded a row ahead into registers
    // (lane + 64 k holds float4 k), then split into the three bf16 terms the
    // producers' B operands take.  (A direct-to-LDS copy would make every
    // later LDS access of this wave wait for all its outstanding loads.)
    f32x4 qv[4];
    auto q_row = [&](int r) {
        return reinterpret_cast<const f32x4*>(a.q + ((size_t)un.s * dm.L * dm.Hq + qrow0(dm, r)) * kHeadDim);
    };
    // Loads are unconditional (indices clamped into the row): loads under
    // lane conditions make the compiler wait for every outstanding load
    // before each of them.
    auto load_q = [&](int r) {
        const f32x4* qr = q_row(r);
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (64 * k < G * 32) qv[k] = qr[min(lane + 64 * k, G * 32 - 1)];   // uniform condition
    };
    auto split_store = [&](uint32_t* qb, int f, const f32x4& x, bool& bad) {
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
    };
    auto store_q = [&](int r) {
        uint32_t* qb = sm.qs + (size_t)(r % kQBufs) * 3 * G * 64;
        bool bad = false;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int f = lane + 64 * k;
            if (f < G * 32) split_store(qb, f, qv[k], bad);
            __builtin_amdgcn_sched_barrier(0);   // one float4 at a time: few live registers
        }
        // heads past the eighth (G > 8) are loaded here
        const f32x4* qr = q_row(r);
        for (int f = lane + 256; f < G * 32; f += 64) split_store(qb, f, qr[f], bad);
        if (bad) atomicOr(a.status, MD_DEV_NONFINITE);
    };

    auto set_norm = [&](int rc, int hd, float M, float inv) {
        sm.norm[(rc % kNormBufs) * 16 + hd] = make_float2(M, inv);
    };
    auto tag_ok = [&](unsigned long long v) { return (uint32_t)(v >> 32) == tag; };
    // Requests for the other units' words go out at one row's publication
    // and are checked at the next, so the manager never waits on a global
    // round trip while it has LDS work: lane k holds unit k of the first 64,
    // its first eight heads.
    unsigned long long w[8][2];
    // p: the unit's words of head h0 (a valid unit for every lane)
    auto load_words = [&](const unsigned long long* p, int h0) {
#pragma unroll
        for (int hd = 0; hd < 8; ++hd) {
            if (h0 + hd < G) {   // uniform condition
                w[hd][0] = __hip_atomic_load(p + 2 * hd, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                w[hd][1] = __hip_atomic_load(p + 2 * hd + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    };
    auto words_ok = [&](int h0, bool act) {
        bool ok = true;
#pragma unroll
        for (int hd = 0; hd < 8; ++hd)
            if (h0 + hd < G && act) ok &= tag_ok(w[hd][0]) && tag_ok(w[hd][1]);
        return ok;
    };
    auto unit_words = [&](int x, int k, int h0) {
        return a.ustat + (((size_t)(un.us + k) * dm.R + qrow0(dm, x) + h0) << 1);
    };
    auto issue = [&](int x) {
        const bool act = lane < un.nu;
        load_words(unit_words(x, act ? lane : 0, 0), 0);
    };
    auto ready = [&]() -> bool { return __all(words_ok(0, lane < un.nu)); };

    // Row x's normaliser: per head, a wave max of the units' maxima, then a
    // wave sum of their sums rescaled to it (one exp2 per unit), both with
    // DPP; eight heads at a time (the first eight of the first 64 units came
    // with the request; the rest are fetched here with bounded waits).  Lane h
    // keeps head h's running result.
    auto finish = [&](int x) {
        float run_m = -INFINITY, run_l = 0.0f;
        for (int h0 = 0; h0 < G; h0 += 8) {
            for (int c0 = 0; c0 < un.nu; c0 += 64) {
                const int k = c0 + lane;
                const bool act = k < un.nu;
                if (c0 > 0 || h0 > 0) {
                    const unsigned long long* p = unit_words(x, act ? k : 0, h0);
                    const uint64_t t0 = now_ticks();
                    while (true) {
                        load_words(p, h0);
                        if (__all(words_ok(h0, act)) || lds_get(flags + kFlagStop)) break;
                        const uint64_t t = now_ticks();
                        if (t - t0 > kGlobalWaitTicks || t > un.deadline) {
                            stop_all(flags, a.status);
                            break;
                        }
                        __builtin_amdgcn_s_sleep(8);
                    }
                }
#pragma unroll
                for (int hd = 0; hd < 8; ++hd) {
                    if (h0 + hd < G) {
                        const float m = act ? __uint_as_float((uint32_t)w[hd][0]) : -INFINITY;
                        const float l = act ? __uint_as_float((uint32_t)w[hd][1]) : 0.0f;
                        const float M = wave_max_dpp(m);
                        const float L = wave_sum_dpp(m == -INFINITY ? 0.0f : l * hw_exp2(m - M));
                        if (lane == h0 + hd) merge_stat(run_m, run_l, M, L);
                    }
                }
            }
        }
        if (lane < G) set_norm(x, lane, run_m, 1.0f / run_l);
        lds_publish(flags + kFlagNorm, x + 1);
    };

    // the first kQBufs query rows up front, the next one in flight
    for (int r = 0; r < min(kQBufs, dm.LHkv); ++r) {
        load_q(r);
        store_q(r);
    }
    lds_publish(flags + kFlagQ, min(kQBufs, dm.LHkv));
    if (dm.LHkv > kQBufs) load_q(kQBufs);

    // Event loop, driven by the producers' progress.  Loads come back in
    // issue order, so every load this wave waits on must be about a row old:
    // the next query row and the request for the units' words go out
    // together when a row is published, and both are consumed when the next
    // row is.  The request for row x goes out at the publication of row
    // x + 1 (every unit has had about a row to publish row x) and normally
    // completes at the publication of row x + 2, kConsumeLag - 2 rows before
    // the producers need it.  If the producers stop (they may be waiting
    // for that very row), an unanswered request is checked and re-sent every
    // kRecheckTicks on its own.  Only publishing and finishing rows count as
    // progress for the time limit.
    const int ahead = 2;
    int r_pub = 0, x_next = 0, x_pend = -1, n_done = 0;
    uint64_t last_prog = now_ticks(), issued_t = 0;
    auto check = [&]() {   // x_pend >= 0; its words are a row or kRecheckTicks old
        if (ready()) {
            finish(x_pend);
            ++n_done;
            x_pend = -1;
            last_prog = now_ticks();
            return true;
        }
        return false;
    };
    while (n_done < dm.LHkv) {
        bool all = r_pub < dm.LHkv;
        if (all) {
#pragma unroll
            for (int pw = 0; pw < kProducers; ++pw) all &= lds_get(flags + kFlagProd + pw) > r_pub;
        }
        if (all) {
            const int r = r_pub;
            // query row r + kQBufs (loaded at the previous publication) into
            // the buffer row r used: every producer has read row r's terms
            if (r + kQBufs < dm.LHkv) {
                store_q(r + kQBufs);
                lds_publish(flags + kFlagQ, r + kQBufs + 1);
            }
            const bool resend = x_pend >= 0 && !check();
            r_pub = r + 1;
            last_prog = now_ticks();
            if (r + kQBufs + 1 < dm.LHkv) load_q(r + kQBufs + 1);
            if (resend) {
                issue(x_pend);
                issued_t = now_ticks();
            } else if (x_pend < 0 && x_next < dm.LHkv && (x_next + ahead <= r_pub || r_pub == dm.LHkv)) {
                issue(x_next);
                x_pend = x_next++;
                issued_t = now_ticks();
            }
            continue;
        }
        if (x_pend >= 0) {
            if (now_ticks() - issued_t > kRecheckTicks && !check()) {
                issue(x_pend);
                issued_t = now_ticks();
            }
        } else if (x_next < dm.LHkv && (x_next + ahead <= r_pub || r_pub == dm.LHkv)) {
            issue(x_next);
            x_pend = x_next++;
            issued_t = now_ticks();
            continue;
        }
        const uint64_t t = now_ticks();
        if (lds_get(flags + kFlagStop) || t - last_prog > kGlobalWaitTicks || t > un.deadline) {
            // give up on the step: release the producers
            if (!lds_get(flags + kFlagStop)) stop_all(flags, a.status);
            lds_publish(flags + kFlagQ, dm.LHkv + kQBufs);
            lds_publish(flags + kFlagNorm, dm.LHkv);
            break;
        }
        __builtin_amdgcn_s_sleep(1);
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
        un.deadline = now_ticks() + kUnitTicks;
        // The lane index is made opaque here so that per-lane address
        // arithmetic stays inside each role instead of being hoisted to the
        // kernel entry and kept live (and spilled) across both roles.
        int lane = (int)threadIdx.x & 63;
        asm volatile("" : "+v"(lane));
        if (wv < kProducers) producer(dm, a, sm, un, wv, lane, tag);
        else manager(dm, a, sm, un, tag, lane);
    }
}

}  // namespace

size_t attend_lds_bytes(int G, int Tstride) {
    return rowbuf_bytes(G, Tstride) + qs_bytes(G) + kWstatBytes + kNormBytes + kFlagBytes;
}

const void* attend_kernel() { return reinterpret_cast<const void*>(&k_attend); }

hipError_t launch_attend(const Dims& dm, const View& v, const Scratch& sc, const float* q, float* abar_out,
                         hipStream_t st) {
    AttendDims ad{dm.L, dm.Hq, dm.Hkv, dm.G, dm.P, dm.Pshift, dm.MP, dm.NP, dm.R, dm.LHkv, dm.Tstride, dm.U_cap,
                  dm.rho, dm.tau_scale};
    AttendArgs aa{v.k_pool, v.page_table, v.n_tokens, v.clock, v.imp, v.t_ref, q, abar_out,
                  sc.ustart, sc.plan, sc.epoch, sc.ustat, sc.status, nullptr};
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
