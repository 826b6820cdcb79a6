// gfx950 fused observation kernel: attention mass (Sec. III-C), EWMA (Eq. 2)
// and refresh (Eq. 3) of every cached token in one pass over the key cache,
// with the logits of the step held in LDS instead of HBM.
//
// The attention mass of token i averages, over every (layer, query head) row,
// the token's softmax weight in that row.  A row's softmax needs the row's
// maximum and sum over all of the session's tokens, so the logits of a block
// of tokens cannot be normalised where they are produced.  Here a session's
// tokens are split into units of T tokens, one workgroup per unit,
// all units of a session resident at once.  Each workgroup walks the
// (layer, KV head) rows in order: it computes the logits of its tokens for
// the G query heads of the row on MFMA, keeps them in an LDS ring of
// kRowBufs rows, publishes the row's (max, sum) to the other units of the
// session, and kConsumeLag rows later, when every unit's statistics of that
// row are in, turns the held logits into softmax weights and adds them to
// its tokens' mass.  The key cache is read once and nothing per
// (token, row) is written back.
//
// Workgroup = four waves with the same job; wave w owns the unit's tiles
// 4w .. 4w + 3 (16 tokens each), i.e. tokens 64w .. 64w + 63.  Each wave
// streams its K tiles through registers two rows ahead of the row it works
// on, so its loads never wait for a row boundary.
// At a row boundary the waves meet once (s_barrier, no memory fence: a fence
// would wait for the load ring) and split the row's bookkeeping:
//   * every wave merges its own (max, sum) of the row into LDS; after the
//     barrier, wave w merges the four partials of heads w, w + 4, ... and
//     publishes them for the other units;
//   * wave w also gathers every unit's statistics of heads w, w + 4, ... of
//     the row kConsumeLag back (the loads go out at one barrier and are used
//     in the next row, after loads that the ring does not wait for) and
//     writes that row's normalisers to LDS before the next barrier; the row
//     is normalised in the row after that;
//   * wave w stages its quarter of the query of the next row (three bf16
//     terms per float, loaded at the last barrier).
// All of it but the barrier runs between the tiles of the following row.
// Unit <-> unit hand-offs are 64-bit words (tag << 32 | float bits, the tag
// being the step's epoch) written and polled with agent-scope atomics, so a
// word is either absent or complete.  A unit waits only for words of rows
// kConsumeLag or more behind its own, which every unit publishes before it
// can wait on anything later, so the waits form no cycle.  Every wait is
// bounded; a wait that runs out sets MD_DEV_TIMEOUT, and the wave stops
// waiting for the rest of the step, so the grid always drains.

#include <hip/hip_ext.h>

#include "md_device.h"

namespace md {

namespace {

struct AttendDims {
    int L, Hq, Hkv, G, P, Pshift, MP, NP, R, LHkv;
    int wg_per_cu, n_cu, S, n_regions, norm_attn;
    uint32_t pin_mask;
    float rho, tau_scale, alpha;
    int aligned;
    int Gq, Wn;   // window (WN instantiations): query heads per KV head and window
                  // queries; G above counts the MFMA columns, Gq * Wn
    int rg;       // row groups (RS instantiations): a unit covers one of rg
                  // consecutive ranges of the L * Hkv rows; 1 = every row
};

struct AttendArgs {
    const uint16_t* k_pool;
    const int32_t* page_table;
    const int32_t* n_tokens;
    const int32_t* clock;
    const uint8_t* region;
    const float* b;
    const float* lam;
    float* imp;
    int32_t* t_ref;
    float* pscore;
    const float* q;
    float* abar_out;
    const int32_t* ustart;
    const int32_t* plan;
    const int32_t* epoch;
    unsigned long long* claim;
    unsigned long long* lane_box;
    unsigned long long* ustat;
    unsigned long long* unorm;
    int32_t* status;
    int32_t* probe;    // check mode only: [arrivals, least seen]
    const int32_t* n_live;   // tokens |K_t| (the n_tokens array unless pages are region-aligned)
    const uint8_t* page_format;   // quantised tier: 1 = the page holds E4M3 codes
    const int32_t* t_ins;         // window: insertion steps, for the causal mask
    int32_t* valid;               // [S] cleared for a session whose step is void
    unsigned long long* upart;    // row groups: [units][T] tagged partial masses
};

// LDS row stride (floats) of a head's values: W waves of KT tiles
__host__ __device__ constexpr int tstride(int W, int KT) { return 16 * W * KT + 4; }

struct Lds {
    float* rowbuf;    // [kRowBufs][G][tstride] 2^(logit - wave max) of the held rows
    uint32_t* qs;     // [2][3][G][64] hi, mid, lo bf16 query terms (pairs) of two rows
    float2* wstat;    // [2][W][16] per-wave row statistics
    float2* norm;     // [2][16] row normalisers (M, 1 / Lambda)
    int* vflag;       // [1] the unit's step is void: a non-finite query, or a wait ran out
    int* claim;       // [32] lane mode: the next pass claimed early (sessions [0], [1];
                      // [24] set when it was), and claim_sessions' bookkeeping
    float* wmax;      // [kRowBufs][W][head slots] each wave's maximum of the held rows per head
};

__host__ __device__ inline size_t rowbuf_bytes(int G, int W, int KT) {
    return (size_t)kRowBufs * G * tstride(W, KT) * sizeof(float);
}
__host__ __device__ inline size_t qs_bytes(int G) { return (size_t)2 * 3 * G * 64 * sizeof(uint32_t); }
__host__ __device__ inline size_t wstat_bytes(int W) { return (size_t)2 * W * 16 * sizeof(float2); }
constexpr size_t kNormBytes = (size_t)2 * 16 * sizeof(float2);
constexpr size_t kFlagBytes = 16;
constexpr size_t kClaimBytes = 32 * sizeof(int);
// head slots of a wave's row maxima: W NH of the instantiation for G columns
__host__ __device__ inline int head_slots(int G) { return G <= 4 ? 4 : G <= 8 ? 8 : 16; }
__host__ __device__ inline size_t wmax_bytes(int G, int W) {
    return (size_t)kRowBufs * W * head_slots(G) * sizeof(float);
}

__device__ __forceinline__ Lds carve(unsigned char* smem, int G, int W, int KT) {
    Lds l;
    size_t o = 0;
    l.rowbuf = reinterpret_cast<float*>(smem + o);
    o += rowbuf_bytes(G, W, KT);
    l.qs = reinterpret_cast<uint32_t*>(smem + o);
    o += qs_bytes(G);
    l.wstat = reinterpret_cast<float2*>(smem + o);
    o += wstat_bytes(W);
    l.norm = reinterpret_cast<float2*>(smem + o);
    o += kNormBytes;
    l.vflag = reinterpret_cast<int*>(smem + o);
    o += kFlagBytes;
    l.claim = reinterpret_cast<int*>(smem + o);
    o += kClaimBytes;
    l.wmax = reinterpret_cast<float*>(smem + o);
    return l;
}

// Workgroup meeting point for LDS hand-offs.  A wave's LDS writes are done
// once lgkmcnt is zero; the barrier carries no fence, so the waves' global
// loads stay in flight across it.  The empty asm statements keep the
// compiler from moving memory accesses over the barrier.
__device__ __forceinline__ void lds_sync() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Time limits, in ticks of the 100 MHz real-time counter.
constexpr uint64_t kGlobalWaitTicks = 5000000ull;    // 50 ms for one row's statistics
constexpr uint64_t kUnitTicks = 100000000ull;        // 1 s: a unit stops waiting after this

__device__ __forceinline__ uint64_t now_ticks() { return __builtin_amdgcn_s_memrealtime(); }

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
    int s, j, ntok, nt_s, nu, us;
    uint64_t deadline;   // real-time tick after which the unit stops waiting
    int nl_s;            // region-aligned pages: the session's tokens |K_t| (nt_s counts holes too)
    // row groups (RS): the unit covers rows [r0, r1) of group grp of rg; nu,
    // j and us count the units of that group, ubase is the session's first
    // unit (group 0)
    int r0, r1, grp, rg, ubase;
};

__device__ void claim_sessions(const AttendArgs& a, int* xs, int lane_no, int cap);

// First query row (layer * Hq + KV head * G) of (layer, KV head) row r:
// with Hq = Hkv * G that is r * G.
__device__ __forceinline__ int qrow0(const AttendDims& dm, int r) { return r * dm.G; }

// One wave's part of a unit.  W = waves per workgroup, NH = normaliser
// heads per wave (G <= W NH), KT = tiles per wave (units of 16 W KT tokens),
// AL = region-aligned pages (hole slots are masked), QT = quantised tier
// (tiles of quantised pages hold 8-bit codes), WN = a window of several
// decode queries (column c of a row is window query c / Gq, head c % Gq, and
// a causal mask keeps each query to the tokens inserted by its step);
// separate instantiations keep the plain kernel's register budget.
// RS = row groups: the unit walks only its group's rows, and the groups'
// partial masses meet in the unit of group 0, which alone finishes the
// tokens (the plain instantiations walk every row).
// next_box (lane mode, the lane's first workgroup; else NULL): the lane's
// next pass is claimed with claim_lane and cap once the unit's rows are
// done, and published there.
template <int W, int NH, int KT, bool AL, bool QT, bool WN, bool RS>
__device__ __forceinline__ void attend_wave(const AttendDims& dm, const AttendArgs& a, const Lds& sm,
                                            const Unit& un, int wv, int lane, uint32_t tag, int claim_lane,
                                            int cap, unsigned long long* next_box) {
    constexpr int KQ = (W * NH * 32 + 64 * W - 1) / (64 * W);   // float4 of the query row per lane
    const int G = dm.G;
    const int h = lane & 15;          // MFMA column: query head of the group
    const int g = lane >> 4;          // k-group of A/B, row quad of C
    const int hh = min(h, G - 1);     // in-bounds head for the unused columns
    const uint32_t voff = 16u * lane;   // piece (8-dim block 4j + g, token h) of a 16-token block
    constexpr int kT = 16 * W * KT;   // tokens per unit
    constexpr int kTs = tstride(W, KT);
    constexpr int kTok = KT / 4;          // tokens per lane
    const int wtok0 = wv * 16 * KT;       // unit-local token of this wave's first tile
    bool dead = false;                    // a wait of this wave ran out: stop waiting
    // the unit's rows [r_beg, r_end)
    const int r_beg = RS ? un.r0 : 0;
    const int r_end = RS ? un.r1 : dm.LHkv;

    // lane i < KT: slot (physical page * P + offset) of tile i's first token
    int myslot = 0;
    bool myok = false;
    if (lane < KT) {
        const int tok = un.j * kT + wtok0 + 16 * lane;
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
    constexpr unsigned long long kAll = (1ull << KT) - 1;
    // Region-aligned pages: a page's holes follow its last token, so the
    // holes of a 16-slot tile are a suffix of it; byte u of `lims` is the
    // number of slots of tile u before its first hole (16: none).  Lane
    // u < KT counts them for tile u.  Wave-uniform.
    uint32_t lims = 0x10101010u;
    if constexpr (AL) {
        int mylim = 16;
        if (myok) {
            const u32x4 rb = *reinterpret_cast<const u32x4*>(a.region + myslot);
            for (int k = 15; k >= 0; --k)
                if (((rb[k >> 2] >> (8 * (k & 3))) & 0xffu) == (uint32_t)kHole) mylim = k;
        }
        lims = 0;
#pragma unroll
        for (int u = 0; u < KT; ++u) lims |= (uint32_t)__builtin_amdgcn_readlane(mylim, u) << (8 * u);
    }
    // Window: bit 4u + i marks this lane's logit column (window query
    // h / Gq) of tile u, token 4g + i, as inserted after that query's step.
    uint32_t unseen = 0;
    if constexpr (WN) {
        const int t_lim = a.clock[un.s] - (dm.Wn - 1 - min(h / dm.Gq, dm.Wn - 1));
#pragma unroll
        for (int u = 0; u < KT; ++u) {
            const int slot = __builtin_amdgcn_readlane(myslot, u);
            if ((vmask >> u) & 1ull) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    unseen |= (a.t_ins[slot + 4 * g + i] > t_lim) ? 1u << (4 * u + i) : 0u;
            }
        }
    }
    const bool wave_full = (vmask & kAll) == kAll && wtok0 + 16 * KT <= un.ntok && (!AL || lims == 0x10101010u) &&
                           (!WN || !__any(unseen != 0));
    // Quantised tier: bit u of qmask marks tile u as 8-bit codes (its page's
    // format); wave-uniform.
    uint32_t qmask = 0;
    if constexpr (QT) {
        const bool qz = myok && a.page_format[myslot >> dm.Pshift] != 0;
        qmask = (uint32_t)(__ballot(qz) & kAll);
    }

    // K tile u of row r in the MFMA A layout: the pool keeps each block of
    // 16 tokens as [d / 8][16][8], so load j reads 1 KiB contiguous and lane
    // (h, g) gets token h's dims 32j + 8g .. +7.  A tile without cached
    // tokens, or past the last row, reads the pool's first tile (its logits
    // are masked), so loads never branch.
    auto load_tile = [&](u32x4 (&rg)[4], int r, int u) {
        const bool ok = r < r_end && ((vmask >> u) & 1ull);
        const int slot = __builtin_amdgcn_readlane(myslot, u);
        const size_t e = ok ? ((size_t)(slot >> dm.Pshift) * dm.LHkv + r) * dm.P + (slot & (dm.P - 1)) : 0;
        gbytes base = uni_ptr(a.k_pool + e * kHeadDim);
        if constexpr (QT) {
            // a quantised block: codes in its first 2 KiB (rg[0], rg[1]), the
            // scale at byte 2048 (rg[2]); rg[3] takes the next 16 bytes of
            // the same line, which the widening overwrites.  Two loads of
            // one address would be merged into one and a register copy,
            // and the copy of a load in flight waits for every load.
            const bool qt = (qmask >> u) & 1u;
#pragma unroll
            for (int j = 0; j < 4; ++j)
                rg[j] = __builtin_nontemporal_load(
                    reinterpret_cast<gvec>(base + ((qt && j >= 2) ? 2048u + 16u * (j - 2) : voff + 1024u * j)));
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
                rg[j] = __builtin_nontemporal_load(reinterpret_cast<gvec>(base + voff + 1024 * j));
        }
    };


    // ---- query staging: this wave's float4 f = lane + 64 (wv + W k) of a row
    f32x4 qv[KQ];
    auto q_row = [&](int r) {
        return reinterpret_cast<const f32x4*>(a.q + ((size_t)un.s * dm.L * dm.Hq + qrow0(dm, r)) * kHeadDim);
    };
    auto load_q = [&](int r) {   // unconditional loads, indices clamped into the row
        if constexpr (WN) {
            // queries [S][Wn][L][Hq][d]: column c is query c / Gq, head c % Gq
            const int l = r / dm.Hkv, kv = r - l * dm.Hkv;
#pragma unroll
            for (int k = 0; k < KQ; ++k) {
                const int f = min(lane + 64 * (wv + W * k), G * 32 - 1);
                const int c = f >> 5, w = c / dm.Gq, hd = c - w * dm.Gq;
                qv[k] = reinterpret_cast<const f32x4*>(
                    a.q + ((((size_t)un.s * dm.Wn + w) * dm.L + l) * dm.Hq + kv * dm.Gq + hd) * kHeadDim)[f & 31];
            }
        } else {
            const f32x4* qr = q_row(r);
#pragma unroll
            for (int k = 0; k < KQ; ++k) qv[k] = qr[min(lane + 64 * (wv + W * k), G * 32 - 1)];
        }
    };
    auto store_q = [&](int r) {
        uint32_t* qb = sm.qs + (size_t)(r & 1) * 3 * G * 64;
        bool bad = false;
#pragma unroll
        for (int k = 0; k < KQ; ++k) {
            const int f = lane + 64 * (wv + W * k);
            if (f < G * 32) {
                const int hd = f >> 5, d2 = 2 * (f & 31);
                uint32_t t[3][4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    bad |= !isfinite(qv[k][e]);
                    split3(qv[k][e], t[0][e], t[1][e], t[2][e]);
                }
#pragma unroll
                for (int p = 0; p < 3; ++p)
                    *reinterpret_cast<uint2*>(qb + (p * G + hd) * 64 + d2) =
                        make_uint2(t[p][0] | (t[p][1] << 16), t[p][2] | (t[p][3] << 16));
            }
        }
        if (bad) {   // the step of the session is void
            atomicOr(a.status, MD_DEV_NONFINITE);
            *sm.vflag = 1;
        }
    };
    // ---- cross-unit words.  Every unit publishes its (max, sum) of each
    // (row, query head); the leader of row x (unit x mod nu of the session)
    // gathers them into the row's normaliser words (M, 1 / Lambda), which
    // every unit reads.  Wave wv looks after heads wv + W i (i < NH).
    const int last = r_end - 1;
    const unsigned long long tag_hi = (unsigned long long)tag << 32;
    auto tag_ok = [&](unsigned long long v) { return (uint32_t)(v >> 32) == tag; };
    auto stat_word = [&](int x, int k, int hd) {
        return a.ustat + ((((size_t)(un.us + k)) * dm.R + qrow0(dm, x) + hd) << 1);
    };
    auto norm_word = [&](int x, int hd) {
        return a.unorm + ((((size_t)un.s) * dm.R + qrow0(dm, x) + hd) << 1);
    };
    // Rows this unit leads are j, j + nu, j + 2 nu, ...: lead_next is the
    // next one to request, lead_now says whether the previous request was
    // this unit's (both advance once per iteration).
    int lead_next = RS ? r_beg + ((un.j - r_beg) % un.nu + un.nu) % un.nu : un.j;
    bool lead_now = false;
    // Re-read until every active lane's words carry the step's tag (bounded).
    auto await_tags = [&](auto&& ready, auto&& reload) {
        if (__all(ready()) || dead) return;
        const uint64_t t0 = now_ticks();
        while (true) {
            __builtin_amdgcn_s_sleep(4);
            reload();
            if (__all(ready())) return;
            const uint64_t t = now_ticks();
            if (t - t0 > kGlobalWaitTicks || t > un.deadline) {
                atomicOr(a.status, MD_DEV_TIMEOUT);
                dead = true;
                *sm.vflag = 1;
                return;
            }
        }
    };

    // Normaliser words of row x: wave x mod 4 reads them (lane h: head h)
    // and, once they carry the tag, writes them to LDS.
    const bool hd_lane = lane < NH && wv + W * lane < G;
    unsigned long long nw[2];
    auto load_norm = [&](int x) {
        const unsigned long long* p = norm_word(x, min(lane, G - 1));
        nw[0] = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        nw[1] = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    auto check_norm = [&](int x) {
        await_tags([&] { return lane >= G || (tag_ok(nw[0]) && tag_ok(nw[1])); }, [&] { load_norm(x); });
        if (lane < G)
            sm.norm[(x & 1) * 16 + lane] =
                make_float2(__uint_as_float((uint32_t)nw[0]), __uint_as_float((uint32_t)nw[1]));
    };

    // Leader: the units' words of heads wv + W i, lane k = unit k (the first
    // 64 units are requested a row ahead; further units are read here).
    unsigned long long w[NH][2];
    auto load_stats = [&](int x, int c0) {
        const int k = c0 + lane < un.nu ? c0 + lane : 0;
#pragma unroll
        for (int i = 0; i < NH; ++i) {
            const unsigned long long* p = stat_word(x, k, min(wv + W * i, G - 1));
            w[i][0] = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            w[i][1] = __hip_atomic_load(p + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    };
    // A wave max over the units' maxima, then a wave sum of their sums
    // rescaled to it; heads past the group are reduced too (their words are a
    // valid head's) so that the NH reductions run side by side.
    auto lead = [&](int x) {
        float run_m[NH], run_l[NH];
#pragma unroll
        for (int i = 0; i < NH; ++i) {
            run_m[i] = -INFINITY;
            run_l[i] = 0.0f;
        }
        auto fold = [&](int c0) {
            const bool act = c0 + lane < un.nu;
            await_tags(
                [&] {
                    bool ok = true;
#pragma unroll
                    for (int i = 0; i < NH; ++i) ok &= !act || (tag_ok(w[i][0]) && tag_ok(w[i][1]));
                    return ok;
                },
                [&] { load_stats(x, c0); });
#pragma unroll
            for (int i = 0; i < NH; ++i) {
                const float m = act ? __uint_as_float((uint32_t)w[i][0]) : -INFINITY;
                const float l = act ? __uint_as_float((uint32_t)w[i][1]) : 0.0f;
                const float M = wave_max_dpp(m);
                const float S = wave_sum_dpp(m == -INFINITY ? 0.0f : l * hw_exp2(m - M));
                merge_stat(run_m[i], run_l[i], M, S);
            }
        };
        // The first 64 units' words were requested an iteration earlier and
        // are folded outside the loop: inside it, the wait for them would
        // also wait for every tile load issued since.
        fold(0);
        for (int c0 = 64; c0 < un.nu; c0 += 64) {
            load_stats(x, c0);
            fold(c0);
        }
        // a leader whose wait ran out publishes nothing: every unit of the
        // session then runs out of time on this row too, and all of them
        // leave the step void
        if (hd_lane && !dead) {
            float M = run_m[0], Ls = run_l[0];
#pragma unroll
            for (int i = 1; i < NH; ++i)
                if (lane == i) {
                    M = run_m[i];
                    Ls = run_l[i];
                }
            // a row with no live token gives zero weights, never NaN
            M = M == -INFINITY ? 0.0f : M;
            const float inv = Ls > 0.0f ? 1.0f / Ls : 0.0f;
            unsigned long long* p = norm_word(x, wv + W * lane);
            __hip_atomic_store(p, tag_hi | __float_as_uint(M), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(p + 1, tag_hi | __float_as_uint(inv), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    };

    // The unit's (max, sum) of row r, merged over the four waves; wave r mod 4
    // publishes all heads (lane h = head h).
    auto publish = [&](int r) {
        if (wv == (r & (W - 1)) && lane < G) {
            float um = -INFINITY, ul = 0.0f;
#pragma unroll
            for (int pw = 0; pw < W; ++pw) {
                const float2 st = sm.wstat[((r & 1) * W + pw) * 16 + lane];
                merge_stat(um, ul, st.x, st.y);
            }
            unsigned long long* p = stat_word(r, un.j, lane);
            __hip_atomic_store(p, tag_hi | __float_as_uint(um), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(p + 1, tag_hi | __float_as_uint(ul), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    };

    // Row x's softmax weights of this wave's tokens, added to their mass.
    // The held values are 2^(logit - m_w), m_w being the wave's maximum of
    // the row for head h, so a weight is the held value times
    // f_h = 2^(m_w - M_h) / Lambda_h: lane h works f_h out once, and every
    // lane reads it from lane h.
    float acc[kTok];   // attention mass of tokens wtok0 + lane + 64 k, summed over rows
#pragma unroll
    for (int k = 0; k < kTok; ++k) acc[k] = 0.0f;
    // The wave's maximum of held row x for head h (the values it held are
    // 2^(logit - that maximum)) sits in LDS next to the row, not in
    // registers: kRowBufs rows of it would cost the plain kernel seven
    // registers and push the quantised and window instantiations into spills.
    constexpr int kSlots = W * NH;
    float* const wm_wave = sm.wmax + (size_t)wv * kSlots;
    auto consume = [&](int x) {
        const float* rb = sm.rowbuf + (size_t)(x % kRowBufs) * G * kTs + wtok0 + lane;
        const float mw = wm_wave[(size_t)(x % kRowBufs) * W * kSlots + min(h, kSlots - 1)];
        const float2 n = sm.norm[(x & 1) * 16 + hh];
        const float f = h < G ? hw_exp2(mw - n.x) * n.y : 0.0f;
#pragma unroll
        for (int hd = 0; hd < W * NH; ++hd) {   // heads past the group read a valid row and weigh zero
            const float fh = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), hd));
#pragma unroll
            for (int k = 0; k < kTok; ++k) acc[k] = fmaf(rb[min(hd, G - 1) * kTs + 64 * k], fh, acc[k]);
        }
    };

    // Bookkeeping of iteration r (a row of tiles for r < LHkv, then
    // kConsumeLag iterations without tiles).  Row x's words travel:
    //   iteration x + 1  its unit statistics are published;
    //   iteration x + 3  the leader requests them (a row and a half after the
    //                    last unit can have published);
    //   iteration x + 4  the leader publishes the normalisers;
    //   iteration x + 5  every unit requests them;
    //   iteration x + 6  they go to LDS, before the barrier;
    //   iteration x + 7  row x's held logits are normalised.
    // Requests are the loads of iteration r: they go out before the tiles of
    // row r + 2 and are used at iteration r + 1, after the tiles of row
    // r + 1 came in, so no wait ever holds the tile loads up (loads come back
    // in issue order).
    auto use_loads = [&](int r) {   // steps of iteration r that use iteration r - 1's loads
        const int xa = r - 6;
        if (xa >= r_beg && xa <= last && (xa & (W - 1)) == wv) check_norm(xa);
        if (lead_now) lead(r - 4);
    };
    auto issue_loads = [&](int r) {
        if (((r - 5) & (W - 1)) == wv) load_norm(min(max(r - 5, r_beg), last));
        const int xd = r - 3;
        lead_now = xd == lead_next && xd <= last;
        if (lead_now) {
            load_stats(xd, 0);
            lead_next += un.nu;
        }
    };
    auto after_tiles = [&](int r) {   // publish row r - 1, normalise row r - 7
        if (r - 1 >= r_beg && r - 1 <= last) publish(r - 1);
        const int xf = r - kConsumeLag;
        if (xf >= r_beg && xf <= last) consume(xf);
    };

    // ---- prologue: query row 0 staged; then the loads in the order every
    // iteration issues them: row 0's tiles, the requests and row 1's query,
    // row 1's tiles
    load_q(r_beg);
    store_q(r_beg);
    lds_sync();
    // Two rings of four tiles: row r's tiles sit in ring r & 1, and the
    // loads of row r + 2 go out as soon as row r's tiles have been through
    // MFMA, so two rows of loads are in flight while a wave works on a row.
    u32x4 ringA[KT][4], ringB[KT][4];
#pragma unroll
    for (int u = 0; u < KT; ++u) load_tile(ringA[u], r_beg, u);
    if (((r_beg - 5) & (W - 1)) == wv) load_norm(r_beg);
    load_q(min(r_beg + 1, last));
#pragma unroll
    for (int u = 0; u < KT; ++u) load_tile(ringB[u], min(r_beg + 1, last + 2), u);

    // Row r:
    //   1. logits of the four tiles on MFMA, k-chunk by k-chunk (the chunk's
    //      query terms are read from LDS once, the four accumulations run
    //      side by side);
    //   2. bookkeeping on the last iteration's loads; the query of row r + 1
    //      into LDS; this iteration's requests and row r + 2's query;
    //   3. softmax statistics of row r, its logits into LDS;
    //   4. publish row r - 1, normalise row r - 7; row r's statistics into
    //      LDS; barrier.
    // The four tiles of row r + 2 go out one by one between these steps
    // rather than in one burst: a burst of all waves' loads at once stalls
    // every wave at issue, while spread out the issue waits overlap the
    // work of the row.
    auto do_row = [&](u32x4 (&ring)[KT][4], int row) {
        const uint32_t* qb = sm.qs + (size_t)(row & 1) * 3 * G * 64 + hh * 64 + 4 * g;
        // Quantised tiles: the scale (the same 16 bytes in every lane) goes
        // to a scalar, and the codes are widened to bf16 (exact) in place,
        // so the MFMA loop below is the plain one and holds no second copy
        // of the tile; the scale multiplies the finished sums.
        float qsc[KT];
        if constexpr (QT) {
#pragma unroll
            for (int u = 0; u < KT; ++u) {
                qsc[u] = 1.0f;
                if ((qmask >> u) & 1u) {
                    qsc[u] = __uint_as_float(__builtin_amdgcn_readfirstlane(ring[u][2][0]));
                    // last slot first: each widened slot takes the place of
                    // one whose contents are no longer needed
                    ring[u][3] = codes_to_bf16<1>(ring[u][1]);
                    ring[u][2] = codes_to_bf16<0>(ring[u][1]);
                    ring[u][1] = codes_to_bf16<1>(ring[u][0]);
                    ring[u][0] = codes_to_bf16<0>(ring[u][0]);
                }
            }
        }
        f32x4 c[KT];
#pragma unroll
        for (int u = 0; u < KT; ++u) c[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            u32x4 bq[3];
#pragma unroll
            for (int p = 0; p < 3; ++p) bq[p] = *reinterpret_cast<const u32x4*>(qb + p * G * 64 + 16 * j);
#pragma unroll
            for (int u = 0; u < KT; ++u) {
#pragma unroll
                for (int p = 0; p < 3; ++p)
                    c[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        __builtin_bit_cast(bf16x8, ring[u][j]), __builtin_bit_cast(bf16x8, bq[p]), c[u], 0, 0, 0);
            }
        }
        if constexpr (QT) {
#pragma unroll
            for (int u = 0; u < KT; ++u)
                if ((qmask >> u) & 1u) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) c[u][i] *= qsc[u];
                }
        }
        load_tile(ring[0], row + 2, 0);
        use_loads(row);
        load_tile(ring[1], row + 2, 1);
        if (row + 1 < r_end) store_q(row + 1);
        issue_loads(row);
        load_q(min(row + 2, last));
        load_tile(ring[2], row + 2, 2);

        // Base-2 logits of the wave's 64 tokens (lane: head h, tokens
        // 16 u + 4 g + i), their maximum and the sum of 2^(logit - max) per
        // head; the LDS row keeps 2^(logit - max).
        float xs[KT][4];
#pragma unroll
        for (int u = 0; u < KT; ++u)
#pragma unroll
            for (int i = 0; i < 4; ++i) xs[u][i] = c[u][i] * kLogitScale;
        if (!wave_full) {   // tokens past the unit's end, tiles without a page
#pragma unroll
            for (int u = 0; u < KT; ++u)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (!((vmask >> u) & 1ull) || wtok0 + 16 * u + 4 * g + i >= un.ntok ||
                        (AL && 4 * g + i >= (int)((lims >> (8 * u)) & 0xffu)) ||
                        (WN && ((unseen >> (4 * u + i)) & 1u)))
                        xs[u][i] = -INFINITY;
        }
        float mx = -INFINITY;
#pragma unroll
        for (int u = 0; u < KT; ++u)
            mx = fmaxf(mx, fmaxf(fmaxf(xs[u][0], xs[u][1]), fmaxf(xs[u][2], xs[u][3])));
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float ms = mx == -INFINITY ? 0.0f : mx;
        float ls = 0.0f;
        float* rbw = sm.rowbuf + ((size_t)(row % kRowBufs) * G + h) * kTs + wtok0 + 4 * g;
#pragma unroll
        for (int u = 0; u < KT; ++u) {
            f32x4 pv;
#pragma unroll
            for (int i = 0; i < 4; ++i) pv[i] = hw_exp2(xs[u][i] - ms);
            ls += (pv[0] + pv[1]) + (pv[2] + pv[3]);
            if (h < G) *reinterpret_cast<f32x4*>(rbw + 16 * u) = pv;
        }
        load_tile(ring[3], row + 2, 3);
        ls += __shfl_xor(ls, 16);
        ls += __shfl_xor(ls, 32);
        after_tiles(row);
        if (g == 0 && h < kSlots) wm_wave[(size_t)(row % kRowBufs) * W * kSlots + h] = ms;
        if (g == 0 && h < G) sm.wstat[((row & 1) * W + wv) * 16 + h] = make_float2(mx, ls);
        lds_sync();
    };
    int row = r_beg;
    for (; row + 1 < r_end; row += 2) {
        do_row(ringA, row);
        do_row(ringB, row + 1);
    }
    if (row < r_end) do_row(ringA, row);

    // ---- lane mode: the lane's next pass, claimed before this unit's
    // drain, so that the lane's other workgroups find it published as they
    // finish (claimed after the drain, they waited for it about 10 us)
    if (next_box != nullptr) {
        claim_sessions(a, sm.claim, claim_lane, cap);
        if (threadIdx.x == 0) {
            __hip_atomic_store(next_box,
                               ((unsigned long long)tag << 32) | ((uint32_t)sm.claim[0] << 16) | (uint32_t)sm.claim[1],
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            sm.claim[24] = 1;
        }
    }

    // ---- iterations without tiles, until the last row is normalised
    for (int r = r_end; r < r_end + kConsumeLag; ++r) {
        use_loads(r);
        issue_loads(r);
        after_tiles(r);
        lds_sync();
    }

    // ---- row groups: every group but the first hands its tokens' partial
    // masses to the unit of group 0 (same tokens) as tagged words, a NaN
    // payload marking a void step; that unit adds them in group order and
    // finishes the tokens alone.
    if constexpr (RS) {
        if (un.rg > 1) {
            const bool void_here = *sm.vflag != 0;
            unsigned long long* pbase = a.upart + (size_t)(un.ubase + un.j) * kT + wtok0 + lane;
            const size_t gstride = (size_t)un.nu * kT;   // the words of one group's units
            if (un.grp != 0) {
#pragma unroll
                for (int k = 0; k < kTok; ++k)
                    __hip_atomic_store(pbase + un.grp * gstride + 64 * k,
                                       tag_hi | (void_here ? 0x7fc00000u : __float_as_uint(acc[k])),
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (void_here && threadIdx.x == 0) a.valid[un.s] = 0;
                return;
            }
            if (!void_here) {
                unsigned long long pw[kMaxRowGroups - 1][kTok];
                auto load_parts = [&] {
#pragma unroll
                    for (int g2 = 1; g2 < kMaxRowGroups; ++g2)
#pragma unroll
                        for (int k = 0; k < kTok; ++k)
                            pw[g2 - 1][k] = g2 < un.rg ? __hip_atomic_load(pbase + g2 * gstride + 64 * k, __ATOMIC_RELAXED,
                                                                           __HIP_MEMORY_SCOPE_AGENT)
                                                       : tag_hi;
                };
                load_parts();
                await_tags(
                    [&] {
                        bool ok = true;
#pragma unroll
                        for (int g2 = 1; g2 < kMaxRowGroups; ++g2)
#pragma unroll
                            for (int k = 0; k < kTok; ++k) ok &= tag_ok(pw[g2 - 1][k]);
                        return ok;
                    },
                    load_parts);
                bool bad = false;
#pragma unroll
                for (int g2 = 1; g2 < kMaxRowGroups; ++g2)
#pragma unroll
                    for (int k = 0; k < kTok; ++k) {
                        if (g2 < un.rg) {
                            const float pv = __uint_as_float((uint32_t)pw[g2 - 1][k]);
                            bad |= pv != pv;
                            acc[k] += pv;
                        }
                    }
                if (bad) *sm.vflag = 1;
            }
            lds_sync();   // every wave sees the unit's void flag
        }
    }

    // ---- Eq. 2 and Eq. 3 for this wave's tokens, then their retention
    // scores (Eq. 4) and the scores of their pages (Eq. 5): a page's P
    // tokens are P consecutive lanes of one wave, since units and waves
    // start at multiples of 64 tokens.
    // A void step (a non-finite query, or a wait that ran out) changes no
    // token's state and leaves the session out of this step's selection and
    // compaction.
    if (*sm.vflag != 0) {
        if (threadIdx.x == 0) a.valid[un.s] = 0;
        return;
    }
    // Every load first, then the stores: a wait for a load also waits for
    // the stores issued before it.  The session's region priors are read
    // once per wave (lane r holds region r's) and picked by shuffles.
    const int t_now = a.clock[un.s];
    const size_t rbase = (size_t)un.s * dm.n_regions;
    const float b_l = lane < dm.n_regions ? a.b[rbase + lane] : 0.0f;
    const float lam_l = lane < dm.n_regions ? a.lam[rbase + lane] : 0.0f;
    const int n_tok = AL ? un.nl_s : un.nt_s;   // |K_t|
    const float aw = attention_weight(dm.alpha, dm.norm_attn, n_tok);
    bool live[kTok];
    size_t si[kTok];
    float a_old[kTok];
    int tr_old[kTok], reg[kTok];
#pragma unroll
    for (int k = 0; k < kTok; ++k) {
        const int lt = lane + 64 * k;   // wave-local token
        const int tile = lt >> 4;
        const int slot0 = __shfl(myslot, tile);
        // holes hold no token
        live[k] = wtok0 + lt < un.ntok && ((vmask >> tile) & 1ull) &&
                  (!AL || (lt & 15) < (int)((lims >> (8 * tile)) & 0xffu));
        si[k] = (size_t)slot0 + (lt & 15);
        a_old[k] = 0.0f;
        tr_old[k] = reg[k] = 0;
        if (live[k]) {
            a_old[k] = a.imp[si[k]];
            tr_old[k] = a.t_ref[si[k]];
            reg[k] = a.region[si[k]];
        }
    }
#pragma unroll
    for (int k = 0; k < kTok; ++k) {
        const int lt = lane + 64 * k;
        int r = reg[k];
        if (live[k] && r >= dm.n_regions) {
            atomicOr(a.status, kDevCorrupt);
            r = dm.n_regions - 1;
        }
        const float br = __shfl(b_l, r), lamr = __shfl(lam_l, r);
        float sc = 0.0f;
        bool pin = false;
        if (live[k]) {
            const float abar = acc[k] / (float)dm.R;
            const float an = fmaf(dm.rho, a_old[k], (1.0f - dm.rho) * abar);
            a.imp[si[k]] = an;
            int tr = tr_old[k];
            if (abar >= dm.tau_scale / (float)n_tok) {
                tr = t_now;
                a.t_ref[si[k]] = tr;
            }
            if (a.abar_out != nullptr) a.abar_out[si[k]] = abar;
            pin = (dm.pin_mask >> r) & 1u;
            sc = pin ? INFINITY : retention_score(br, lamr, t_now, tr, aw, an);
        }
        float ps;
        const bool has = page_score_of(sc, live[k], pin, dm.P, &ps);
        const int tok = un.j * kT + wtok0 + lt;
        if ((lt & (dm.P - 1)) == 0 && has) a.pscore[(size_t)un.s * dm.MP + (tok >> dm.Pshift)] = ps;
    }
}

// ------------------------------------------------------------ passes

// Number of threads of the workgroup with p set (tmp: 17 ints of LDS).
// Contains barriers.
__device__ int count_true(bool p, int* tmp) {
    const int k = __popcll(__ballot(p));
    if (threadIdx.x == 0) tmp[16] = 0;
    __syncthreads();
    if (lane_id() == 0 && k > 0) atomicAdd(&tmp[16], k);
    __syncthreads();
    const int total = tmp[16];
    __syncthreads();
    return total;
}

// Number of i < n with v[i] <= x, for non-decreasing v, counted by the whole
// workgroup in chunks of blockDim.x (tmp: 17 ints of LDS).  Wave-uniform
// result; contains barriers.
__device__ int count_at_most(const int32_t* v, int n, int x, int* tmp) {
    int total = 0;
    for (int c = 0; c < n; c += blockDim.x) {
        const int i = c + (int)threadIdx.x;
        total += count_true(i < n && v[i] <= x, tmp);
    }
    return uni(total);
}

// Lane mode: the lane's first workgroup claims the next sessions of the
// step for one pass of its lane: consecutive sessions whose units add up to
// at most cap, from the front of the unclaimed range (lane 0) or from its
// back (lane 1), by compare-and-swap on the (first, end) word.  Writes the
// claimed [first, end) to xs[0], xs[1] (both 0 when nothing is left).
// Whole workgroup; contains barriers.
__device__ void claim_sessions(const AttendArgs& a, int* xs, int lane_no, int cap) {
    const bool front = (lane_no & 1) == 0;
    int* tmp = xs + 2;
    while (true) {
        if (threadIdx.x == 0) {
            const unsigned long long c = __hip_atomic_load(a.claim, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            xs[4 + 17] = (int)(c >> 32);
            xs[5 + 17] = (int)(c & 0xffffffffu);
        }
        __syncthreads();
        const int f = xs[4 + 17], e = xs[5 + 17];
        if (f >= e) {
            if (threadIdx.x == 0) xs[0] = xs[1] = 0;
            __syncthreads();
            return;
        }
        // units of the t-th session from the claiming end (one window of
        // blockDim.x sessions; a pass never holds more sessions than that
        // unless some have no units, and then the next pass takes the rest)
        const int t = (int)threadIdx.x;
        const int s = front ? f + t : e - 1 - t;
        const int u = (t < e - f) ? a.ustart[s + 1] - a.ustart[s] : (cap + 1);
        int tot;
        const int before = block_exclusive_scan(u, tmp, &tot);
        const bool take = t < e - f && before + u <= cap;
        const int k = count_true(take, tmp);   // sessions taken (a prefix)
        if (threadIdx.x == 0) {
            const int nf = front ? f + k : f, ne = front ? e : e - k;
            const unsigned long long want = ((unsigned long long)(uint32_t)nf << 32) | (uint32_t)ne;
            const unsigned long long seen = ((unsigned long long)(uint32_t)f << 32) | (uint32_t)e;
            const unsigned long long got = atomicCAS(a.claim, seen, want);
            xs[4 + 17] = got == seen;
            xs[0] = front ? f : e - k;
            xs[1] = front ? f + k : e;
        }
        __syncthreads();
        const bool done = xs[4 + 17] != 0;
        __syncthreads();
        if (done) return;
    }
}

// ------------------------------------------------------------ kernel

// Two workgroups per CU (two waves per SIMD) for groups of up to eight query
// heads; larger groups need a CU's LDS for one workgroup, which then may use
// the whole register file.  (Workgroups that take a whole CU, with eight
// waves or with eight tiles per wave, measured slower: the two workgroups'
// row barriers fall at different times and fill each other's gaps.)
template <int W, int NH, int KT, bool AL, bool QT, bool WN, bool RS>
__global__ void __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(NH == 4 ? 1 : 2)))
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
    const Lds sm = carve(smem, dm.G, W, KT);
    const int wv = uni(threadIdx.x >> 6);
    const uint32_t tag = (uint32_t)a.epoch[0];
    // Between units the row buffer is free: it holds the pass bookkeeping.
    int* xs = reinterpret_cast<int*>(sm.rowbuf);
    const int n_pass = a.plan[0];
    const bool lanes = n_pass < 0;
    // Lane mode.  The first workgroup dispatched to each CU (blocks
    // 0 .. n_cu - 1) wins most memory issue slots over the second, so the
    // two kinds run at different speeds.  Each kind forms a lane with one
    // workgroup per CU; a lane runs passes of whole sessions that it claims
    // itself, lane 0 from the front of the session list and lane 1 from the
    // back, so the units of one session always share a lane and start
    // together, and the faster lane takes more sessions.  The first pass of
    // each lane is claimed and published before the kernel starts (by the
    // append kernel), so no workgroup waits to begin.
    const int lane_no = lanes ? (int)blockIdx.x / dm.n_cu : 0;
    const int w = lanes ? (int)blockIdx.x % dm.n_cu : (int)blockIdx.x;
    const int cap = lanes ? dm.n_cu : 0;
    if (threadIdx.x == 0) sm.claim[24] = 0;   // ordered before its reads by the barrier below
    for (int ps = 0;; ++ps) {
        lds_sync();   // the previous unit is done with the LDS
        if (threadIdx.x == 0) *sm.vflag = 0;   // ordered before the unit by the barriers below
        int sb, se;
        if (!lanes) {
            if (ps >= n_pass) break;
            sb = a.plan[2 + 3 * ps];
            se = a.plan[3 + 3 * ps];
        } else {
            // the lane's first workgroup claimed this pass during its last
            // unit (unless that pass gave it no unit)
            const bool ahead = w == 0 && ps > 0 && sm.claim[24] != 0;
            if (w == 0 && ps > 0 && !ahead) claim_sessions(a, xs, lane_no, cap);
            if (threadIdx.x == 0) {
                unsigned long long* box = a.lane_box + (size_t)lane_no * (dm.S + 1) + ps;
                if (ahead) {
                    xs[0] = sm.claim[0];
                    xs[1] = sm.claim[1];
                } else if (w == 0 && ps > 0) {
                    __hip_atomic_store(box, ((unsigned long long)tag << 32) | ((uint32_t)xs[0] << 16) | (uint32_t)xs[1],
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                } else {
                    // the lane's first workgroup publishes the pass once its
                    // own unit of the last pass is done (bounded wait)
                    const uint64_t t0 = now_ticks();
                    unsigned long long v = __hip_atomic_load(box, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    while ((uint32_t)(v >> 32) != tag) {
                        if (now_ticks() - t0 > kUnitTicks) {
                            atomicOr(a.status, MD_DEV_TIMEOUT);
                            v = 0;
                            break;
                        }
                        __builtin_amdgcn_s_sleep(8);
                        v = __hip_atomic_load(box, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                    xs[0] = (int)((v >> 16) & 0xffff);
                    xs[1] = (int)(v & 0xffff);
                }
            }
            __syncthreads();
            sb = xs[0];
            se = xs[1];
            if (threadIdx.x == 0 && ahead) sm.claim[24] = 0;   // read by all threads before the barrier above
            if (sb >= se) break;
        }
        const int u0 = a.ustart[sb];
        if (w >= a.ustart[se] - u0) continue;
        // session of unit u0 + w: the last s in [sb, se) with ustart[s] <= u0 + w
        const int s = sb + count_at_most(a.ustart + sb, se - sb, u0 + w, xs + 2) - 1;
        Unit un;
        un.s = s;
        un.us = a.ustart[s];
        un.nu = a.ustart[s + 1] - un.us;
        un.j = u0 + w - un.us;
        if constexpr (RS) {
            // the session's units are rg groups of nu / rg units, group g
            // covering rows [g L Hkv / rg, (g + 1) L Hkv / rg)
            const int rg = min(max(dm.rg, 1), kMaxRowGroups);
            const int nut = max(un.nu / rg, 1);
            if (un.nu != nut * rg && threadIdx.x == 0) atomicOr(a.status, kDevCorrupt);
            un.rg = rg;
            un.ubase = un.us;
            un.grp = min(un.j / nut, rg - 1);
            un.j -= un.grp * nut;
            un.nu = nut;
            un.us += un.grp * nut;
            un.r0 = un.grp * dm.LHkv / rg;
            un.r1 = (un.grp + 1) * dm.LHkv / rg;
        }
        un.nt_s = a.n_tokens[s];
        un.nl_s = AL ? a.n_live[s] : 0;
        constexpr int kT = 16 * W * KT;
        un.ntok = min(kT, un.nt_s - un.j * kT);
        un.deadline = now_ticks() + kUnitTicks;
        // The lane index is made opaque here so that per-lane address
        // arithmetic is not hoisted out of the pass loop and kept live.
        int lane = (int)threadIdx.x & 63;
        asm volatile("" : "+v"(lane));
        unsigned long long* next_box =
            (lanes && w == 0) ? a.lane_box + (size_t)lane_no * (dm.S + 1) + ps + 1 : nullptr;
        attend_wave<W, NH, KT, AL, QT, WN, RS>(dm, a, sm, un, wv, lane, tag, lane_no, cap, next_box);
    }
}

}  // namespace

size_t attend_lds_bytes(int G) {
    const int W = attend_threads(G) / 64;
    return rowbuf_bytes(G, W, attend_unit_tokens(G) / (16 * W)) + qs_bytes(G) + wstat_bytes(W) + kNormBytes +
           kFlagBytes + kClaimBytes + wmax_bytes(G, W);
}

namespace {
template <bool AL, bool QT, bool WN, bool RS = false>
const void* attend_for(int G) {
    if (G <= 4) return reinterpret_cast<const void*>(&k_attend<4, 1, 4, AL, QT, WN, RS>);
    if (G <= 8) return reinterpret_cast<const void*>(&k_attend<4, 2, 4, AL, QT, WN, RS>);
    return reinterpret_cast<const void*>(&k_attend<4, 4, 4, AL, QT, WN, RS>);
}
}  // namespace

// G: MFMA columns (query heads per KV head times window queries).  Row
// groups run only on plain pages in full precision with one query.
const void* attend_kernel(int G, int aligned, int quant, int window, int row_groups) {
    if (window > 1) {
        if (aligned) return quant ? attend_for<true, true, true>(G) : attend_for<true, false, true>(G);
        return quant ? attend_for<false, true, true>(G) : attend_for<false, false, true>(G);
    }
    if (aligned) return quant ? attend_for<true, true, false>(G) : attend_for<true, false, false>(G);
    if (quant) return attend_for<false, true, false>(G);
    return row_groups > 1 ? attend_for<false, false, false, true>(G) : attend_for<false, false, false>(G);
}

// The grid as one launch: cooperative (the runtime keeps the device to it)
// with MD_FLAG_COOPERATIVE, an ordinary one otherwise (measured 15-20 us
// less per step; residency is checked at init with the same launch kind).
// With an event pair (t0, t1), an ordinary launch records the events with
// the kernel's dispatch itself.
static hipError_t launch_grid(const Dims& dm, int n_wg, int rg, void** args, hipStream_t st, hipEvent_t t0 = nullptr,
                              hipEvent_t t1 = nullptr) {
    const void* fn = attend_kernel(dm.G * dm.W, dm.aligned, dm.quant, dm.W, rg);
    const dim3 grid(n_wg), block(attend_threads(dm.G * dm.W));
    const unsigned lds = (unsigned)attend_lds_bytes(dm.G * dm.W);
    if (dm.coop) return hipLaunchCooperativeKernel(fn, grid, block, args, lds, st);
    if (t0 != nullptr && t1 != nullptr) return hipExtLaunchKernel(fn, grid, block, args, lds, st, t0, t1, 0);
    return hipLaunchKernel(fn, grid, block, args, lds, st);
}

hipError_t launch_attend(const Dims& dm, const View& v, const Scratch& sc, const float* q, float* abar_out,
                         int rg, hipStream_t st, hipEvent_t t0, hipEvent_t t1) {
    AttendDims ad{dm.L, dm.Hq, dm.Hkv, dm.G * dm.W, dm.P, dm.Pshift, dm.MP, dm.NP, dm.R, dm.LHkv,
                  dm.wg_per_cu, dm.n_wg / dm.wg_per_cu, dm.S, dm.n_regions, dm.norm_attn, dm.pin_mask,
                  dm.rho, dm.tau_scale, dm.alpha, dm.aligned, dm.G, dm.W, rg};
    AttendArgs aa{v.k_pool, v.page_table, v.n_tokens, v.clock, v.region, v.b, v.lam, v.imp, v.t_ref,
                  sc.pscore, q, abar_out, sc.ustart, sc.plan, sc.epoch, sc.claim, sc.lane_box, sc.ustat,
                  sc.unorm, sc.status, nullptr, v.n_live, v.page_format, v.t_ins, sc.valid, sc.upart};
    void* args[] = {&ad, &aa};
    return launch_grid(dm, dm.n_wg, rg, args, st, t0, t1);
}

hipError_t launch_attend_check(const Dims& dm, int32_t* probe, int n_wg, int rg, hipStream_t st) {
    AttendDims ad{};
    AttendArgs aa{};
    aa.probe = probe;
    hipError_t e = hipMemsetD32Async(reinterpret_cast<hipDeviceptr_t>(probe), 0, 1, st);
    if (e == hipSuccess) e = hipMemsetD32Async(reinterpret_cast<hipDeviceptr_t>(probe + 1), 1 << 30, 1, st);
    if (e != hipSuccess) return e;
    void* args[] = {&ad, &aa};
    return launch_grid(dm, n_wg, rg, args, st);
}

}  // namespace md
