// gfx950 kernels of the MemDecay observation step.
//
// A step over a batch of sessions runs these kernels on the caller's stream (the
// fused observation kernel of md_attend.hip replaces k_logits, k_rowstats,
// k_mass and, for the library's own page scores, k_score):
//   k_append    one block per session: clock, append into the tail page or a
//               page popped from the free list, copy of the new key rows; the
//               last block builds the step's work lists.
//   k_logits    HOT: every cached token's logits q.k/sqrt(d) for all query heads
//               (Sec. III-C), one 128-token chunk of one (layer, KV head) per
//               wave, on MFMA; chunk softmax statistics; logits spilled for
//               the normalisation pass.
//   k_rowstats  per (session, layer, query head): softmax max and 1/sum over
//               the chunk statistics, in a fixed order.
//   k_mass      per token: attention mass A_i, EWMA (Eq. 2), refresh (Eq. 3).
//   k_score     per token: retention score (Eq. 4); per page: mean (Eq. 5).
//   k_select    one block per session: weighted radix select of the pages to
//               evict (Sec. III-D, Alg. 1).
//   k_compact   one block per session: page-table compaction, free-list push.
//   k_evict     k_select and the compaction of its selection in one launch
//               (md_select_compact without a tier).
// Every reduction is in a fixed order; no float atomics are used.

#include <mutex>

#include "md_device.h"

namespace md {

// Scratch of handles made by md_init_static, for callers that cannot
// allocate device memory.  Host code must not pass the array's name to a
// kernel or a copy (it stands for the host-side shadow); static_scratch
// hands out the device address instead.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

hipError_t static_scratch(void** ptr) {
    constexpr int kMaxDevices = 64;
    static void* addr[kMaxDevices];   // device address of the array, per device
    static std::mutex mu;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (addr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

// ---------------------------------------------------------------- append

// Whether the append of session s2 opens a page (takes one from the free
// list), judged on the counters as they stand before the append: the last
// page is full, or with region-aligned pages the token's region differs
// from the last token's; and the page table has room.
__device__ bool opens_page(const Dims& dm, const View& v, int s2, const uint8_t* __restrict__ new_region) {
    const int np = v.n_pages[s2];
    const int nt = v.n_tokens[s2];
    if (!counters_ok(np, nt, dm) || np >= dm.MP) return false;
    if (!(np > 0 && nt < np * dm.P)) return true;
    if (!dm.aligned) return false;
    const int p = v.page_table[(size_t)s2 * dm.MP + np - 1];
    if (p < 0 || p >= dm.NP) return false;
    const int slot = nt - (np - 1) * dm.P;
    return v.region[(size_t)p * dm.P + slot - 1] != new_region[s2];
}

// One block per session: the append.  The last block (highest index) also
// lays out the step's work lists.
// Pages leave the free list in session order: session s takes the entry
// below those of the sessions before it that open a page at this append.
// No block but the last changes a session's page or token count (each block
// hands its session's new counts to the last one), so every block judges
// the earlier sessions on the counts before the append.
//
// Each block hands its session's new counts to the last block as one 64-bit
// word stored at device scope and tagged with the launch (`tag`, different
// for consecutive launches), so the hand-off needs no memory fence: the last
// block reads the words and waits, bounded, for any that still carries an
// older tag.  (A device-scope fence writes back the L2 of the block's XCD.)
__device__ __forceinline__ unsigned long long append_word(uint32_t tag, bool bad, bool appended, int np, int nt) {
    return ((unsigned long long)(tag & kWordTagMask) << 37) | ((unsigned long long)bad << 36) |
           ((unsigned long long)appended << 34) | ((unsigned long long)(np & 0x3FFF) << 20) |
           (unsigned long long)(nt & 0xFFFFF);
}

__global__ void __launch_bounds__(256) k_append(Dims dm, View v, Scratch sc,
                                                const uint16_t* __restrict__ new_k,
                                                const uint8_t* __restrict__ new_region, int fused,
                                                int observe, int rg, uint32_t tag) {
    const int s = blockIdx.x;
    __shared__ int sh_phys, sh_slot, sh_rank;
    __shared__ int lds[5 * 17];
    // The step's key rows (16 pieces of 16 bytes per (layer, KV head) row)
    // do not depend on the slot: waves 1.. read their first kPre pieces now
    // and write them once the slot is known, while wave 0 finds the slot
    // (its loads are then not queued behind the copy's).
    constexpr int kPre = 8;
    const int n_pieces = new_k != nullptr ? dm.LHkv * 16 : 0;
    const u32x4* src = new_k != nullptr ? reinterpret_cast<const u32x4*>(new_k) + (size_t)s * dm.LHkv * 16 : nullptr;
    const int ct = (int)threadIdx.x - 64, nct = (int)blockDim.x - 64;   // copy threads
    u32x4 kr[kPre];
    if (ct >= 0) {
#pragma unroll
        for (int c = 0; c < kPre; ++c) {
            const int i = ct + c * nct;
            if (i < n_pieces) kr[c] = src[i];
        }
    }
    // Thread 0's own counters go out with the other sessions' below (the
    // pages the sessions before this one take at this append), and the last
    // page's table entry right behind them, so the chain to the slot is
    // three round trips to memory rather than six.
    int t0_clock = 0, np = 0, nt = 0, fc0 = 0, ep0 = 0, ns0 = 0, last_p = -1, wants_page = 0;
    uint8_t rg_new = 0;
    if (threadIdx.x == 0) {
        t0_clock = v.clock[s];
        np = v.n_pages[s];
        nt = v.n_tokens[s];
        fc0 = v.free_count[0];   // the free count and the epoch change only in the last block
        ep0 = *sc.epoch;
        ns0 = v.next_serial[s];
        if (new_k != nullptr) rg_new = new_region[s];
    }
    if (threadIdx.x == 0) sh_rank = 0;
    int rank_mine = 0;
    if (new_k != nullptr)
        for (int s2 = threadIdx.x; s2 < s; s2 += blockDim.x) rank_mine += opens_page(dm, v, s2, new_region) ? 1 : 0;
    if (threadIdx.x == 0 && np > 0 && np <= dm.MP) last_p = v.page_table[(size_t)s * dm.MP + np - 1];
    __syncthreads();
    if (new_k != nullptr) {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) rank_mine += __shfl_xor(rank_mine, o);
        if (lane_id() == 0 && rank_mine > 0) atomicAdd(&sh_rank, rank_mine);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        // Every load first, then the stores: a wait for a load also waits
        // for the stores issued before it.
        const int t = t0_clock + 1;
        const size_t row = (size_t)s * dm.MP;
        int phys = -1, slot = 0, new_p = -1, close_from = -1;
        bool appended = false;
        wants_page = 0;
        const bool bad = !counters_ok(np, nt, dm);
        if (new_k != nullptr && !bad) {
            bool open = !(np > 0 && nt < np * dm.P);
            if (!open) {
                if (last_p >= 0 && last_p < dm.NP) {
                    phys = last_p;
                    slot = nt - (np - 1) * dm.P;
                    // region-aligned pages: a new region closes the last
                    // page, its unused slots becoming holes
                    if (dm.aligned && slot > 0 && v.region[(size_t)last_p * dm.P + slot - 1] != rg_new) {
                        close_from = slot;
                        phys = -1;
                        open = true;
                    }
                } else {
                    atomicOr(sc.status, kDevCorrupt);
                }
            }
            if (!open) {
                // the token joins the last page (or the page was corrupt)
            } else if (np < dm.MP) {
                // the free list is a stack: this session takes the entry
                // below the earlier sessions' ones
                wants_page = 1;
                const int idx = min(fc0, dm.NP) - 1 - sh_rank;
                if (idx >= 0) {
                    const int p = v.free_list[idx];
                    if (p >= 0 && p < dm.NP) {
                        new_p = phys = p;
                        slot = 0;
                    } else {
                        atomicOr(sc.status, kDevCorrupt);
                    }
                } else {
                    atomicOr(sc.status, MD_DEV_CAPACITY);
                }
            } else {
                atomicOr(sc.status, MD_DEV_CAPACITY);
            }
        }
        v.clock[s] = t;
        if (close_from >= 0) {
            const size_t s0 = (size_t)last_p * dm.P;
            for (int o = close_from; o < dm.P; ++o) {
                v.region[s0 + o] = (uint8_t)kHole;
                v.t_ins[s0 + o] = 0;
                v.t_ref[s0 + o] = 0;
                v.imp[s0 + o] = 0.0f;
            }
            nt = np * dm.P;
        }
        if (new_p >= 0) {
            v.page_table[row + np] = new_p;
            v.page_serial[row + np] = ns0;
            if (dm.quant) v.page_format[new_p] = 0;   // a reused page holds bf16 keys again
            v.next_serial[s] = ns0 + 1;
            np += 1;
        }
        if (phys >= 0) {
            nt += 1;
            appended = true;
            const size_t si = (size_t)phys * dm.P + slot;
            v.region[si] = rg_new;
            v.t_ins[si] = t;
            v.t_ref[si] = t;
            v.imp[si] = 0.0f;
        }
        sh_phys = phys;
        sh_slot = slot;
        // the session's counts after the append, applied by the last block
        __hip_atomic_store(sc.app_word + s, append_word(tag, bad, appended, np, nt), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    const int phys = sh_phys;
    if (phys >= 0) {
        // piece b of row r goes to its 16-token block's [b][slot mod 16] place
        const int slot = sh_slot;
        auto place = [&](int i) {
            const int r = i >> 4, part = i & 15;
            u32x4* blk = reinterpret_cast<u32x4*>(
                v.k_pool + (((size_t)phys * dm.LHkv + r) * dm.P + (slot & ~15)) * kHeadDim);
            return blk + part * 16 + (slot & 15);
        };
        if (ct >= 0) {
#pragma unroll
            for (int c = 0; c < kPre; ++c) {
                const int i = ct + c * nct;
                if (i < n_pieces) *place(i) = kr[c];
            }
            for (int i = ct + kPre * nct; i < n_pieces; i += nct) *place(i) = src[i];
        }
    }

    // The last block (the highest index: blocks are dispatched in index
    // order, so every other block has started before it) lays out the step's
    // work lists once every session's word carries this launch's tag.  A
    // block stores its word after all its reads of the counters have
    // returned (the word is computed from them), so no block reads a count
    // the last block has already changed.
    if (s != (int)gridDim.x - 1) return;
    __shared__ int s_n[kMaxSessions];      // token slots in use (0 for a skipped session)
    __shared__ int s_live[kMaxSessions];   // live tokens (with region-aligned pages, holes left out)
    __shared__ int s_pass[kMaxSessions];   // fused pass of the session, -1 on the spill path
    __shared__ int s_pb[kMaxSessions], s_pe[kMaxSessions], s_pl[kMaxSessions];   // pass mode: sessions, units
    __syncthreads();
    for (int s2 = threadIdx.x; s2 < dm.S; s2 += blockDim.x) {
        // loads before the stores (a wait for a load also waits for them)
        const int live0 = dm.aligned ? v.n_live[s2] : 0;
        unsigned long long wd = __hip_atomic_load(sc.app_word + s2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        bool stale = (uint32_t)(wd >> 37) != (tag & kWordTagMask);
        while (stale && __builtin_amdgcn_s_memrealtime() - t0 < kWordWaitTicks) {
            __builtin_amdgcn_s_sleep(2);
            wd = __hip_atomic_load(sc.app_word + s2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            stale = (uint32_t)(wd >> 37) != (tag & kWordTagMask);
        }
        const int np = (int)((wd >> 20) & 0x3FFF), nt = (int)(wd & 0xFFFFF);
        const bool ok = !stale && !((wd >> 36) & 1ull) && counters_ok(np, nt, dm);
        int live = nt;
        if (ok) {
            v.n_pages[s2] = np;
            v.n_tokens[s2] = nt;
            if (dm.aligned) {
                live = live0 + (int)((wd >> 34) & 1ull);
                v.n_live[s2] = live;
            }
        } else {
            atomicOr(sc.status, kDevCorrupt);
        }
        sc.valid[s2] = ok ? 1 : 0;
        s_n[s2] = ok ? nt : 0;
        s_live[s2] = (ok && nt > 0) ? live : 0;
        s_pass[s2] = -1;
    }
    __syncthreads();
    // Entries off the free list: one per session that wants a page, as every
    // block ranked them from the counts before the append (sh_rank counts
    // the other sessions here), whether or not its word arrived in time; a
    // session whose word did not keeps its old counts, and its page, if it
    // took one, is lost to the list rather than handed out twice.
    if (threadIdx.x == 0) v.free_count[0] = max(min(fc0, dm.NP) - (sh_rank + wants_page), 0);
    // Lane mode when every fused session fits half a lane (one workgroup
    // per CU): each lane then claims whole sessions as it goes (see
    // k_attend), at least two per pass.  A larger session would leave the
    // rest of its lane idle for the whole pass (a 32,769-token session is
    // 129 units: one per lane pass, half of the grid idle), so steps with
    // such sessions, typically the first observation of long prompts, run
    // the plan's passes over the whole grid instead, which pack them closer
    // and let each workgroup start its next unit as soon as it is done.
    __shared__ int s_lane_ok;
    if (threadIdx.x == 0) s_lane_ok = fused && dm.wg_per_cu >= 2;
    __syncthreads();
    // With row groups a session's units are rg groups of its token units.
    if (fused) {
        for (int s2 = threadIdx.x; s2 < dm.S; s2 += blockDim.x) {
            const int u = (s_n[s2] + dm.T - 1) / dm.T * rg;
            if (2 * u > dm.lane_cap) atomicExch(&s_lane_ok, 0);
            if (u <= dm.n_wg) s_pass[s2] = 0;
        }
    }
    __syncthreads();
    const bool lane_mode = fused && s_lane_ok;
    __shared__ int sh_f0, sh_e1;
    if (threadIdx.x == 0) {
        sh_f0 = min(dm.S, (int)blockDim.x);
        sh_e1 = max(0, dm.S - (int)blockDim.x);
    }
    if (threadIdx.x == 0 && fused && !lane_mode) {
        // Pass mode: sessions in order, packed greedily into passes of at
        // most n_wg units (a session's units wait for each other row by row,
        // so all of them run in the same pass).  A session larger than a
        // whole pass takes the spill path.  (The lane plan follows the work
        // lists below.)
        // Then neighbouring passes are evened out from the back: greedy
        // packing can leave the last pass nearly empty (16 sessions of 129
        // units give five passes of three and one of one), and a pass of few
        // units streams at a fraction of the bandwidth (a quarter of the grid
        // reads at about 2.5 TB/s, half of it at about 6.4), so the previous
        // pass's last sessions move into the next one while that lowers the
        // larger of the two passes' units.
        auto units = [&](int s2) { return (s_n[s2] + dm.T - 1) / dm.T * rg; };
        for (int s2 = 0; s2 < dm.S; ++s2) s_pass[s2] = -1;
        int np = 0, s0 = 0;
        while (s0 < dm.S) {
            int used = 0, e = s0;
            while (e < dm.S) {
                const int u = units(e);
                if (used + u > dm.n_wg) break;
                used += u;
                ++e;
            }
            if (e == s0) {   // too large for any pass
                ++s0;
                continue;
            }
            s_pb[np] = s0;
            s_pe[np] = e;
            s_pl[np] = used;
            ++np;
            s0 = e;
        }
        for (int p = np - 1; p >= 1; --p) {
            while (s_pe[p - 1] == s_pb[p] && s_pe[p - 1] - s_pb[p - 1] > 1) {
                const int u = units(s_pe[p - 1] - 1);
                if (s_pl[p] + u > dm.n_wg || s_pl[p] + u >= s_pl[p - 1]) break;
                s_pl[p - 1] -= u;
                s_pl[p] += u;
                s_pe[p - 1] -= 1;
                s_pb[p] -= 1;
            }
        }
        for (int p = 0; p < np; ++p) {
            for (int s2 = s_pb[p]; s2 < s_pe[p]; ++s2) s_pass[s2] = p;
            sc.plan[1 + 3 * p] = dm.T;
            sc.plan[2 + 3 * p] = s_pb[p];
            sc.plan[3 + 3 * p] = s_pe[p];
        }
        sc.plan[0] = np;
        *sc.epoch = ep0 + 1;
    }
    __syncthreads();
    // Work lists: fused units; attention items, chunks and mass tiles of the
    // spill path; score tiles for every session.
    int uu[4], it[4], ti[4], si[4];
    int my_units = 0, my_items = 0, my_tiles = 0, my_stiles = 0, my_tokens = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int s2 = threadIdx.x * 4 + k;
        uu[k] = it[k] = ti[k] = si[k] = 0;
        if (s2 < dm.S) {
            const int nt = s_n[s2];
            const int ps = s_pass[s2];
            const bool spill = ps < 0;
            const int ch = spill ? (nt + kChunk - 1) / kChunk : 0;
            sc.chunks[s2] = ch;
            uu[k] = spill ? 0 : (nt + dm.T - 1) / dm.T * rg;
            it[k] = ch * dm.LHkv;
            ti[k] = spill ? (nt + kTile - 1) / kTile : 0;
            si[k] = (nt + kTile - 1) / kTile;
            my_tokens += s_live[s2];
        }
        my_units += uu[k];
        my_items += it[k];
        my_tiles += ti[k];
        my_stiles += si[k];
    }
    const int mine[5] = {my_units, my_items, my_tiles, my_stiles, my_tokens};
    int ex[5], tot[5];
    block_exclusive_scan_n<5>(mine, lds, ex, tot);
    int ex_u = ex[0], ex_i = ex[1], ex_t = ex[2], ex_s = ex[3];
    const int tot_u = tot[0], tot_i = tot[1], tot_t = tot[2], tot_s = tot[3], tot_n = tot[4];
    // Lane mode: the first pass of each lane, claimed here: lane 0 the
    // longest prefix of sessions, lane 1 the longest suffix of the rest, each
    // within one workgroup per CU (lane_cap units) and at most blockDim.x
    // sessions (what the kernel's own claims take); the rest stays to be
    // claimed.  The prefix ends at the first session whose inclusive unit
    // count exceeds lane_cap, the suffix starts after the last session whose
    // suffix count does (both counts are monotone), each found by the one
    // thread that sees the crossing.
    const int cap = dm.lane_cap;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int s2 = threadIdx.x * 4 + k;
        if (s2 < dm.S) {
            sc.ustart[s2] = ex_u;
            sc.item_prefix[s2] = ex_i;
            sc.tile_prefix[s2] = ex_t;
            sc.score_prefix[s2] = ex_s;
            if (lane_mode) {
                const int incl = ex_u + uu[k];
                if (s2 < (int)blockDim.x && ex_u <= cap && cap < incl) atomicMin(&sh_f0, s2);
                if (tot_u - ex_u > cap && tot_u - incl <= cap) atomicMax(&sh_e1, s2 + 1);
            }
        }
        ex_u += uu[k];
        ex_i += it[k];
        ex_t += ti[k];
        ex_s += si[k];
    }
    if (lane_mode) __syncthreads();
    if (threadIdx.x == 0) {
        if (lane_mode) {
            const int f0 = sh_f0, e1 = max(sh_e1, f0);
            const int ep = ep0 + 1;
            sc.plan[0] = -1;
            *sc.epoch = ep;
            const unsigned long long tag = (unsigned long long)(uint32_t)ep << 32;
            sc.lane_box[0] = tag | ((unsigned long long)0 << 16) | (unsigned long long)f0;
            sc.lane_box[dm.S + 1] = tag | ((unsigned long long)e1 << 16) | (unsigned long long)dm.S;
            *sc.claim = ((unsigned long long)(uint32_t)f0 << 32) | (uint32_t)e1;
        }
        if (tot_u > dm.U_cap) {            // cannot happen for consistent counters
            atomicOr(sc.status, kDevCorrupt);
            sc.plan[0] = 0;
        }
        sc.ustart[dm.S] = tot_u;
        sc.item_prefix[dm.S] = tot_i;
        sc.tile_prefix[dm.S] = tot_t;
        sc.score_prefix[dm.S] = tot_s;
        if (observe) {
            atomicAdd(&sc.counters[0], (unsigned long long)tot_n);
            atomicAdd(&sc.counters[1], 1ull);
        }
    }
}

hipError_t launch_append(const Dims& dm, const View& v, const Scratch& sc,
                         const uint16_t* new_k, const uint8_t* new_region, int fused, int observe,
                         int rg, uint32_t tag, hipStream_t st) {
    hipLaunchKernelGGL(k_append, dim3(dm.S), dim3(256), 0, st, dm, v, sc, new_k, new_region, fused, observe,
                       max(rg, 1), tag);
    return hipGetLastError();
}

// ---------------------------------------------------------------- logits

// Position of an attention work item: chunk c (128 tokens) of row (s, lkv),
// lkv = layer * Hkv + KV head.  Items are ordered session, row, chunk.
struct Cursor {
    int s, lkv, c, nch;
};

// find_session with every LDS read made wave-uniform.
__device__ __forceinline__ int find_session_uni(const int* pref, int S, int x) {
    int lo = 0, hi = S;
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (uni(pref[mid]) <= x) lo = mid; else hi = mid;
    }
    return lo;
}

__device__ __forceinline__ void cursor_next(Cursor& cu, const int* s_pref, int S, int LHkv) {
    if (++cu.c == cu.nch) {
        cu.c = 0;
        if (++cu.lkv == LHkv) {
            cu.lkv = 0;
            do { ++cu.s; } while (cu.s < S && uni(s_pref[cu.s + 1]) == uni(s_pref[cu.s]));
            if (cu.s < S) cu.nch = uni((uni(s_pref[cu.s + 1]) - uni(s_pref[cu.s])) / LHkv);
        }
    }
}

// What the logits kernel reads besides its pointers.
struct LogitsDims {
    int L, Hq, Hkv, G, P, Pshift, S, MP, NP, R, LHkv, max_chunks;
    int W, Gw;   // window queries per observation; MFMA columns G * W
    int aligned; // region-aligned pages: hole slots are masked
    int quant;   // quantised tier: tiles of quantised pages hold 8-bit codes
};

// B operands of one row (session s, lkv = layer * Hkv + KV head) in
// registers: lane column c = lane & 15 is window query w = c / G, query head
// kv * G + c % G (zero past G W); k-group g = lane >> 4 holds dims
// 32j + 8g .. +7; each float32 term is split into hi, mid and lo bf16 terms.
__device__ __forceinline__ void split_query_regs(u32x4 (&bq)[4][3], const float* __restrict__ q,
                                                 const LogitsDims& dm, int s, int lkv, int h, int g,
                                                 int32_t* status, int32_t* valid) {
    const int l = lkv / dm.Hkv, kv = lkv - l * dm.Hkv;
    const int w = h / dm.G, hh = h - w * dm.G;
    const float* qh = q + ((((size_t)s * dm.W + w) * dm.L + l) * dm.Hq + kv * dm.G + hh) * kHeadDim;
    bool bad = false;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        f32x4 u0 = f32x4{0.f, 0.f, 0.f, 0.f}, u1 = u0;
        if (h < dm.Gw) {
            const f32x4* p = reinterpret_cast<const f32x4*>(qh + 32 * j + 8 * g);
            u0 = p[0];
            u1 = p[1];
        }
        const float xs[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
        for (int e = 0; e < 8; e += 2) {
            uint32_t h0, m0, l0, h1, m1, l1;
            bad |= !isfinite(xs[e]) || !isfinite(xs[e + 1]);
            split3(xs[e], h0, m0, l0);
            split3(xs[e + 1], h1, m1, l1);
            bq[j][0][e >> 1] = h0 | (h1 << 16);
            bq[j][1][e >> 1] = m0 | (m1 << 16);
            bq[j][2][e >> 1] = l0 | (l1 << 16);
        }
    }
    if (bad) {   // a non-finite query voids the session's step
        atomicOr(status, MD_DEV_NONFINITE);
        valid[s] = 0;
    }
}

// The eight 16-token row tiles of an item: slot index (physical page * P +
// offset in the page) of each tile's first token, and a mask of the tiles
// that hold cached tokens.  Page-table reads are clamped into the session's
// table, so the lookup never branches; out-of-range entries drop the tile
// and report MD_DEV_CORRUPT once per item.
struct ItemTiles {
    int slot0[8];
    unsigned vmask;
    unsigned qmask;   // quantised tier: tiles holding 8-bit codes
    int nt;
};

template <bool QT>
__device__ __forceinline__ void item_tiles(ItemTiles& it, const Cursor& cu, const LogitsDims& dm,
                                           const int32_t* __restrict__ page_table,
                                           const int32_t* __restrict__ n_tokens, int32_t* status,
                                           int lane, const uint8_t* __restrict__ page_format) {
    const int nt = n_tokens[cu.s];
    const int np = (nt + dm.P - 1) >> dm.Pshift;
    const int* ptab = page_table + (size_t)cu.s * dm.MP;
    unsigned vm = 0, bad = 0;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        const int tok = cu.c * kChunk + 16 * t;
        const int pg = min(tok >> dm.Pshift, max(np - 1, 0));
        const int p = ptab[pg];
        const bool in_seq = tok < nt;
        const bool in_pool = (unsigned)p < (unsigned)dm.NP;
        vm |= (in_seq && in_pool) ? 1u << t : 0u;
        bad |= (in_seq && !in_pool) ? 1u : 0u;
        it.slot0[t] = (in_seq && in_pool) ? (p << dm.Pshift) + (tok & (dm.P - 1)) : 0;
    }
    it.vmask = vm;
    it.qmask = 0;
    if constexpr (QT) {
#pragma unroll
        for (int t = 0; t < 8; ++t)
            if ((vm & (1u << t)) && page_format[it.slot0[t] >> dm.Pshift]) it.qmask |= 1u << t;
    }
    it.nt = nt;
    if (bad && lane == 0) atomicOr(status, kDevCorrupt);
}

// Four 16-byte pieces of one K row tile in the MFMA A layout: lane (h, g)
// holds token h's dims 32j + 8g .. +7 for j = 0..3.  The pool keeps each
// block of 16 tokens as [d / 8][16][8], so piece j of all 64 lanes is 1 KiB
// contiguous (voff = 16 lane).
// A tile without cached tokens reads the pool's first row tile instead
// (always in bounds; its logits are masked), so loads never branch.
template <bool QT>
__device__ __forceinline__ void load_tile(u32x4 (&a)[4], const LogitsDims& dm,
                                          const uint16_t* __restrict__ k_pool, const ItemTiles& it,
                                          int t, int lkv, uint32_t voff) {
    const bool ok = it.vmask & (1u << t);
    const int slot = it.slot0[t];
    const size_t tile = ok ? ((size_t)(slot >> dm.Pshift) * dm.LHkv + lkv) * dm.P + (slot & (dm.P - 1)) : 0;
    gbytes base = uni_ptr(k_pool + tile * kHeadDim);
    if constexpr (QT) {
        // a quantised block: codes in its first 2 KiB (a[0], a[1]), the
        // scale at byte 2048 (a[2]; a[3] the next 16 bytes of that line:
        // one address loaded twice becomes one load and a copy, and the copy
        // waits for every load in flight)
        const bool qt = it.qmask & (1u << t);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            a[j] = __builtin_nontemporal_load(
                reinterpret_cast<gvec>(base + ((qt && j >= 2) ? 2048u + 16u * (j - 2) : voff + 1024u * j)));
    } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            a[j] = __builtin_nontemporal_load(reinterpret_cast<gvec>(base + voff + 1024 * j));
    }
}

// Each wave streams a contiguous run of work items (128-token chunks of one
// (session, layer, KV head) row) tile by tile through a ring of four 16-token
// K tiles held in registers: while tile t is multiplied, tiles t+1..t+3 are in
// flight, and the slot tile t frees is refilled with tile t+4, which may
// belong to the next item (whose page-table entries are fetched one item
// ahead).  Per tile: one 16x16x32 bf16 MFMA row tile, A = 16 tokens x 32 dims
// of K, B = 32 dims x 16 columns holding the G heads' query terms (hi, mid
// and lo accumulate into the same C), C = 16 tokens x 16 heads in float32.
// Lane layout (16x16x32): A/B lane l holds row/column l & 15 and the eight
// consecutive k = 8 (l >> 4) .. +7; C lane l holds column l & 15, rows
// 4 (l >> 4) .. +3.  Softmax statistics of the chunk are kept online per
// lane and merged across the four row quads at the end of the chunk.
template <bool QT>
__global__ void __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 3)))
k_logits(LogitsDims dm, const uint16_t* __restrict__ k_pool, const int32_t* __restrict__ page_table,
         const int32_t* __restrict__ n_tokens, const float* __restrict__ q,
         float* __restrict__ logits, float2* __restrict__ cstats, int32_t* status,
         const int32_t* __restrict__ item_prefix, const int32_t* __restrict__ t_ins,
         const int32_t* __restrict__ clock, const uint8_t* __restrict__ region,
         const uint8_t* __restrict__ page_format, int32_t* valid) {
    __shared__ int s_pref[kMaxSessions + 1];
    const int S = dm.S;
    for (int i = threadIdx.x; i <= S; i += blockDim.x) s_pref[i] = item_prefix[i];
    __syncthreads();
    const int total = uni(s_pref[S]);
    const int lane = lane_id();
    const int n_waves = gridDim.x * (blockDim.x >> 6);
    const int gw = uni(blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6));
    const int per = uni((total + n_waves - 1) / n_waves);
    int it = gw * per;
    const int end = min(total, it + per);
    if (it >= end) return;

    const int h = lane & 15;         // MFMA column = query head within the group
    const int g = lane >> 4;         // k-group of A/B, row quad of C
    const uint32_t voff = 16u * lane;
    Cursor cu;
    cu.s = find_session_uni(s_pref, S, it);
    const int base_it = uni(s_pref[cu.s]);
    cu.nch = uni((uni(s_pref[cu.s + 1]) - base_it) / dm.LHkv);
    cu.lkv = uni((it - base_it) / cu.nch);
    cu.c = uni((it - base_it) - cu.lkv * cu.nch);
    u32x4 ring[4][4];
    u32x4 bq[4][3];

    // Outer loop: one row segment (items of one (session, layer, KV head) row)
    // at a time; the query operands load once per segment.
    while (it < end) {
        const int seg_end = min(end, it + (cu.nch - cu.c));
        split_query_regs(bq, q, dm, cu.s, cu.lkv, h, g, status, valid);
        const int l = uni(cu.lkv / dm.Hkv);
        const int kv = cu.lkv - l * dm.Hkv;
        const int row0 = uni(cu.lkv * dm.Gw);   // first logits row of the group: (lkv, w, h)
        // window query of this lane's column sees tokens inserted up to
        // step t - (W - 1 - w) (W = 1: every token)
        const int t_lim = dm.W > 1 ? clock[cu.s] - (dm.W - 1 - h / dm.G) : 0;
        (void)l;
        (void)kv;
        ItemTiles cur;
        item_tiles<QT>(cur, cu, dm, page_table, n_tokens, status, lane, page_format);
#pragma unroll
        for (int t = 0; t < 4; ++t) load_tile<QT>(ring[t], dm, k_pool, cur, t, cu.lkv, voff);

        // Inner loop: the segment's items, streamed without a break.
        for (; it < seg_end; ++it) {
            ItemTiles nxt;
            if (it + 1 < seg_end) {
                Cursor nx = cu;
                ++nx.c;
                item_tiles<QT>(nxt, nx, dm, page_table, n_tokens, status, lane, page_format);
            } else {
                nxt = cur;
                nxt.vmask = 0;
                nxt.qmask = 0;
            }
            const int tok0 = cu.c * kChunk;
            float m = -INFINITY, lsum = 0.0f;
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
                if (QT && (cur.qmask & (1u << t))) {
                    // quantised tile: codes as bf16 (exact), the scale after the sum
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const u32x4 av = (j & 1) ? codes_to_bf16<1>(ring[t & 3][j >> 1]) : codes_to_bf16<0>(ring[t & 3][j >> 1]);
#pragma unroll
                        for (int p = 0; p < 3; ++p)
                            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8, av), __builtin_bit_cast(bf16x8, bq[j][p]), acc, 0, 0, 0);
                    }
                    const float qs = __uint_as_float(ring[t & 3][2][0]);
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[i] *= qs;
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
#pragma unroll
                        for (int p = 0; p < 3; ++p)
                            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                                __builtin_bit_cast(bf16x8, ring[t & 3][j]), __builtin_bit_cast(bf16x8, bq[j][p]),
                                acc, 0, 0, 0);
                    }
                }
                // refill the slot with the tile four ahead
                if (t < 4) load_tile<QT>(ring[t & 3], dm, k_pool, cur, t + 4, cu.lkv, voff);
                else load_tile<QT>(ring[t & 3], dm, k_pool, nxt, t - 4, cu.lkv, voff);

                // base-2 logits; tokens past the session's count, tokens
                // newer than the column's window query, and hole slots are
                // masked out
                const bool tvalid = cur.vmask & (1u << t);
                int tins[4] = {0, 0, 0, 0};
                if (dm.W > 1 && tvalid) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) tins[i] = t_ins[cur.slot0[t] + 4 * g + i];
                }
                uint32_t rb = 0;   // region codes of this lane's four tokens
                if (dm.aligned && tvalid) rb = *reinterpret_cast<const uint32_t*>(region + cur.slot0[t] + 4 * g);
                float x[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int tok = tok0 + 16 * t + 4 * g + i;
                    const bool seen = dm.W == 1 || tins[i] <= t_lim;
                    const bool hole = dm.aligned && ((rb >> (8 * i)) & 0xffu) == (uint32_t)kHole;
                    x[i] = (tvalid && tok < cur.nt && seen && !hole) ? acc[i] * kLogitScale : -INFINITY;
                }
                const float mn = fmaxf(m, fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])));
                const bool live = mn != -INFINITY;
                const float ms = live ? mn : 0.0f;
                const float part = (hw_exp2(x[0] - ms) + hw_exp2(x[1] - ms)) +
                                   (hw_exp2(x[2] - ms) + hw_exp2(x[3] - ms));
                lsum = live ? lsum * hw_exp2(m - ms) + part : lsum;
                m = live ? mn : m;
                if (tvalid && h < dm.Gw) {
                    const int slot = cur.slot0[t];
                    gbytes base = uni_ptr(logits + ((size_t)(slot >> dm.Pshift) * dm.R + row0) * dm.P +
                                          (slot & (dm.P - 1)));
                    const uint32_t so = 4u * (h * dm.P + 4 * g);
                    *(__attribute__((address_space(1))) f32x4*)(base + so) = f32x4{x[0], x[1], x[2], x[3]};
                }
            }
            // merge the four row quads' (max, sum) pairs; the merge is
            // symmetric, so every lane of a column ends with the same values
#pragma unroll
            for (int o = 16; o <= 32; o <<= 1) {
                const float m2 = __shfl_xor(m, o);
                const float l2 = __shfl_xor(lsum, o);
                const float M = fmaxf(m, m2);
                lsum = (M == -INFINITY) ? 0.0f : lsum * hw_exp2(m - M) + l2 * hw_exp2(m2 - M);
                m = M;
            }
            if (h < dm.Gw && g == 0)
                cstats[((size_t)cu.s * dm.R + row0 + h) * dm.max_chunks + cu.c] = make_float2(m, lsum);
            ++cu.c;
            cur = nxt;
        }
        // next row
        cu.c = cu.nch - 1;
        cursor_next(cu, s_pref, S, dm.LHkv);
    }
}

hipError_t launch_logits(const Dims& dm, const View& v, const Scratch& sc, const float* q, int n_blocks,
                         hipStream_t st) {
    LogitsDims ld{dm.L, dm.Hq, dm.Hkv, dm.G, dm.P, dm.Pshift, dm.S, dm.MP, dm.NP, dm.R, dm.LHkv, dm.max_chunks,
                  dm.W, dm.G * dm.W, dm.aligned, dm.quant};
    hipLaunchKernelGGL(dm.quant ? k_logits<true> : k_logits<false>, dim3(n_blocks), dim3(256), 0, st, ld, v.k_pool, v.page_table,
                       v.n_tokens, q, sc.logits, sc.cstats, sc.status, sc.item_prefix, v.t_ins, v.clock,
                       v.region, v.page_format, sc.valid);
    return hipGetLastError();
}

// ---------------------------------------------------------------- row statistics

__global__ void __launch_bounds__(256) k_rowstats(Dims dm, Scratch sc) {
    const int w = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = lane_id();
    if (w >= dm.S * dm.R) return;
    const int s = w / dm.R, row = w - s * dm.R;
    const int nch = sc.chunks[s];
    if (nch == 0) return;
    const float2* cs = sc.cstats + ((size_t)s * dm.R + row) * dm.max_chunks;
    float m = -INFINITY;
    for (int c = lane; c < nch; c += 64) m = fmaxf(m, cs[c].x);
    m = wave_max(m);
    float l = 0.0f;
    for (int c = lane; c < nch; c += 64) {
        const float2 st = cs[c];
        l += st.y * hw_exp2(st.x - m);
    }
    l = wave_sum(l);
    // a window query that sees none of the session's tokens gives them no
    // weight (its row has no live logit)
    if (lane == 0) sc.rstats[(size_t)s * dm.R + row] = m == -INFINITY ? make_float2(0.0f, 0.0f)
                                                                       : make_float2(m, 1.0f / l);
}

hipError_t launch_rowstats(const Dims& dm, const Scratch& sc, hipStream_t st) {
    const int waves = dm.S * dm.R;
    hipLaunchKernelGGL(k_rowstats, dim3((waves + 3) / 4), dim3(256), 0, st, dm, sc);
    return hipGetLastError();
}

// ---------------------------------------------------------------- mass, EWMA, refresh

// One block per 64-token tile at a time: 4 row groups x 64 tokens; each
// thread sums its rows' softmax weights 2^(x - M) / Lambda, the four partials
// add in a fixed order; then wave 0 applies Eq. 2 and Eq. 3 to the tile's
// tokens and scores them and their pages (Eq. 4, Eq. 5: the scoring
// kernel's work, with the same device functions and reduction, so the
// selection reads the page scores the scoring kernel would have written).
// FOLD: each block works its session's row statistics (M, 1 / Lambda) out
// from the chunk statistics itself, in a fixed order (sessions of at most
// kFoldChunks chunks: a few KB read per block), instead of a separate
// row-statistics kernel.
template <bool FOLD>
__global__ void __launch_bounds__(256) k_mass(Dims dm, View v, Scratch sc, float* abar_out) {
    __shared__ int s_pref[kMaxSessions + 1];
    __shared__ float2 s_rs[kMaxRows];
    __shared__ float s_part[4][kTile];
    const int S = dm.S;
    for (int i = threadIdx.x; i <= S; i += blockDim.x) s_pref[i] = sc.tile_prefix[i];
    __syncthreads();
    const int total = s_pref[S];
    const int tl = threadIdx.x & 63, rg = threadIdx.x >> 6;
    const float one_m_rho = 1.0f - dm.rho;
    int cur = -1;
    for (int tile = blockIdx.x; tile < total; tile += gridDim.x) {
        const int s = find_session(s_pref, S, tile);
        if (s != cur) {
            __syncthreads();
            if constexpr (FOLD) {
                // the session's rows: max over its chunks, then the sum of
                // their sums rescaled to it, chunk by chunk
                const int nch = min(sc.chunks[s], kFoldChunks);
                for (int i = threadIdx.x; i < dm.R; i += blockDim.x) {
                    const float2* cs = sc.cstats + ((size_t)s * dm.R + i) * dm.max_chunks;
                    float2 st[kFoldChunks];
                    float m = -INFINITY;
#pragma unroll
                    for (int c = 0; c < kFoldChunks; ++c) {
                        st[c] = c < nch ? cs[c] : make_float2(-INFINITY, 0.0f);
                        m = fmaxf(m, st[c].x);
                    }
                    float l = 0.0f;
#pragma unroll
                    for (int c = 0; c < kFoldChunks; ++c)
                        if (c < nch) l += st[c].y * hw_exp2(st[c].x - m);
                    // a window query that sees none of the session's tokens
                    // gives them no weight (its row has no live logit)
                    s_rs[i] = m == -INFINITY ? make_float2(0.0f, 0.0f) : make_float2(m, 1.0f / l);
                }
            } else {
                for (int i = threadIdx.x; i < dm.R; i += blockDim.x) s_rs[i] = sc.rstats[(size_t)s * dm.R + i];
            }
            __syncthreads();
            cur = s;
        }
        const int nt = v.n_tokens[s];
        const int tok = (tile - s_pref[s]) * kTile + tl;
        bool valid = tok < nt;
        int phys = 0, slot = 0;
        float acc = 0.0f;
        if (valid) {
            const int pg = tok >> dm.Pshift;
            slot = tok - (pg << dm.Pshift);
            phys = v.page_table[(size_t)s * dm.MP + pg];
            if ((unsigned)phys >= (unsigned)dm.NP) {
                valid = false;
                atomicOr(sc.status, kDevCorrupt);
            } else if (dm.aligned && v.region[(size_t)phys * dm.P + slot] == kHole) {
                valid = false;   // a hole holds no token
            } else {
                const float* lp = sc.logits + (size_t)phys * dm.R * dm.P + slot;
#pragma unroll 16
                for (int row = rg; row < dm.R; row += 4) {
                    const float2 rs = s_rs[row];
                    acc += hw_exp2(lp[(size_t)row * dm.P] - rs.x) * rs.y;
                }
            }
        }
        s_part[rg][tl] = acc;
        __syncthreads();
        if (rg == 0) {
            // every load before the stores (a wait for a load also waits for them)
            const size_t si = (size_t)phys * dm.P + slot;
            const bool keep = sc.valid[s] != 0;   // a void step writes nothing
            const int t = v.clock[s];
            const int n_live = v.n_live[s];
            float a = 0.0f;
            int tr = 0, r = 0;
            if (valid) {
                a = v.imp[si];
                tr = v.t_ref[si];
                r = v.region[si];
            }
            if (valid && r >= dm.n_regions) {
                atomicOr(sc.status, kDevCorrupt);
                r = dm.n_regions - 1;
            }
            const size_t ri = (size_t)s * dm.n_regions + r;
            const float br = valid ? v.b[ri] : 0.0f, lamr = valid ? v.lam[ri] : 0.0f;
            if (valid && keep) {
                const float abar =
                    (((s_part[0][tl] + s_part[1][tl]) + s_part[2][tl]) + s_part[3][tl]) / (float)dm.R;
                a = fmaf(dm.rho, a, one_m_rho * abar);
                v.imp[si] = a;
                if (abar >= dm.tau_scale / (float)n_live) {
                    tr = t;
                    v.t_ref[si] = tr;
                }
                if (abar_out != nullptr) abar_out[si] = abar;
            }
            const bool pin = valid && ((dm.pin_mask >> r) & 1u);
            const float sc_i = pin ? INFINITY
                                   : (valid ? retention_score(br, lamr, t, tr, attention_weight(dm.alpha, dm.norm_attn, n_live), a)
                                            : 0.0f);
            float ps;
            const bool has = page_score_of(sc_i, valid, pin, dm.P, &ps);
            if ((tl & (dm.P - 1)) == 0 && has) sc.pscore[(size_t)s * dm.MP + (tok >> dm.Pshift)] = ps;
        }
        __syncthreads();
    }
}

hipError_t launch_mass(const Dims& dm, const View& v, const Scratch& sc, float* abar_out,
                       int n_blocks, bool fold, hipStream_t st) {
    hipLaunchKernelGGL(fold ? k_mass<true> : k_mass<false>, dim3(n_blocks), dim3(256), 0, st, dm, v, sc, abar_out);
    return hipGetLastError();
}

// ---------------------------------------------------------------- scores

// One wave per 64-token tile (4 pages of 16 or one page of 64); a page's
// members are P consecutive lanes, reduced with a butterfly; lane 0 of the
// page writes its score.
__global__ void __launch_bounds__(256) k_score(Dims dm, View v, Scratch sc, float* page_score,
                                               float* token_score) {
    __shared__ int s_pref[kMaxSessions + 1];
    const int S = dm.S;
    for (int i = threadIdx.x; i <= S; i += blockDim.x) s_pref[i] = sc.score_prefix[i];
    __syncthreads();
    const int total = s_pref[S];
    const int lane = lane_id();
    const int n_waves = gridDim.x * (blockDim.x >> 6);
    const int gw = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6);
    for (int tile = gw; tile < total; tile += n_waves) {
        const int s = find_session(s_pref, S, tile);
        const int nt = v.n_tokens[s];
        const int t = v.clock[s];
        const int tok = (tile - s_pref[s]) * kTile + lane;
        const int pg = tok >> dm.Pshift;
        bool valid = tok < nt;
        bool pin = false;
        float sc_i = 0.0f;
        if (valid) {
            const int phys = v.page_table[(size_t)s * dm.MP + pg];
            if ((unsigned)phys >= (unsigned)dm.NP) {
                valid = false;
                atomicOr(sc.status, kDevCorrupt);
            } else {
                const size_t si = (size_t)phys * dm.P + (tok - (pg << dm.Pshift));
                int r = v.region[si];
                if (dm.aligned && r == kHole) {
                    valid = false;   // a hole holds no token
                } else {
                    if (r >= dm.n_regions) {
                        atomicOr(sc.status, kDevCorrupt);
                        r = dm.n_regions - 1;
                    }
                    pin = (dm.pin_mask >> r) & 1u;
                    if (pin) {
                        sc_i = INFINITY;
                    } else {
                        const size_t ri = (size_t)s * dm.n_regions + r;
                        sc_i = retention_score(v.b[ri], v.lam[ri], t, v.t_ref[si],
                                               attention_weight(dm.alpha, dm.norm_attn, v.n_live[s]), v.imp[si]);
                    }
                    if (token_score != nullptr) token_score[si] = sc_i;
                }
            }
        }
        float ps;
        const bool has = page_score_of(sc_i, valid, pin, dm.P, &ps);
        if ((lane & (dm.P - 1)) == 0 && has) {
            sc.pscore[(size_t)s * dm.MP + pg] = ps;
            if (page_score != nullptr) page_score[(size_t)s * dm.MP + pg] = ps;
        }
    }
}

hipError_t launch_score(const Dims& dm, const View& v, const Scratch& sc, float* page_score,
                        float* token_score, int n_blocks, hipStream_t st) {
    hipLaunchKernelGGL(k_score, dim3(n_blocks), dim3(256), 0, st, dm, v, sc, page_score, token_score);
    return hipGetLastError();
}

// ---------------------------------------------------------------- select

// Tokens of page i (physical id phys) of a session with np pages and nt
// slots in use: P, or the last page's slots; with region-aligned pages the
// slots that are not holes.
__device__ int page_tokens(const Dims& dm, const View& v, int phys, int i, int np, int nt) {
    const int used = (i == np - 1) ? nt - (np - 1) * dm.P : dm.P;
    if (!dm.aligned) return used;
    if ((unsigned)phys >= (unsigned)dm.NP) return 0;
    const uint32_t* w = reinterpret_cast<const uint32_t*>(v.region + (size_t)phys * dm.P);
    int holes = 0;
    for (int k = 0; k < dm.P / 4; ++k) {
        const uint32_t x = w[k];
#pragma unroll
        for (int b = 0; b < 4; ++b)
            holes += (4 * k + b < used && ((x >> (8 * b)) & 0xffu) == (uint32_t)kHole) ? 1 : 0;
    }
    return used - holes;
}

// Radix select over the float bit patterns of the page scores (non-negative,
// so the unsigned order of the bits is the numeric order), weighted by each
// page's live token count: the threshold key T is where the ascending
// cumulative weight first reaches need = n - B.  Pages with key < T go; pages
// with key == T go in serial order until the need is met.  Pinned pages
// (+inf) never enter.  Each thread owns a contiguous run of page indices, so
// per-thread runs in thread order are the serial order.
// When the pages holding the smallest key already weigh at least the need
// (the usual decode step: one token over the budget), T is that key and the
// radix passes are skipped.
//
// Apply: the selection is also carried out by the same block (k_evict, the
// compaction of k_compact for this step's own selection).  Freed ids go
// onto the free list in (session, serial) order: each block publishes its
// count as a 64-bit word tagged with the launch (`tag`) and adds up the
// words of the sessions before it (a look-back; blocks are dispatched in
// index order, so every block it waits for has started), bounded in time.
// Each block then tells the last one (highest index) whether it applied its
// selection; the last block sets the free count only if all did, so a
// block that gave up waiting (its session left as it was, MD_DEV_CORRUPT)
// never has unwritten places counted.  Every block has read the free count
// before publishing its word (the word is computed from it), so none reads
// the new value.
template <bool Apply>
__device__ __forceinline__ void select_session(const Dims& dm, const View& v, const Scratch& sc,
                                               int32_t* ev_serial, int32_t* ev_count, uint8_t* infeasible,
                                               uint32_t tag) {
    const int s = blockIdx.x;
    __shared__ int lds[2 * 17];
    __shared__ uint32_t s_min[16];
    __shared__ int hist[256];
    __shared__ int sh_digit, sh_before, sh_fc, sh_prior, sh_bad;
    const int tid = threadIdx.x;
    const uint32_t kInf = 0x7F800000u;
    const float* ps = sc.pscore + (size_t)s * dm.MP;
    int* ser = v.page_serial + (size_t)s * dm.MP;
    int* ptab = v.page_table + (size_t)s * dm.MP;
    // The runs split the page-table capacity, not the session's pages, so
    // the scores, serials and table entries go out with the counters rather
    // than after them; entries past the session's pages are read but not used.
    const int per = (dm.MP + kSelThreads - 1) / kSelThreads;
    const int i0 = min(dm.MP, tid * per), ie = min(dm.MP, i0 + per);
    float sv[kPerThread];
    int pv[kPerThread], sr[kPerThread];
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        sv[k] = 0.0f;
        pv[k] = sr[k] = 0;
        if (i0 + k < ie) {
            sv[k] = ps[i0 + k];
            sr[k] = ser[i0 + k];
            if (Apply || dm.aligned) pv[k] = ptab[i0 + k];
        }
    }
    if (Apply && tid == 0) sh_fc = v.free_count[0];
    const int np = v.n_pages[s], nt = v.n_tokens[s], B = v.budget[s];
    const int need = v.n_live[s] - B;
    const bool active = sc.valid[s] && need > 0 && np > 0;
    if (!Apply && !active) {
        if (tid == 0) {
            ev_count[s] = 0;
            infeasible[s] = 0;
        }
        return;
    }
    const int i1 = active ? min(np, ie) : i0;
    uint32_t key[kPerThread];
    int wt[kPerThread];
    int wsum = 0;
    uint32_t kmin = kInf;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        const int i = i0 + k;
        key[k] = kInf;
        wt[k] = 0;
        if (i < i1) {
            key[k] = __float_as_uint(sv[k]);
            wt[k] = page_tokens(dm, v, pv[k], i, np, nt);
            if (key[k] < kInf) wsum += wt[k];
            kmin = min(kmin, key[k]);
        }
    }
    kmin = wave_min_u32(kmin);
    if (lane_id() == 0) s_min[tid >> 6] = kmin;
    int total;
    block_exclusive_scan(wsum, lds, &total);   // its barriers publish s_min too
    const bool infeas = active && total < need;
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) kmin = min(kmin, s_min[w]);
    // the smallest key's weight, and each thread's share of it before its run
    int teq = 0;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k)
        if (key[k] == kmin && key[k] < kInf) teq += wt[k];
    int at_min;
    int run = block_exclusive_scan(teq, lds, &at_min);
    uint32_t T = kmin;
    int rem = need;
    if (active && !infeas && at_min < need) {
        uint32_t prefix = 0, pmask = 0;
        for (int shift = 24; shift >= 0; shift -= 8) {
            if (tid < 256) hist[tid] = 0;
            __syncthreads();
#pragma unroll
            for (int k = 0; k < kPerThread; ++k) {
                if (key[k] < kInf && (key[k] & pmask) == prefix)
                    atomicAdd(&hist[(key[k] >> shift) & 255u], wt[k]);
            }
            __syncthreads();
            // inclusive scan of the 256 bins by the first four waves; every
            // thread of the block reaches both barriers
            int hv = 0, incl = 0;
            if (tid < 256) {
                const int lane = lane_id();
                hv = hist[tid];
                incl = hv;
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const int t2 = __shfl_up(incl, o);
                    if (lane >= o) incl += t2;
                }
                if (lane == 63) lds[tid >> 6] = incl;
            }
            __syncthreads();
            if (tid < 256) {
                const int wid = tid >> 6;
                for (int w = 0; w < wid; ++w) incl += lds[w];
                const int excl = incl - hv;
                if (excl < rem && rem <= incl) {
                    sh_digit = tid;
                    sh_before = excl;
                }
            }
            __syncthreads();
            prefix |= (uint32_t)sh_digit << shift;
            pmask |= 0xFFu << shift;
            rem -= sh_before;
            __syncthreads();
        }
        T = prefix;
        // weights of the key == T pages before this thread's run
        teq = 0;
#pragma unroll
        for (int k = 0; k < kPerThread; ++k)
            if (key[k] == T) teq += wt[k];
        int dummy;
        run = block_exclusive_scan(teq, lds, &dummy);
    }
    bool ev[kPerThread];
    int my_ev = 0, my_live = 0;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        bool e = false;
        if (i0 + k < i1 && key[k] < kInf) {
            if (infeas) {
                e = true;
            } else if (key[k] < T) {
                e = true;
            } else if (key[k] == T) {
                e = run < rem;
                run += wt[k];
            }
        }
        ev[k] = e;
        my_ev += e ? 1 : 0;
        my_live += e ? wt[k] : 0;
    }
    int ex[2], tot[2];
    {
        const int m[2] = {my_ev, my_live};
        block_exclusive_scan_n<2>(m, lds, ex, tot);
    }
    const int n_ev = tot[0];
    int pos = ex[0];
    int32_t* out = ev_serial + (size_t)s * dm.MP;
#pragma unroll
    for (int k = 0; k < kPerThread; ++k)
        if (ev[k]) out[pos++] = sr[k];
    if (tid == 0) {
        ev_count[s] = n_ev;
        infeasible[s] = infeas ? 1 : 0;
        if (infeas) atomicOr(sc.warn, 1);
    }
    if (!Apply) return;

    // ---- the compaction of this session, and the free list
    const int fc = sh_fc;   // read by thread 0 before the barriers of the scans
    const int last = (int)gridDim.x - 1;
    if (tid == 0) {
        sh_prior = 0;
        sh_bad = 0;
        __hip_atomic_store(sc.ev_word + s,
                           ((unsigned long long)(tag & kWordTagMask) << 32) |
                               ((unsigned long long)(fc < 0 ? 1 : 0) << 31) | (unsigned long long)n_ev,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    // look-back: the counts of the sessions before this one (all of them for
    // the last block)
    int prior = 0, bad = 0;
    for (int s2 = tid; s2 < s; s2 += blockDim.x) {
        unsigned long long wd = __hip_atomic_load(sc.ev_word + s2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        bool stale = (uint32_t)(wd >> 32) != (tag & kWordTagMask);
        while (stale && __builtin_amdgcn_s_memrealtime() - t0 < kWordWaitTicks) {
            __builtin_amdgcn_s_sleep(1);
            wd = __hip_atomic_load(sc.ev_word + s2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            stale = (uint32_t)(wd >> 32) != (tag & kWordTagMask);
        }
        if (stale || ((wd >> 31) & 1ull)) bad = 1;
        prior += (int)(wd & 0x7FFFFFFFull);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        prior += __shfl_xor(prior, o);
        bad |= __shfl_xor(bad, o);
    }
    if (lane_id() == 0 && prior > 0) atomicAdd(&sh_prior, prior);
    if (lane_id() == 0 && bad) sh_bad = 1;
    __syncthreads();
    const int base = fc + sh_prior;
    const bool ok = !sh_bad && fc >= 0 && base + n_ev <= dm.NP;
    // Whether this block applies its selection, told to the last block
    // (which commits the free count only if every block does: a block that
    // gave up waiting leaves its session as it was and its places unwritten,
    // and the count must not cover them).
    if (tid == 0) {
        __hip_atomic_store(sc.ev_done + s, ((unsigned long long)(tag & kWordTagMask) << 32) | (ok ? 1ull : 0ull),
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (!ok) atomicOr(sc.status, kDevCorrupt);
        sc.freed[s] = ok ? n_ev : 0;
    }
    if (ok && n_ev > 0) {
        // kept pages move down in order; the evicted ones' ids go onto the
        // free list at the session's places.  Every table entry was read
        // before the scans' barriers.
        int kpos = min(i0, np) - ex[0], gpos = ex[0];
#pragma unroll
        for (int k = 0; k < kPerThread; ++k) {
            if (i0 + k < i1) {
                if (!ev[k]) {
                    ptab[kpos] = pv[k];
                    ser[kpos] = sr[k];
                    ++kpos;
                } else {
                    if (ok && base + gpos >= 0 && base + gpos < dm.NP) v.free_list[base + gpos] = pv[k];
                    ++gpos;
                }
            }
        }
        // the thread owning the last page knows whether it survived; all
        // pages but the last are full
        if (i1 == np && i1 > i0) {
            const int k_last = np - 1 - i0;
            bool last_kept = false;
#pragma unroll
            for (int k = 0; k < kPerThread; ++k)
                if (k == k_last) last_kept = !ev[k];
            const int kept = np - n_ev;
            v.n_pages[s] = kept;
            v.n_tokens[s] = last_kept ? nt - n_ev * dm.P : kept * dm.P;
            if (dm.aligned) v.n_live[s] -= tot[1];
            atomicAdd(&sc.counters[2], (unsigned long long)n_ev);
            atomicAdd(&sc.counters[3], (unsigned long long)tot[1]);
        }
    }
    if (s != last) return;
    // the last block: every block applied its selection, so the list grew
    // by the sum of the counts
    int all_ok = ok ? 1 : 0;
    for (int s2 = tid; s2 < s; s2 += blockDim.x) {
        unsigned long long wd = __hip_atomic_load(sc.ev_done + s2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        bool stale = (uint32_t)(wd >> 32) != (tag & kWordTagMask);
        while (stale && __builtin_amdgcn_s_memrealtime() - t0 < kWordWaitTicks) {
            __builtin_amdgcn_s_sleep(1);
            wd = __hip_atomic_load(sc.ev_done + s2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            stale = (uint32_t)(wd >> 32) != (tag & kWordTagMask);
        }
        if (stale || !(wd & 1ull)) all_ok = 0;
    }
    all_ok = __syncthreads_and(all_ok);
    if (tid == 0) {
        if (all_ok) v.free_count[0] = base + n_ev;
        else atomicOr(sc.status, kDevCorrupt);
    }
}

__global__ void __launch_bounds__(kSelThreads) k_select(Dims dm, View v, Scratch sc, int32_t* ev_serial,
                                                        int32_t* ev_count, uint8_t* infeasible) {
    select_session<false>(dm, v, sc, ev_serial, ev_count, infeasible, 0);
}

__global__ void __launch_bounds__(kSelThreads) k_evict(Dims dm, View v, Scratch sc, int32_t* ev_serial,
                                                       int32_t* ev_count, uint8_t* infeasible, uint32_t tag) {
    select_session<true>(dm, v, sc, ev_serial, ev_count, infeasible, tag);
}

hipError_t launch_select(const Dims& dm, const View& v, const Scratch& sc, int32_t* ev_serial,
                         int32_t* ev_count, uint8_t* infeasible, hipStream_t st) {
    hipLaunchKernelGGL(k_select, dim3(dm.S), dim3(kSelThreads), 0, st, dm, v, sc, ev_serial,
                       ev_count, infeasible);
    return hipGetLastError();
}

hipError_t launch_evict(const Dims& dm, const View& v, const Scratch& sc, int32_t* ev_serial,
                        int32_t* ev_count, uint8_t* infeasible, uint32_t tag, hipStream_t st) {
    hipLaunchKernelGGL(k_evict, dim3(dm.S), dim3(kSelThreads), 0, st, dm, v, sc, ev_serial,
                       ev_count, infeasible, tag);
    return hipGetLastError();
}

// ---------------------------------------------------------------- compact

// Pages listed for eviction in a session whose step stands (0 otherwise):
// the places the session's freed ids take on the free list.
__device__ __forceinline__ int evict_listed(const Dims& dm, const Scratch& sc, const int32_t* ev_count, int s) {
    const int valid = sc.valid[s], c = ev_count[s];   // both loads issued together
    return valid ? min(max(c, 0), dm.MP) : 0;
}

// One block per session.  Freed physical ids go onto the free list in
// (session, serial) order: session s pushes above the places of the
// sessions before it, which reserve one place per listed serial; the last
// block to finish sets the new count and, if some list named serials its
// session does not hold, closes the gaps they left, keeping the order.
//
// trusted: the lists are this step's selection (md_compact without lists),
// which names only pages the sessions hold.  Then no gaps can arise, and the
// blocks hand the last one nothing but a count, folded into the completion
// counter itself: no memory fence (a device-scope fence writes back the L2
// of the block's XCD, about 3 us each).  Should a session's table have
// changed since the selection after all, its unused places get -1 (an id
// the append refuses, setting MD_DEV_CORRUPT) rather than stale ids.
__global__ void __launch_bounds__(kSelThreads) k_compact(Dims dm, View v, Scratch sc,
                                                         const int32_t* __restrict__ ev_serial,
                                                         const int32_t* __restrict__ ev_count, int trusted) {
    const int s = blockIdx.x;
    __shared__ int lds[3 * 17];
    __shared__ int sh_last, sh_before, sh_listed;
    __shared__ int s_evs[kMaxPages];   // the session's list, searched in LDS
    const int tid = threadIdx.x;
    // Every load that depends on nothing else goes out at once: the
    // session's list length and counters, the free count (it changes only in
    // the last block, after every block has read it), the list lengths of
    // all sessions (those before this one give its places on the free list,
    // all of them the growth of the list), and the thread's run of the table
    // and of the list.  The runs split the page-table capacity, so they need
    // no count first; entries past the session's pages or list are not used.
    const int cnt = evict_listed(dm, sc, ev_count, s);
    const int np = v.n_pages[s], nt = v.n_tokens[s];
    const int fc = v.free_count[0];
    const int* evs = ev_serial + (size_t)s * dm.MP;
    int* ptab = v.page_table + (size_t)s * dm.MP;
    int* pser = v.page_serial + (size_t)s * dm.MP;
    const int per = (dm.MP + kSelThreads - 1) / kSelThreads;
    const int i0 = min(dm.MP, tid * per), ie = min(dm.MP, i0 + per);
    int ph[kPerThread], se[kPerThread];
#pragma unroll
    for (int k = 0; k < kPerThread; ++k) {
        ph[k] = se[k] = 0;
        if (i0 + k < ie) {
            ph[k] = ptab[i0 + k];
            se[k] = pser[i0 + k];
            s_evs[i0 + k] = evs[i0 + k];
        }
    }
    int mine = 0, all = 0;
    for (int s2 = tid; s2 < dm.S; s2 += blockDim.x) {
        const int c = evict_listed(dm, sc, ev_count, s2);
        mine += s2 < s ? c : 0;
        all += c;
    }
    if (tid == 0) sh_before = sh_listed = 0;
    __syncthreads();
    {
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            mine += __shfl_xor(mine, o);
            all += __shfl_xor(all, o);
        }
        if (lane_id() == 0 && mine > 0) atomicAdd(&sh_before, mine);
        if (lane_id() == 0 && all > 0) atomicAdd(&sh_listed, all);
    }
    __syncthreads();
    int gone_total = 0;
    if (cnt > 0 && np == 0) {
        if (tid == 0) atomicOr(sc.status, MD_DEV_BAD_EVICT);
    } else if (cnt > 0) {
        const int i1 = min(np, ie);
        bool keep[kPerThread];
        int n_keep = 0, n_gone = 0, live_gone = 0;
#pragma unroll
        for (int k = 0; k < kPerThread; ++k) {
            const int i = i0 + k;
            keep[k] = false;
            if (i < i1) {
                int lo = 0, hi = cnt;
                while (lo < hi) {  // serials in the list ascend
                    const int mid = (lo + hi) >> 1;
                    if (s_evs[mid] < se[k]) lo = mid + 1; else hi = mid;
                }
                const bool gone = lo < cnt && s_evs[lo] == se[k];
                keep[k] = !gone;
                n_keep += gone ? 0 : 1;
                n_gone += gone ? 1 : 0;
                if (gone) live_gone += page_tokens(dm, v, ph[k], i, np, nt);
            }
        }
        int kept_total;
        const int mine[3] = {n_keep, n_gone, live_gone};
        int ex[3], tot[3];
        block_exclusive_scan_n<3>(mine, lds, ex, tot);   // ends with a barrier: the old table is read
        int kpos = ex[0], gpos = ex[1];
        kept_total = tot[0];
        gone_total = tot[1];
        const int live_gone_total = tot[2];
        const int base = fc + sh_before;
        if (tid == 0) {
            if (gone_total != cnt) atomicOr(sc.status, MD_DEV_BAD_EVICT);
            if (fc < 0 || base + gone_total > dm.NP) atomicOr(sc.status, kDevCorrupt);
        }
#pragma unroll
        for (int k = 0; k < kPerThread; ++k) {
            if (i0 + k < i1) {
                if (keep[k]) {
                    ptab[kpos] = ph[k];
                    pser[kpos] = se[k];
                    ++kpos;
                } else {
                    if (base + gpos >= 0 && base + gpos < dm.NP) v.free_list[base + gpos] = ph[k];
                    ++gpos;
                }
            }
        }
        // The thread owning the last page knows whether it survived; all pages
        // but the last are full, so the token count follows from that.
        if (i1 == np && i1 > i0) {
            const int k_last = np - 1 - i0;
            bool last_kept = false;
#pragma unroll
            for (int k = 0; k < kPerThread; ++k)
                if (k == k_last) last_kept = keep[k];
            const int nt_new = last_kept ? nt - gone_total * dm.P : kept_total * dm.P;
            v.n_pages[s] = kept_total;
            v.n_tokens[s] = nt_new;
            if (dm.aligned) v.n_live[s] -= live_gone_total;
            atomicAdd(&sc.counters[2], (unsigned long long)gone_total);
            atomicAdd(&sc.counters[3], (unsigned long long)live_gone_total);
        }
    }
    if (tid == 0) sc.freed[s] = gone_total;

    if (trusted) {
        const int base = fc + sh_before;
        for (int i = gone_total + tid; i < cnt; i += blockDim.x)
            if (base + i >= 0 && base + i < dm.NP) v.free_list[base + i] = -1;
        __syncthreads();   // every thread is past its reads of the free count
        if (tid == 0) {
            const unsigned long long old =
                atomicAdd(sc.compact_acc, (1ull << 40) | (unsigned long long)(cnt - gone_total));
            sh_last = (int)(old >> 40) == (int)gridDim.x - 1;
        }
        __syncthreads();
        if (!sh_last) return;
        // the last block: every block has read the free count; the list grew
        // by one place per listed page
        if (tid == 0) {
            v.free_count[0] = min(max(fc, 0) + sh_listed, dm.NP);
            *sc.compact_acc = 0;
        }
        return;
    }

    // The last block to finish: the new free count; gaps left by listed
    // serials a session did not hold are closed session by session, each
    // chunk read before it is written (destinations never pass sources).
    __threadfence();
    __syncthreads();
    if (tid == 0) sh_last = (atomicAdd(sc.done_compact, 1) == (int)gridDim.x - 1);
    __syncthreads();
    if (!sh_last) return;
    __threadfence();
    int pushed = 0, listed = 0;
    for (int s2 = tid; s2 < dm.S; s2 += blockDim.x) {
        pushed += load_agent(sc.freed + s2);
        listed += evict_listed(dm, sc, ev_count, s2);
    }
    int tot2[2];
    {
        const int m2[2] = {pushed, listed};
        int ex2[2];
        block_exclusive_scan_n<2>(m2, lds, ex2, tot2);
    }
    if (tot2[0] != tot2[1] && fc >= 0) {
        int src = fc, dst = fc;
        for (int s2 = 0; s2 < dm.S; ++s2) {
            const int g = load_agent(sc.freed + s2);
            if (dst != src) {
                for (int c = 0; c < g; c += blockDim.x) {
                    const int i = c + tid;
                    const bool in = i < g && src + i < dm.NP && dst + i >= 0;
                    const int id = in ? load_agent(v.free_list + src + i) : 0;
                    __syncthreads();
                    if (in) v.free_list[dst + i] = id;
                    __syncthreads();
                }
            }
            src += evict_listed(dm, sc, ev_count, s2);
            dst += g;
        }
    }
    if (tid == 0) {
        v.free_count[0] = min(max(fc, 0) + tot2[0], dm.NP);
        *sc.done_compact = 0;
    }
}

// ---------------------------------------------------------------- quantised tier

// Quantised tier (Sec. III-E), before the compaction of the same lists:
// every page that survives the eviction, is not pinned (its score is +inf),
// is not the session's last page, is still bf16 and scores below the
// threshold becomes FP8 E4M3 codes with a float32 scale max|k| / 448 per
// 16-token block and row.  Grid (blocks, S): block x takes the page
// indices x, x + gridDim.x, ...; an eligible page's (row, 16-token block)
// pairs go to the four waves in turn.  A wave reads its block's 4 KiB (lane
// l: 16 bytes at 16 l + 1024 j, i.e. token l % 16, dims 32 j + 8 (l / 16)
// .. +7), reduces max|k| over the block's tokens, and writes the codes over
// the block's first 2 KiB (lane l: 16 bytes at 16 l + 1024 j', the codes of
// its chunks 2 j' and 2 j' + 1) and the scale (four copies) at byte 2048,
// once every lane has read (the reduction needs them all).
__global__ void __launch_bounds__(256) k_quant(Dims dm, View v, Scratch sc, const int32_t* __restrict__ ev_serial,
                                               const int32_t* __restrict__ ev_count) {
    const int s = blockIdx.y;
    const int np = v.n_pages[s];
    if (!sc.valid[s] || np < 2) return;
    const int cnt = min(max(ev_count[s], 0), dm.MP);
    const int32_t* evs = ev_serial + (size_t)s * dm.MP;
    const int32_t* ptab = v.page_table + (size_t)s * dm.MP;
    const int32_t* pser = v.page_serial + (size_t)s * dm.MP;
    const int lane = lane_id(), wv = threadIdx.x >> 6;
    const int nblk = dm.P >> 4;
    for (int i = blockIdx.x; i < np - 1; i += gridDim.x) {   // never the last page
        const float ps = sc.pscore[(size_t)s * dm.MP + i];
        const int phys = ptab[i];
        bool ok = ps < dm.quant_thr && (unsigned)phys < (unsigned)dm.NP;
        if (ok) ok = v.page_format[phys] == 0;
        if (ok) {   // not evicted by this step (the serials in the list ascend)
            const int se = pser[i];
            int lo = 0, hi = cnt;
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (evs[mid] < se) lo = mid + 1; else hi = mid;
            }
            ok = !(lo < cnt && evs[lo] == se);
        }
        if (!ok) continue;   // uniform over the block
        for (int b = wv; b < dm.LHkv * nblk; b += 4) {
            const int r = b / nblk, blk = b - r * nblk;
            char* base = reinterpret_cast<char*>(v.k_pool + (((size_t)phys * dm.LHkv + r) * dm.P + 16 * blk) * kHeadDim);
            u32x4 x[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) x[j] = *reinterpret_cast<const u32x4*>(base + 16 * lane + 1024 * j);
            // a hole (region-aligned pages) holds no token
            const bool tok = !dm.aligned || v.region[(size_t)phys * dm.P + 16 * blk + (lane & 15)] != kHole;
            float m = 0.0f;
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    m = fmaxf(m, fabsf(__uint_as_float(x[j][w] << 16)));
                    m = fmaxf(m, fabsf(__uint_as_float(x[j][w] & 0xffff0000u)));
                }
            m = wave_max(tok ? m : 0.0f);
            const float scale = m > 0.0f ? __fdiv_rn(m, 448.0f) : 0.0f;
            u32x4 out[2] = {u32x4{0u, 0u, 0u, 0u}, u32x4{0u, 0u, 0u, 0u}};
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    uint32_t pair = 0;
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const float f = __uint_as_float(e ? (x[j][w] & 0xffff0000u) : (x[j][w] << 16));
                        const uint32_t c = (tok && m > 0.0f) ? e4m3_encode(__fdiv_rn(f, scale)) : 0u;
                        pair |= c << (8 * e);
                    }
                    // dims 2w, 2w + 1 of chunk j: bytes 8 (j & 1) + 2w, +1 of out[j >> 1]
                    out[j >> 1][2 * (j & 1) + (w >> 1)] |= pair << (16 * (w & 1));
                }
#pragma unroll
            for (int j = 0; j < 2; ++j) *reinterpret_cast<u32x4*>(base + 16 * lane + 1024 * j) = out[j];
            if (lane == 0) {
                const uint32_t sb = __float_as_uint(scale);
                *reinterpret_cast<u32x4*>(base + 2048) = u32x4{sb, sb, sb, sb};
            }
        }
        __syncthreads();
        if (threadIdx.x == 0) v.page_format[phys] = 1;
    }
}

hipError_t launch_quant(const Dims& dm, const View& v, const Scratch& sc, const int32_t* ev_serial,
                        const int32_t* ev_count, hipStream_t st) {
    hipLaunchKernelGGL(k_quant, dim3(64, dm.S), dim3(256), 0, st, dm, v, sc, ev_serial, ev_count);
    return hipGetLastError();
}

hipError_t launch_compact(const Dims& dm, const View& v, const Scratch& sc,
                          const int32_t* ev_serial, const int32_t* ev_count, int trusted, hipStream_t st) {
    hipLaunchKernelGGL(k_compact, dim3(dm.S), dim3(kSelThreads), 0, st, dm, v, sc, ev_serial, ev_count,
                       trusted);
    return hipGetLastError();
}

// ---------------------------------------------------------------- calibration

// Lifetime statistics (Sec. IV-B): one thread per token position of one
// session (blockIdx.y); tokens past the session's count do nothing.  The
// lanes of a wave that share a (region, age bucket) bin add their mass,
// count and age sum with wave reductions, and one lane adds them to the bin
// with 64-bit integer atomics (mass in fixed point, A * 2^40), so the sums
// do not depend on the order of the additions.
__global__ void __launch_bounds__(256) k_calib(Dims dm, View v, Scratch sc, const float* __restrict__ abar,
                                               int bucket_steps, int n_buckets,
                                               unsigned long long* mass_fx, unsigned long long* count,
                                               unsigned long long* age_sum) {
    const int s = blockIdx.y;
    const int tok = blockIdx.x * blockDim.x + threadIdx.x;
    const int nt = sc.valid[s] ? v.n_tokens[s] : 0;   // a void step adds nothing
    int key = -1;
    unsigned long long fx = 0, ag = 0;
    if (tok < nt && tok < dm.MP * dm.P) {
        const int p = v.page_table[(size_t)s * dm.MP + (tok >> dm.Pshift)];
        if ((unsigned)p < (unsigned)dm.NP) {
            const size_t si = (size_t)p * dm.P + (tok & (dm.P - 1));
            const int r = v.region[si];
            const int age = v.clock[s] - v.t_ins[si];
            const int b = age >= 0 ? age / bucket_steps : n_buckets;
            if (r < dm.n_regions && b < n_buckets) {
                key = r * n_buckets + b;
                fx = (unsigned long long)llrint((double)abar[si] * 1099511627776.0);   // 2^40
                ag = (unsigned long long)age;
            }
        } else {
            atomicOr(sc.status, kDevCorrupt);
        }
    }
    bool todo = key >= 0;
    while (__ballot(todo) != 0ull) {
        const int first = __ffsll((long long)__ballot(todo)) - 1;
        const int k = __shfl(key, first);
        const bool mine = todo && key == k;
        unsigned long long m = mine ? fx : 0ull, a = mine ? ag : 0ull;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            m += __shfl_xor(m, o);
            a += __shfl_xor(a, o);
        }
        const int c = __popcll(__ballot(mine));
        if (lane_id() == first) {
            const size_t bin = (size_t)s * dm.n_regions * n_buckets + k;
            atomicAdd(mass_fx + bin, m);
            atomicAdd(count + bin, (unsigned long long)c);
            atomicAdd(age_sum + bin, a);
        }
        todo = todo && !mine;
    }
}

hipError_t launch_calib(const Dims& dm, const View& v, const Scratch& sc, const float* abar, int bucket_steps,
                        int n_buckets, unsigned long long* mass_fx, unsigned long long* count,
                        unsigned long long* age_sum, hipStream_t st) {
    const int per_session = dm.MP * dm.P;
    hipLaunchKernelGGL(k_calib, dim3((per_session + 255) / 256, dm.S), dim3(256), 0, st, dm, v, sc, abar,
                       bucket_steps, n_buckets, mass_fx, count, age_sum);
    return hipGetLastError();
}

// ---------------------------------------------------------------- scratch layout

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

size_t scratch_bytes(const Dims& dm) {
    size_t n = 0;
    const size_t spill = dm.multi ? 1 : 0;   // the logits spill exists only when used
    n += align256(spill * dm.NP * dm.R * dm.P * sizeof(float));
    n += align256(spill * dm.S * dm.R * dm.max_chunks * sizeof(float2));
    n += align256((size_t)dm.S * dm.R * sizeof(float2));
    n += align256((size_t)dm.S * dm.MP * sizeof(float));
    n += 7 * align256((size_t)(dm.S + 1) * sizeof(int32_t));
    n += align256((size_t)(1 + 3 * (dm.S + 1)) * sizeof(int32_t));
    n += align256(sizeof(int32_t));
    n += align256((1 + (size_t)kAttendPerCu * (dm.S + 1)) * sizeof(unsigned long long));
    n += align256((size_t)dm.R * dm.U_cap * 2 * sizeof(unsigned long long));
    n += align256((dm.fused ? (size_t)dm.S * dm.R : 0) * 2 * sizeof(unsigned long long));
    n += align256((dm.rg_max > 1 ? (size_t)dm.U_cap * dm.T : 0) * sizeof(unsigned long long));
    n += align256(4 * sizeof(int32_t));
    n += align256(9 * sizeof(unsigned long long));
    n += 3 * align256((size_t)dm.S * sizeof(unsigned long long));
    n += align256((size_t)dm.S * dm.H * sizeof(int32_t));
    n += align256((size_t)(dm.S + 1) * sizeof(int32_t));
    return n;
}

void scratch_carve(const Dims& dm, void* base, Scratch* sc) {
    char* p = static_cast<char*>(base);
    auto take = [&](size_t bytes) {
        char* r = p;
        p += align256(bytes);
        return r;
    };
    const size_t spill = dm.multi ? 1 : 0;
    sc->logits = reinterpret_cast<float*>(take(spill * dm.NP * dm.R * dm.P * sizeof(float)));
    sc->cstats = reinterpret_cast<float2*>(take(spill * dm.S * dm.R * dm.max_chunks * sizeof(float2)));
    sc->rstats = reinterpret_cast<float2*>(take((size_t)dm.S * dm.R * sizeof(float2)));
    sc->pscore = reinterpret_cast<float*>(take((size_t)dm.S * dm.MP * sizeof(float)));
    sc->item_prefix = reinterpret_cast<int32_t*>(take((size_t)(dm.S + 1) * sizeof(int32_t)));
    sc->tile_prefix = reinterpret_cast<int32_t*>(take((size_t)(dm.S + 1) * sizeof(int32_t)));
    sc->chunks = reinterpret_cast<int32_t*>(take((size_t)(dm.S + 1) * sizeof(int32_t)));
    sc->valid = reinterpret_cast<int32_t*>(take((size_t)(dm.S + 1) * sizeof(int32_t)));
    sc->freed = reinterpret_cast<int32_t*>(take((size_t)(dm.S + 1) * sizeof(int32_t)));
    sc->score_prefix = reinterpret_cast<int32_t*>(take((size_t)(dm.S + 1) * sizeof(int32_t)));
    sc->ustart = reinterpret_cast<int32_t*>(take((size_t)(dm.S + 1) * sizeof(int32_t)));
    sc->plan = reinterpret_cast<int32_t*>(take((size_t)(1 + 3 * (dm.S + 1)) * sizeof(int32_t)));
    sc->epoch = reinterpret_cast<int32_t*>(take(sizeof(int32_t)));
    sc->claim = reinterpret_cast<unsigned long long*>(
        take((1 + (size_t)kAttendPerCu * (dm.S + 1)) * sizeof(unsigned long long)));
    sc->lane_box = sc->claim + 1;
    sc->ustat = reinterpret_cast<unsigned long long*>(
        take((size_t)dm.R * dm.U_cap * 2 * sizeof(unsigned long long)));
    sc->unorm = reinterpret_cast<unsigned long long*>(
        take((dm.fused ? (size_t)dm.S * dm.R : 0) * 2 * sizeof(unsigned long long)));
    sc->upart = reinterpret_cast<unsigned long long*>(
        take((dm.rg_max > 1 ? (size_t)dm.U_cap * dm.T : 0) * sizeof(unsigned long long)));
    int32_t* words = reinterpret_cast<int32_t*>(take(4 * sizeof(int32_t)));
    sc->status = words;      // the warning word follows the status word (read together)
    sc->warn = words + 1;
    sc->done_compact = words + 2;
    sc->opened = words + 3;
    sc->counters = reinterpret_cast<unsigned long long*>(take(9 * sizeof(unsigned long long)));
    sc->compact_acc = sc->counters + 8;
    sc->app_word = reinterpret_cast<unsigned long long*>(take((size_t)dm.S * sizeof(unsigned long long)));
    sc->ev_word = reinterpret_cast<unsigned long long*>(take((size_t)dm.S * sizeof(unsigned long long)));
    sc->ev_done = reinterpret_cast<unsigned long long*>(take((size_t)dm.S * sizeof(unsigned long long)));
    sc->recall = reinterpret_cast<int32_t*>(take((size_t)dm.S * dm.H * sizeof(int32_t)));
    sc->rcount = reinterpret_cast<int32_t*>(take((size_t)(dm.S + 1) * sizeof(int32_t)));
}

}  // namespace md
